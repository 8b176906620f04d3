"""Argument checks of the tensor-level Python calls (CPU): a host tensor, a wrong dtype or a short
index array is refused before anything reaches the library, since a host address handed to a
kernel would fault the GPU."""
import pytest
import torch

from paper_2606_17107_amd import pkv


def test_host_tensors_are_refused():
    k = torch.zeros(1, 2, 8, 64, dtype=torch.bfloat16)
    pos = torch.zeros(8, dtype=torch.int32)
    with pytest.raises(ValueError, match="live on the GPU"):
        pkv.reposition_splice(k, k, k.clone(), k.clone(), pos, pos, 1e4, 64)
    with pytest.raises(ValueError, match="live on the GPU"):
        pkv.reposition_splice_freqs(k, k, k.clone(), k.clone(), pos, pos, [1.0] * 32, 64)
    with pytest.raises(ValueError, match="live on the GPU"):
        pkv.reposition_splice_batched(k, k, k.clone(), k.clone(), torch.zeros(64, dtype=torch.uint8), 1, 8, 1e4, 64)
    q = torch.zeros(1, 4, 4, 64, dtype=torch.bfloat16)
    with pytest.raises(ValueError, match="live on the GPU"):
        pkv.suffix_attention(q, k, k, q.clone(), torch.zeros(4, dtype=torch.int32), torch.tensor([8], dtype=torch.int32),
                             0.125, 8)
    with pytest.raises(TypeError, match="torch.Tensor"):
        pkv.suffix_attention(None, k, k, q, None, None, 0.125, 8)


def test_need_checks_type_dtype_size_and_device():
    cpu, meta = torch.device("cpu"), torch.device("meta")
    pos = torch.zeros(10, dtype=torch.int32)
    pkv._need(None, "x", cpu, torch.int32, 5)                               # optional argument absent
    pkv._need(pos, "src_pos", cpu, torch.int32, 10, contiguous=True)
    with pytest.raises(TypeError, match="src_pos must be torch.int32"):
        pkv._need(pos.long(), "src_pos", cpu, torch.int32, 10)
    with pytest.raises(ValueError, match="holds 10 elements, the call reads 11"):
        pkv._need(pos, "src_pos", cpu, torch.int32, 11)
    with pytest.raises(ValueError, match="must be contiguous"):
        pkv._need(torch.zeros(20, dtype=torch.int32)[::2], "q_pos", cpu, torch.int32, 10, contiguous=True)
    with pytest.raises(ValueError, match="is on cpu, the call runs on meta"):
        pkv._need(pos, "kv_len", meta, torch.int32, 1)
    with pytest.raises(TypeError, match="must be a torch.Tensor"):
        pkv._need([0] * 10, "dst_pos", cpu, torch.int32, 10)
