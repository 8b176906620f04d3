"""The stream-copy reference kernel the benchmark times beside the splice: bit-exact copies, and
the argument checks of its entry point."""
import pytest
import torch

import bench

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("nbytes", [8192, 3 * 8192, 64 << 20])
def test_copies_bytes(nbytes):
    g = torch.Generator(device="cuda").manual_seed(nbytes)
    src = torch.randint(0, 256, (nbytes,), dtype=torch.uint8, device="cuda", generator=g)
    dst = torch.zeros(nbytes + 4096, dtype=torch.uint8, device="cuda")
    bench.stream_copy(dst[:nbytes], src, torch.cuda.current_stream().cuda_stream)
    torch.cuda.synchronize()
    assert torch.equal(dst[:nbytes], src)
    assert int(dst[nbytes:].count_nonzero()) == 0          # nothing written past the end


def test_rejects_bad_sizes():
    src = torch.ones(8192 + 16, dtype=torch.uint8, device="cuda")
    dst = torch.empty_like(src)
    with pytest.raises(RuntimeError):
        bench.stream_copy(dst, src, torch.cuda.current_stream().cuda_stream)   # not a multiple of 8192
