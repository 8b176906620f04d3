"""pkv_suffix_attention_noalloc, the allocation-free variant of pkv_suffix_attention
for callers that cannot allocate (graph capture, serving loops), against the
existing entry point with a caller workspace: two calls in a row, the second
smaller, on the same static scratch; a planned split count lowered to fit the
scratch; an explicit one that does not fit rejected.  Outputs must equal the
workspace entry point's at the same split count bit for bit, and meet the
attention bar against the oracle on sampled rows."""
import math

import numpy as np
import pytest
import torch

import oracle
from helpers import Guarded, check_attention_close, host_bits, log
from paper_2606_17107_amd import pkv, synth

pytestmark = pytest.mark.gpu


def case(L, H, Hkv, d, dv, n_q, kv, seed, mla=False):
    g = synth.Draws(seed, "cuda")
    k = g.normal((L, Hkv, kv, d))
    v = k[..., :dv] if mla else g.normal((L, Hkv, kv, dv))
    q = g.normal((L, n_q, H, d))
    q_pos = torch.arange(kv - n_q, kv, dtype=torch.int32, device="cuda")
    return dict(q=q, k=k, v=v, q_pos=q_pos, kv_len=torch.tensor([kv], dtype=torch.int32, device="cuda"), kv=kv,
                H=H, Hkv=Hkv, d=d, dv=dv, scale=1 / math.sqrt(192 if mla else d),
                variant=pkv.PKV_ATTN_MLA if mla else pkv.PKV_ATTN_GQA)


def with_workspace(c, n_splits):
    out = torch.zeros(c["q"].shape[:3] + (c["dv"],), dtype=torch.bfloat16, device="cuda")
    desc = pkv.make_attn_desc(c["q"], c["k"], c["v"], out, c["kv"], variant=c["variant"], n_splits=n_splits)
    need = pkv.pkv_attention_workspace_size(desc, c["H"], c["Hkv"], c["d"])
    ws = torch.empty(max(need, 16), dtype=torch.uint8, device="cuda")
    st = pkv.pkv_suffix_attention(c["q"], c["k"], c["v"], out, c["q_pos"], c["kv_len"], c["H"], c["Hkv"], c["d"],
                                  c["scale"], desc, ws, need)
    assert st == pkv.PKV_OK, pkv.pkv_last_error()
    torch.cuda.synchronize()
    return out, need


def no_alloc(c, n_splits):
    out = Guarded(c["q"].shape[:3] + (c["dv"],), torch.bfloat16)
    desc = pkv.make_attn_desc(c["q"], c["k"], c["v"], out.t, c["kv"], variant=c["variant"], n_splits=n_splits)
    st = pkv.pkv_suffix_attention_noalloc(c["q"], c["k"], c["v"], out.t, c["q_pos"], c["kv_len"], c["H"], c["Hkv"],
                                          c["d"], c["scale"], desc)
    return st, out


def check_against_oracle(c, out, layers, rows):
    q, k, v = host_bits(c["q"]), host_bits(c["k"]), host_bits(c["v"])
    got = host_bits(out)
    for l in layers:
        want, _ = oracle.attention(np.ascontiguousarray(q[l][rows]), k[l], np.ascontiguousarray(v[l]),
                                   c["q_pos"].cpu().numpy()[rows], c["kv"], c["scale"])
        log("   layer %d vs oracle" % l, check_attention_close(got[l][rows], want))


def test_two_calls_in_a_row_second_smaller():
    big = case(1, 32, 8, 128, 128, 64, 8256, seed=31)       # one gqa8b layer: the planner splits it 16 ways
    small = case(1, 8, 2, 128, 128, 20, 3000, seed=32)
    for c, name in ((big, "one gqa8b-shaped layer"), (small, "a smaller layer")):
        want, need = with_workspace(c, 0)
        assert 0 < need <= pkv.PKV_NOALLOC_SCRATCH_BYTES, need
        st, out = no_alloc(c, 0)
        assert st == pkv.PKV_OK, pkv.pkv_last_error()
        torch.cuda.synchronize()
        out.check("no-alloc output")
        log("  %s: %d bytes of partials in the scratch" % (name, need))
        assert torch.equal(out.t, want), "differs from pkv_suffix_attention at the same split count"
        check_against_oracle(c, out.t, [0], np.array([0, 1, c["q"].shape[1] // 2, c["q"].shape[1] - 1]))


def test_mla_split_count_lowered_to_fit():
    """The 27-layer MLA workload in one call: the planner's 2 splits need 227 MB of partials, more than
    the scratch, so the allocation-free call runs 1 split; it equals the workspace call with
    n_splits = 1."""
    c = case(27, 16, 1, 576, 512, 128, 32896, seed=33, mla=True)
    _, need_auto = with_workspace(c, 0)
    assert need_auto > pkv.PKV_NOALLOC_SCRATCH_BYTES
    _, need2 = with_workspace(c, 2)
    assert need2 > pkv.PKV_NOALLOC_SCRATCH_BYTES
    want, need1 = with_workspace(c, 1)
    assert need1 == 0
    st, out = no_alloc(c, 0)
    assert st == pkv.PKV_OK, pkv.pkv_last_error()
    torch.cuda.synchronize()
    out.check("no-alloc output")
    assert torch.equal(out.t, want)
    check_against_oracle(c, out.t, [0, 26], np.array([0, 63, 127]))


def test_explicit_split_count_beyond_the_scratch_is_rejected():
    c = case(27, 16, 1, 576, 512, 128, 32896, seed=34, mla=True)
    st, out = no_alloc(c, 2)
    assert st == pkv.PKV_ERR_SHAPE
    assert "scratch" in pkv.pkv_last_error()
    torch.cuda.synchronize()
    assert out.untouched(slice(None)), "a rejected call must not write"
