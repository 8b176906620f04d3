"""Every compiled variant of the splice kernel against the oracle (paper Sec. 5; Fig. "Two cache
operations" (b); Sec. 8 paged caches and scaled / multimodal RoPE): storage type (bf16, fp32) x
pairing (HALF, INTERLEAVED) x entry point (per-token positions, explicit frequency table, paged
destination, batched segments).  Each case is small (2 layers x 2 KV heads, d 64, 70 tokens) with
scattered source positions, so both the shared-delta and the per-lane coefficient paths run where
the entry point allows them.  Bars as elsewhere: V bit-exact, bf16 K within one ulp (with the
near-zero floor), fp32 K within 1e-6 relative per pair; destination slots outside the splice
untouched."""
import types

import numpy as np
import pytest
import torch

import oracle
from helpers import dev, host_bits
from paper_2606_17107_amd import pkv, synth
from test_gpu_paged import block_table, gather
from test_gpu_splice import compare

pytestmark = pytest.mark.gpu

L, H, D, N, CAP, THETA = 2, 2, 64, 70, 320, 1e4


def draw(shape, seed, dtype):
    t = synth.Draws(seed, "cpu").normal(shape, torch.bfloat16 if dtype == "bf16" else torch.float32)
    return host_bits(t)


def spec(dtype, style):
    return types.SimpleNamespace(dtype=dtype, rope_style=style, rope_dim=D, rope_offset=0)


def positions(seed):
    rng = np.random.default_rng(seed)
    src = rng.integers(0, 5000, N).astype(np.int32)
    dst = rng.permutation(CAP)[:N].astype(np.int32)
    return src, dst


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
@pytest.mark.parametrize("style", [synth.HALF, synth.INTERLEAVED])
def test_per_token(dtype, style):
    sk, sv = draw((L, H, N, D), 1, dtype), draw((L, H, N, D), 2, dtype)
    ck, cv = draw((L, H, CAP, D), 3, dtype), draw((L, H, CAP, D), 4, dtype)
    src, dst = positions(5)
    gk, gv = dev(ck), dev(cv)
    pkv.reposition_splice(dev(sk), dev(sv), gk, gv, torch.from_numpy(src).cuda(), torch.from_numpy(dst).cuda(),
                          THETA, D, 0, style)
    torch.cuda.synchronize()
    ok, ov = ck.copy(), cv.copy()
    oracle.reposition_splice(sk, sv, ok, ov, src, dst, THETA, D, 0, style)
    compare(spec(dtype, style), host_bits(gk), host_bits(gv), ok, ov)


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
@pytest.mark.parametrize("style", [synth.HALF, synth.INTERLEAVED])
def test_frequency_table(dtype, style):
    sk, sv = draw((L, H, N, D), 11, dtype), draw((L, H, N, D), 12, dtype)
    ck, cv = draw((L, H, CAP, D), 13, dtype), draw((L, H, CAP, D), 14, dtype)
    src, dst = positions(15)
    # a scaled schedule: the theta frequencies with the low half divided by 8
    omega = THETA ** (-2.0 * np.arange(D // 2) / D)
    omega[D // 4:] /= 8.0
    gk, gv = dev(ck), dev(cv)
    pkv.reposition_splice_freqs(dev(sk), dev(sv), gk, gv, torch.from_numpy(src).cuda(),
                                torch.from_numpy(dst).cuda(), omega, D, 0, style)
    torch.cuda.synchronize()
    ok, ov = ck.copy(), cv.copy()
    oracle.reposition_splice(sk, sv, ok, ov, src, dst, THETA, D, 0, style, omega=omega)
    compare(spec(dtype, style), host_bits(gk), host_bits(gv), ok, ov)


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
@pytest.mark.parametrize("style", [synth.HALF, synth.INTERLEAVED])
def test_paged_destination(dtype, style):
    B, max_pages = 32, CAP // 32
    P = max_pages + 3
    pk, pv = draw((L, P, B, H, D), 21, dtype), draw((L, P, B, H, D), 22, dtype)
    sk, sv = draw((L, H, N, D), 23, dtype), draw((L, H, N, D), 24, dtype)
    bt = block_table(1, max_pages, P, 25)
    src, dst = positions(26)
    gk, gv = dev(pk), dev(pv)
    pkv.reposition_splice_paged(dev(sk), dev(sv), gk, gv, torch.from_numpy(src).cuda(), torch.from_numpy(dst).cuda(),
                                torch.from_numpy(bt).cuda(), THETA, D, 0, style)
    torch.cuda.synchronize()
    hk, hv = host_bits(gk), host_bits(gv)
    ok, ov = gather(pk, bt[0], CAP), gather(pv, bt[0], CAP)
    oracle.reposition_splice(sk, sv, ok, ov, src, dst, THETA, D, 0, style)
    compare(spec(dtype, style), gather(hk, bt[0], CAP), gather(hv, bt[0], CAP), ok, ov)
    spare = np.setdiff1d(np.arange(P), bt[0])
    np.testing.assert_array_equal(hk[:, spare], pk[:, spare])


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
@pytest.mark.parametrize("style", [synth.HALF, synth.INTERLEAVED])
def test_batched_segments(dtype, style):
    """One source chunk spliced into two sequences (different deltas, one of them negative) and a
    second chunk into the first sequence."""
    sk, sv = draw((L, H, N, D), 31, dtype), draw((L, H, N, D), 32, dtype)
    ck, cv = draw((L, H, CAP, D), 33, dtype), draw((L, H, CAP, D), 34, dtype)
    seq_len = CAP // 2
    segs = [dict(src_slot0=0, dst_seq_base=0, n_tokens=40, src_pos0=300, dst_pos0=10, dst_seq_len=seq_len),
            dict(src_slot0=0, dst_seq_base=seq_len, n_tokens=40, src_pos0=300, dst_pos0=1000 - 900, dst_seq_len=seq_len),
            dict(src_slot0=40, dst_seq_base=0, n_tokens=30, src_pos0=7, dst_pos0=90, dst_seq_len=seq_len)]
    gk, gv = dev(ck), dev(cv)
    pkv.reposition_splice_batched(dev(sk), dev(sv), gk, gv, pkv.make_segments(segs, "cuda"), len(segs), 40, THETA,
                                  D, 0, style)
    torch.cuda.synchronize()
    ok, ov = ck.copy(), cv.copy()
    for s in segs:
        n = s["n_tokens"]
        base = s["dst_seq_base"]
        seq_k = ok[:, :, base: base + s["dst_seq_len"]]
        seq_v = ov[:, :, base: base + s["dst_seq_len"]]
        sl = slice(s["src_slot0"], s["src_slot0"] + n)
        oracle.reposition_splice(np.ascontiguousarray(sk[:, :, sl]), np.ascontiguousarray(sv[:, :, sl]), seq_k, seq_v,
                                 np.arange(s["src_pos0"], s["src_pos0"] + n, dtype=np.int32),
                                 np.arange(s["dst_pos0"], s["dst_pos0"] + n, dtype=np.int32), THETA, D, 0, style)
    compare(spec(dtype, style), host_bits(gk), host_bits(gv), ok, ov)
