"""Pins for the oracle's causal suffix attention (paper Sec. 5 "Linear-time
TTFT": the transplant costs a re-rotation pass plus the suffix; Sec. 6: the
agent prefills only the delta over the reused cache) and its MLA absorbed
form (Sec. 8 MLA adapter: the cache holds a latent plus a decoupled k_pe).

Checked against a library routine (torch's scaled_dot_product_attention in
fp64 with an explicit mask), closed-form special cases, invariances, the
explicit (non-absorbed) MLA formulation, and the end-to-end transplant
identity."""
import math

import numpy as np
import pytest
import torch
import torch.nn.functional as F

from paper_2606_17107_amd import synth


def bits_to_f64(b):
    if b.dtype == np.uint16:
        return (b.astype(np.uint32) << 16).view(np.float32).astype(np.float64)
    return b.astype(np.float64)


def randn(shape, seed, dtype=torch.bfloat16, mult=1.0):
    g = torch.Generator().manual_seed(seed)
    return synth.to_numpy_bits((torch.randn(shape, generator=g) * mult).to(dtype))


def sdpa_reference(q, k, v, q_pos, kv_len, scale):
    """torch SDPA (fp64, CPU) with an explicit boolean causal mask and repeated KV heads."""
    qd = torch.from_numpy(bits_to_f64(q)).permute(1, 0, 2)          # [H][n_q][d]
    kd = torch.from_numpy(bits_to_f64(k[:, :kv_len]))               # [Hkv][kv][d]
    vd = torch.from_numpy(bits_to_f64(v[:, :kv_len]))
    G = qd.shape[0] // kd.shape[0]
    kd = kd.repeat_interleave(G, dim=0)
    vd = vd.repeat_interleave(G, dim=0)
    j = torch.arange(kv_len)
    mask = j[None, :] <= torch.from_numpy(q_pos.astype(np.int64))[:, None]
    o = F.scaled_dot_product_attention(qd, kd, vd, attn_mask=mask, scale=scale)
    return o.permute(1, 0, 2).numpy()


@pytest.mark.parametrize("dtype", [torch.bfloat16, torch.float32])
@pytest.mark.parametrize("H,Hkv,d,n_q,slots,kv_len", [(4, 2, 64, 16, 528, 528), (6, 3, 32, 9, 70, 61),
                                                     (8, 1, 128, 5, 300, 300), (2, 2, 16, 3, 40, 17)])
def test_matches_sdpa(ref, dtype, H, Hkv, d, n_q, slots, kv_len):
    q = randn((n_q, H, d), 1, dtype, 2.0)
    k = randn((Hkv, slots, d), 2, dtype)
    v = randn((Hkv, slots, d), 3, dtype)
    q_pos = (kv_len - n_q + np.arange(n_q)).astype(np.int32)
    q_pos[0] = min(q_pos[0], 3)    # one query that sees only a few slots
    out, lse = ref.attention(q, k, v, q_pos, kv_len, 1 / math.sqrt(d))
    want = sdpa_reference(q, k, v, q_pos, kv_len, 1 / math.sqrt(d))
    np.testing.assert_allclose(out, want, rtol=1e-12, atol=1e-12)
    # lse: log-sum-exp of the visible scaled scores, via torch.logsumexp
    qd, kd = bits_to_f64(q), bits_to_f64(k)
    G = H // Hkv
    for i in range(n_q):
        for h in range(H):
            nv = min(kv_len, q_pos[i] + 1)
            s = kd[h // G, :nv] @ qd[i, h] / math.sqrt(d)
            assert abs(lse[i, h] - torch.logsumexp(torch.from_numpy(s), 0).item()) < 1e-12


def test_special_cases(ref):
    H, Hkv, d, slots = 4, 2, 64, 50
    q = randn((3, H, d), 4)
    k = randn((Hkv, slots, d), 5)
    v = randn((Hkv, slots, d), 6)
    # a query at position 0 sees only slot 0: output is v_0 exactly
    out, _ = ref.attention(q, k, v, np.array([0, 0, 0], np.int32), slots, 0.125)
    for h in range(H):
        np.testing.assert_array_equal(out[:, h], np.broadcast_to(bits_to_f64(v[h // 2, 0]), (3, d)))
    # every V row equal: output is that row
    v_eq = np.broadcast_to(v[:, :1], v.shape).copy()
    out, _ = ref.attention(q, k, v_eq, np.array([10, 30, 49], np.int32), slots, 0.125)
    for h in range(H):
        np.testing.assert_allclose(out[:, h], np.broadcast_to(bits_to_f64(v[h // 2, 0]), (3, d)),
                                   rtol=1e-14, atol=1e-14)
    # scale 0: the mean of the visible values
    qp = np.array([9, 20, 49], np.int32)
    out, lse = ref.attention(q, k, v, qp, slots, 0.0)
    for i, p in enumerate(qp):
        for h in range(H):
            np.testing.assert_allclose(out[i, h], bits_to_f64(v[h // 2, : p + 1]).mean(0), rtol=1e-13,
                                       atol=1e-14)
            assert abs(lse[i, h] - math.log(p + 1)) < 1e-13
    # a row with no visible slot (kv_len 0) is zero with lse -inf
    out, lse = ref.attention(q, k, v, qp, 0, 0.125)
    assert np.all(out == 0) and np.all(np.isneginf(lse))


def test_gqa_equals_mha_with_repeated_kv_and_permutation_invariance(ref):
    H, Hkv, d, slots, n_q = 8, 2, 32, 64, 4
    q = randn((n_q, H, d), 7, mult=3.0)
    k = randn((Hkv, slots, d), 8)
    v = randn((Hkv, slots, d), 9)
    qp = np.full(n_q, slots - 1, np.int32)
    out, _ = ref.attention(q, k, v, qp, slots, 0.2)
    k_rep = np.repeat(k, H // Hkv, axis=0)
    v_rep = np.repeat(v, H // Hkv, axis=0)
    out_mha, _ = ref.attention(q, k_rep, v_rep, qp, slots, 0.2)
    np.testing.assert_allclose(out, out_mha, rtol=1e-13, atol=1e-15)
    perm = np.random.default_rng(0).permutation(slots)
    out_p, _ = ref.attention(q, np.ascontiguousarray(k[:, perm]), np.ascontiguousarray(v[:, perm]), qp,
                             slots, 0.2)
    np.testing.assert_allclose(out, out_p, rtol=1e-12, atol=1e-14)


def test_causality_and_kv_len(ref):
    """Slots beyond a query's position, or beyond kv_len, never influence it."""
    H, Hkv, d, slots = 2, 1, 16, 40
    q = randn((2, H, d), 10)
    k = randn((Hkv, slots, d), 11)
    v = randn((Hkv, slots, d), 12)
    qp = np.array([19, 29], np.int32)
    out, _ = ref.attention(q, k, v, qp, 30, 0.3)
    k2, v2 = k.copy(), v.copy()
    k2[:, 30:] = randn((Hkv, 10, d), 13)
    v2[:, 30:] = randn((Hkv, 10, d), 14)
    out2, _ = ref.attention(q, k2, v2, qp, 30, 0.3)
    np.testing.assert_array_equal(out, out2)
    k2[:, 20:30] = randn((Hkv, 10, d), 15)
    out3, _ = ref.attention(q, k2, v, qp, 30, 0.3)
    np.testing.assert_array_equal(out3[0], out[0])        # query 0 at position 19 unaffected
    assert not np.allclose(out3[1], out[1])


def test_planted_needle(ref):
    """One key aligned with the query and much larger than the rest: the output
    is (almost exactly) that slot's value."""
    H, Hkv, d, slots = 1, 1, 64, 200
    q = randn((1, H, d), 16)
    k = randn((Hkv, slots, d), 17)
    v = randn((Hkv, slots, d), 18)
    k_needle = (bits_to_f64(q[0, 0]) * 8.0).astype(np.float32)
    k[0, 123] = synth.to_numpy_bits(torch.from_numpy(k_needle).to(torch.bfloat16))
    out, _ = ref.attention(q, k, v, np.array([199], np.int32), slots, 1 / 8)
    np.testing.assert_allclose(out[0, 0], bits_to_f64(v[0, 123]), atol=1e-6)


def test_mla_absorbed_equals_explicit(ref):
    """Absorbed MLA (scores over [c_kv | k_pe] with q = [W_UK^T q_nope | q_pe],
    values from c_kv) followed by the value up-projection equals explicit
    per-head attention with k_h = [W_UK c | k_pe] and v_h = W_UV c."""
    n_q, H, d_c, d_nope, d_pe, d_v, slots = 4, 3, 32, 16, 8, 12, 45
    rng = np.random.default_rng(19)
    c = rng.standard_normal((slots, d_c)).astype(np.float32)
    k_pe = rng.standard_normal((slots, d_pe)).astype(np.float32)
    W_UK = rng.standard_normal((H, d_nope, d_c)) * 0.2
    W_UV = rng.standard_normal((H, d_v, d_c)) * 0.2
    q_nope = rng.standard_normal((n_q, H, d_nope))
    q_pe = rng.standard_normal((n_q, H, d_pe)).astype(np.float32)
    scale = 1 / math.sqrt(d_nope + d_pe)
    q_pos = np.array([10, 20, 30, 44], np.int32)
    # absorbed form through the oracle (fp32 storage of the absorbed query)
    q_lat = np.einsum("hnc,ihn->ihc", W_UK, q_nope).astype(np.float32)
    q_abs = np.concatenate([q_lat, q_pe], axis=-1)
    rows = np.concatenate([c, k_pe], axis=-1)[None]           # [1][slots][d_c+d_pe]
    o_lat, _ = ref.attention(np.ascontiguousarray(q_abs), rows, rows[..., :d_c], q_pos, slots, scale)
    o_abs = np.einsum("hvc,ihc->ihv", W_UV, o_lat)
    # explicit form with torch SDPA in fp64 (using the fp32-stored absorbed query's
    # exact inner products: q_lat . c == q_nope . (W_UK c) up to the fp32 storage of q_lat)
    cd = torch.from_numpy(c.astype(np.float64))
    k_h = torch.cat([torch.einsum("hnc,jc->hjn", torch.from_numpy(W_UK), cd),
                     torch.from_numpy(k_pe.astype(np.float64))[None].expand(H, -1, -1)], -1)
    v_h = torch.einsum("hvc,jc->hjv", torch.from_numpy(W_UV), cd)
    q_h = torch.cat([torch.from_numpy(q_nope), torch.from_numpy(q_pe.astype(np.float64))], -1).permute(1, 0, 2)
    mask = torch.arange(slots)[None, :] <= torch.from_numpy(q_pos.astype(np.int64))[:, None]
    o_exp = F.scaled_dot_product_attention(q_h, k_h, v_h, attn_mask=mask, scale=scale).permute(1, 0, 2)
    np.testing.assert_allclose(o_abs, o_exp.numpy(), rtol=1e-5, atol=1e-6)


def test_transplant_then_attend_equals_recompute(ref):
    """End to end: attention over splice(RoPE(k, src)) equals attention over a
    cache holding RoPE(k, dst) directly (fp32 storage)."""
    L, H, Hkv, d, T, theta = 1, 4, 2, 64, 128, 10000.0
    cap, n_q = 512, 16
    k_pre = randn((L, Hkv, T, d), 20, torch.float32)
    v = randn((L, Hkv, T, d), 21, torch.float32)
    ctx_k = ref.rope_rows(randn((L, Hkv, cap + n_q, d), 22, torch.float32),
                          np.broadcast_to(np.arange(cap + n_q, dtype=np.int32), (L, Hkv, cap + n_q)),
                          theta, d)
    ctx_v = randn((L, Hkv, cap + n_q, d), 23, torch.float32)
    src = np.arange(T, dtype=np.int32)
    dst = (300 + src).astype(np.int32)
    k_src = ref.rope_rows(k_pre, np.broadcast_to(src, (L, Hkv, T)), theta, d)
    spliced_k, spliced_v = ctx_k.copy(), ctx_v.copy()
    ref.reposition_splice(k_src, v, spliced_k, spliced_v, src, dst, theta, d)
    direct_k, direct_v = ctx_k.copy(), ctx_v.copy()
    direct_k[:, :, dst] = ref.rope_rows(k_pre, np.broadcast_to(dst, (L, Hkv, T)), theta, d)
    direct_v[:, :, dst] = v
    q = ref.rope_rows(randn((n_q, H, d), 24, torch.float32),
                      np.broadcast_to((cap + np.arange(n_q)).astype(np.int32)[:, None], (n_q, H)),
                      theta, d)
    q_pos = (cap + np.arange(n_q)).astype(np.int32)
    o1, _ = ref.attention(q, spliced_k[0], spliced_v[0], q_pos, cap + n_q, 0.125)
    o2, _ = ref.attention(q, direct_k[0], direct_v[0], q_pos, cap + n_q, 0.125)
    np.testing.assert_allclose(o1, o2, rtol=1e-5, atol=1e-6)
    # without the rotation the outputs differ clearly
    bad_k = ctx_k.copy()
    bad_k[:, :, dst] = k_src
    o3, _ = ref.attention(q, bad_k[0], spliced_v[0], q_pos, cap + n_q, 0.125)
    assert np.abs(o3 - o2).max() > 1e-3


def sdpa_window_reference(q, k, v, q_pos, kv_len, scale, window):
    """torch SDPA (fp64) with an explicit banded mask: q_pos - window < j <= q_pos, j < kv_len."""
    qd = torch.from_numpy(bits_to_f64(q)).permute(1, 0, 2)
    kd = torch.from_numpy(bits_to_f64(k[:, :kv_len]))
    vd = torch.from_numpy(bits_to_f64(v[:, :kv_len]))
    G = qd.shape[0] // kd.shape[0]
    kd = kd.repeat_interleave(G, dim=0)
    vd = vd.repeat_interleave(G, dim=0)
    j = torch.arange(kv_len)[None, :]
    p = torch.from_numpy(q_pos.astype(np.int64))[:, None]
    mask = (j <= p) & (j > p - window)
    o = F.scaled_dot_product_attention(qd, kd, vd, attn_mask=mask, scale=scale)
    return o.permute(1, 0, 2).numpy()


@pytest.mark.parametrize("window", [1, 7, 33, 100, 1000])
def test_sliding_window_matches_banded_sdpa(ref, window):
    """Sliding-window layers keep the full cache; the mask alone enforces the window (Sec. 8 config fix)."""
    H, Hkv, d, n_q, slots = 4, 2, 64, 12, 300
    q = randn((n_q, H, d), 21, torch.bfloat16, 2.0)
    k = randn((Hkv, slots, d), 22)
    v = randn((Hkv, slots, d), 23)
    q_pos = np.array([0, 5, 31, 32, 64, 99, 150, 200, 250, 280, 290, 299], dtype=np.int32)
    out, _ = ref.attention(q, k, v, q_pos, slots, 1 / math.sqrt(d), window=window)
    want = sdpa_window_reference(q, k, v, q_pos, slots, 1 / math.sqrt(d), window)
    np.testing.assert_allclose(out, want, rtol=1e-12, atol=1e-12)


def test_sliding_window_limits(ref):
    H, Hkv, d, n_q, slots = 4, 1, 32, 6, 80
    q = randn((n_q, H, d), 24, torch.bfloat16, 3.0)
    k = randn((Hkv, slots, d), 25)
    v = randn((Hkv, slots, d), 26)
    q_pos = np.array([0, 3, 17, 40, 70, 79], dtype=np.int32)
    full, lse_full = ref.attention(q, k, v, q_pos, slots, 0.2)
    # a window covering every visible slot is plain causal attention, to the bit
    wide, lse_wide = ref.attention(q, k, v, q_pos, slots, 0.2, window=80)
    assert np.array_equal(full, wide) and np.array_equal(lse_full, lse_wide)
    # window 1: only the query's own slot is visible, so the output is that value row
    one, lse_one = ref.attention(q, k, v, q_pos, slots, 0.2, window=1)
    vd = bits_to_f64(v)
    for i, p in enumerate(q_pos):
        np.testing.assert_array_equal(one[i], np.broadcast_to(vd[0, p], (H, d)))
    # windowed attention equals causal attention over the sliced cache with shifted positions
    for W in (5, 16, 50):
        win, _ = ref.attention(q, k, v, q_pos, slots, 0.2, window=W)
        for i, p in enumerate(q_pos):
            lo = max(0, int(p) - W + 1)
            sl, _ = ref.attention(np.ascontiguousarray(q[i:i + 1]), np.ascontiguousarray(k[:, lo:]),
                                  np.ascontiguousarray(v[:, lo:]), np.array([p - lo], np.int32), slots - lo, 0.2)
            np.testing.assert_allclose(win[i], sl[0], rtol=1e-13, atol=1e-13)
