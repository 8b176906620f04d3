"""GPU edge cases against the oracle: deltas at the limit the ABI states
(|delta| < 2^24) on the uniform and the per-lane coefficient paths, GQA group
sizes 1 (MHA) and 8, calls with nothing to do, and a sequence with no cache
slots.  Bars as in the other parity tests."""
import numpy as np
import pytest
import torch

import oracle
from helpers import bits_to_f64, check_attention_close, check_rotated_keys, dev, host_bits, log
from paper_2606_17107_amd import pkv, synth

pytestmark = pytest.mark.gpu

LIMIT = (1 << 24) - 1


def bits(shape, seed):
    return host_bits(synth.Draws(seed, "cpu").normal(shape))


def splice_case(deltas, d=128, v_dim=128, r=128, offset=0, style=0, theta=5e5, seed=0):
    n = len(deltas)
    L, H = 2, 2
    sk = bits((L, H, n, d), seed)
    sv = bits((L, H, n, v_dim), seed + 1) if v_dim else None
    dk = bits((L, H, n, d), seed + 2)
    dv = bits((L, H, n, v_dim), seed + 3) if v_dim else None
    dst = np.arange(n, dtype=np.int64)
    src = dst - np.asarray(deltas, np.int64)
    assert src.min() >= -(1 << 31) and src.max() < (1 << 31)
    src, dst = src.astype(np.int32), dst.astype(np.int32)
    gk, gv = dev(dk), (dev(dv) if v_dim else None)
    pkv.reposition_splice(dev(sk), dev(sv) if v_dim else None, gk, gv, torch.from_numpy(src).cuda(),
                          torch.from_numpy(dst).cuda(), theta, r, offset, style)
    torch.cuda.synchronize()
    ok, ov = dk.copy(), (dv.copy() if v_dim else None)
    oracle.reposition_splice(sk, sv, ok, ov, src, dst, theta, r, offset, style)
    if v_dim:
        np.testing.assert_array_equal(host_bits(gv), ov)
    return check_rotated_keys(host_bits(gk), ok, offset, r, style)


def test_uniform_delta_at_the_limit():
    """Every token moves by 2^24 - 1 (the wave-uniform coefficient path), and by -(2^24 - 1)."""
    for sign in (1, -1):
        n_diff, n_floor = splice_case([sign * LIMIT] * 96, seed=10)
        log("  delta %+d: K not bit-equal %d, floor %d" % (sign * LIMIT, n_diff, n_floor))


def test_mixed_large_deltas():
    """Per-token deltas spread over (-2^24, 2^24) (the per-lane path), GQA rows and MLA k_pe."""
    rng = np.random.default_rng(11)
    deltas = np.concatenate([[LIMIT, -LIMIT, 1 << 23, -(1 << 23), 1, -1, 0],
                             rng.integers(-LIMIT, LIMIT + 1, 121)])
    splice_case(deltas, seed=12)
    splice_case(deltas, d=576, v_dim=0, r=64, offset=512, style=1, theta=1e4, seed=13)


@pytest.mark.parametrize("H,Hkv,d", [(4, 4, 128), (16, 2, 128), (8, 8, 64), (16, 2, 64), (12, 4, 128), (40, 8, 128),
                                     (32, 2, 64), (64, 2, 128)])
def test_group_sizes(H, Hkv, d):
    """GQA groups of 1 (multi-head attention), 3 and 5 (a 32-row MFMA block then holds rows of
    several queries with the group split across blocks), 8, 16 and 32 query heads per KV head."""
    L, n_q, kv = 2, 37, 611
    g = synth.Draws(20 + H + d, "cpu")
    q = host_bits(g.normal((L, n_q, H, d)))
    k = host_bits(g.normal((L, Hkv, kv, d)))
    v = host_bits(g.normal((L, Hkv, kv, d)))
    q_pos = np.arange(kv - n_q, kv, dtype=np.int32)
    scale = 1 / np.sqrt(d)
    for splits in (1, 3):
        out = torch.zeros(L, n_q, H, d, dtype=torch.bfloat16, device="cuda")
        pkv.suffix_attention(dev(q), dev(k), dev(v), out, torch.from_numpy(q_pos).cuda(),
                             torch.tensor([kv], dtype=torch.int32, device="cuda"), scale, max_kv_len=kv,
                             n_splits=splits)
        torch.cuda.synchronize()
        got = host_bits(out)
        for l in range(L):
            want, _ = oracle.attention(q[l], k[l], v[l], q_pos, kv, scale)
            check_attention_close(got[l], want)


def test_calls_with_nothing_to_do():
    """n_tokens = 0 splices nothing; total_q = 0 attends nothing; both return OK and touch nothing."""
    g = synth.Draws(30, "cuda")
    sk, sv = g.normal((1, 2, 4, 128)), g.normal((1, 2, 4, 128))
    dk, dv = g.normal((1, 2, 16, 128)), g.normal((1, 2, 16, 128))
    before = (dk.clone(), dv.clone())
    pos = torch.zeros(4, dtype=torch.int32, device="cuda")
    layout = pkv.make_layout(sk, sv, dk, dv, n_tokens=0)
    assert pkv.pkv_reposition_splice(sk, sv, dk, dv, pos, pos, 1e4, 128, layout) == pkv.PKV_OK
    q = g.normal((1, 3, 4, 128))
    out = torch.full((1, 3, 4, 128), 5.0, dtype=torch.bfloat16, device="cuda")
    desc = pkv.make_attn_desc(q, dk, dv, out, 16)
    desc.total_q = desc.max_q = 0
    kl = torch.tensor([16], dtype=torch.int32, device="cuda")
    assert pkv.pkv_suffix_attention(q, dk, dv, out, pos, kl, 4, 2, 128, 0.1, desc, None, 0) == pkv.PKV_OK
    torch.cuda.synchronize()
    assert torch.equal(dk, before[0]) and torch.equal(dv, before[1])
    assert bool((out == 5.0).all())


def test_sequence_without_slots():
    """In a ragged call a sequence with kv_len 0 gets zero rows and LSE -inf; its neighbours are exact."""
    H, Hkv, d, L = 8, 2, 128, 1
    nqs, kvls = [5, 9, 7], [300, 0, 450]
    caps = [max(kl, 1) + 3 for kl in kvls]
    bases = np.concatenate([[0], np.cumsum(caps)[:-1]]).astype(np.int64)
    g = synth.Draws(31, "cpu")
    k = host_bits(g.normal((L, Hkv, int(sum(caps)), d)))
    v = host_bits(g.normal((L, Hkv, int(sum(caps)), d)))
    q = host_bits(g.normal((L, sum(nqs), H, d)))
    q_pos = np.concatenate([np.arange(max(kl - n, 0), max(kl - n, 0) + n) for n, kl in zip(nqs, kvls)]).astype(
        np.int32)
    cu = np.concatenate([[0], np.cumsum(nqs)]).astype(np.int32)
    out = torch.full((L, sum(nqs), H, d), 7.0, dtype=torch.bfloat16, device="cuda")
    lse = torch.zeros(L, sum(nqs), H, dtype=torch.float32, device="cuda")
    pkv.suffix_attention(dev(q), dev(k), dev(v), out, torch.from_numpy(q_pos).cuda(),
                         torch.tensor(kvls, dtype=torch.int32, device="cuda"), 1 / np.sqrt(d), max_kv_len=max(kvls),
                         n_seqs=3, cu_q=torch.from_numpy(cu).cuda(), kv_base=torch.from_numpy(bases).cuda(),
                         max_q=max(nqs), lse_out=lse)
    torch.cuda.synchronize()
    got, lse = host_bits(out), lse.cpu().numpy()
    empty = slice(cu[1], cu[2])
    assert np.all(bits_to_f64(got[:, empty]) == 0) and np.all(np.isneginf(lse[:, empty]))
    for s in (0, 2):
        rows = slice(cu[s], cu[s + 1])
        ks = slice(bases[s], bases[s] + caps[s])
        want, _ = oracle.attention(np.ascontiguousarray(q[0, rows]), np.ascontiguousarray(k[0][:, ks]),
                                   np.ascontiguousarray(v[0][:, ks]), q_pos[rows], kvls[s], 1 / np.sqrt(d))
        check_attention_close(got[0, rows], want)


@pytest.mark.parametrize("splits,window,d", [(0, 0, 64), (0, 150, 64), (5, 150, 64), (0, 0, 128), (3, 150, 128)])
def test_fp32_ragged_split(splits, window, d):
    """fp32 attention over ragged sequences, split over the keys (0: the planner's count) with and
    without a sliding window, at fp32 tolerance against the oracle; both head sizes of the fp32
    kernel."""
    H, Hkv, L = 4, 2, 2
    nqs, kvls = [7, 16, 3], [530, 300, 700]
    caps = [kl + 5 for kl in kvls]
    bases = np.concatenate([[0], np.cumsum(caps)[:-1]]).astype(np.int64)
    g = synth.Draws(40 + splits + window + d, "cpu")
    k = g.normal((L, Hkv, int(sum(caps)), d), torch.float32).numpy()
    v = g.normal((L, Hkv, int(sum(caps)), d), torch.float32).numpy()
    q = g.normal((L, sum(nqs), H, d), torch.float32).numpy()
    q_pos = np.concatenate([np.arange(kl - n, kl) for n, kl in zip(nqs, kvls)]).astype(np.int32)
    cu = np.concatenate([[0], np.cumsum(nqs)]).astype(np.int32)
    out = torch.zeros(L, sum(nqs), H, d, dtype=torch.float32, device="cuda")
    lse = torch.zeros(L, sum(nqs), H, dtype=torch.float32, device="cuda")
    log("fp32 ragged, splits %d, window %d, d %d" % (splits, window, d))
    pkv.suffix_attention(torch.from_numpy(q).cuda(), torch.from_numpy(k).cuda(), torch.from_numpy(v).cuda(), out,
                         torch.from_numpy(q_pos).cuda(), torch.tensor(kvls, dtype=torch.int32, device="cuda"),
                         1 / np.sqrt(d), max_kv_len=max(kvls), n_seqs=3, cu_q=torch.from_numpy(cu).cuda(),
                         kv_base=torch.from_numpy(bases).cuda(), max_q=max(nqs), n_splits=splits, lse_out=lse,
                         window=window)
    torch.cuda.synchronize()
    got, lse = out.cpu().numpy().astype(np.float64), lse.cpu().numpy()
    for l in range(L):
        for s in range(3):
            rows = slice(cu[s], cu[s + 1])
            ks = slice(bases[s], bases[s] + caps[s])
            want, want_lse = oracle.attention(np.ascontiguousarray(q[l, rows]), np.ascontiguousarray(k[l][:, ks]),
                                              np.ascontiguousarray(v[l][:, ks]), q_pos[rows], kvls[s],
                                              1 / np.sqrt(d), window=window)
            assert np.abs(got[l, rows] - want).max() <= 1e-5
            np.testing.assert_allclose(lse[l, rows], want_lse, rtol=1e-5, atol=1e-5)


@pytest.mark.parametrize("scale", [0.0, -1 / 192 ** 0.5])
def test_mla_zero_and_negative_scale(scale):
    """Absorbed MLA attention with scale 0 (every visible slot weighs the same: the mean of the
    visible latent rows) and a negative scale, one pass and split, against the oracle."""
    L, H, n_q, kv = 2, 16, 7, 500
    g = synth.Draws(41, "cpu")
    q = host_bits(g.normal((L, n_q, H, 576)))
    rows = host_bits(g.normal((L, 1, kv, 576)))
    q_pos = np.array([0, 3, 31, 32, 250, 498, 499], np.int32)
    for splits in (1, 3):
        out = torch.zeros(L, n_q, H, 512, dtype=torch.bfloat16, device="cuda")
        rd = dev(rows)
        pkv.suffix_attention(dev(q), rd, rd[..., :512], out, torch.from_numpy(q_pos).cuda(),
                             torch.tensor([kv], dtype=torch.int32, device="cuda"), scale, max_kv_len=kv,
                             variant=pkv.PKV_ATTN_MLA, n_splits=splits)
        torch.cuda.synchronize()
        got = host_bits(out)
        for l in range(L):
            want, _ = oracle.attention(q[l], rows[l], rows[l][..., :512], q_pos, kv, scale)
            log("  mla scale %g splits %d layer %d" % (scale, splits, l), check_attention_close(got[l], want))


def test_mla_score_spike_reruns_the_key_range():
    """A latent row whose k_pe (32x one row's q_pe) puts that row's score about 200 (log2 units) above
    every score before it, past the fp32 range of a probability taken against the earlier maximum:
    the workgroup must run its key range a second time with exact maxima.  The row returns that
    slot's latent and the other rows still match the oracle."""
    L, H, n_q, kv = 1, 16, 8, 900
    g = synth.Draws(42, "cpu")
    q = g.normal((L, n_q, H, 576))
    rows = g.normal((L, 1, kv, 576))
    rows[0, 0, 700, 512:] = (q[0, 5, 7, 512:].float() * 32).to(torch.bfloat16)
    qh, rh = host_bits(q), host_bits(rows)
    q_pos = np.arange(kv - n_q, kv, dtype=np.int32)
    scale = 1 / 192 ** 0.5
    for splits in (1, 2):
        out = torch.zeros(L, n_q, H, 512, dtype=torch.bfloat16, device="cuda")
        rd = rows.cuda()
        pkv.suffix_attention(q.cuda(), rd, rd[..., :512], out, torch.from_numpy(q_pos).cuda(),
                             torch.tensor([kv], dtype=torch.int32, device="cuda"), scale, max_kv_len=kv,
                             variant=pkv.PKV_ATTN_MLA, n_splits=splits)
        torch.cuda.synchronize()
        got = host_bits(out)
        want, _ = oracle.attention(qh[0], rh[0], rh[0][..., :512], q_pos, kv, scale)
        log("  spike splits %d" % splits, check_attention_close(got[0], want))
        np.testing.assert_allclose(bits_to_f64(got[0, 5, 7]), bits_to_f64(rh[0, 0, 700, :512]), atol=3e-2)


def test_more_sequences_than_one_combine_grid():
    """65,537 one-query sequences split over the keys: the split merge runs as two grids (at most
    65,535 sequences each); sequences on both sides of the boundary match the oracle."""
    n_seqs, kv, H, Hkv, d = 65537, 128, 2, 1, 64
    g = synth.Draws(61, "cuda")
    k = g.normal((1, Hkv, n_seqs * kv, d))
    v = g.normal((1, Hkv, n_seqs * kv, d))
    q = g.normal((1, n_seqs, H, d))
    out = torch.zeros(1, n_seqs, H, d, dtype=torch.bfloat16, device="cuda")
    q_pos = torch.full((n_seqs,), kv - 1, dtype=torch.int32, device="cuda")
    kv_len = torch.full((n_seqs,), kv, dtype=torch.int32, device="cuda")
    cu = torch.arange(n_seqs + 1, dtype=torch.int32, device="cuda")
    base = torch.arange(n_seqs, dtype=torch.int64, device="cuda") * kv
    log("65537 sequences, 2 splits")
    pkv.suffix_attention(q, k, v, out, q_pos, kv_len, d ** -0.5, max_kv_len=kv, n_seqs=n_seqs, cu_q=cu,
                         kv_base=base, max_q=1, n_splits=2)
    torch.cuda.synchronize()
    for s in (0, 1, 65534, 65535, 65536):
        ks = slice(s * kv, (s + 1) * kv)
        want, _ = oracle.attention(host_bits(q[0, s: s + 1]), host_bits(k[0, :, ks]), host_bits(v[0, :, ks]),
                                   np.array([kv - 1], dtype=np.int32), kv, d ** -0.5)
        check_attention_close(host_bits(out[0, s: s + 1]), want)


EXTREME_POS = np.array([2 ** 31 - 1, 2 ** 31 - 40, -2 ** 31, -1, 0, 1, 31, 32, 299, 300, 301, 5000], np.int32)


@pytest.mark.parametrize("variant,dtype,d,window", [
    ("gqa", "bf16", 128, 0), ("gqa", "bf16", 128, 1), ("gqa", "bf16", 64, 37), ("gqa", "bf16", 128, 2 ** 31 - 1),
    ("gqa", "f32", 64, 0), ("gqa", "f32", 128, 37), ("mla", "bf16", 576, 0), ("mla", "bf16", 576, 2 ** 31 - 40)])
def test_extreme_positions(variant, dtype, d, window):
    """Query positions at both ends of the int32 range (far past the cache, before it) and windows up
    to 2^31 - 1: each row sees exactly the slots the contract names (j < kv_len, j <= q_pos,
    j > q_pos - window), in one pass and split, against the oracle.  (The oracle forms the bounds in
    64-bit integers; q_pos + 1 and q_pos - window + 1 overflow int32 at these values.)"""
    L, kv, n_q = 1, 300, EXTREME_POS.size
    H, Hkv = (16, 1) if variant == "mla" else (8, 2)
    dv = 512 if variant == "mla" else d
    g = synth.Draws(43 + d + (window % 1000), "cpu")
    tdt = torch.float32 if dtype == "f32" else torch.bfloat16
    q = g.normal((L, n_q, H, d), tdt)
    k = g.normal((L, Hkv, kv + 4, d), tdt)
    v = k[..., :512] if variant == "mla" else g.normal((L, Hkv, kv + 4, d), tdt)
    scale = 1 / np.sqrt(192.0 if variant == "mla" else d)
    host = (lambda t: t.numpy().astype(np.float64)) if dtype == "f32" else host_bits
    qh, kh = host(q), host(k)
    vh = kh[..., :512] if variant == "mla" else host(v)
    for splits in (1, 3):
        out = torch.zeros(L, n_q, H, dv, dtype=tdt, device="cuda")
        lse = torch.zeros(L, n_q, H, dtype=torch.float32, device="cuda")
        kd = k.cuda()
        vd = kd[..., :512] if variant == "mla" else v.cuda()
        log("extreme positions: %s %s d %d window %d splits %d" % (variant, dtype, d, window, splits))
        pkv.suffix_attention(q.cuda(), kd, vd, out, torch.from_numpy(EXTREME_POS).cuda(),
                             torch.tensor([kv], dtype=torch.int32, device="cuda"), scale, max_kv_len=kv,
                             variant=pkv.PKV_ATTN_MLA if variant == "mla" else pkv.PKV_ATTN_GQA, n_splits=splits,
                             lse_out=lse, window=window)
        torch.cuda.synchronize()
        if dtype == "f32":
            want, want_lse = oracle.attention(q[0].numpy(), k[0].numpy(), v[0].contiguous().numpy(), EXTREME_POS, kv,
                                              scale, window=window)
            assert np.abs(out[0].cpu().numpy() - want).max() <= 1e-5
        else:
            want, want_lse = oracle.attention(qh[0], kh[0], np.ascontiguousarray(vh[0]), EXTREME_POS, kv, scale,
                                              window=window)
            check_attention_close(host_bits(out)[0], want)
        got_lse = lse[0].cpu().numpy()
        empty = np.isneginf(want_lse)
        assert np.array_equal(np.isneginf(got_lse), empty)
        np.testing.assert_allclose(got_lse[~empty], want_lse[~empty], rtol=1e-4, atol=1e-4)
