"""GPU parity of pkv_reposition_splice / pkv_reposition_splice_batched against
the fp64 oracle (paper Sec. 5 compose path; Sec. 8 MLA adapter).

Bar: V, the MLA latent, non-rotary channels and untouched slots bit-exact;
re-rotated bf16 keys within one bf16 ulp (floor 2^-12 of the pair norm for
values that cancel to near zero); fp32 keys within 1e-6 relative per pair."""
import numpy as np
import pytest
import torch

import oracle
from helpers import (bits_to_f64, check_rotated_keys, dev, host_bits, log, rope_cache, small_workload)
from paper_2606_17107_amd import pkv, synth

pytestmark = pytest.mark.gpu

SENTINEL = 0x7fa5


def run_gpu_splice(w, skill_k, skill_v, ctx_k, ctx_v, src_pos, dst_pos, err_flag=None):
    """Upload, splice on the GPU, return host copies of dst K / V."""
    dk, dv = dev(ctx_k), (dev(ctx_v) if ctx_v is not None else None)
    sk, sv = dev(skill_k), (dev(skill_v) if skill_v is not None else None)
    sp = torch.from_numpy(src_pos.astype(np.int32)).cuda()
    dp = torch.from_numpy(dst_pos.astype(np.int32)).cuda()
    pkv.reposition_splice(sk, sv, dk, dv, sp, dp, w.theta, w.rope_dim, w.rope_offset, w.rope_style,
                          err_flag=err_flag)
    torch.cuda.synchronize()
    return host_bits(dk), (host_bits(dv) if dv is not None else None)


def oracle_splice(w, skill_k, skill_v, ctx_k, ctx_v, src_pos, dst_pos):
    ok, ov = ctx_k.copy(), (ctx_v.copy() if ctx_v is not None else None)
    oracle.reposition_splice(skill_k, skill_v, ok, ov, src_pos, dst_pos, w.theta, w.rope_dim, w.rope_offset,
                             w.rope_style)
    return ok, ov


def compare(w, got_k, got_v, want_k, want_v):
    if want_v is not None:
        np.testing.assert_array_equal(got_v, want_v)
    if w.dtype == "f32":
        assert np.array_equal(got_k.view(np.uint32)[..., : w.rope_offset], want_k.view(np.uint32)[..., : w.rope_offset])
        g, o = got_k.astype(np.float64), want_k.astype(np.float64)
        # per-pair relative error (HALF pairing over the full row)
        h = w.rope_dim // 2
        sl = slice(w.rope_offset, w.rope_offset + w.rope_dim)
        gg, oo = g[..., sl], o[..., sl]
        if w.rope_style == synth.HALF:
            num = np.hypot(gg[..., :h] - oo[..., :h], gg[..., h:] - oo[..., h:])
            den = np.hypot(oo[..., :h], oo[..., h:])
        else:
            num = np.hypot(gg[..., 0::2] - oo[..., 0::2], gg[..., 1::2] - oo[..., 1::2])
            den = np.hypot(oo[..., 0::2], oo[..., 1::2])
        rel = num / np.maximum(den, 1e-30)
        assert rel.max() <= 1e-6, rel.max()
        return 0, 0
    return check_rotated_keys(got_k, want_k, w.rope_offset, w.rope_dim, w.rope_style)


def build_inputs(w, seed=0, layers=None, device="cpu", rope_skill=True):
    """Host bit arrays for a single-sequence splice of workload w."""
    c = synth.gqa_case(w, seed=seed, device=device, layers=layers)
    ctx_k = host_bits(c["ctx_k"])
    ctx_v = host_bits(c["ctx_v"]) if "ctx_v" in c else None
    src = c["src_pos"].numpy()
    dst = c["dst_pos"].numpy()
    k_pre = host_bits(c["skill_k_pre"])
    skill_k = rope_cache(k_pre, src[None, None, :], w) if rope_skill else k_pre
    skill_v = host_bits(c["skill_v"]) if "skill_v" in c else None
    return dict(ctx_k=ctx_k, ctx_v=ctx_v, skill_k=skill_k, skill_v=skill_v, src=src, dst=dst, k_pre=k_pre)


def test_tiny_fp32_config():
    """The tiny fp32 reference: 128-token skill RoPE'd at 0..127 moved to 300..427 of 528 slots."""
    w = synth.TINY
    x = build_inputs(w)
    log("tiny fp32 splice", w)
    gk, gv = run_gpu_splice(w, x["skill_k"], x["skill_v"], x["ctx_k"], x["ctx_v"], x["src"], x["dst"])
    ok, ov = oracle_splice(w, x["skill_k"], x["skill_v"], x["ctx_k"], x["ctx_v"], x["src"], x["dst"])
    compare(w, gk, gv, ok, ov)
    # untouched slots bit-exact, spliced slots equal RoPE(k, dst) within 1e-5 relative
    mask = np.ones(w.kv_len, bool)
    mask[x["dst"]] = False
    np.testing.assert_array_equal(gk[:, :, mask], x["ctx_k"][:, :, mask])
    direct = rope_cache(x["k_pre"], x["dst"][None, None, :], w)
    got = gk[:, :, x["dst"]].astype(np.float64)
    rel = np.linalg.norm(got - direct, axis=-1) / np.linalg.norm(direct, axis=-1)
    assert rel.max() <= 1e-5


CASES = [
    dict(d=128, style=0, rope_dim=128, rope_offset=0, skill=200, L=3, Hkv=2, theta=5e5),
    dict(d=128, style=1, rope_dim=128, rope_offset=0, skill=200, L=3, Hkv=2, theta=5e5),
    dict(d=64, style=0, rope_dim=64, rope_offset=0, skill=77, L=2, Hkv=5, theta=1e4),
    dict(d=128, style=0, rope_dim=64, rope_offset=32, skill=130, L=2, Hkv=3, theta=1e6),
    dict(d=128, style=1, rope_dim=32, rope_offset=96, skill=33, L=4, Hkv=1, theta=1e4),
    # head size 256: 128 rotary pairs (the most a row may rotate; more pairs than lanes in a wave, so
    # every wave forms its own coefficients), and a partial interleaved slice
    dict(d=256, style=0, rope_dim=256, rope_offset=0, skill=70, L=2, Hkv=2, theta=1e4),
    dict(d=256, style=1, rope_dim=128, rope_offset=64, skill=45, L=2, Hkv=2, theta=1e6),
]


@pytest.mark.parametrize("case", CASES, ids=lambda c: "d%d_s%d_r%d_o%d" % (c["d"], c["style"], c["rope_dim"],
                                                                          c["rope_offset"]))
def test_small_bf16(case):
    w = small_workload(L=case["L"], H=case["Hkv"] * 2, Hkv=case["Hkv"], d=case["d"], theta=case["theta"],
                       style=case["style"], skill=case["skill"], dst0=1000, ctx=1300, n_q=5,
                       rope_dim=case["rope_dim"], rope_offset=case["rope_offset"])
    w = synth.Workload(w.name, w.n_layers, w.n_heads, w.n_kv_heads, w.head_dim, w.v_dim, w.theta, w.rope_dim,
                       w.rope_offset, w.rope_style, w.dtype, w.skill_tokens, 11, 1000, w.ctx_slots, w.n_q,
                       w.scale)
    x = build_inputs(w, seed=3)
    log("small bf16 splice", case)
    gk, gv = run_gpu_splice(w, x["skill_k"], x["skill_v"], x["ctx_k"], x["ctx_v"], x["src"], x["dst"])
    ok, ov = oracle_splice(w, x["skill_k"], x["skill_v"], x["ctx_k"], x["ctx_v"], x["src"], x["dst"])
    n_diff, n_floor = compare(w, gk, gv, ok, ov)
    log("  elements not bit-equal:", n_diff, "needing the floor:", n_floor)


@pytest.mark.parametrize("style", [0, 1])
@pytest.mark.parametrize("d,v_dim,rope_dim,rope_offset", [(128, 128, 128, 0), (576, 0, 64, 512)])
def test_scattered_positions(style, d, v_dim, rope_dim, rope_offset):
    """Per-token source and destination positions with no common delta (every wave takes the per-lane
    coefficient path), destinations a random permutation of a larger cache, token count not a tile multiple."""
    n, cap, L, Hkv = 333, 1500, 2, (2 if v_dim else 1)
    rng = np.random.default_rng(11 + style)
    g = synth.Draws(12, "cpu")
    skill_k = host_bits(g.normal((L, Hkv, n, d)))
    skill_v = host_bits(g.normal((L, Hkv, n, v_dim))) if v_dim else None
    ctx_k = host_bits(g.normal((L, Hkv, cap, d)))
    ctx_v = host_bits(g.normal((L, Hkv, cap, v_dim))) if v_dim else None
    src = rng.integers(-40000, 40000, n).astype(np.int32)
    dst = rng.permutation(cap)[:n].astype(np.int32)
    w = synth.Workload("scatter", L, Hkv, Hkv, d, v_dim, 5e5, rope_dim, rope_offset, style, "bf16", n, 0, 0, cap,
                       1, 1.0, mla=not v_dim)
    log("scattered positions", dict(style=style, d=d, rope_dim=rope_dim))
    gk, gv = run_gpu_splice(w, skill_k, skill_v, ctx_k, ctx_v, src, dst)
    ok, ov = oracle_splice(w, skill_k, skill_v, ctx_k, ctx_v, src, dst)
    if ov is not None:
        np.testing.assert_array_equal(gv, ov)
    np.testing.assert_array_equal(gk[..., :rope_offset], ok[..., :rope_offset])
    compare(w, gk, gv, ok, ov)


@pytest.mark.parametrize("d", [64, 256])
def test_scattered_positions_fp32(d):
    n, cap, L, Hkv = 200, 700, 1, 2
    rng = np.random.default_rng(5)
    g = synth.Draws(13, "cpu")
    skill_k = g.normal((L, Hkv, n, d), torch.float32).numpy()
    skill_v = g.normal((L, Hkv, n, d), torch.float32).numpy()
    ctx_k = g.normal((L, Hkv, cap, d), torch.float32).numpy()
    ctx_v = g.normal((L, Hkv, cap, d), torch.float32).numpy()
    src = rng.integers(0, 20000, n).astype(np.int32)
    dst = rng.permutation(cap)[:n].astype(np.int32)
    w = synth.Workload("scatter32", L, Hkv, Hkv, d, d, 1e4, d, 0, synth.HALF, "f32", n, 0, 0, cap, 1, 1.0)
    gk, gv = run_gpu_splice(w, skill_k, skill_v, ctx_k, ctx_v, src, dst)
    ok, ov = oracle_splice(w, skill_k, skill_v, ctx_k, ctx_v, src, dst)
    np.testing.assert_array_equal(gv.view(np.uint32), ov.view(np.uint32))
    compare(w, gk, gv, ok, ov)


def test_mla_rows_small():
    w = synth.Workload("mla_small", 3, 16, 1, 576, 512, 1e4, 64, 512, synth.INTERLEAVED, "bf16", 150, 0, 900,
                       1200, 4, 1 / 192 ** 0.5, mla=True)
    x = build_inputs(w, seed=4)
    gk, _ = run_gpu_splice(w, x["skill_k"], None, x["ctx_k"], None, x["src"], x["dst"])
    ok, _ = oracle_splice(w, x["skill_k"], None, x["ctx_k"], None, x["src"], x["dst"])
    np.testing.assert_array_equal(gk[..., :512], ok[..., :512])
    compare(w, gk, None, ok, None)


def test_token_major_strides():
    """[L][slot][H][d] caches (token-major) through the same entry point."""
    w = small_workload(L=2, H=8, Hkv=4, d=128, theta=5e5, skill=90, dst0=10, ctx=300, n_q=3)
    x = build_inputs(w, seed=5)
    sk = dev(np.ascontiguousarray(x["skill_k"].transpose(0, 2, 1, 3))).permute(0, 2, 1, 3)
    sv = dev(np.ascontiguousarray(x["skill_v"].transpose(0, 2, 1, 3))).permute(0, 2, 1, 3)
    dk = dev(np.ascontiguousarray(x["ctx_k"].transpose(0, 2, 1, 3))).permute(0, 2, 1, 3)
    dv = dev(np.ascontiguousarray(x["ctx_v"].transpose(0, 2, 1, 3))).permute(0, 2, 1, 3)
    pkv.reposition_splice(sk, sv, dk, dv, torch.from_numpy(x["src"]).cuda(), torch.from_numpy(x["dst"]).cuda(),
                          w.theta, w.rope_dim)
    torch.cuda.synchronize()
    gk = host_bits(dk.permute(0, 2, 1, 3).contiguous()).transpose(0, 2, 1, 3)
    gv = host_bits(dv.permute(0, 2, 1, 3).contiguous()).transpose(0, 2, 1, 3)
    ok, ov = oracle_splice(w, x["skill_k"], x["skill_v"], x["ctx_k"], x["ctx_v"], x["src"], x["dst"])
    compare(w, np.ascontiguousarray(gk), np.ascontiguousarray(gv), ok, ov)


def test_inplace_rope_and_delta_zero():
    """In place with dst_pos[t] == t: rotating pre-RoPE keys by their positions is RoPE; delta 0 is the
    identity bit-exact."""
    w = small_workload(L=2, H=4, Hkv=2, d=128, theta=5e5, skill=300)
    g = synth.Draws(6, "cpu")
    k = host_bits(g.normal((2, 2, 300, 128)))
    t = dev(k)
    zero = torch.zeros(300, dtype=torch.int32, device="cuda")
    pos = torch.arange(300, dtype=torch.int32, device="cuda")
    pkv.reposition_splice(t, None, t, None, pos, pos, w.theta, 128)        # delta 0
    torch.cuda.synchronize()
    np.testing.assert_array_equal(host_bits(t), k)
    pkv.reposition_splice(t, None, t, None, zero, pos, w.theta, 128)       # RoPE at 0..299 in place
    torch.cuda.synchronize()
    want = oracle.rope_rows(k, np.broadcast_to(np.arange(300, dtype=np.int32), (2, 2, 300)), w.theta, 128)
    check_rotated_keys(host_bits(t), want, 0, 128, 0)


def test_round_trip_and_determinism():
    w = small_workload(L=2, H=4, Hkv=2, d=128, theta=5e5, skill=256)
    g = synth.Draws(7, "cpu")
    k = dev(host_bits(g.normal((2, 2, 256, 128))))
    mid = torch.zeros(2, 2, 20256, 128, dtype=torch.bfloat16, device="cuda")
    back = torch.zeros_like(k)
    pos = torch.arange(256, dtype=torch.int32, device="cuda")
    pkv.reposition_splice(k, None, mid, None, pos, pos + 20000, w.theta, 128)
    mid2 = mid[:, :, 20000:].contiguous()
    pkv.reposition_splice(mid2, None, back, None, pos + 20000, pos, w.theta, 128)
    again = torch.zeros_like(mid)
    pkv.reposition_splice(k, None, again, None, pos, pos + 20000, w.theta, 128)
    torch.cuda.synchronize()
    assert torch.equal(mid.view(torch.int16), again.view(torch.int16))
    a, b = bits_to_f64(host_bits(back)), bits_to_f64(host_bits(k))
    err = np.linalg.norm(a - b, axis=-1) / np.linalg.norm(b, axis=-1)
    assert err.max() < 2 * 2.0 ** -8
    assert not torch.equal(mid2.view(torch.int16), k.view(torch.int16))


def test_out_of_range_destinations_flagged():
    w = small_workload(L=2, H=4, Hkv=2, d=64, theta=1e4, skill=6)
    g = synth.Draws(8, "cpu")
    sk = dev(host_bits(g.normal((2, 2, 6, 64))))
    sv = dev(host_bits(g.normal((2, 2, 6, 64))))
    dk = torch.full((2, 2, 10, 64), SENTINEL, dtype=torch.int16, device="cuda").view(torch.bfloat16)
    dv = torch.full((2, 2, 10, 64), SENTINEL, dtype=torch.int16, device="cuda").view(torch.bfloat16)
    flag = torch.zeros(1, dtype=torch.int32, device="cuda")
    src = torch.arange(6, dtype=torch.int32, device="cuda")
    dst = torch.tensor([0, -1, 9, 10, 5, 2 ** 30], dtype=torch.int32, device="cuda")
    pkv.reposition_splice(sk, sv, dk, dv, src, dst, w.theta, 64, err_flag=flag)
    torch.cuda.synchronize()
    assert int(flag.item()) == 1
    hk = host_bits(dk)
    assert np.all(hk[:, :, [1, 2, 3, 4, 6, 7, 8]] == SENTINEL)
    assert not np.any(hk[:, :, [0, 5, 9]] == SENTINEL)
    flag.zero_()
    pkv.reposition_splice(sk, sv, dk, dv, src, torch.arange(6, dtype=torch.int32, device="cuda"), w.theta, 64,
                          err_flag=flag)
    torch.cuda.synchronize()
    assert int(flag.item()) == 0


def batched_small_plan():
    bw = synth.BatchedWorkload(n_seqs=3, skills=(40, 100, 257), ctx_min=600, ctx_max=900, src_pos_max=300,
                               n_layers=2, n_heads=8, n_kv_heads=2, head_dim=128, n_q=19)
    return bw, synth.batched_plan(bw, seed=1)


def run_batched(bw, plan, case, segs, max_tok):
    sk, sv = dev(case["skill_k"]), dev(case["skill_v"])
    dk, dv = dev(case["ctx_k"]), dev(case["ctx_v"])
    segs_dev = pkv.make_segments(segs, "cuda")
    flag = torch.zeros(1, dtype=torch.int32, device="cuda")
    pkv.reposition_splice_batched(sk, sv, dk, dv, segs_dev, len(segs), max_tok, bw.theta, bw.head_dim,
                                  err_flag=flag)
    torch.cuda.synchronize()
    return host_bits(dk), host_bits(dv), int(flag.item())


def oracle_batched(bw, plan, case, segs):
    ok, ov = case["ctx_k"].copy(), case["ctx_v"].copy()
    for s in segs:
        n = s["n_tokens"]
        src_sl = slice(s["src_slot0"], s["src_slot0"] + n)
        base = s["dst_seq_base"]
        # the destination sequence viewed on its own slot axis
        seq_k = ok[:, :, base: base + s["dst_seq_len"]]
        seq_v = ov[:, :, base: base + s["dst_seq_len"]]
        oracle.reposition_splice(np.ascontiguousarray(case["skill_k"][:, :, src_sl]),
                                 np.ascontiguousarray(case["skill_v"][:, :, src_sl]), seq_k, seq_v,
                                 np.arange(s["src_pos0"], s["src_pos0"] + n, dtype=np.int32),
                                 np.arange(s["dst_pos0"], s["dst_pos0"] + n, dtype=np.int32), bw.theta,
                                 bw.head_dim)
    return ok, ov


def segments_of(plan):
    segs = []
    for sq in plan["seqs"]:
        for sg in sq["segs"]:
            segs.append(dict(src_slot0=sg["src_slot0"], dst_seq_base=sq["seq_base"], n_tokens=sg["n_tokens"],
                             src_pos0=sg["src_pos0"], dst_pos0=sg["dst_pos0"], dst_seq_len=sq["kv_len"]))
    return segs


def batched_inputs(bw, plan, seed=0, device="cpu", layers=None):
    c = synth.batched_case(bw, plan, seed=seed, device=device, layers=layers)
    return dict(ctx_k=host_bits(c["ctx_k"]), ctx_v=host_bits(c["ctx_v"]), skill_k=host_bits(c["skill_k_pre"]),
                skill_v=host_bits(c["skill_v"]))


def test_batched_segments_small():
    bw, plan = batched_small_plan()
    case = batched_inputs(bw, plan, seed=2)
    segs = segments_of(plan)
    gk, gv, flag = run_batched(bw, plan, case, segs, max(s["n_tokens"] for s in segs))
    assert flag == 0
    ok, ov = oracle_batched(bw, plan, case, segs)
    np.testing.assert_array_equal(gv, ov)
    check_rotated_keys(gk, ok, 0, bw.head_dim, 0)


def test_batched_out_of_range_segment_flagged():
    bw, plan = batched_small_plan()
    case = batched_inputs(bw, plan, seed=2)
    segs = segments_of(plan)[:2]
    bad = dict(segs[0])
    bad["dst_pos0"] = bad["dst_seq_len"] - 5        # runs past the end of its sequence
    segs = segs + [bad]
    gk, gv, flag = run_batched(bw, plan, case, segs, max(s["n_tokens"] for s in segs))
    assert flag == 1
    # the in-range tokens of the bad segment were written, the rest skipped
    ok, ov = case["ctx_k"].copy(), case["ctx_v"].copy()
    good = segs[:2] + [dict(bad, n_tokens=5)]
    ok, ov = oracle_batched(bw, plan, dict(case, ctx_k=ok, ctx_v=ov), good)
    np.testing.assert_array_equal(gv, ov)
    check_rotated_keys(gk, ok, 0, bw.head_dim, 0)


def test_batched_long_segments_whole_rows_per_xcd():
    """8 (layer, head) rows (the launch then gives each XCD whole rows) and segments long enough that a
    block walks five tiles of 16 tokens (two batches of up to four in-flight tiles); three sequences
    share each skill."""
    bw = synth.BatchedWorkload(n_seqs=3, skills=(40, 700, 2100), ctx_min=3000, ctx_max=3400, src_pos_max=300,
                               n_layers=4, n_heads=8, n_kv_heads=2, head_dim=128, n_q=19)
    plan = synth.batched_plan(bw, seed=4)
    case = batched_inputs(bw, plan, seed=5)
    segs = segments_of(plan)
    gk, gv, flag = run_batched(bw, plan, case, segs, max(s["n_tokens"] for s in segs))
    assert flag == 0
    ok, ov = oracle_batched(bw, plan, case, segs)
    np.testing.assert_array_equal(gv, ov)
    check_rotated_keys(gk, ok, 0, bw.head_dim, 0)


def test_batched_source_out_of_range():
    """A segment whose source slots lie past the end of the source tensor writes nothing and sets the
    flag; a segment straddling the end writes only its in-range tokens."""
    bw = synth.BatchedWorkload(n_seqs=3, skills=(40, 100, 257), ctx_min=600, ctx_max=900, src_pos_max=300,
                               n_layers=4, n_heads=8, n_kv_heads=2, head_dim=128, n_q=19)
    plan = synth.batched_plan(bw, seed=1)
    case = batched_inputs(bw, plan, seed=2)
    n_src = case["skill_k"].shape[2]
    segs = segments_of(plan)[:1]
    outside = dict(segments_of(plan)[8], src_slot0=n_src + 10)
    straddle = dict(segments_of(plan)[4], src_slot0=n_src - 7)
    gk, gv, flag = run_batched(bw, plan, case, segs + [outside, straddle], 300)
    assert flag == 1
    ok, ov = oracle_batched(bw, plan, case, segs + [dict(straddle, n_tokens=7)])
    np.testing.assert_array_equal(gv, ov)
    check_rotated_keys(gk, ok, 0, bw.head_dim, 0)


# ---- full-size workloads (the launch configuration the benchmark times) -----

def full_size(w, layers=None, seed=0):
    torch.cuda.synchronize()
    c = synth.gqa_case(w, seed=seed, device="cuda")
    L = w.n_layers
    sk = c["skill_k_pre"]
    # post-RoPE skill keys: rotate the pre-RoPE draws to their source positions with the oracle
    sel = list(range(L)) if layers is None else layers
    log("full-size", w.name, "layers checked:", "all" if layers is None else sel)
    sk_host = host_bits(sk[sel])
    skill_k = rope_cache(sk_host, c["src_pos"].numpy()[None, None, :], w)
    sk[sel] = dev(skill_k)
    dk = c["ctx_k"].clone()
    dv = c["ctx_v"].clone() if "ctx_v" in c else None
    sv = c.get("skill_v")
    pkv.reposition_splice(sk, sv, dk, dv, c["src_pos"].cuda(), c["dst_pos"].cuda(), w.theta, w.rope_dim,
                          w.rope_offset, w.rope_style)
    torch.cuda.synchronize()
    ok = host_bits(c["ctx_k"][sel])
    ov = host_bits(c["ctx_v"][sel]) if dv is not None else None
    oracle.reposition_splice(skill_k, host_bits(sv[sel]) if sv is not None else None, ok, ov,
                             c["src_pos"].numpy(), c["dst_pos"].numpy(), w.theta, w.rope_dim, w.rope_offset,
                             w.rope_style)
    if dv is not None:
        np.testing.assert_array_equal(host_bits(dv[sel]), ov)
    n_diff, n_floor = check_rotated_keys(host_bits(dk[sel]), ok, w.rope_offset, w.rope_dim, w.rope_style)
    log("  K elements not bit-equal:", n_diff, "needing the floor:", n_floor)


def test_full_gqa8b():
    full_size(synth.GQA8B)


def test_full_mla():
    full_size(synth.MLA)


def test_full_long32k_sampled_layers():
    full_size(synth.LONG32K, layers=[0, 13, 27])
