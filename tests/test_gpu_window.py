"""GPU parity of sliding-window suffix attention: the cache keeps every
token's K/V and the mask alone enforces the window, slot j visible iff
q_pos - W < j <= q_pos and j < kv_len (paper Sec. 8, the sliding-window
configuration fix; Fig. "attention-variant adapters" (c)).

Same bars as the causal tests: bf16 max-abs 2e-2 / mean-abs 2e-3 / rel-L2
1e-2 (with sharpened queries so the check is not vacuous), fp32 rel-L2 1e-5."""
import numpy as np
import pytest
import torch

import oracle
from helpers import bits_to_f64, check_attention_close, dev, host_bits, log, small_workload
from paper_2606_17107_amd import pkv, synth
from test_gpu_attention import assemble_cache

pytestmark = pytest.mark.gpu


def run(w, q, k, v, q_pos, kv_len, window, n_splits=0, variant=pkv.PKV_ATTN_GQA, lse=False):
    qd, kd = dev(q), dev(k)
    vd = kd[..., : w.v_dim] if v is None else dev(v)
    L, nq, H = q.shape[:3]
    dt = torch.bfloat16 if w.dtype == "bf16" else torch.float32
    out = torch.zeros(L, nq, H, w.v_dim, dtype=dt, device="cuda")
    lse_t = torch.zeros(L, nq, H, dtype=torch.float32, device="cuda") if lse else None
    pkv.suffix_attention(qd, kd, vd, out, torch.from_numpy(q_pos.astype(np.int32)).cuda(),
                         torch.tensor([kv_len], dtype=torch.int32, device="cuda"), w.scale, max_kv_len=kv_len,
                         variant=variant, n_splits=n_splits, lse_out=lse_t, window=window)
    torch.cuda.synchronize()
    return (host_bits(out), lse_t.cpu().numpy()) if lse else host_bits(out)


def want(w, q, k, v, q_pos, kv_len, window):
    outs, lses = [], []
    for l in range(q.shape[0]):
        vv = k[l][..., : w.v_dim] if v is None else v[l]
        o, s = oracle.attention(q[l], k[l], vv, q_pos, kv_len, w.scale, window=window)
        outs.append(o)
        lses.append(s)
    return np.stack(outs), np.stack(lses)


@pytest.mark.parametrize("d", [64, 128])
@pytest.mark.parametrize("window", [1, 17, 32, 100, 5000])
def test_window_gqa_bf16(d, window):
    w = small_workload(L=2, H=8, Hkv=2, d=d, theta=1e4, skill=200, dst0=30, ctx=700, n_q=45)
    c = synth.gqa_case(w, seed=7)
    q, k, v, q_pos = assemble_cache(w, c)
    q4 = synth.to_numpy_bits(synth.from_numpy_bits(q).float().mul(4).to(torch.bfloat16))
    ref, ref_lse = want(w, q4, k, v, q_pos, w.kv_len, window)
    for splits in (1, 3):
        got, lse = run(w, q4, k, v, q_pos, w.kv_len, window, n_splits=splits, lse=True)
        stats = check_attention_close(got, ref)
        np.testing.assert_allclose(lse, ref_lse, atol=2e-2)
        log("  window %d d %d splits %d" % (window, d, splits), stats)


def test_window_one_is_own_value_row():
    """W = 1: each query sees only its own slot, so the output is that slot's value row."""
    w = small_workload(L=1, H=8, Hkv=2, d=128, theta=1e4, skill=100, dst0=10, ctx=300, n_q=20)
    c = synth.gqa_case(w, seed=8)
    q, k, v, q_pos = assemble_cache(w, c)
    got = bits_to_f64(run(w, q, k, v, q_pos, w.kv_len, 1))
    vv = bits_to_f64(v[0])[np.repeat(np.arange(2), 4)][:, q_pos].transpose(1, 0, 2)   # [n_q][H][d]
    np.testing.assert_allclose(got[0], vv, atol=1e-6)


def test_window_mla():
    w = synth.Workload("mla_small", 2, 16, 1, 576, 512, 1e4, 64, 512, synth.INTERLEAVED, "bf16", 150, 0, 100,
                       500, 12, 1 / 192 ** 0.5, mla=True)
    c = synth.gqa_case(w, seed=9)
    q, k, _, q_pos = assemble_cache(w, c)
    for window in (20, 200):
        ref, _ = want(w, q, k, None, q_pos, w.kv_len, window)
        for splits in (1, 2):
            got = run(w, q, k, None, q_pos, w.kv_len, window, n_splits=splits, variant=pkv.PKV_ATTN_MLA)
            log("  mla window %d splits %d" % (window, splits), check_attention_close(got, ref))


@pytest.mark.parametrize("window", [1, 50, 600])
def test_window_fp32(window):
    w = synth.TINY
    c = synth.gqa_case(w, seed=0)
    q, k, v, q_pos = assemble_cache(w, c)
    got = run(w, q, k, v, q_pos, w.kv_len, window)
    ref, _ = want(w, q, k, v, q_pos, w.kv_len, window)
    rl2 = np.linalg.norm(got - ref) / np.linalg.norm(ref)
    assert rl2 <= 1e-5, rl2


def test_window_full_size_gqa8b_sampled():
    """The Llama-3-8B-shaped workload (32 layers, 32/8 heads, 8256 slots, 64 queries) with a 4096-token
    window, as a sliding-window layer of a Gemma-style model would see it: layers 0 and 31 checked."""
    w = synth.GQA8B
    c = synth.gqa_case(w, seed=0, device="cuda")
    layers = [0, 31]
    # oracle-built inputs for the checked layers, device draws elsewhere
    sub = {k: v[layers].cpu() for k, v in c.items() if k in ("ctx_k", "ctx_v", "skill_k_pre", "skill_v", "q_pre",
                                                            "suf_k_pre", "suf_v")}
    sub.update({k: c[k] for k in ("src_pos", "dst_pos", "q_pos")})
    wl = synth.Workload(w.name, len(layers), w.n_heads, w.n_kv_heads, w.head_dim, w.v_dim, w.theta, w.rope_dim,
                        w.rope_offset, w.rope_style, w.dtype, w.skill_tokens, w.src_pos0, w.dst_pos0, w.ctx_slots,
                        w.n_q, w.scale)
    q, k, v, q_pos = assemble_cache(wl, sub)
    qd = c["q_pre"].clone()
    kd, vd = c["ctx_k"].clone(), c["ctx_v"].clone()
    for i, l in enumerate(layers):
        qd[l], kd[l], vd[l] = dev(q[i]), dev(k[i]), dev(v[i])
    out = torch.zeros(w.n_layers, w.n_q, w.n_heads, w.head_dim, dtype=torch.bfloat16, device="cuda")
    pkv.suffix_attention(qd, kd, vd, out, c["q_pos"].cuda(), torch.tensor([w.kv_len], dtype=torch.int32,
                         device="cuda"), w.scale, max_kv_len=w.kv_len, window=4096)
    torch.cuda.synchronize()
    got = host_bits(out[layers])
    ref, _ = want(wl, q, k, v, q_pos, w.kv_len, 4096)
    log("  gqa8b window 4096", check_attention_close(got, ref))


@pytest.mark.parametrize("window", [40, 300])
def test_window_ragged_sequences(window):
    """Windows over several packed sequences (per-sequence query ranges, cache bases and lengths)."""
    H, Hkv, d, L = 8, 2, 128, 2
    nqs, kvls = [17, 40, 1, 64], [300, 1000, 77, 513]
    caps = [kl + 11 for kl in kvls]
    bases = np.concatenate([[0], np.cumsum(caps)[:-1]]).astype(np.int64)
    g = synth.Draws(60, "cpu")
    k = host_bits(g.normal((L, Hkv, int(sum(caps)), d)))
    v = host_bits(g.normal((L, Hkv, int(sum(caps)), d)))
    q = host_bits(g.normal((L, sum(nqs), H, d)))
    q_pos = np.concatenate([np.arange(kl - n, kl) for n, kl in zip(nqs, kvls)]).astype(np.int32)
    cu = np.concatenate([[0], np.cumsum(nqs)]).astype(np.int32)
    scale = 1 / np.sqrt(d)
    for splits in (1, 3):
        out = torch.zeros(L, sum(nqs), H, d, dtype=torch.bfloat16, device="cuda")
        pkv.suffix_attention(dev(q), dev(k), dev(v), out, torch.from_numpy(q_pos).cuda(),
                             torch.tensor(kvls, dtype=torch.int32, device="cuda"), scale, max_kv_len=max(kvls),
                             n_seqs=len(nqs), cu_q=torch.from_numpy(cu).cuda(),
                             kv_base=torch.from_numpy(bases).cuda(), max_q=max(nqs), n_splits=splits,
                             window=window)
        torch.cuda.synchronize()
        got = host_bits(out)
        for s in range(len(nqs)):
            rows = slice(cu[s], cu[s + 1])
            ks = slice(bases[s], bases[s] + caps[s])
            for l in range(L):
                o, _ = oracle.attention(np.ascontiguousarray(q[l, rows]), np.ascontiguousarray(k[l][:, ks]),
                                        np.ascontiguousarray(v[l][:, ks]), q_pos[rows], kvls[s], scale,
                                        window=window)
                check_attention_close(got[l, rows], o)


def test_window_paged_mla():
    """A windowed MLA layer over a paged latent pool."""
    L, H, n_q, kv, B, window = 2, 16, 9, 700, 64, 150
    g = synth.Draws(61, "cpu")
    q = host_bits(g.normal((L, n_q, H, 576)))
    rows = host_bits(g.normal((L, 1, kv, 576)))
    q_pos = np.arange(kv - n_q, kv, dtype=np.int32)
    scale = 1 / 192 ** 0.5
    max_pages = (kv + B - 1) // B
    P = max_pages + 3
    bt = np.random.default_rng(62).permutation(P)[:max_pages].astype(np.int32)[None, :]
    pool = host_bits(g.normal((L, P, B, 1, 576)))
    p = np.arange(kv)
    pool[:, bt[0, p // B], p % B] = rows.transpose(0, 2, 1, 3)
    want = np.stack([oracle.attention(q[l], rows[l], rows[l][..., :512], q_pos, kv, scale, window=window)[0]
                     for l in range(L)])
    for splits in (1, 2):
        out = torch.zeros(L, n_q, H, 512, dtype=torch.bfloat16, device="cuda")
        pd = dev(pool)
        pkv.suffix_attention_paged(dev(q), pd, pd[..., :512], out, torch.from_numpy(q_pos).cuda(),
                                   torch.tensor([kv], dtype=torch.int32, device="cuda"), torch.from_numpy(bt).cuda(),
                                   scale, max_kv_len=kv, variant=pkv.PKV_ATTN_MLA, n_splits=splits, window=window)
        torch.cuda.synchronize()
        check_attention_close(host_bits(out), want)
