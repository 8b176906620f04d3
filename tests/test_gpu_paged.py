"""GPU parity of the paged-cache entry points (paper Sec. 8: paged attention
keeps per-token KV, so reposition, splice and the suffix attention carry over
unchanged; the cache is a pool of fixed-size pages addressed through a
per-sequence block table, as in vLLM).

The expected values come from the oracle run on the logical (contiguous)
view of the pool: sequence s's slot p is row p % page_size of page
block_table[s][p // page_size].  Pools here are [layer][page][slot][kv_head][d]
with the block table a random permutation of the pool's pages, so logically
adjacent pages are far apart.  Bars as for the contiguous tests (values
bit-exact, bf16 keys within one ulp, attention max-abs 2e-2 / mean-abs 2e-3 /
rel-L2 1e-2); in addition the paged kernels, which differ from the
contiguous ones only in where a tile is read from or a row written to, must
agree with them bit for bit."""
import numpy as np
import pytest
import torch

import oracle
from helpers import check_attention_close, check_rotated_keys, dev, host_bits, log, rope_cache, small_workload
from paper_2606_17107_amd import pkv, synth
from test_gpu_attention import assemble_cache

pytestmark = pytest.mark.gpu


def bits(shape, seed):
    return host_bits(synth.Draws(seed, "cpu").normal(shape))


def gather(pool, bt_row, n_slots):
    """Logical view [L][H][n_slots][d] of pool [L][P][B][H][d] through one block-table row."""
    B = pool.shape[2]
    p = np.arange(n_slots)
    return np.ascontiguousarray(pool[:, bt_row[p // B], p % B].transpose(0, 2, 1, 3))


def scatter(pool, bt_row, logical):
    """Write logical [L][H][n][d] into pool through one block-table row (in place)."""
    B = pool.shape[2]
    p = np.arange(logical.shape[2])
    pool[:, bt_row[p // B], p % B] = logical.transpose(0, 2, 1, 3)


def block_table(n_seqs, max_pages, n_pages, seed):
    """Disjoint random pages for every sequence."""
    perm = np.random.default_rng(seed).permutation(n_pages)[: n_seqs * max_pages]
    return perm.reshape(n_seqs, max_pages).astype(np.int32)


# ---- paged splice -------------------------------------------------------------

@pytest.mark.parametrize("B", [32, 128])
@pytest.mark.parametrize("scatter_pos", [False, True])
def test_paged_splice_gqa(B, scatter_pos):
    L, H, d, n, th = 2, 4, 128, 300, 5e5
    max_pages = 24                       # logical capacity 24 B
    P = max_pages + 9                    # spare pages the table never names
    cap = max_pages * B
    pk, pv = bits((L, P, B, H, d), 1), bits((L, P, B, H, d), 2)
    sk, sv = bits((L, H, n, d), 3), bits((L, H, n, d), 4)
    bt = block_table(1, max_pages, P, 5)
    rng = np.random.default_rng(6)
    if scatter_pos:
        src = rng.integers(0, 20000, n).astype(np.int32)
        dst = rng.permutation(cap)[:n].astype(np.int32)
    else:
        src = (np.arange(n) + 17).astype(np.int32)
        dst = (np.arange(n) + cap - n - 5).astype(np.int32)
    gk, gv = dev(pk), dev(pv)
    pkv.reposition_splice_paged(dev(sk), dev(sv), gk, gv, torch.from_numpy(src).cuda(), torch.from_numpy(dst).cuda(),
                                torch.from_numpy(bt).cuda(), th, d)
    torch.cuda.synchronize()
    hk, hv = host_bits(gk), host_bits(gv)
    ok, ov = gather(pk, bt[0], cap), gather(pv, bt[0], cap)
    oracle.reposition_splice(sk, sv, ok, ov, src, dst, th, d)
    np.testing.assert_array_equal(gather(hv, bt[0], cap), ov)
    n_diff, n_floor = check_rotated_keys(gather(hk, bt[0], cap), ok, 0, d, 0)
    spare = np.setdiff1d(np.arange(P), bt[0])
    np.testing.assert_array_equal(hk[:, spare], pk[:, spare])      # pages outside the table untouched
    np.testing.assert_array_equal(hv[:, spare], pv[:, spare])
    log("  paged splice B %d scatter %s: K not bit-equal %d, floor %d" % (B, scatter_pos, n_diff, n_floor))


def test_paged_splice_mla():
    """MLA latent rows (one head, 576 channels, interleaved k_pe at 512): latent bit-exact."""
    L, n, B, max_pages, P = 3, 200, 64, 8, 13
    cap = B * max_pages
    pool = bits((L, P, B, 1, 576), 7)
    src_rows = bits((L, 1, n, 576), 8)
    bt = block_table(1, max_pages, P, 9)
    src = np.arange(n, dtype=np.int32)
    dst = (np.arange(n) + 211).astype(np.int32)
    g = dev(pool)
    pkv.reposition_splice_paged(dev(src_rows), None, g, None, torch.from_numpy(src).cuda(),
                                torch.from_numpy(dst).cuda(), torch.from_numpy(bt).cuda(), 1e4, 64, 512,
                                pkv.PKV_ROPE_INTERLEAVED)
    torch.cuda.synchronize()
    want = gather(pool, bt[0], cap)
    oracle.reposition_splice(src_rows, None, want, None, src, dst, 1e4, 64, 512, 1)
    got = gather(host_bits(g), bt[0], cap)
    np.testing.assert_array_equal(got[..., :512], want[..., :512])
    check_rotated_keys(got, want, 512, 64, 1)


def test_paged_splice_bad_page_entries_skip_tokens():
    """A block-table entry outside the pool: its tokens are skipped and the error flag is set; every
    other token lands as in the contiguous case."""
    L, H, d, n, B, max_pages, P = 1, 2, 128, 100, 32, 6, 8
    cap = B * max_pages
    pk, pv = bits((L, P, B, H, d), 10), bits((L, P, B, H, d), 11)
    sk, sv = bits((L, H, n, d), 12), bits((L, H, n, d), 13)
    bt = block_table(1, max_pages, P, 14)
    bt[0, 2] = P + 3              # logical slots 64..95 map outside the pool
    src = np.arange(n, dtype=np.int32)
    dst = (np.arange(n) + 40).astype(np.int32)      # slots 40..139
    flag = torch.zeros(1, dtype=torch.int32, device="cuda")
    gk, gv = dev(pk), dev(pv)
    pkv.reposition_splice_paged(dev(sk), dev(sv), gk, gv, torch.from_numpy(src).cuda(), torch.from_numpy(dst).cuda(),
                                torch.from_numpy(bt).cuda(), 1e4, d, err_flag=flag)
    torch.cuda.synchronize()
    assert int(flag.item()) == 1
    keep = (dst // B) != 2
    good_pages = np.array([0, 1, 3, 4, 5])
    bt_ok = bt[0].copy()
    bt_ok[2] = 0                                     # placeholder so the gather stays in range
    ok, ov = gather(pk, bt_ok, cap), gather(pv, bt_ok, cap)
    oracle.reposition_splice(np.ascontiguousarray(sk[:, :, keep]), np.ascontiguousarray(sv[:, :, keep]), ok, ov,
                             src[keep], dst[keep], 1e4, d)
    hk, hv = host_bits(gk), host_bits(gv)
    for pg in good_pages:
        sl = slice(pg * B, (pg + 1) * B)
        np.testing.assert_array_equal(gather(hv, bt_ok, cap)[:, :, sl], ov[:, :, sl])
        check_rotated_keys(gather(hk, bt_ok, cap)[:, :, sl], ok[:, :, sl], 0, d, 0)
    others = np.setdiff1d(np.arange(P), bt[0, good_pages])
    np.testing.assert_array_equal(hk[:, others], pk[:, others])


def test_paged_splice_full_size_matches_contiguous():
    """The Llama-3-8B-shaped splice (32 layers, 8 KV heads, 4096 tokens moved 2000 positions) into a
    shuffled pool of 64-slot pages equals the contiguous splice bit for bit."""
    w = synth.GQA8B
    B = 64
    max_pages = (w.kv_len + B - 1) // B
    P = max_pages + 16
    c = synth.gqa_case(w, seed=3, device="cuda")
    bt = torch.from_numpy(block_table(1, max_pages, P, 15)).cuda()
    pool_k = synth.Draws(16, "cuda").normal((w.n_layers, P, B, w.n_kv_heads, w.head_dim))
    pool_v = synth.Draws(17, "cuda").normal((w.n_layers, P, B, w.n_kv_heads, w.head_dim))
    p = torch.arange(w.kv_len, device="cuda")
    rows = (bt[0, p // B].long(), p % B)
    ctx_k = pool_k[:, rows[0], rows[1]].permute(0, 2, 1, 3).contiguous()   # logical view before the splice
    ctx_v = pool_v[:, rows[0], rows[1]].permute(0, 2, 1, 3).contiguous()
    src_k = c["skill_k_pre"]
    src_v = c["skill_v"]
    sp, dp = c["src_pos"].cuda(), c["dst_pos"].cuda()
    log("  full-size paged splice")
    pkv.reposition_splice_paged(src_k, src_v, pool_k, pool_v, sp, dp, bt, w.theta, w.rope_dim)
    pkv.reposition_splice(src_k, src_v, ctx_k, ctx_v, sp, dp, w.theta, w.rope_dim)
    torch.cuda.synchronize()
    assert torch.equal(pool_k[:, rows[0], rows[1]].permute(0, 2, 1, 3), ctx_k)
    assert torch.equal(pool_v[:, rows[0], rows[1]].permute(0, 2, 1, 3), ctx_v)


# ---- paged attention -------------------------------------------------------------

def paged_inputs(k, v, B, seed, extra_pages=5):
    """Pools holding logical caches k, v [L][Hkv][slots][d] (one sequence) behind a shuffled table."""
    L, Hkv, S, d = k.shape
    max_pages = (S + B - 1) // B
    P = max_pages + extra_pages
    bt = block_table(1, max_pages, P, seed)
    pk = bits((L, P, B, Hkv, d), seed + 1)
    scatter(pk, bt[0], k)
    pv = None
    if v is not None:
        pv = bits((L, P, B, Hkv, v.shape[3]), seed + 2)
        scatter(pv, bt[0], v)
    return pk, pv, bt


def gpu_paged(q, pk, pv, bt, q_pos, kv_len, scale, dv, n_splits=0, variant=pkv.PKV_ATTN_GQA, window=0, lse=False):
    L, nq, H = q.shape[:3]
    kd = dev(pk)
    vd = kd[..., :dv] if pv is None else dev(pv)
    out = torch.zeros(L, nq, H, dv, dtype=torch.bfloat16, device="cuda")
    lse_t = torch.zeros(L, nq, H, dtype=torch.float32, device="cuda") if lse else None
    pkv.suffix_attention_paged(dev(q), kd, vd, out, torch.from_numpy(q_pos.astype(np.int32)).cuda(),
                               torch.tensor([kv_len], dtype=torch.int32, device="cuda"), torch.from_numpy(bt).cuda(),
                               scale, max_kv_len=kv_len, variant=variant, n_splits=n_splits, window=window,
                               lse_out=lse_t)
    torch.cuda.synchronize()
    return (host_bits(out), lse_t.cpu().numpy()) if lse else host_bits(out)


def gpu_contiguous(q, k, v, q_pos, kv_len, scale, dv, n_splits=0, variant=pkv.PKV_ATTN_GQA, window=0):
    L, nq, H = q.shape[:3]
    kd = dev(k)
    vd = kd[..., :dv] if v is None else dev(v)
    out = torch.zeros(L, nq, H, dv, dtype=torch.bfloat16, device="cuda")
    pkv.suffix_attention(dev(q), kd, vd, out, torch.from_numpy(q_pos.astype(np.int32)).cuda(),
                         torch.tensor([kv_len], dtype=torch.int32, device="cuda"), scale, max_kv_len=kv_len,
                         variant=variant, n_splits=n_splits, window=window)
    torch.cuda.synchronize()
    return host_bits(out)


def oracle_out(q, k, v, q_pos, kv_len, scale, dv, window=0):
    outs, lses = [], []
    for l in range(q.shape[0]):
        vv = k[l][..., :dv] if v is None else v[l]
        o, s = oracle.attention(q[l], k[l], vv, q_pos, kv_len, scale, window=window)
        outs.append(o)
        lses.append(s)
    return np.stack(outs), np.stack(lses)


@pytest.mark.parametrize("d", [64, 128])
@pytest.mark.parametrize("B", [32, 64, 256])
def test_paged_attention_gqa(d, B):
    w = small_workload(L=2, H=8, Hkv=2, d=d, theta=1e4, skill=200, dst0=30, ctx=700, n_q=45)
    c = synth.gqa_case(w, seed=21)
    q, k, v, q_pos = assemble_cache(w, c)
    pk, pv, bt = paged_inputs(k, v, B, 22)
    want, want_lse = oracle_out(q, k, v, q_pos, w.kv_len, w.scale, d)
    for splits in (1, 3):
        got, lse = gpu_paged(q, pk, pv, bt, q_pos, w.kv_len, w.scale, d, n_splits=splits, lse=True)
        stats = check_attention_close(got, want)
        np.testing.assert_allclose(lse, want_lse, atol=2e-2)
        np.testing.assert_array_equal(got, gpu_contiguous(q, k, v, q_pos, w.kv_len, w.scale, d, n_splits=splits))
        log("  paged d %d B %d splits %d" % (d, B, splits), stats)


def test_paged_attention_window():
    w = small_workload(L=1, H=8, Hkv=2, d=128, theta=1e4, skill=300, dst0=30, ctx=1500, n_q=40)
    c = synth.gqa_case(w, seed=23)
    q, k, v, q_pos = assemble_cache(w, c)
    pk, pv, bt = paged_inputs(k, v, 32, 24)
    for window in (50, 700):
        want, _ = oracle_out(q, k, v, q_pos, w.kv_len, w.scale, 128, window=window)
        for splits in (1, 2):
            got = gpu_paged(q, pk, pv, bt, q_pos, w.kv_len, w.scale, 128, n_splits=splits, window=window)
            check_attention_close(got, want)
            np.testing.assert_array_equal(got, gpu_contiguous(q, k, v, q_pos, w.kv_len, w.scale, 128,
                                                              n_splits=splits, window=window))


def test_paged_attention_window_reload():
    """More than 256 pages in one split: the kernel's block-table window moves forward mid-loop."""
    L, H, Hkv, d, kv, n_q, B = 1, 4, 1, 64, 9000, 20, 32
    g = synth.Draws(25, "cpu")
    q = host_bits(g.normal((L, n_q, H, d)))
    k = host_bits(g.normal((L, Hkv, kv, d)))
    v = host_bits(g.normal((L, Hkv, kv, d)))
    q_pos = np.arange(kv - n_q, kv, dtype=np.int32)
    pk, pv, bt = paged_inputs(k, v, B, 26)
    assert bt.shape[1] > 256
    want, _ = oracle_out(q, k, v, q_pos, kv, 1 / 8, d)
    got = gpu_paged(q, pk, pv, bt, q_pos, kv, 1 / 8, d, n_splits=1)
    check_attention_close(got, want)
    np.testing.assert_array_equal(got, gpu_contiguous(q, k, v, q_pos, kv, 1 / 8, d, n_splits=1))


def test_paged_attention_ragged_sequences():
    """Several sequences, each with its own block-table row and length."""
    H, Hkv, d, L, B = 8, 2, 128, 2, 64
    nqs = [17, 40, 1, 64]
    kvls = [300, 1000, 77, 513]
    max_pages = max((kl + B - 1) // B for kl in kvls)
    P = len(nqs) * max_pages + 3
    g = synth.Draws(27, "cpu")
    pk = host_bits(g.normal((L, P, B, Hkv, d)))
    pv = host_bits(g.normal((L, P, B, Hkv, d)))
    q = host_bits(g.normal((L, sum(nqs), H, d)))
    q_pos = np.concatenate([np.arange(kl - n, kl) for n, kl in zip(nqs, kvls)]).astype(np.int32)
    cu = np.concatenate([[0], np.cumsum(nqs)]).astype(np.int32)
    bt = block_table(len(nqs), max_pages, P, 28)
    scale = 1 / np.sqrt(d)
    for splits in (1, 4):
        out = torch.zeros(L, sum(nqs), H, d, dtype=torch.bfloat16, device="cuda")
        pkv.suffix_attention_paged(dev(q), dev(pk), dev(pv), out, torch.from_numpy(q_pos).cuda(),
                                   torch.tensor(kvls, dtype=torch.int32, device="cuda"), torch.from_numpy(bt).cuda(),
                                   scale, max_kv_len=max(kvls), n_seqs=len(nqs), cu_q=torch.from_numpy(cu).cuda(),
                                   max_q=max(nqs), n_splits=splits)
        torch.cuda.synchronize()
        got = host_bits(out)
        for s in range(len(nqs)):
            rows = slice(cu[s], cu[s + 1])
            ks, vs = gather(pk, bt[s], kvls[s]), gather(pv, bt[s], kvls[s])
            for l in range(L):
                want, _ = oracle.attention(np.ascontiguousarray(q[l, rows]), ks[l], vs[l], q_pos[rows], kvls[s],
                                           scale)
                check_attention_close(got[l, rows], want)


def test_paged_attention_clamps_out_of_pool_entries():
    """Entries outside [0, n_pages) are clamped into the pool: the result is attention over the clamped
    pages' rows (computed here by the oracle on that gather), and nothing is read outside the pool."""
    L, H, Hkv, d, kv, n_q, B = 1, 8, 2, 128, 400, 16, 32
    g = synth.Draws(29, "cpu")
    max_pages = (kv + B - 1) // B
    P = max_pages + 2
    pk = host_bits(g.normal((L, P, B, Hkv, d)))
    pv = host_bits(g.normal((L, P, B, Hkv, d)))
    q = host_bits(g.normal((L, n_q, H, d)))
    q_pos = np.arange(kv - n_q, kv, dtype=np.int32)
    bt = block_table(1, max_pages, P, 30)
    bt[0, 3] = -7
    bt[0, 5] = P + 100
    clamped = np.clip(bt[0], 0, P - 1)
    want, _ = oracle_out(q, gather(pk, clamped, kv), gather(pv, clamped, kv), q_pos, kv, 1 / np.sqrt(d), d)
    got = gpu_paged(q, pk, pv, bt, q_pos, kv, 1 / np.sqrt(d), d, n_splits=1)
    check_attention_close(got, want)


@pytest.mark.parametrize("splits", [1, 3])
def test_paged_attention_mla(splits):
    L, H, n_q, kv, B = 2, 16, 9, 700, 64
    g = synth.Draws(31, "cpu")
    q = host_bits(g.normal((L, n_q, H, 576)))
    rows = host_bits(g.normal((L, 1, kv, 576)))
    q_pos = np.arange(kv - n_q, kv, dtype=np.int32)
    scale = 1 / 192 ** 0.5
    pk, _, bt = paged_inputs(rows, None, B, 32)
    want, _ = oracle_out(q, rows, None, q_pos, kv, scale, 512)
    got = gpu_paged(q, pk, None, bt, q_pos, kv, scale, 512, n_splits=splits, variant=pkv.PKV_ATTN_MLA)
    check_attention_close(got, want)
    np.testing.assert_array_equal(got, gpu_contiguous(q, rows, None, q_pos, kv, scale, 512, n_splits=splits,
                                                      variant=pkv.PKV_ATTN_MLA))


def test_paged_attention_full_gqa8b():
    """The Llama-3-8B-shaped attention (32 layers, 32/8 heads, 8256 slots, 64 queries) over a shuffled pool
    of 32-slot pages (258 pages: the table window moves mid-loop): bit-identical to the contiguous kernel
    on every layer, and layer 0 against the oracle."""
    w = synth.GQA8B
    B = 32
    c = synth.gqa_case(w, seed=4, device="cuda")
    k, v, q = c["ctx_k"], c["ctx_v"], c["q_pre"]
    max_pages = (w.kv_len + B - 1) // B
    P = max_pages + 8
    bt = torch.from_numpy(block_table(1, max_pages, P, 33)).cuda()
    pool_k = torch.zeros(w.n_layers, P, B, w.n_kv_heads, w.head_dim, dtype=torch.bfloat16, device="cuda")
    pool_v = torch.zeros_like(pool_k)
    p = torch.arange(w.kv_len, device="cuda")
    pool_k[:, bt[0, p // B].long(), p % B] = k.permute(0, 2, 1, 3)
    pool_v[:, bt[0, p // B].long(), p % B] = v.permute(0, 2, 1, 3)
    qp = c["q_pos"].cuda()
    kl = torch.tensor([w.kv_len], dtype=torch.int32, device="cuda")
    out_p = torch.zeros(w.n_layers, w.n_q, w.n_heads, w.head_dim, dtype=torch.bfloat16, device="cuda")
    out_c = torch.zeros_like(out_p)
    log("  full-size paged attention")
    for splits in (0, 1):
        pkv.suffix_attention_paged(q, pool_k, pool_v, out_p, qp, kl, bt, w.scale, max_kv_len=w.kv_len,
                                   n_splits=splits)
        pkv.suffix_attention(q, k, v, out_c, qp, kl, w.scale, max_kv_len=w.kv_len, n_splits=splits)
        torch.cuda.synchronize()
        assert torch.equal(out_p, out_c), "splits %d" % splits
    want, _ = oracle.attention(host_bits(q[0]), host_bits(k[0]), host_bits(v[0]), c["q_pos"].numpy(), w.kv_len,
                               w.scale)
    log("  layer 0", check_attention_close(host_bits(out_p[0]), want))


# ---- separate value table: value pages referenced in place -------------------------

def test_paged_splice_separate_v_table():
    """Keys and values through their own block tables."""
    L, H, d, n, B, max_pages, P = 2, 4, 128, 200, 32, 12, 30
    cap = B * max_pages
    pk, pv = bits((L, P, B, H, d), 40), bits((L, P, B, H, d), 41)
    sk, sv = bits((L, H, n, d), 42), bits((L, H, n, d), 43)
    bt_k, bt_v = block_table(1, max_pages, P, 44), block_table(1, max_pages, P, 45)
    src = (np.arange(n) + 9).astype(np.int32)
    dst = np.random.default_rng(46).permutation(cap)[:n].astype(np.int32)
    gk, gv = dev(pk), dev(pv)
    pkv.reposition_splice_paged(dev(sk), dev(sv), gk, gv, torch.from_numpy(src).cuda(), torch.from_numpy(dst).cuda(),
                                torch.from_numpy(bt_k).cuda(), 1e4, d, v_block_table=torch.from_numpy(bt_v).cuda())
    torch.cuda.synchronize()
    ok, ov = gather(pk, bt_k[0], cap), gather(pv, bt_v[0], cap)
    oracle.reposition_splice(sk, sv, ok, ov, src, dst, 1e4, d)
    np.testing.assert_array_equal(gather(host_bits(gv), bt_v[0], cap), ov)
    check_rotated_keys(gather(host_bits(gk), bt_k[0], cap), ok, 0, d, 0)


@pytest.mark.parametrize("d", [64, 128])
def test_paged_attention_separate_v_table(d):
    w = small_workload(L=2, H=8, Hkv=2, d=d, theta=1e4, skill=200, dst0=30, ctx=700, n_q=45)
    c = synth.gqa_case(w, seed=47)
    q, k, v, q_pos = assemble_cache(w, c)
    B = 64
    pk, _, bt_k = paged_inputs(k, None, B, 48)
    pv, _, bt_v = paged_inputs(v, None, B, 49)
    want, _ = oracle_out(q, k, v, q_pos, w.kv_len, w.scale, d)
    for splits in (1, 3):
        L, nq, H = q.shape[:3]
        out = torch.zeros(L, nq, H, d, dtype=torch.bfloat16, device="cuda")
        pkv.suffix_attention_paged(dev(q), dev(pk), dev(pv), out, torch.from_numpy(q_pos).cuda(),
                                   torch.tensor([w.kv_len], dtype=torch.int32, device="cuda"),
                                   torch.from_numpy(bt_k).cuda(), w.scale, max_kv_len=w.kv_len, n_splits=splits,
                                   v_block_table=torch.from_numpy(bt_v).cuda())
        torch.cuda.synchronize()
        got = host_bits(out)
        check_attention_close(got, want)
        np.testing.assert_array_equal(got, gpu_contiguous(q, k, v, q_pos, w.kv_len, w.scale, d, n_splits=splits))


def test_value_pages_remapped_not_copied():
    """A precompiled skill whose K/V sit in library pages is composed into a new context: its keys
    are re-rotated into the context's own K pages, its value pages are not copied at all, the
    context's V table points at the library pages (values are position-free).  Attention then equals
    the oracle on the cache a full copy would have built."""
    L, H, Hkv, d, B = 2, 8, 2, 128, 64
    theta, n_skill, src0, dst0 = 1e4, 256, 0, 320           # skill: 4 whole pages, page-aligned at 320
    ctx, n_q = 700, 40
    kv_len = ctx + n_q
    max_pages = (kv_len + B - 1) // B
    w = synth.Workload("remap", L, H, Hkv, d, d, theta, d, 0, synth.HALF, "bf16", n_skill, src0, dst0, ctx, n_q,
                       1 / np.sqrt(d))
    c = synth.gqa_case(w, seed=50)
    # logical cache a full copy builds (oracle), and the queries
    q, k_log, v_log, q_pos = assemble_cache(w, c)
    # library: the skill's post-RoPE keys (at their source positions) and its values, in pages
    # P_lib .. P_lib + 3 of both pools
    skill_k = rope_cache(host_bits(c["skill_k_pre"]), np.arange(src0, src0 + n_skill)[None, None, :], w)
    skill_v = host_bits(c["skill_v"])
    n_ctx_pages = max_pages
    P = n_ctx_pages + n_skill // B + 3
    lib_pages = np.arange(n_ctx_pages, n_ctx_pages + n_skill // B, dtype=np.int32)
    perm = np.random.default_rng(51).permutation(n_ctx_pages).astype(np.int32)
    bt_k = perm[None, :].copy()
    pk = bits((L, P, B, Hkv, d), 52)
    pv = bits((L, P, B, Hkv, d), 53)
    # the context's own pages hold the logical cache except the skill range (K is spliced there below)
    ctx_k = k_log.copy()
    ctx_k[:, :, dst0:dst0 + n_skill] = bits((L, Hkv, n_skill, d), 54)   # stale content to be overwritten
    scatter(pk, bt_k[0], ctx_k)
    ctx_v = v_log.copy()
    ctx_v[:, :, dst0:dst0 + n_skill] = bits((L, Hkv, n_skill, d), 55)   # the context's own V pages there: unused
    scatter(pv, perm, ctx_v)
    pv[:, lib_pages] = skill_v.transpose(0, 2, 1, 3).reshape(L, n_skill // B, B, Hkv, d)
    # values: the skill's logical pages map to the library pages
    bt_v = bt_k.copy()
    bt_v[0, dst0 // B: (dst0 + n_skill) // B] = lib_pages
    # keys: re-rotate the skill into the context's K pages (no values moved)
    gk = dev(pk)
    pkv.reposition_splice_paged(dev(skill_k), None, gk, None, c["src_pos"].cuda(), c["dst_pos"].cuda(),
                                torch.from_numpy(bt_k).cuda(), theta, d)
    out = torch.zeros(L, n_q, H, d, dtype=torch.bfloat16, device="cuda")
    pkv.suffix_attention_paged(dev(q), gk, dev(pv), out, torch.from_numpy(q_pos).cuda(),
                               torch.tensor([kv_len], dtype=torch.int32, device="cuda"), torch.from_numpy(bt_k).cuda(),
                               w.scale, max_kv_len=kv_len, v_block_table=torch.from_numpy(bt_v).cuda())
    torch.cuda.synchronize()
    # the spliced keys equal the oracle's splice (one bf16 ulp), the attention the oracle's
    check_rotated_keys(gather(host_bits(gk), bt_k[0], kv_len)[:, :, dst0:dst0 + n_skill],
                       k_log[:, :, dst0:dst0 + n_skill], 0, d, 0)
    want, _ = oracle_out(q, k_log, v_log, q_pos, kv_len, w.scale, d)
    log("  remapped values", check_attention_close(host_bits(out), want))


def test_paged_ragged_separate_v_tables_window():
    """Several sequences, each with its own K and V block-table rows, under a sliding window."""
    H, Hkv, d, L, B, window = 8, 2, 128, 2, 32, 200
    nqs, kvls = [17, 40, 1, 64], [300, 1000, 77, 513]
    max_pages = max((kl + B - 1) // B for kl in kvls)
    P = len(nqs) * max_pages + 5
    g = synth.Draws(63, "cpu")
    pk = host_bits(g.normal((L, P, B, Hkv, d)))
    pv = host_bits(g.normal((L, P, B, Hkv, d)))
    q = host_bits(g.normal((L, sum(nqs), H, d)))
    q_pos = np.concatenate([np.arange(kl - n, kl) for n, kl in zip(nqs, kvls)]).astype(np.int32)
    cu = np.concatenate([[0], np.cumsum(nqs)]).astype(np.int32)
    bt_k = block_table(len(nqs), max_pages, P, 64)
    bt_v = block_table(len(nqs), max_pages, P, 65)
    scale = 1 / np.sqrt(d)
    for splits in (1, 4):
        out = torch.zeros(L, sum(nqs), H, d, dtype=torch.bfloat16, device="cuda")
        pkv.suffix_attention_paged(dev(q), dev(pk), dev(pv), out, torch.from_numpy(q_pos).cuda(),
                                   torch.tensor(kvls, dtype=torch.int32, device="cuda"), torch.from_numpy(bt_k).cuda(),
                                   scale, max_kv_len=max(kvls), n_seqs=len(nqs), cu_q=torch.from_numpy(cu).cuda(),
                                   max_q=max(nqs), n_splits=splits, window=window,
                                   v_block_table=torch.from_numpy(bt_v).cuda())
        torch.cuda.synchronize()
        got = host_bits(out)
        for s in range(len(nqs)):
            rows = slice(cu[s], cu[s + 1])
            ks, vs = gather(pk, bt_k[s], kvls[s]), gather(pv, bt_v[s], kvls[s])
            for l in range(L):
                want, _ = oracle.attention(np.ascontiguousarray(q[l, rows]), ks[l], vs[l], q_pos[rows], kvls[s],
                                           scale, window=window)
                check_attention_close(got[l, rows], want)
