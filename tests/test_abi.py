"""The C ABI: libpkv.so loads, exports every function include/pkv.h declares,
and rejects bad arguments on the host before any device work.

These tests pass fake device addresses, so they only run where no GPU is
visible: every call here must be refused by host-side validation."""
import ctypes
import os
import re

import numpy as np
import pytest
import torch

from paper_2606_17107_amd import pkv

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))

pytestmark = pytest.mark.skipif(torch.cuda.is_available(),
                                reason="fake-pointer validation tests run only without a GPU")


def declared_functions():
    with open(os.path.join(ROOT, "include", "pkv.h")) as f:
        text = f.read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(pkv_[a-z_]+)\s*\(", text)))


def test_exports_every_declared_symbol():
    names = declared_functions()
    assert set(names) == set(pkv.SYMBOLS)
    lib = pkv.lib()
    for n in names:
        assert hasattr(lib, n), n
    assert pkv.pkv_version() == 1


def test_struct_sizes_match_header():
    # pkv_layout: 10 int32 + 4 x int64[3] + pointer; pkv_segment: 32 bytes
    assert ctypes.sizeof(pkv.pkv_segment) == 32
    assert ctypes.sizeof(pkv.pkv_layout) == 40 + 96 + 8
    assert ctypes.sizeof(pkv.pkv_attn_desc) == 40 + 16 + 8 + 96 + 8
    assert ctypes.sizeof(pkv.pkv_paged_cache) == 8 + 8 + 24 + 8


BASE = 1 << 40   # fake, 16-byte aligned device addresses; never dereferenced


def good_layout(**kw):
    L = pkv.pkv_layout()
    L.dtype, L.n_layers, L.n_kv_heads, L.head_dim, L.v_dim = 0, 2, 4, 128, 128
    L.n_tokens, L.rope_offset, L.rope_style, L.dst_capacity, L.reserved = 16, 0, 0, 64, 0
    L.src_k_stride = pkv._i64x3(4 * 16 * 128, 16 * 128, 128)
    L.src_v_stride = pkv._i64x3(4 * 16 * 128, 16 * 128, 128)
    L.dst_k_stride = pkv._i64x3(4 * 64 * 128, 64 * 128, 128)
    L.dst_v_stride = pkv._i64x3(4 * 64 * 128, 64 * 128, 128)
    for k, v in kw.items():
        setattr(L, k, v)
    return L


SK, SV, DK, DV, SP, DP = (BASE + i * (1 << 32) for i in range(6))


def splice(L, sk=SK, sv=SV, dk=DK, dv=DV, sp=SP, dp=DP, theta=1e4, r=128):
    st = pkv.pkv_reposition_splice(sk, sv, dk, dv, sp, dp, theta, r, L, 0)
    return st, pkv.pkv_last_error()


@pytest.mark.parametrize("kw,args,want", [
    ({}, dict(sk=None), pkv.PKV_ERR_NULL),
    ({}, dict(dv=None), pkv.PKV_ERR_NULL),
    ({}, dict(sp=None), pkv.PKV_ERR_NULL),
    (dict(v_dim=0), {}, pkv.PKV_ERR_SHAPE),                 # V pointers given without V
    ({}, dict(r=127), pkv.PKV_ERR_SHAPE),                   # odd rope_dim
    ({}, dict(r=0), pkv.PKV_ERR_SHAPE),
    (dict(rope_offset=16), {}, pkv.PKV_ERR_SHAPE),          # slice past the row
    (dict(n_tokens=-1), {}, pkv.PKV_ERR_SHAPE),
    (dict(reserved=1), {}, pkv.PKV_ERR_SHAPE),
    ({}, dict(theta=0.0), pkv.PKV_ERR_SHAPE),
    ({}, dict(theta=float("inf")), pkv.PKV_ERR_SHAPE),
    (dict(dtype=7), {}, pkv.PKV_ERR_UNSUPPORTED),
    (dict(rope_style=3), {}, pkv.PKV_ERR_UNSUPPORTED),
    ({}, dict(r=8), pkv.PKV_ERR_UNSUPPORTED),               # rope_dim not a multiple of 16 (bf16)
    (dict(head_dim=120, v_dim=120), dict(r=96), pkv.PKV_ERR_UNSUPPORTED),
    (dict(head_dim=512, v_dim=512), dict(r=288), pkv.PKV_ERR_UNSUPPORTED),   # rotary slice > 256 channels
    ({}, dict(sk=SK + 8), pkv.PKV_ERR_ALIGN),
    (dict(src_k_stride=pkv._i64x3(4 * 16 * 128, 16 * 128, 132)), {}, pkv.PKV_ERR_ALIGN),
    ({}, dict(dk=SK + 4096), pkv.PKV_ERR_ALIAS),             # dst_k partially overlaps src_k
    ({}, dict(dv=DK + 256), pkv.PKV_ERR_ALIAS),              # dst_k and dst_v overlap
])
def test_splice_validation(kw, args, want):
    st, msg = splice(good_layout(**kw), **args)
    assert st == want, (st, msg)
    assert msg


def test_splice_null_layout():
    assert pkv.pkv_reposition_splice(SK, SV, DK, DV, SP, DP, 1e4, 128, None, 0) == pkv.PKV_ERR_NULL


def test_inplace_needs_identical_strides():
    L = good_layout(dst_k_stride=pkv._i64x3(4 * 16 * 128, 16 * 128, 128),
                    dst_v_stride=pkv._i64x3(4 * 16 * 128, 16 * 128, 128), dst_capacity=16)
    # exact in-place passes validation; refuse it through an odd rope_dim so nothing launches
    st, _ = splice(L, dk=SK, dv=SV, r=3)
    assert st == pkv.PKV_ERR_SHAPE
    L.dst_k_stride = pkv._i64x3(4 * 16 * 128, 16 * 128, 256)
    st, _ = splice(L, dk=SK, dv=SV)
    assert st == pkv.PKV_ERR_ALIAS


def test_batched_validation():
    L = good_layout()
    seg = BASE + 9 * (1 << 32)
    f = pkv.pkv_reposition_splice_batched
    assert f(SK, SV, DK, DV, seg, -1, 16, 1e4, 128, L, 0) == pkv.PKV_ERR_SHAPE
    assert f(SK, SV, DK, DV, None, 2, 16, 1e4, 128, L, 0) == pkv.PKV_ERR_NULL
    assert f(SK, SV, DK, DV, seg + 4, 2, 16, 1e4, 128, L, 0) == pkv.PKV_ERR_ALIGN
    assert f(SK, SV, DK, DV, seg, 70000, 16, 1e4, 128, L, 0) == pkv.PKV_ERR_UNSUPPORTED
    assert f(SK, SV, SK + 2048, DV, seg, 2, 16, 1e4, 128, L, 0) == pkv.PKV_ERR_ALIAS


def attn_desc(**kw):
    d = pkv.pkv_attn_desc()
    d.dtype, d.variant, d.n_layers, d.n_seqs, d.head_dim_v = 0, 0, 2, 1, 128
    d.total_q, d.max_q, d.max_kv_len, d.n_splits, d.window = 64, 64, 1000, 0, 0
    d.cache_slots = 1000
    d.q_stride = pkv._i64x3(64 * 32 * 128, 32 * 128, 128)
    d.k_stride = pkv._i64x3(8 * 1000 * 128, 1000 * 128, 128)
    d.v_stride = pkv._i64x3(8 * 1000 * 128, 1000 * 128, 128)
    d.o_stride = pkv._i64x3(64 * 32 * 128, 32 * 128, 128)
    for k, v in kw.items():
        setattr(d, k, v)
    return d


Q, K, V, O, QP, KL, WS = (BASE + i * (1 << 34) for i in range(7))


def attend(d, H=32, Hkv=8, D=128, q=Q, k=K, v=V, o=O, qp=QP, kl=KL, ws=None, wsb=0, scale=0.08):
    return pkv.pkv_suffix_attention(q, k, v, o, qp, kl, H, Hkv, D, scale, d, ws, wsb, 0)


@pytest.mark.parametrize("kw,args,want", [
    ({}, dict(q=None), pkv.PKV_ERR_NULL),
    ({}, dict(kl=None), pkv.PKV_ERR_NULL),
    ({}, dict(H=30), pkv.PKV_ERR_SHAPE),                      # not a multiple of n_kv_heads
    (dict(n_seqs=2), {}, pkv.PKV_ERR_NULL),                   # cu_q required
    (dict(max_q=10), {}, pkv.PKV_ERR_SHAPE),
    (dict(window=-1), {}, pkv.PKV_ERR_SHAPE),
    ({}, dict(D=96), pkv.PKV_ERR_UNSUPPORTED),
    (dict(head_dim_v=64), {}, pkv.PKV_ERR_SHAPE),
    (dict(variant=1), {}, pkv.PKV_ERR_SHAPE),                 # MLA needs 1 KV head, 576/512
    (dict(variant=1, dtype=1, head_dim_v=512), dict(Hkv=1, D=576), pkv.PKV_ERR_UNSUPPORTED),
    (dict(variant=1, head_dim_v=512), dict(Hkv=1, D=576), pkv.PKV_ERR_SHAPE),   # MLA values must come from k_cache
    (dict(dtype=5), {}, pkv.PKV_ERR_UNSUPPORTED),
    ({}, dict(o=O + 8), pkv.PKV_ERR_ALIGN),
    (dict(q_stride=pkv._i64x3(64 * 32 * 128, 32 * 128, 100)), {}, pkv.PKV_ERR_ALIGN),
    ({}, dict(o=K + 4096), pkv.PKV_ERR_ALIAS),
    ({}, dict(scale=float("nan")), pkv.PKV_ERR_SHAPE),
    # slot strides above 64 MiB (a tile's keys are addressed by 32-bit offsets); exactly 64 MiB passes
    # that check and fails the later alias check instead
    (dict(k_stride=pkv._i64x3(8 * 1000 * 128, 1000 * 128, (1 << 25) + 8)), {}, pkv.PKV_ERR_SHAPE),
    (dict(v_stride=pkv._i64x3(8 * 1000 * 128, 1000 * 128, (1 << 25) + 8)), {}, pkv.PKV_ERR_SHAPE),
    (dict(k_stride=pkv._i64x3(8 * 1000 * 128, 1000 * 128, 1 << 25)), dict(o=K + 4096), pkv.PKV_ERR_ALIAS),
    (dict(max_kv_len=(1 << 30) + 1), {}, pkv.PKV_ERR_SHAPE),       # key arithmetic stays inside int32
    (dict(max_kv_len=1 << 30), dict(o=K + 4096), pkv.PKV_ERR_ALIAS),
])
def test_attention_validation(kw, args, want):
    st = attend(attn_desc(**kw), **args)
    assert st == want, (st, pkv.pkv_last_error())


def test_workspace_size_and_requirement():
    d = attn_desc(n_splits=4)
    need = pkv.pkv_attention_workspace_size(d, 32, 8, 128)
    rows = 4 * 2 * 64 * 32
    assert need == rows * 128 * 4 + rows * 4
    assert attend(d, ws=None, wsb=0) == pkv.PKV_ERR_NULL
    assert attend(d, ws=WS, wsb=need - 1) == pkv.PKV_ERR_SHAPE
    assert attend(d, ws=WS + 4, wsb=need) == pkv.PKV_ERR_ALIGN
    assert pkv.pkv_attention_workspace_size(attn_desc(n_splits=1), 32, 8, 128) == 0
    # fp32: 64 workgroups (2 layers x 8 KV heads x 4 row blocks of 64) split 4 ways to reach the 256 CUs
    rows = 4 * 2 * 64 * 32
    assert pkv.pkv_attention_workspace_size(attn_desc(dtype=1), 32, 8, 128) == rows * 128 * 4 + rows * 4
    assert pkv.pkv_attention_workspace_size(attn_desc(dtype=1, n_splits=1), 32, 8, 128) == 0
    assert pkv.pkv_attention_workspace_size(None, 32, 8, 128) == 0
    assert pkv.pkv_attention_workspace_size(d, 30, 8, 128) == 0


def test_freqs_validation():
    L = good_layout()
    f = pkv.pkv_reposition_splice_freqs
    w = [0.5] * 64
    assert f(SK, SV, DK, DV, SP, DP, None, None, 128, L, 0) == pkv.PKV_ERR_NULL        # omega required
    assert f(SK, SV, DK, DV, None, DP, None, w, 128, L, 0) == pkv.PKV_ERR_NULL
    bad = list(w)
    bad[7] = float("nan")
    assert f(SK, SV, DK, DV, SP, DP, None, bad, 128, L, 0) == pkv.PKV_ERR_SHAPE
    assert "omega[7]" in pkv.pkv_last_error()
    assert f(SK, SV, DK, DV, SP, DP, None, w, 127, L, 0) == pkv.PKV_ERR_SHAPE          # odd rope_dim
    assert f(SK, SV, DK + 4096 - 4096 + 8, DV, SP, DP, None, w, 128, L, 0) == pkv.PKV_ERR_ALIGN


def good_paging(**kw):
    pg = pkv.pkv_paged_cache()
    pg.page_size, pg.max_pages, pg.block_table, pg.n_pages = 32, 4, BASE + 11 * (1 << 32), 8
    pg.page_stride_k = pg.page_stride_v = 32 * 4 * 128
    for k, v in kw.items():
        setattr(pg, k, v)
    return pg


def paged_layout(**kw):
    # pools [layer 2][page 8][slot 32][kv_head 4][128]
    pool = pkv._i64x3(8 * 32 * 4 * 128, 128, 4 * 128)
    L = good_layout(dst_k_stride=pool, dst_v_stride=pool, dst_capacity=128)
    for k, v in kw.items():
        setattr(L, k, v)
    return L


@pytest.mark.parametrize("lkw,pkw,args,want", [
    ({}, None, {}, pkv.PKV_ERR_NULL),
    ({}, dict(block_table=None), {}, pkv.PKV_ERR_NULL),
    ({}, dict(page_size=16), {}, pkv.PKV_ERR_SHAPE),
    ({}, dict(page_size=48), {}, pkv.PKV_ERR_SHAPE),           # not a power of two
    ({}, dict(page_size=1 << 21), {}, pkv.PKV_ERR_SHAPE),
    ({}, dict(max_pages=0), {}, pkv.PKV_ERR_SHAPE),
    ({}, dict(n_pages=0), {}, pkv.PKV_ERR_SHAPE),
    ({}, dict(n_pages=1 << 31), {}, pkv.PKV_ERR_SHAPE),
    ({}, dict(page_stride_k=-4096), {}, pkv.PKV_ERR_SHAPE),
    ({}, dict(page_stride_v=4100), {}, pkv.PKV_ERR_ALIGN),
    (dict(dst_capacity=129), {}, {}, pkv.PKV_ERR_SHAPE),         # beyond max_pages * page_size
    ({}, {}, dict(dk=SK + 2048), pkv.PKV_ERR_ALIAS),
    ({}, {}, dict(dv=DK + 7 * 32 * 4 * 128 * 2), pkv.PKV_ERR_ALIAS),   # V pool starts inside K's last page
    ({}, {}, dict(sp=None), pkv.PKV_ERR_NULL),
    ({}, {}, dict(r=127), pkv.PKV_ERR_SHAPE),
])
def test_paged_splice_validation(lkw, pkw, args, want):
    L = paged_layout(**lkw)
    pg = None if pkw is None else good_paging(**pkw)
    a = dict(sk=SK, sv=SV, dk=DK, dv=DV, sp=SP, dp=DP, theta=1e4, r=128)
    a.update(args)
    st = pkv.pkv_reposition_splice_paged(a["sk"], a["sv"], a["dk"], a["dv"], a["sp"], a["dp"], a["theta"], a["r"],
                                         L, pg, 0)
    assert st == want, (st, pkv.pkv_last_error())
    assert pkv.pkv_last_error()


def paged_attn_desc(**kw):
    pool = pkv._i64x3(8 * 32 * 8 * 128, 128, 8 * 128)   # [layer][page 8][slot 32][kv_head 8][128]
    d = attn_desc(k_stride=pool, v_stride=pool, cache_slots=128, max_kv_len=128)
    for k, v in kw.items():
        setattr(d, k, v)
    return d


def paged_paging(**kw):
    return good_paging(page_stride_k=32 * 8 * 128, page_stride_v=32 * 8 * 128, **kw)


@pytest.mark.parametrize("dkw,pkw,args,want", [
    ({}, None, {}, pkv.PKV_ERR_NULL),
    ({}, dict(block_table=None), {}, pkv.PKV_ERR_NULL),
    ({}, dict(page_size=64 + 32), {}, pkv.PKV_ERR_SHAPE),
    (dict(dtype=1), {}, {}, pkv.PKV_ERR_UNSUPPORTED),           # paged attention is bf16 only
    (dict(kv_base=BASE), {}, {}, pkv.PKV_ERR_SHAPE),
    (dict(cache_slots=129), {}, {}, pkv.PKV_ERR_SHAPE),
    ({}, {}, dict(o=K + 5 * 32 * 8 * 128 * 2), pkv.PKV_ERR_ALIAS),   # out inside page 5 of the K pool
    ({}, {}, dict(D=96), pkv.PKV_ERR_UNSUPPORTED),
    ({}, {}, dict(scale=float("nan")), pkv.PKV_ERR_SHAPE),
])
def test_paged_attention_validation(dkw, pkw, args, want):
    d = paged_attn_desc(**dkw)
    pg = None if pkw is None else paged_paging(**pkw)
    a = dict(H=32, Hkv=8, D=128, q=Q, k=K, v=V, o=O, qp=QP, kl=KL, scale=0.08)
    a.update(args)
    st = pkv.pkv_suffix_attention_paged(a["q"], a["k"], a["v"], a["o"], a["qp"], a["kl"], a["H"], a["Hkv"], a["D"],
                                        a["scale"], d, pg, None, 0, 0)
    assert st == want, (st, pkv.pkv_last_error())


def test_paged_mla_page_strides_must_match():
    pool = pkv._i64x3(8 * 32 * 576, 576, 576)
    d = attn_desc(variant=1, head_dim_v=512, k_stride=pool, v_stride=pool, cache_slots=128, max_kv_len=128)
    pg = good_paging(page_stride_k=32 * 576, page_stride_v=32 * 576 + 8)
    st = pkv.pkv_suffix_attention_paged(Q, K, K, O, QP, KL, 16, 1, 576, 0.07, d, pg, None, 0, 0)
    assert st == pkv.PKV_ERR_SHAPE and "page_stride_v" in pkv.pkv_last_error()
    pg = good_paging(page_stride_k=32 * 576, page_stride_v=32 * 576, v_block_table=BASE + 12 * (1 << 32))
    st = pkv.pkv_suffix_attention_paged(Q, K, K, O, QP, KL, 16, 1, 576, 0.07, d, pg, None, 0, 0)
    assert st == pkv.PKV_ERR_SHAPE and "v_block_table" in pkv.pkv_last_error()


def planned_splits(L, H, Hkv, d, dv, total_q, kv, variant=0, dtype=0, window=0):
    """Split count the library picks, read back through the workspace size."""
    d_ = pkv.pkv_attn_desc()
    d_.dtype, d_.variant, d_.n_layers, d_.n_seqs, d_.head_dim_v = dtype, variant, L, 1, dv
    d_.total_q, d_.max_q, d_.max_kv_len, d_.n_splits, d_.window = total_q, total_q, kv, 0, window
    d_.cache_slots = kv
    d_.q_stride = pkv._i64x3(total_q * H * d, H * d, d)
    d_.k_stride = d_.v_stride = pkv._i64x3(Hkv * kv * d, kv * d, d)
    d_.o_stride = pkv._i64x3(total_q * H * dv, H * dv, dv)
    n = pkv.pkv_attention_workspace_size(d_, H, Hkv, d)
    per_split = L * total_q * H * (dv + 1) * 4
    assert n % per_split == 0
    return max(1, n // per_split)


def test_split_planner_choices():
    """The planner weighs workgroup rounds over the 256 CUs (each with a fixed cost) against the
    combine pass's traffic: the 8B workload fills the GPU in one round (no split), the 32k prefill
    splits 2 ways and the MLA workload (128-row workgroups) 4 ways; launched one layer at a time
    they split 16, 2 and 16 ways (each the measured best, or tied with it, on MI355X); short caches
    never split below 512 keys per split."""
    assert planned_splits(32, 32, 8, 128, 128, 64, 8256) == 1
    assert planned_splits(28, 28, 4, 128, 128, 1024, 50176) == 2
    assert planned_splits(27, 16, 1, 576, 512, 128, 32896, variant=1) == 4
    assert planned_splits(1, 32, 8, 128, 128, 64, 8256) == 16
    assert planned_splits(1, 28, 4, 128, 128, 1024, 50176) == 2
    assert planned_splits(1, 16, 1, 576, 512, 128, 32896, variant=1) == 16
    assert planned_splits(1, 8, 2, 128, 128, 16, 300) == 1
    assert planned_splits(1, 8, 2, 128, 128, 16, 1000) == 1    # under 2 x 512 keys: no split
    assert planned_splits(1, 8, 2, 128, 128, 16, 4096) > 1     # one layer, one KV head pair: split to fill CUs


def test_split_planner_sizes_windowed_work_by_the_window():
    """With a sliding window a workgroup sees about window + queries keys, not the whole cache: the
    32k prefill with a 4096-key window runs unsplit (its rounds already fill the CUs; 1.67 ms against
    1.94 ms split 2 ways on MI355X), one 8B layer splits by its window (2 ways for 1024 keys, 8 for
    4096, 16 without a window)."""
    assert planned_splits(28, 28, 4, 128, 128, 1024, 50176, window=4096) == 1
    assert planned_splits(1, 32, 8, 128, 128, 64, 8256, window=1024) == 2
    assert planned_splits(1, 32, 8, 128, 128, 64, 8256, window=4096) == 8
    assert planned_splits(1, 32, 8, 128, 128, 64, 8256, window=10000) == 16   # window past the cache


def test_split_planner_fp32():
    """fp32: split until there is about one workgroup per CU, at least 64 keys per split, at most 32."""
    assert planned_splits(1, 4, 2, 64, 64, 16, 528, dtype=1) == 8       # tiny: 2 workgroups, 528 keys
    assert planned_splits(1, 4, 2, 64, 64, 16, 100, dtype=1) == 1       # under 2 x 64 keys
    assert planned_splits(1, 4, 2, 64, 64, 16, 100000, dtype=1) == 32   # capped
    assert planned_splits(8, 32, 8, 128, 128, 64, 4096, dtype=1) == 1   # 256 workgroups already


def test_stream_copy_library_exports():
    """The stream-copy reference library (timed by bench.py beside the splice) is built and exports its
    one entry point."""
    import ctypes
    import os
    from paper_2606_17107_amd import build as B
    assert os.path.exists(B.COPY_LIB)
    lib = ctypes.CDLL(B.COPY_LIB)
    assert hasattr(lib, "pkv_stream_copy")


def test_workspace_size_over_random_descriptors():
    """The split planner over 3000 seeded descriptors (layer, head, length, window and split counts of
    every size the ABI accepts, plus invalid ones): the size is 0 for an invalid descriptor or an
    unsplit plan, otherwise a whole number of per-split records: 2..32 splits of the library's own
    choice, and an explicit split count kept unless it exceeds ceil(max_kv_len / 64).  Host code
    only: nothing launches."""
    rng = np.random.default_rng(2024)
    for _ in range(3000):
        variant = int(rng.integers(0, 2))
        dtype = 0 if variant else int(rng.integers(0, 2))
        if variant:
            Hkv, H, D, dv = 1, int(rng.choice([8, 16, 128])), 576, 512
        else:
            Hkv = int(rng.choice([1, 2, 4, 8]))
            H = Hkv * int(rng.choice([1, 3, 4, 7, 8]))
            D = int(rng.choice([64, 128, 96]))   # 96 is unsupported
            dv = D
        L, n_seqs = int(rng.integers(1, 65)), int(rng.integers(1, 9))
        total_q = int(rng.integers(0, 4097))
        max_q = int(rng.integers(0, total_q + 1)) if n_seqs > 1 else total_q
        kv = int(rng.integers(0, 1 << 17))
        splits = int(rng.choice([0, 0, 1, 2, 3, 16, 33]))
        window = int(rng.choice([0, 0, 1, 100, 4096, 1 << 20]))
        d_ = pkv.pkv_attn_desc()
        d_.dtype, d_.variant, d_.n_layers, d_.n_seqs, d_.head_dim_v = dtype, variant, L, n_seqs, dv
        d_.total_q, d_.max_q, d_.max_kv_len, d_.n_splits, d_.window = total_q, max_q, kv, splits, window
        d_.cu_q = BASE + (1 << 33) if n_seqs > 1 else None
        d_.cache_slots = kv
        d_.q_stride = pkv._i64x3(max(total_q, 1) * H * D, H * D, D)
        d_.k_stride = d_.v_stride = pkv._i64x3(Hkv * max(kv, 1) * D, max(kv, 1) * D, D)
        d_.o_stride = pkv._i64x3(max(total_q, 1) * H * dv, H * dv, dv)
        n = pkv.pkv_attention_workspace_size(d_, H, Hkv, D)
        valid = D != 96
        if not valid:
            assert n == 0
            continue
        per_split = L * total_q * H * (dv + 1) * 4
        if n == 0:
            continue
        assert per_split > 0 and n % per_split == 0, (n, per_split)
        s = n // per_split
        if splits > 1:
            assert s == min(splits, (kv + 63) // 64), (s, splits, kv)   # explicit: kept, or lowered
        else:
            assert splits == 0 and 2 <= s <= 32, (s, splits)           # the library's own choice
