"""Benchmark of the compose hot path on one MI355X: reposition+splice of a
precompiled skill's KV into a destination cache, then causal suffix attention
over the spliced cache (paper Sec. 5: a re-rotation pass plus the suffix).

One step = pkv_reposition_splice over every layer and KV head, then
pkv_suffix_attention over every layer, on synthetic seeded inputs resident in
HBM.  Default workload: Llama-3-8B-shaped single sequence (32 layers, 32/8
heads, d 128, RoPE theta 5e5, 4096-token skill spliced at 2000 into 8192
slots, 64-token suffix over 8256 slots, bf16).

Prints one JSON line: the splice GB/s as `value`, the attention time and
TFLOP/s beside it, the roofline of the dominant kernel (timed with HIP events
on the library's stream), and the CPU oracle timed on a bounded sample.
"""
from __future__ import annotations

import argparse
import json
import math
import os
import sys
import time

import torch

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

from paper_2606_17107_amd import pkv, synth  # noqa: E402

METRIC = "KV reposition+splice GB/s; suffix prefix-attention µs and TFLOP/s"
HBM_PEAK_GBS = 8000.0
BF16_PEAK_TFLOPS = 2500.0
FP32_PEAK_TFLOPS = 157.3


def log(*a):
    print(*a, file=sys.stderr, flush=True)


class GqaStep:
    """Inputs and launches of one workload (single sequence, GQA or MLA)."""

    def __init__(self, w: synth.Workload, n_splits: int, seed: int = 0, window: int = 0, rope: str = "theta",
                 page_size: int = 0):
        self.w = w
        self.window = window
        self.rope = rope
        self.page_size = page_size
        if page_size and rope != "theta":
            raise SystemExit("--paged takes the theta schedule (no --rope table)")
        # explicit per-pair frequencies for pkv_reposition_splice_freqs (None: the theta schedule)
        tables = {"mrope_sectioned": lambda: synth.mrope_temporal_omega(w.theta, w.rope_dim, (16, 24, 24)),
                  "mrope_interleaved": lambda: synth.mrope_temporal_omega(w.theta, w.rope_dim, (24, 20, 20),
                                                                           "interleaved"),
                  "llama31": lambda: synth.llama31_omega(w.theta, w.rope_dim)}
        self.omega = None
        if rope != "theta":
            import ctypes
            t = tables[rope]()
            self.omega = (ctypes.c_double * len(t))(*[float(x) for x in t])
        dev = torch.device("cuda")
        c = synth.gqa_case(w, seed=seed, device=dev)
        self.cache_k = c["ctx_k"]
        self.cache_v = c.get("ctx_v")
        self.skill_k = c["skill_k_pre"]
        self.skill_v = c.get("skill_v")
        self.src_pos = c["src_pos"].to(dev)
        self.dst_pos = c["dst_pos"].to(dev)
        self.q_pos = c["q_pos"].to(dev)
        n, nq = w.skill_tokens, w.n_q
        # Post-RoPE skill keys: rotate the pre-RoPE draws from position 0 to their
        # source positions, in place (dst_pos[t] == t keeps slot t).
        zeros = torch.zeros(n, dtype=torch.int32, device=dev)
        pkv.reposition_splice(self.skill_k, None, self.skill_k, None, zeros, self.src_pos, w.theta, w.rope_dim,
                              w.rope_offset, w.rope_style)
        # Suffix keys sit in cache slots ctx..kv_len-1 at positions equal to their slots.
        suf = self.cache_k[:, :, w.ctx_slots:]
        t_idx = torch.arange(nq, dtype=torch.int32, device=dev)
        pkv.reposition_splice(suf, None, suf, None, torch.full((nq,), -w.ctx_slots, dtype=torch.int32,
                              device=dev), t_idx, w.theta, w.rope_dim, w.rope_offset, w.rope_style)
        # Post-RoPE queries [L][n_q][H][d], rotated in place per (query, head) row.
        self.q = c["q_pre"]
        qv = self.q.permute(0, 2, 1, 3)          # [L][H][n_q][d] view for the rotation
        pkv.reposition_splice(qv, None, qv, None, torch.full((nq,), -w.ctx_slots, dtype=torch.int32,
                              device=dev), t_idx, w.theta, w.rope_dim, w.rope_offset, w.rope_style)
        self.out = torch.zeros(w.n_layers, nq, w.n_heads, w.v_dim, dtype=self.q.dtype, device=dev)
        self.kv_len = torch.tensor([w.kv_len], dtype=torch.int32, device=dev)
        self.v_view = self.cache_k[..., : w.v_dim] if w.mla else self.cache_v
        self.splice_layout = pkv.make_layout(self.skill_k, self.skill_v, self.cache_k, self.cache_v,
                                             w.rope_offset, w.rope_style)
        variant = pkv.PKV_ATTN_MLA if w.mla else pkv.PKV_ATTN_GQA
        self.desc = pkv.make_attn_desc(self.q, self.cache_k, self.v_view, self.out, w.kv_len, variant=variant,
                                       n_splits=n_splits, window=window)
        if page_size:
            self._to_pages(page_size, seed)
        self.ws_bytes = pkv.pkv_attention_workspace_size(self.desc, w.n_heads, w.n_kv_heads, w.head_dim)
        self.ws = torch.empty(max(self.ws_bytes, 16), dtype=torch.uint8, device=dev)
        torch.cuda.synchronize()

    def _to_pages(self, B: int, seed: int):
        """Move the cache into a pool [layer][page][slot][kv_head][d] (the vLLM layout) whose pages the
        block table hands out in a random order, and describe both calls over the pool."""
        w = self.w
        dev = self.cache_k.device
        max_pages = (w.kv_len + B - 1) // B
        n_pages = max_pages + 64
        perm = torch.randperm(n_pages, generator=torch.Generator().manual_seed(seed + 101))[:max_pages]
        self.block_table = perm.to(torch.int32).reshape(1, max_pages).to(dev)
        p = torch.arange(w.kv_len, device=dev)
        page, slot = self.block_table[0, p // B].long(), p % B
        self.pool_k = torch.zeros(w.n_layers, n_pages, B, w.n_kv_heads, w.head_dim, dtype=self.cache_k.dtype,
                                  device=dev)
        self.pool_k[:, page, slot] = self.cache_k.permute(0, 2, 1, 3)
        self.pool_v = None
        if self.cache_v is not None:
            self.pool_v = torch.zeros(w.n_layers, n_pages, B, w.n_kv_heads, w.v_dim, dtype=self.cache_v.dtype,
                                      device=dev)
            self.pool_v[:, page, slot] = self.cache_v.permute(0, 2, 1, 3)
        self.cache_k = self.cache_v = self.v_view = None
        self.pool_v_view = self.pool_k[..., : w.v_dim] if w.mla else self.pool_v
        self.paging = pkv.make_paging(self.block_table, self.pool_k, self.pool_v_view)
        L = self.splice_layout
        L.dst_capacity = max_pages * B
        L.dst_k_stride = pkv.pool_strides3(self.pool_k)
        L.dst_v_stride = pkv.pool_strides3(self.pool_v)
        d = self.desc
        d.cache_slots = max_pages * B
        d.k_stride = pkv.pool_strides3(self.pool_k)
        d.v_stride = pkv.pool_strides3(self.pool_v_view)
        torch.cuda.synchronize()

    def splice(self, stream):
        w = self.w
        if self.page_size:
            st = pkv.pkv_reposition_splice_paged(self.skill_k, self.skill_v, self.pool_k, self.pool_v, self.src_pos,
                                                 self.dst_pos, w.theta, w.rope_dim, self.splice_layout, self.paging,
                                                 stream)
            if st != 0:
                raise pkv.PkvError(st, pkv.pkv_last_error())
            return
        if self.omega is not None:
            import ctypes
            st = pkv.lib().pkv_reposition_splice_freqs(
                pkv._ptr(self.skill_k), pkv._ptr(self.skill_v), pkv._ptr(self.cache_k), pkv._ptr(self.cache_v),
                pkv._ptr(self.src_pos), pkv._ptr(self.dst_pos), None, self.omega, w.rope_dim,
                ctypes.byref(self.splice_layout), stream)
        else:
            st = pkv.pkv_reposition_splice(self.skill_k, self.skill_v, self.cache_k, self.cache_v, self.src_pos,
                                           self.dst_pos, w.theta, w.rope_dim, self.splice_layout, stream)
        if st != 0:
            raise pkv.PkvError(st, pkv.pkv_last_error())

    def attention(self, stream):
        w = self.w
        if self.page_size:
            st = pkv.pkv_suffix_attention_paged(self.q, self.pool_k, self.pool_v_view, self.out, self.q_pos,
                                                self.kv_len, w.n_heads, w.n_kv_heads, w.head_dim, w.scale, self.desc,
                                                self.paging, self.ws, self.ws_bytes, stream)
            if st != 0:
                raise pkv.PkvError(st, pkv.pkv_last_error())
            return
        st = pkv.pkv_suffix_attention(self.q, self.cache_k, self.v_view, self.out, self.q_pos, self.kv_len,
                                      w.n_heads, w.n_kv_heads, w.head_dim, w.scale, self.desc, self.ws,
                                      self.ws_bytes, stream)
        if st != 0:
            raise pkv.PkvError(st, pkv.pkv_last_error())

    def layer_calls_setup(self):
        """Per-layer launches (one call per layer, as a model that interleaves layers makes them):
        one descriptor for a single layer, the library's own split choice for it, and its workspace."""
        w = self.w
        variant = pkv.PKV_ATTN_MLA if w.mla else pkv.PKV_ATTN_GQA
        self.layer_desc = pkv.make_attn_desc(self.q[:1], self.cache_k[:1], self.v_view[:1], self.out[:1], w.kv_len,
                                             variant=variant, n_splits=self.desc.n_splits, window=self.window)
        self.layer_ws_bytes = pkv.pkv_attention_workspace_size(self.layer_desc, w.n_heads, w.n_kv_heads,
                                                               w.head_dim)
        self.layer_ws = torch.empty(max(self.layer_ws_bytes, 16), dtype=torch.uint8, device=self.q.device)

    def attention_layer_calls(self, stream):
        w = self.w
        for l in range(w.n_layers):
            st = pkv.pkv_suffix_attention(self.q[l:l + 1], self.cache_k[l:l + 1], self.v_view[l:l + 1],
                                          self.out[l:l + 1], self.q_pos, self.kv_len, w.n_heads, w.n_kv_heads,
                                          w.head_dim, w.scale, self.layer_desc, self.layer_ws, self.layer_ws_bytes,
                                          stream)
            if st != 0:
                raise pkv.PkvError(st, pkv.pkv_last_error())

    def splice_bytes(self):
        return self.w.splice_bytes()

    def describe(self):
        w = self.w
        return ("%s: %d layers, %d/%d heads, d %d, %d-token skill %d->%d, %d-token suffix over %d slots%s%s"
                % (w.name, w.n_layers, w.n_heads, w.n_kv_heads, w.head_dim, w.skill_tokens, w.src_pos0, w.dst_pos0,
                   w.n_q, w.kv_len, ", sliding window %d" % self.window if self.window else "",
                   ", splice frequencies %s" % self.rope if self.rope != "theta" else "")
                + (", paged cache (%d-slot pages, shuffled block table, [layer][page][slot][kv_head][d] pool)"
                   % self.page_size if self.page_size else ""))

    def attn_flops(self):
        return self.w.attn_flops(self.window)

    def attn_bytes(self):
        return self.w.attn_bytes(self.window)


class BatchedStep:
    """Batched composition: 16 sequences each splice the same three library skills
    (1024, 2048, 4096 tokens) at their own offsets, then run a 256-query causal
    suffix over their own cache length (ragged).  One splice launch covers all
    48 segments and one attention launch covers all sequences and layers."""

    def __init__(self, bw: synth.BatchedWorkload, n_splits: int, seed: int = 0):
        self.bw = bw
        dev = torch.device("cuda")
        self.plan = plan = synth.batched_plan(bw, seed)
        c = synth.batched_case(bw, plan, seed=seed, device=dev)
        self.cache_k, self.cache_v = c["ctx_k"], c["ctx_v"]
        L, Hkv, H, d, nq = bw.n_layers, bw.n_kv_heads, bw.n_heads, bw.head_dim, bw.n_q
        n_seqs = bw.n_seqs
        # Post-RoPE library keys: skill k's tokens sit at positions src_pos0[k] + t.
        self.skill_v = c["skill_v"]
        self.skill_k = torch.empty_like(c["skill_k_pre"])
        lib_segs = [dict(src_slot0=plan["skill_base"][k], dst_seq_base=plan["skill_base"][k] - plan["src_pos0"][k],
                         n_tokens=bw.skills[k], src_pos0=0, dst_pos0=plan["src_pos0"][k],
                         dst_seq_len=plan["src_pos0"][k] + bw.skills[k]) for k in range(len(bw.skills))]
        pkv.reposition_splice_batched(c["skill_k_pre"], None, self.skill_k, None, pkv.make_segments(lib_segs, dev),
                                      len(lib_segs), max(bw.skills), bw.theta, d)
        del c["skill_k_pre"]
        # Suffix keys (rotated to their positions) and values into each sequence's cache slots.
        suf_segs, q_segs, q_pos, cu, bases, kvl = [], [], [], [0], [], []
        for s_i, sq in enumerate(plan["seqs"]):
            C = sq["ctx"]
            suf_segs.append(dict(src_slot0=s_i * nq, dst_seq_base=sq["seq_base"], n_tokens=nq, src_pos0=0,
                                 dst_pos0=C, dst_seq_len=sq["kv_len"]))
            q_segs.append(dict(src_slot0=s_i * nq, dst_seq_base=s_i * nq - C, n_tokens=nq, src_pos0=0, dst_pos0=C,
                               dst_seq_len=C + nq))
            q_pos.extend(range(C, C + nq))
            cu.append(cu[-1] + nq)
            bases.append(sq["seq_base"])
            kvl.append(sq["kv_len"])
            self.cache_v[:, :, sq["seq_base"] + C: sq["seq_base"] + C + nq] = c["suf_v"][:, :, s_i * nq:(s_i + 1) * nq]
        pkv.reposition_splice_batched(c["suf_k_pre"], None, self.cache_k, None, pkv.make_segments(suf_segs, dev),
                                      len(suf_segs), nq, bw.theta, d)
        # Post-RoPE queries [L][rows][H][d], rotated through a [L][H][rows][d] view.
        self.q = torch.empty_like(c["q_pre"])
        pkv.reposition_splice_batched(c["q_pre"].permute(0, 2, 1, 3), None, self.q.permute(0, 2, 1, 3), None,
                                      pkv.make_segments(q_segs, dev), len(q_segs), nq, bw.theta, d)
        del c
        self.segs = synth.batched_segments(plan)
        self.segs_dev = pkv.make_segments(self.segs, dev)
        self.max_seg = max(sg["n_tokens"] for sg in self.segs)
        self.q_pos = torch.tensor(q_pos, dtype=torch.int32, device=dev)
        self.cu_q = torch.tensor(cu, dtype=torch.int32, device=dev)
        self.kv_base = torch.tensor(bases, dtype=torch.int64, device=dev)
        self.kv_len = torch.tensor(kvl, dtype=torch.int32, device=dev)
        self.out = torch.zeros(L, n_seqs * nq, H, d, dtype=torch.bfloat16, device=dev)
        self.splice_layout = pkv.make_layout(self.skill_k, self.skill_v, self.cache_k, self.cache_v)
        self.desc = pkv.make_attn_desc(self.q, self.cache_k, self.cache_v, self.out, max(kvl), n_seqs=n_seqs,
                                       cu_q=self.cu_q, kv_base=self.kv_base, max_q=nq, n_splits=n_splits)
        self.ws_bytes = pkv.pkv_attention_workspace_size(self.desc, H, Hkv, d)
        self.ws = torch.empty(max(self.ws_bytes, 16), dtype=torch.uint8, device=dev)
        torch.cuda.synchronize()

    def splice(self, stream):
        bw = self.bw
        st = pkv.pkv_reposition_splice_batched(self.skill_k, self.skill_v, self.cache_k, self.cache_v, self.segs_dev,
                                               len(self.segs), self.max_seg, bw.theta, bw.head_dim,
                                               self.splice_layout, stream)
        if st != 0:
            raise pkv.PkvError(st, pkv.pkv_last_error())

    def attention(self, stream):
        bw = self.bw
        st = pkv.pkv_suffix_attention(self.q, self.cache_k, self.cache_v, self.out, self.q_pos, self.kv_len,
                                      bw.n_heads, bw.n_kv_heads, bw.head_dim, bw.scale, self.desc, self.ws,
                                      self.ws_bytes, stream)
        if st != 0:
            raise pkv.PkvError(st, pkv.pkv_last_error())

    def splice_bytes(self):
        return synth.batched_splice_bytes(self.bw, self.plan)

    def attn_flops(self):
        return synth.batched_attn_flops(self.bw, self.plan)

    def attn_bytes(self):
        return synth.batched_attn_bytes(self.bw, self.plan)

    def describe(self):
        bw = self.bw
        ctx = [sq["ctx"] for sq in self.plan["seqs"]]
        return ("batched: %d layers, %d/%d heads, d %d, %d sequences x skills %s at random offsets in %d-%d-token "
                "contexts, %d-query ragged suffixes" % (bw.n_layers, bw.n_heads, bw.n_kv_heads, bw.head_dim,
                                                        bw.n_seqs, "/".join(map(str, bw.skills)), min(ctx), max(ctx),
                                                        bw.n_q))


def cpu_baseline_batched(bw: synth.BatchedWorkload, budget_s: float = 10.0):
    """Time the fp64 oracle on a bounded sample of the batched workload: the three
    segments of sequence 0 for as many single-layer passes as fit in half the
    budget (scaled to all 48 segments and 32 layers by bytes), and layer 0 of
    sequence 0's suffix attention for as many queries as fit in the other half
    (scaled by visible pairs)."""
    import numpy as np

    import oracle

    oracle.build(force=False)
    threads = oracle.max_threads()
    bits = synth.to_numpy_bits
    plan = synth.batched_plan(bw, 0)
    c = synth.batched_case(bw, plan, seed=1, layers=1)
    sk, sv = bits(c["skill_k_pre"]), bits(c["skill_v"])
    sq = plan["seqs"][0]
    seq_k = bits(c["ctx_k"])[:, :, sq["seq_base"]: sq["seq_base"] + sq["kv_len"]].copy()
    seq_v = bits(c["ctx_v"])[:, :, sq["seq_base"]: sq["seq_base"] + sq["kv_len"]].copy()

    def run_seq0():
        for sg in sq["segs"]:
            n = sg["n_tokens"]
            sl = slice(sg["src_slot0"], sg["src_slot0"] + n)
            oracle.reposition_splice(np.ascontiguousarray(sk[:, :, sl]), np.ascontiguousarray(sv[:, :, sl]), seq_k,
                                     seq_v, np.arange(sg["src_pos0"], sg["src_pos0"] + n, dtype=np.int32),
                                     np.arange(sg["dst_pos0"], sg["dst_pos0"] + n, dtype=np.int32), bw.theta,
                                     bw.head_dim)

    t0 = time.perf_counter()
    run_seq0()
    t_one = time.perf_counter() - t0
    reps = max(1, min(64, int(0.5 * budget_s / max(t_one, 1e-4))))
    t0 = time.perf_counter()
    for _ in range(reps):
        run_seq0()
    t_splice = time.perf_counter() - t0
    per_pass = sum(2 * 2 * sg["n_tokens"] * bw.n_kv_heads * bw.head_dim * 2 for sg in sq["segs"])
    sample_bytes = per_pass * reps
    oracle.set_threads(1)
    reps1, t_splice1 = 0, 0.0
    try:
        while reps1 < 1 or (t_splice1 < 0.1 * budget_s and reps1 < reps):
            t0 = time.perf_counter()
            run_seq0()
            t_splice1 += time.perf_counter() - t0
            reps1 += 1
    finally:
        oracle.set_threads(threads)
    q = bits(c["q_pre"][0])[: bw.n_q]
    q_pos = np.arange(sq["ctx"], sq["ctx"] + bw.n_q, dtype=np.int32)
    t0 = time.perf_counter()
    oracle.attention(np.ascontiguousarray(q[:1]), seq_k[0], seq_v[0], q_pos[:1], sq["kv_len"], bw.scale)
    t_row = max(time.perf_counter() - t0, 1e-4)
    n_rows = max(1, min(bw.n_q, int(0.5 * budget_s / t_row)))
    t0 = time.perf_counter()
    oracle.attention(np.ascontiguousarray(q[:n_rows]), seq_k[0], seq_v[0], q_pos[:n_rows], sq["kv_len"], bw.scale)
    t_attn = time.perf_counter() - t0
    vis = sum(min(sq["kv_len"], int(q_pos[i]) + 1) for i in range(n_rows))
    flops_sample = 4 * bw.head_dim * bw.n_heads * vis
    attn_us_full = t_attn * synth.batched_attn_flops(bw, plan) / flops_sample * 1e6
    return {
        "value": round(sample_bytes / t_splice / 1e9, 4),
        "unit": "GB/s",
        "cores": threads,
        "kind": "oracle",
        "sample": "splice: %d passes over sequence 0's three segments of one layer (%.3f GB moved) in %.2f s; "
                  "attention: layer 0, sequence 0, %d of %d queries in %.2f s, scaled to all sequences and layers "
                  "by visible pairs" % (reps, sample_bytes / 1e9, t_splice, n_rows, bw.n_q, t_attn),
        "attention_us_extrapolated": round(attn_us_full, 1),
        "value_1thread": round(per_pass * reps1 / t_splice1 / 1e9, 4),
        "sample_1thread": "splice: %d pass(es) over sequence 0's segments of one layer in %.2f s on 1 thread"
                          % (reps1, t_splice1),
    }


def cpu_baseline(w: synth.Workload, budget_s: float = 10.0):
    """Time the fp64 oracle on a bounded sample of the same workload on the host cores.

    Splice: the full skill (all tokens) over as many layers as fit in about half
    the budget.  Attention: layer 0, as many suffix queries as fit in the other
    half, scaled to all layers and queries by visible (query, key) pairs."""
    import numpy as np

    import oracle

    oracle.build(force=False)
    threads = oracle.max_threads()
    bits = synth.to_numpy_bits
    # splice: time one layer first, then size the sample
    c1 = synth.gqa_case(w, seed=1, layers=1)
    one = dict(sk=bits(c1["skill_k_pre"]), dk=bits(c1["ctx_k"]),
               sv=bits(c1["skill_v"]) if "skill_v" in c1 else None, dv=bits(c1["ctx_v"]) if "ctx_v" in c1 else None)
    src, dst = c1["src_pos"].numpy(), c1["dst_pos"].numpy()

    def run_splice(x):
        oracle.reposition_splice(x["sk"], x["sv"], x["dk"], x["dv"], src, dst, w.theta, w.rope_dim, w.rope_offset,
                                 w.rope_style)

    t0 = time.perf_counter()
    run_splice(one)
    t_one = time.perf_counter() - t0
    reps = max(1, min(64 * w.n_layers, int(0.5 * budget_s / max(t_one, 1e-4))))
    t0 = time.perf_counter()
    for _ in range(reps):
        run_splice(one)
    t_splice = time.perf_counter() - t0
    sample_bytes = w.splice_bytes() / w.n_layers * reps
    # the same splice on one host thread (a smaller sample: about a tenth of the budget)
    oracle.set_threads(1)
    reps1, t_splice1 = 0, 0.0
    try:
        while reps1 < 1 or (t_splice1 < 0.1 * budget_s and reps1 < reps):
            t0 = time.perf_counter()
            run_splice(one)
            t_splice1 += time.perf_counter() - t0
            reps1 += 1
    finally:
        oracle.set_threads(threads)
    # attention: layer 0 of the same draws
    q = bits(c1["q_pre"][0])
    k = one["dk"][0]
    v = k[..., : w.v_dim] if w.mla else one["dv"][0]
    q_pos = c1["q_pos"].numpy()
    t0 = time.perf_counter()
    oracle.attention(np.ascontiguousarray(q[:1]), k, v, q_pos[:1], w.kv_len, w.scale)
    t_row = max(time.perf_counter() - t0, 1e-4)
    n_rows = max(1, min(w.n_q, int(0.5 * budget_s / t_row)))
    # when every query of a layer fits, repeat the layer (up to the layer count) to fill the budget
    passes = 1
    if n_rows == w.n_q:
        passes = max(1, min(w.n_layers, int(0.5 * budget_s / (t_row * w.n_q))))
    t0 = time.perf_counter()
    for _ in range(passes):
        oracle.attention(np.ascontiguousarray(q[:n_rows]), k, v, q_pos[:n_rows], w.kv_len, w.scale)
    t_attn = time.perf_counter() - t0
    vis = sum(min(w.kv_len, int(q_pos[i]) + 1) for i in range(n_rows))
    vis_all = sum(min(w.kv_len, int(q_pos[i]) + 1) for i in range(w.n_q))
    attn_us_full = t_attn / passes * (vis_all / vis) * w.n_layers * 1e6
    return {
        "value": round(sample_bytes / t_splice / 1e9, 4),
        "unit": "GB/s",
        "cores": threads,
        "kind": "oracle",
        "sample": "splice: %d passes of one layer (all %d skill tokens, %.3f GB moved) in %.2f s; attention: "
                  "%d pass(es) of layer 0, %d of %d queries over %d slots, in %.2f s, scaled to all layers and queries"
                  % (reps, w.skill_tokens, sample_bytes / 1e9, t_splice, passes, n_rows, w.n_q, w.kv_len, t_attn),
        "attention_us_extrapolated": round(attn_us_full, 1),
        "value_1thread": round(w.splice_bytes() / w.n_layers * reps1 / t_splice1 / 1e9, 4),
        "sample_1thread": "splice: %d pass(es) of one layer in %.2f s on 1 thread" % (reps1, t_splice1),
    }


def device_copy_gbps(nbytes: int = 1 << 30, reps: int = 10) -> float:
    """Plain device-to-device copy rate (bytes read + written per second), the practical HBM
    ceiling the splice is compared against: the better of torch's copy (a DMA-engine copy on ROCm,
    about 5 TB/s) and an elementwise fp32 kernel that writes its input unchanged (x * 1)."""
    src = torch.ones(nbytes // 4, dtype=torch.float32, device="cuda")
    dst = torch.empty_like(src)
    best = 0.0
    for f in (lambda: dst.copy_(src), lambda: torch.mul(src, 1.0, out=dst)):
        for _ in range(3):
            f()
        torch.cuda.synchronize()
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record()
        for _ in range(reps):
            f()
        b.record()
        torch.cuda.synchronize()
        best = max(best, 2 * nbytes / (a.elapsed_time(b) / reps * 1e-3) / 1e9)
    del src, dst
    torch.cuda.empty_cache()
    return best


def source_hash(files):
    """Hash of the kernel sources a counter measurement was taken against."""
    import hashlib

    h = hashlib.sha256()
    for f in files:
        with open(os.path.join(ROOT, f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


KERNEL_SOURCES = {   # the sources and compiler options each kernel is built from
    "splice_kernel": ["paper_2606_17107_amd/csrc/splice.hip", "paper_2606_17107_amd/csrc/pkv_internal.h",
                      "paper_2606_17107_amd/build.py"],
    "attn_gqa_bf16": ["paper_2606_17107_amd/csrc/attn_gqa_bf16.hip", "paper_2606_17107_amd/csrc/attn_common.h",
                      "paper_2606_17107_amd/csrc/attention.hip", "paper_2606_17107_amd/csrc/pkv_internal.h",
                      "paper_2606_17107_amd/build.py"],
    "attn_mla_bf16": ["paper_2606_17107_amd/csrc/attn_mla_bf16.hip", "paper_2606_17107_amd/csrc/attn_common.h",
                      "paper_2606_17107_amd/csrc/attention.hip", "paper_2606_17107_amd/csrc/pkv_internal.h",
                      "paper_2606_17107_amd/build.py"],
}


def measured_traffic(kernel: str, workload: str):
    """HBM bytes per launch from the committed rocprofv3 FETCH_SIZE / WRITE_SIZE record
    (profiles/traffic.json), scaled by the plain-copy calibration; None when no record
    exists or the kernel source changed since it was taken."""
    path = os.path.join(ROOT, "profiles", "traffic.json")
    if not os.path.exists(path):
        return None
    with open(path) as f:
        rec = json.load(f)
    r = rec.get("kernels", {}).get(kernel, {}).get(workload)
    if not r or r.get("source_hash") != source_hash(KERNEL_SOURCES[kernel]):
        return None
    return int(r["hbm_bytes_per_launch"])


def copy_calibration():
    """A plain device copy of a known size, for calibrating the FETCH_SIZE / WRITE_SIZE counters."""
    n = 1 << 30
    x = torch.ones(n, dtype=torch.uint8, device="cuda")
    y = torch.empty_like(x)
    for _ in range(3):
        y.copy_(x)
    torch.cuda.synchronize()
    print(json.dumps({"copy_calibration_bytes_read": n, "copy_calibration_bytes_written": n, "launches": 3}))


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=100)
    ap.add_argument("--warmup", type=int, default=30)
    ap.add_argument("--min-warmup-s", type=float, default=0.25,
                    help="keep warming up until this much wall time has passed (clock ramp)")
    ap.add_argument("--workload", default="gqa8b", choices=sorted(synth.WORKLOADS) + ["batched"])
    ap.add_argument("--splits", type=int, default=0, help="KV splits for attention (0 = library choice)")
    ap.add_argument("--rope", default="theta", choices=["theta", "mrope_sectioned", "mrope_interleaved", "llama31"],
                    help="splice frequencies: the theta schedule, or an explicit table through "
                         "pkv_reposition_splice_freqs (M-RoPE temporal move, Llama-3.1 scaling)")
    ap.add_argument("--window", type=int, default=0,
                    help="sliding-window attention over the full cache (0 = causal; single-sequence workloads)")
    ap.add_argument("--paged", type=int, default=0,
                    help="page size of a paged KV cache (0 = contiguous cache)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-budget", type=float, default=10.0)
    ap.add_argument("--copy-calibration", action="store_true",
                    help="run only a 1 GiB device copy (counter calibration for rocprofv3)")
    args = ap.parse_args()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU only: this build has no multi-GPU path "
              "(reposition+splice and suffix attention run on a single MI355X)", file=sys.stderr)
        sys.exit(2)
    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(2)
    if args.copy_calibration:
        copy_calibration()
        return
    pkv.lib()   # fail loudly if libpkv.so is missing

    if args.workload == "batched":
        w = synth.BATCHED
        step = BatchedStep(w, args.splits)
    else:
        w = synth.WORKLOADS[args.workload]
        step = GqaStep(w, args.splits, window=args.window, rope=args.rope, page_size=args.paged)
    log("workload", w)
    stream = torch.cuda.current_stream()
    sh = stream.cuda_stream

    # Attention as one launch per layer, as a model that interleaves layers
    # makes it (a figure beside the layer-batched headline; timed before the
    # headline so that the headline's launches are the last of the run).
    layer_calls = None
    if isinstance(step, GqaStep) and not args.paged:
        step.layer_calls_setup()
        t_warm = time.perf_counter()
        n = 0
        while n < 3 or time.perf_counter() - t_warm < args.min_warmup_s / 2:
            step.attention_layer_calls(sh)
            n += 1
            if n % 8 == 0:
                torch.cuda.synchronize()
        torch.cuda.synchronize()
        reps = max(5, min(args.steps, 50))
        lev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(reps)]
        for a, b in lev:
            a.record(stream)
            step.attention_layer_calls(sh)
            b.record(stream)
        torch.cuda.synchronize()
        lt = sorted(a.elapsed_time(b) for a, b in lev)
        l_ms = sum(lt) / reps
        layer_calls = {
            "launches_per_step": w.n_layers, "us": round(l_ms * 1e3, 2), "us_median": round(lt[reps // 2] * 1e3, 2),
            "us_per_layer": round(l_ms * 1e3 / w.n_layers, 2),
            "tflops": round(step.attn_flops() / (l_ms * 1e-3) / 1e12, 2),
            "workspace_bytes": step.layer_ws_bytes}

    # Untimed warm-up: the requested steps, continued until at least
    # --min-warmup-s of GPU work has run, so the shader clock has left its
    # idle state before the timed region (a few ms of work is not enough).
    t_warm = time.perf_counter()
    n_warm = 0
    while n_warm < args.warmup or time.perf_counter() - t_warm < args.min_warmup_s:
        step.splice(sh)
        step.attention(sh)
        n_warm += 1
        if n_warm % 16 == 0:
            torch.cuda.synchronize()
    torch.cuda.synchronize()

    ev = [[torch.cuda.Event(enable_timing=True) for _ in range(3)] for _ in range(args.steps)]
    start, stop = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    t_wall = time.perf_counter()
    start.record(stream)
    for i in range(args.steps):
        ev[i][0].record(stream)
        step.splice(sh)
        ev[i][1].record(stream)
        step.attention(sh)
        ev[i][2].record(stream)
    stop.record(stream)
    torch.cuda.synchronize()
    t_wall = time.perf_counter() - t_wall
    total_ms = start.elapsed_time(stop)
    splice_t = sorted(e[0].elapsed_time(e[1]) for e in ev)
    attn_t = sorted(e[1].elapsed_time(e[2]) for e in ev)
    # The mean launch duration is the figure rocprofv3's per-kernel average reports; median and min beside it.
    splice_ms = sum(splice_t) / args.steps
    attn_ms = sum(attn_t) / args.steps
    ms_per_step = total_ms / args.steps

    splice_gbs = step.splice_bytes() / (splice_ms * 1e-3) / 1e9
    attn_tflops = step.attn_flops() / (attn_ms * 1e-3) / 1e12
    attn_gbs = step.attn_bytes() / (attn_ms * 1e-3) / 1e9
    ai = step.attn_flops() / step.attn_bytes()
    ridge = BF16_PEAK_TFLOPS * 1e12 / (HBM_PEAK_GBS * 1e9)
    attn_bound = "hbm" if ai < ridge else "mfma"
    if attn_bound == "hbm":
        attn_roof = {"bound": "hbm", "achieved": round(attn_gbs, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": round(attn_gbs / HBM_PEAK_GBS, 4), "traffic": None}
    else:
        attn_roof = {"bound": "mfma", "achieved": round(attn_tflops, 2), "peak": BF16_PEAK_TFLOPS,
                     "unit": "TFLOP/s", "frac": round(attn_tflops / BF16_PEAK_TFLOPS, 4), "traffic": None}
    splice_roof = {"bound": "hbm", "achieved": round(splice_gbs, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                   "frac": round(splice_gbs / HBM_PEAK_GBS, 4), "traffic": None}
    splice_roof["kernel"] = "splice_kernel"
    mla = getattr(w, "mla", False)
    attn_roof["kernel"] = "attn_gqa_bf16" if not mla else "attn_mla_bf16"
    splice_roof["traffic"] = measured_traffic("splice_kernel", w.name)
    attn_roof["traffic"] = measured_traffic(attn_roof["kernel"], w.name)
    splice_roof["algorithmic_bytes"] = step.splice_bytes()
    attn_roof["algorithmic_bytes"] = step.attn_bytes()
    attn_roof["algorithmic_flops"] = step.attn_flops()
    dominant = splice_roof if splice_ms >= attn_ms else attn_roof

    result = {
        "metric": METRIC,
        "value": round(splice_gbs, 1),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "warmup_steps_run": n_warm,
        "ms_per_step": round(ms_per_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16" if w.dtype == "bf16" else "f32",
        "data": "synthetic",
        "config": {
            "workload": step.describe(),
            "splice_bytes": step.splice_bytes(),
            "attention_flops": step.attn_flops(),
            "attention_bytes": step.attn_bytes(),
            "attention_splits": int(step.desc.n_splits) or "auto",
            "workspace_bytes": step.ws_bytes,
        },
        "splice": {"us": round(splice_ms * 1e3, 2), "us_median": round(splice_t[len(splice_t) // 2] * 1e3, 2),
                   "us_min": round(splice_t[0] * 1e3, 2), "gbps": round(splice_gbs, 1)},
        "attention": {"us": round(attn_ms * 1e3, 2), "us_median": round(attn_t[len(attn_t) // 2] * 1e3, 2),
                      "us_min": round(attn_t[0] * 1e3, 2), "tflops": round(attn_tflops, 2),
                      "gbps": round(attn_gbs, 1), "arith_intensity": round(ai, 1), "bound": attn_bound},
        "roofline": dominant,
        "roofline_kernels": [splice_roof, attn_roof],
        "wall_s_timed": round(t_wall, 3),
    }
    if layer_calls is not None:
        result["attention_layer_calls"] = layer_calls
    cp = device_copy_gbps()
    result["device_copy_gbps"] = round(cp, 1)
    result["splice"]["of_device_copy"] = round(splice_gbs / cp, 4)
    if not args.no_cpu_baseline:
        log("timing the CPU oracle on a bounded sample")
        result["cpu_baseline"] = (cpu_baseline_batched(w, args.cpu_budget) if args.workload == "batched"
                                  else cpu_baseline(w, args.cpu_budget))
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
