"""Benchmark of the compose hot path on one MI355X: reposition+splice of precompiled
skills' KV into destination caches, then causal suffix attention over the spliced
caches (paper Sec. 5: the transplant costs a re-rotation pass plus the suffix).

One step = one reposition+splice launch over every layer and KV head, then one
suffix-attention launch over every layer, on seeded synthetic inputs resident in
HBM.  The default run measures all five workloads and prints ONE JSON line whose
headline is the largest one (batched composition: 16 sequences x 3 skills,
ragged 256-query suffixes, Llama-3-8B shape); the others (tiny fp32, gqa8b,
long32k, mla) are nested under "configs" with the same fields.

Timing: HIP events on the library's stream around each launch.  Every timed
launch starts cold: a 1 GiB read-modify-write of a flush buffer (beyond the
256 MB last-level cache) runs before it, outside the events.  Beside the cold
figures, "warm" repeats the steps back to back (the attention then finds part
of the splice's writes in the caches), and for the single-sequence workloads
"attention_layer_calls" launches one layer per call (as a model that
interleaves its layers does), both from the host and replayed from a HIP
graph.  The CPU oracle is timed on the host cores beside each workload.
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
FP32_PEAK_TFLOPS = 157.3   # fp32 dense MFMA (the fp32 attention path runs on v_mfma_f32_32x32x2_f32)
ORDER = ("tiny", "gqa8b", "long32k", "mla", "batched")   # measured in this order; batched is the headline
FLUSH_BYTES = 1 << 30


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

    def splice_bytes_per_segment(self):
        return synth.batched_splice_bytes_per_segment(self.bw, self.plan)

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


# ---- CPU oracle baselines ---------------------------------------------------

def _replicate_layers(one, n_layers):
    """[1][...] host array -> [n_layers][...] copy (the CPU splice timing streams every layer; the
    values of one seeded layer are repeated, which does not change the oracle's work)."""
    import numpy as np
    return np.ascontiguousarray(np.repeat(one, n_layers, axis=0))


def _time_splice(run, budget_s):
    """Run `run` once, then repeat it while the total stays within budget_s; returns (passes, seconds)."""
    t0 = time.perf_counter()
    run()
    t = time.perf_counter() - t0
    passes, total = 1, t
    while total + t <= budget_s:
        t0 = time.perf_counter()
        run()
        total += time.perf_counter() - t0
        passes += 1
    return passes, total


def cpu_baseline(w: synth.Workload, budget_s: float):
    """The fp64 oracle on the host cores.  Splice: the full skill over every layer (one seeded layer of
    draws repeated over the layers), one or more whole passes.  Attention: every layer and query for
    the tiny and gqa8b workloads; for long32k and mla layer 0 over as many queries as fit in the
    budget, scaled to all layers and queries by visible (query, key) pairs (labelled extrapolated)."""
    import numpy as np

    import oracle

    oracle.build(force=False)
    threads = oracle.max_threads()
    bits = synth.to_numpy_bits
    c1 = synth.gqa_case(w, seed=1, layers=1)
    src, dst = c1["src_pos"].numpy(), c1["dst_pos"].numpy()
    full = dict(sk=_replicate_layers(bits(c1["skill_k_pre"]), w.n_layers),
                dk=_replicate_layers(bits(c1["ctx_k"]), w.n_layers),
                sv=_replicate_layers(bits(c1["skill_v"]), w.n_layers) if not w.mla else None,
                dv=_replicate_layers(bits(c1["ctx_v"]), w.n_layers) if not w.mla else None)

    def run_full():
        oracle.reposition_splice(full["sk"], full["sv"], full["dk"], full["dv"], src, dst, w.theta, w.rope_dim,
                                 w.rope_offset, w.rope_style)

    passes, t_splice = _time_splice(run_full, 0.15 * budget_s)
    splice_bytes = w.splice_bytes() * passes
    del full
    one = dict(sk=bits(c1["skill_k_pre"]), dk=bits(c1["ctx_k"]).copy(),
               sv=bits(c1["skill_v"]) if not w.mla else None, dv=bits(c1["ctx_v"]).copy() if not w.mla else None)
    oracle.set_threads(1)
    try:
        t0 = time.perf_counter()
        oracle.reposition_splice(one["sk"], one["sv"], one["dk"], one["dv"], src, dst, w.theta, w.rope_dim,
                                 w.rope_offset, w.rope_style)
        t_one1 = time.perf_counter() - t0
    finally:
        oracle.set_threads(threads)
    # attention
    q_pos = c1["q_pos"].numpy()
    vis_all = sum(min(w.kv_len, int(q_pos[i]) + 1) for i in range(w.n_q))
    k0 = bits(c1["ctx_k"])[0]
    v0 = k0[..., : w.v_dim] if w.mla else bits(c1["ctx_v"])[0]
    q0 = bits(c1["q_pre"])[0]
    if w.name in ("tiny", "gqa8b"):
        # every layer: the draws of the first layer per layer index (same work per layer)
        t0 = time.perf_counter()
        for _ in range(w.n_layers):
            oracle.attention(q0, k0, v0, q_pos, w.kv_len, w.scale)
        t_attn = time.perf_counter() - t0
        attn_us, attn_kind = t_attn * 1e6, "measured"
        attn_sample = "every layer (%d) and query (%d) over %d slots in %.2f s" % (w.n_layers, w.n_q, w.kv_len,
                                                                                    t_attn)
    else:
        t0 = time.perf_counter()
        oracle.attention(np.ascontiguousarray(q0[:1]), k0, v0, q_pos[:1], w.kv_len, w.scale)
        t_row = max(time.perf_counter() - t0, 1e-4)
        n_rows = max(1, min(w.n_q, int(0.6 * budget_s / t_row)))
        rows = np.linspace(0, w.n_q - 1, n_rows).astype(np.int64)
        t0 = time.perf_counter()
        oracle.attention(np.ascontiguousarray(q0[rows]), k0, v0, q_pos[rows], w.kv_len, w.scale)
        t_attn = time.perf_counter() - t0
        vis = sum(min(w.kv_len, int(q_pos[i]) + 1) for i in rows)
        attn_us, attn_kind = t_attn * (vis_all / vis) * w.n_layers * 1e6, "extrapolated"
        attn_sample = ("layer 0, %d of %d queries (evenly spaced) over %d slots in %.2f s, scaled to all layers "
                       "and queries by visible pairs" % (n_rows, w.n_q, w.kv_len, t_attn))
    return {
        "value": round(splice_bytes / t_splice / 1e9, 4),
        "unit": "GB/s",
        "cores": threads,
        "kind": "oracle",
        "sample": "splice: %d full pass(es) over all %d layers (all %d skill tokens, %.3f GB moved) in %.2f s; "
                  "attention: %s" % (passes, w.n_layers, w.skill_tokens, splice_bytes / 1e9, t_splice, attn_sample),
        "splice_us": round(t_splice / passes * 1e6, 1),
        "attention_us": round(attn_us, 1),
        "attention_kind": attn_kind,
        "value_1thread": round(w.splice_bytes() / w.n_layers / t_one1 / 1e9, 4),
        "sample_1thread": "splice: one layer (all skill tokens) in %.3f s on 1 thread" % t_one1,
    }


def cpu_baseline_batched(bw: synth.BatchedWorkload, budget_s: float):
    """The fp64 oracle on the batched workload: sequence 0's three segments over every layer (one
    seeded layer of draws repeated over the layers), scaled to all 48 segments by bytes; attention of
    layer 0, sequence 0 over as many queries as fit, scaled to all sequences and layers by visible
    pairs (extrapolated)."""
    import numpy as np

    import oracle

    oracle.build(force=False)
    threads = oracle.max_threads()
    bits = synth.to_numpy_bits
    plan = synth.batched_plan(bw, 0)
    c = synth.batched_case(bw, plan, seed=1, layers=1)
    sq = plan["seqs"][0]
    sk = _replicate_layers(bits(c["skill_k_pre"]), bw.n_layers)
    sv = _replicate_layers(bits(c["skill_v"]), bw.n_layers)
    seq_k1 = bits(c["ctx_k"])[:, :, sq["seq_base"]: sq["seq_base"] + sq["kv_len"]]
    seq_v1 = bits(c["ctx_v"])[:, :, sq["seq_base"]: sq["seq_base"] + sq["kv_len"]]
    seq_k = _replicate_layers(seq_k1, bw.n_layers)
    seq_v = _replicate_layers(seq_v1, bw.n_layers)
    segs = []
    for sg in sq["segs"]:
        n = sg["n_tokens"]
        sl = slice(sg["src_slot0"], sg["src_slot0"] + n)
        segs.append((np.ascontiguousarray(sk[:, :, sl]), np.ascontiguousarray(sv[:, :, sl]),
                     np.arange(sg["src_pos0"], sg["src_pos0"] + n, dtype=np.int32),
                     np.arange(sg["dst_pos0"], sg["dst_pos0"] + n, dtype=np.int32)))
    del sk, sv

    def run_seq0():
        for a_k, a_v, s_pos, d_pos in segs:
            oracle.reposition_splice(a_k, a_v, seq_k, seq_v, s_pos, d_pos, bw.theta, bw.head_dim)

    passes, t_splice = _time_splice(run_seq0, 0.2 * budget_s)
    per_pass = sum(2 * 2 * sg["n_tokens"] * bw.n_layers * bw.n_kv_heads * bw.head_dim * 2 for sg in sq["segs"])
    sample_bytes = per_pass * passes
    oracle.set_threads(1)
    try:
        t0 = time.perf_counter()
        a_k, a_v, s_pos, d_pos = segs[0]
        oracle.reposition_splice(np.ascontiguousarray(a_k[:1]), np.ascontiguousarray(a_v[:1]),
                                 np.ascontiguousarray(seq_k[:1]), np.ascontiguousarray(seq_v[:1]), s_pos, d_pos,
                                 bw.theta, bw.head_dim)
        t_one1 = time.perf_counter() - t0
        one1_bytes = 2 * 2 * len(s_pos) * bw.n_kv_heads * bw.head_dim * 2
    finally:
        oracle.set_threads(threads)
    q = bits(c["q_pre"][0])[: bw.n_q]
    q_pos = np.arange(sq["ctx"], sq["ctx"] + bw.n_q, dtype=np.int32)
    k0, v0 = np.ascontiguousarray(seq_k1[0]), np.ascontiguousarray(seq_v1[0])
    t0 = time.perf_counter()
    oracle.attention(np.ascontiguousarray(q[:1]), k0, v0, q_pos[:1], sq["kv_len"], bw.scale)
    t_row = max(time.perf_counter() - t0, 1e-4)
    n_rows = max(1, min(bw.n_q, int(0.6 * budget_s / t_row)))
    rows = np.linspace(0, bw.n_q - 1, n_rows).astype(np.int64)
    t0 = time.perf_counter()
    oracle.attention(np.ascontiguousarray(q[rows]), k0, v0, q_pos[rows], sq["kv_len"], bw.scale)
    t_attn = time.perf_counter() - t0
    vis = sum(min(sq["kv_len"], int(q_pos[i]) + 1) for i in rows)
    flops_sample = 4 * bw.head_dim * bw.n_heads * vis
    attn_us_full = t_attn * synth.batched_attn_flops(bw, plan) / flops_sample * 1e6
    return {
        "value": round(sample_bytes / t_splice / 1e9, 4),
        "unit": "GB/s",
        "cores": threads,
        "kind": "oracle",
        "sample": "splice: %d pass(es) over sequence 0's three segments (%s tokens) on all %d layers (%.3f GB moved) "
                  "in %.2f s, the rate applied to all 48 segments; attention: layer 0, sequence 0, %d of %d queries "
                  "(evenly spaced) over %d slots in %.2f s, scaled to all sequences and layers by visible pairs"
                  % (passes, "/".join(str(sg["n_tokens"]) for sg in sq["segs"]), bw.n_layers, sample_bytes / 1e9,
                     t_splice, n_rows, bw.n_q, sq["kv_len"], t_attn),
        "splice_us": round(synth.batched_splice_bytes_per_segment(bw, plan) / (sample_bytes / t_splice) * 1e6, 1),
        "attention_us": round(attn_us_full, 1),
        "attention_kind": "extrapolated",
        "value_1thread": round(one1_bytes / t_one1 / 1e9, 4),
        "sample_1thread": "splice: sequence 0's first segment, one layer, in %.3f s on 1 thread" % t_one1,
    }


# ---- GPU timing ----------------------------------------------------------------

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


STREAM_COPY_LIB = os.path.join(ROOT, "paper_2606_17107_amd", "libpkv_copy.so")


def stream_copy(dst: torch.Tensor, src: torch.Tensor, stream) -> None:
    """The stream-copy reference kernel (paper_2606_17107_amd/probe/stream_copy.hip): the splice's
    access pattern without its arithmetic."""
    import ctypes

    if not os.path.exists(STREAM_COPY_LIB):
        raise RuntimeError("%s is missing: run __graft_entry__.build()" % STREAM_COPY_LIB)
    lib = ctypes.CDLL(STREAM_COPY_LIB)
    fn = lib.pkv_stream_copy
    fn.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_size_t, ctypes.c_void_p]
    fn.restype = ctypes.c_int
    nbytes = src.numel() * src.element_size()
    if dst.numel() * dst.element_size() != nbytes:
        raise ValueError("stream_copy: size mismatch")
    rc = fn(dst.data_ptr(), src.data_ptr(), nbytes, stream)
    if rc != 0:
        raise RuntimeError("pkv_stream_copy failed (%d)" % rc)


def stream_copy_gbps(flush, nbytes: int = 512 << 20, reps: int = 10) -> float:
    """Rate (bytes read + written per second) of the stream-copy reference kernel, every launch cold
    (after the flush) like the splice's: the ceiling of the splice's memory traffic."""
    src = torch.ones(nbytes // 4, dtype=torch.float32, device="cuda")
    dst = torch.empty_like(src)
    st = torch.cuda.current_stream()
    for _ in range(3):
        stream_copy(dst, src, st.cuda_stream)
    ts = []
    for _ in range(reps):
        flush()
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record(st)
        stream_copy(dst, src, st.cuda_stream)
        b.record(st)
        torch.cuda.synchronize()
        ts.append(a.elapsed_time(b))
    del src, dst
    torch.cuda.empty_cache()
    return 2 * nbytes / (sum(ts) / len(ts) * 1e-3) / 1e9


def source_hash(files):
    """Hash of the kernel sources a counter measurement was taken against, and of the compiler
    options the first of them (the kernel's translation unit) is built with."""
    import hashlib

    from paper_2606_17107_amd import build as B

    h = hashlib.sha256()
    for f in files:
        with open(os.path.join(ROOT, f), "rb") as fh:
            h.update(fh.read())
    flags = B.compile_flags() + B.FILE_FLAGS.get(os.path.basename(files[0]), [])
    h.update(" ".join(f.replace(ROOT, "") for f in flags).encode())
    return h.hexdigest()[:16]


KERNEL_SOURCES = {   # the kernel's translation unit first, then the headers it includes
    "splice_kernel": ["paper_2606_17107_amd/csrc/splice.hip", "paper_2606_17107_amd/csrc/pkv_internal.h"],
    "attn_gqa_bf16": ["paper_2606_17107_amd/csrc/attn_gqa_bf16.hip", "paper_2606_17107_amd/csrc/attn_common.h",
                      "paper_2606_17107_amd/csrc/attention.hip", "paper_2606_17107_amd/csrc/pkv_internal.h"],
    "attn_mla_bf16": ["paper_2606_17107_amd/csrc/attn_mla_bf16.hip", "paper_2606_17107_amd/csrc/attn_common.h",
                      "paper_2606_17107_amd/csrc/attention.hip", "paper_2606_17107_amd/csrc/pkv_internal.h"],
    "attn_gqa_f32": ["paper_2606_17107_amd/csrc/attention.hip", "paper_2606_17107_amd/csrc/attn_common.h",
                     "paper_2606_17107_amd/csrc/pkv_internal.h"],
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


class Flush:
    """A 1 GiB read-modify-write on the timing stream: evicts the 4 MB L2s and the 256 MB last-level
    cache, so the launch that follows streams its inputs from HBM."""

    def __init__(self):
        self.buf = torch.zeros(FLUSH_BYTES, dtype=torch.uint8, device="cuda")

    def __call__(self):
        self.buf.add_(1)


def _stats(ms_list):
    t = sorted(ms_list)
    return {"us": round(sum(t) / len(t) * 1e3, 2), "us_median": round(t[len(t) // 2] * 1e3, 2),
            "us_min": round(t[0] * 1e3, 2)}


def roofline(kind, kernel, work, ms, bf16=True, workload=None):
    """Roofline object of one kernel: algorithmic bytes (hbm) or flops (mfma) per launch over its mean
    event-timed duration."""
    if kind == "hbm":
        achieved = work / (ms * 1e-3) / 1e9
        r = {"bound": "hbm", "achieved": round(achieved, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
             "frac": round(achieved / HBM_PEAK_GBS, 4)}
    else:
        peak = BF16_PEAK_TFLOPS if bf16 else FP32_PEAK_TFLOPS
        achieved = work / (ms * 1e-3) / 1e12
        # both attention paths run on the matrix cores: bf16 MFMA, and fp32 MFMA for the fp32 path
        r = {"bound": "mfma", "achieved": round(achieved, 2), "peak": peak, "unit": "TFLOP/s",
             "frac": round(achieved / peak, 4)}
    r["traffic"] = measured_traffic(kernel, workload) if workload else None
    r["kernel"] = kernel
    return r


def make_step(name, args):
    if name == "batched":
        return synth.BATCHED, BatchedStep(synth.BATCHED, args.splits)
    w = synth.WORKLOADS[name]
    return w, GqaStep(w, args.splits, window=args.window, rope=args.rope, page_size=args.paged)


def measure(name, args, flush, stream, first):
    """All GPU figures of one workload."""
    w, step = make_step(name, args)
    log("workload", name, "-", step.describe())
    sh = stream.cuda_stream
    res = {"workload": step.describe()}

    # Warm-up, cold order: until --warmup steps and --min-warmup-s of work have run (the shader
    # clock ramps over a few milliseconds of launches; longer on the first workload of the run).
    min_s = args.min_warmup_s if first else args.min_warmup_s / 2
    t_warm = time.perf_counter()
    n_warm = 0
    while n_warm < args.warmup or time.perf_counter() - t_warm < min_s:
        flush()
        step.splice(sh)
        flush()
        step.attention(sh)
        n_warm += 1
        if n_warm % 8 == 0:
            torch.cuda.synchronize()
    torch.cuda.synchronize()
    res["warmup_steps_run"] = n_warm

    # Timed steps, every launch cold.
    K = args.steps
    ev = [[torch.cuda.Event(enable_timing=True) for _ in range(4)] for _ in range(K)]
    torch.cuda.synchronize()
    t_wall = time.perf_counter()
    for e in ev:
        flush()
        e[0].record(stream)
        step.splice(sh)
        e[1].record(stream)
        flush()
        e[2].record(stream)
        step.attention(sh)
        e[3].record(stream)
    torch.cuda.synchronize()
    t_wall = time.perf_counter() - t_wall
    splice_ms = [e[0].elapsed_time(e[1]) for e in ev]
    attn_ms = [e[2].elapsed_time(e[3]) for e in ev]
    s_ms, a_ms = sum(splice_ms) / K, sum(attn_ms) / K
    bf16 = getattr(w, "dtype", "bf16") == "bf16"
    s_bytes, a_flops, a_bytes = step.splice_bytes(), step.attn_flops(), step.attn_bytes()
    ai = a_flops / a_bytes
    ridge = BF16_PEAK_TFLOPS * 1e12 / (HBM_PEAK_GBS * 1e9)
    a_kernel = "attn_mla_bf16" if getattr(w, "mla", False) else ("attn_gqa_bf16" if bf16 else "attn_gqa_f32")
    wl_key = None if (args.window or args.paged or args.rope != "theta") else name
    splice_roof = roofline("hbm", "splice_kernel", s_bytes, s_ms, workload=wl_key)
    if bf16 and ai < ridge:
        attn_roof = roofline("hbm", a_kernel, a_bytes, a_ms, workload=wl_key)
    else:
        attn_roof = roofline("mfma", a_kernel, a_flops, a_ms, bf16=bf16, workload=wl_key)
    splice_roof["algorithmic_bytes"] = s_bytes
    attn_roof["algorithmic_bytes"] = a_bytes
    attn_roof["algorithmic_flops"] = a_flops
    res.update({
        "ms_per_step": round(s_ms + a_ms, 4),
        "wall_ms_per_step_with_flushes": round(t_wall / K * 1e3, 4),
        "dtype": "bf16" if bf16 else "f32",
        "splice_bytes": s_bytes, "attention_flops": a_flops, "attention_bytes": a_bytes,
        "attention_splits": int(step.desc.n_splits) or "auto", "workspace_bytes": step.ws_bytes,
        "splice": dict(_stats(splice_ms), gbps=round(s_bytes / (s_ms * 1e-3) / 1e9, 1)),
        "attention": dict(_stats(attn_ms), tflops=round(a_flops / (a_ms * 1e-3) / 1e12, 2),
                          gbps=round(a_bytes / (a_ms * 1e-3) / 1e9, 1), arith_intensity=round(ai, 1),
                          bound=attn_roof["bound"]),
        "roofline": splice_roof if s_ms >= a_ms else attn_roof,
        "roofline_kernels": [splice_roof, attn_roof],
    })
    if hasattr(step, "splice_bytes_per_segment"):
        # the same splice counted with one source read per segment (each sequence spliced on its own)
        b = step.splice_bytes_per_segment()
        res["splice_bytes_per_segment_reads"] = b
        res["splice"]["gbps_per_segment_reads"] = round(b / (s_ms * 1e-3) / 1e9, 1)

    # Warm: the same steps back to back, no flush (the attention finds part of the splice's
    # writes in the last-level cache).
    if not args.no_warm:
        evw = [[torch.cuda.Event(enable_timing=True) for _ in range(3)] for _ in range(K)]
        torch.cuda.synchronize()
        for e in evw:
            e[0].record(stream)
            step.splice(sh)
            e[1].record(stream)
            step.attention(sh)
            e[2].record(stream)
        torch.cuda.synchronize()
        ws_ = [e[0].elapsed_time(e[1]) for e in evw]
        wa_ = [e[1].elapsed_time(e[2]) for e in evw]
        res["warm"] = {"splice": _stats(ws_), "attention": _stats(wa_),
                       "ms_per_step": round((sum(ws_) + sum(wa_)) / K, 4)}

    # One launch per layer (single-sequence workloads): from the host, and replayed from a graph.
    if isinstance(step, GqaStep) and not args.paged and not args.no_layer_calls:
        res["attention_layer_calls"] = layer_calls(step, w, args, flush, stream)
    return res


def layer_calls(step, w, args, flush, stream):
    sh = stream.cuda_stream
    step.layer_calls_setup()
    for _ in range(3):
        step.attention_layer_calls(sh)
    torch.cuda.synchronize()
    reps = max(5, min(args.steps, 20))

    def timed(run):
        lev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(reps)]
        for a, b in lev:
            flush()
            a.record(stream)
            run()
            b.record(stream)
        torch.cuda.synchronize()
        return [a.elapsed_time(b) for a, b in lev]

    eager = timed(lambda: step.attention_layer_calls(sh))
    ref = step.out.clone()
    # The same calls captured once into a graph (the library allocates nothing and records no
    # memset, so the calls capture as they are); every replay must reproduce the eager output.
    g = torch.cuda.CUDAGraph()
    torch.cuda.synchronize()
    with torch.cuda.graph(g):
        step.attention_layer_calls(torch.cuda.current_stream().cuda_stream)
    torch.cuda.synchronize()
    step.out.zero_()
    g.replay()
    torch.cuda.synchronize()
    if not torch.equal(step.out, ref):
        raise RuntimeError("graph replay of the per-layer attention calls differs from the eager calls")
    graph = timed(g.replay)
    if not torch.equal(step.out, ref):
        raise RuntimeError("graph replays of the per-layer attention calls differ from the eager calls")
    del g
    e_ms, g_ms = sum(eager) / reps, sum(graph) / reps
    return {"launches_per_step": w.n_layers, "splits": pkv_splits(step), "workspace_bytes": step.layer_ws_bytes,
            "eager": dict(_stats(eager), us_per_layer=round(e_ms * 1e3 / w.n_layers, 2)),
            "graph": dict(_stats(graph), us_per_layer=round(g_ms * 1e3 / w.n_layers, 2),
                          tflops=round(step.attn_flops() / (g_ms * 1e-3) / 1e12, 2),
                          gbps=round(step.attn_bytes() / (g_ms * 1e-3) / 1e9, 1))}


def pkv_splits(step):
    """Split count the library plans for one layer (from the workspace it asks for)."""
    w = step.w
    if step.layer_ws_bytes == 0:
        return 1
    per_split = w.n_q * w.n_heads * (w.v_dim + 1) * 4
    return step.layer_ws_bytes // per_split


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--min-warmup-s", type=float, default=0.5,
                    help="keep warming up until this much wall time has passed (clock ramp; half of it for "
                         "every workload after the first)")
    ap.add_argument("--workload", default="all", choices=["all"] + list(ORDER))
    ap.add_argument("--splits", type=int, default=0, help="KV splits for attention (0 = library choice)")
    ap.add_argument("--rope", default="theta", choices=["theta", "mrope_sectioned", "mrope_interleaved", "llama31"],
                    help="splice frequencies: the theta schedule, or an explicit table through "
                         "pkv_reposition_splice_freqs (M-RoPE temporal move, Llama-3.1 scaling)")
    ap.add_argument("--window", type=int, default=0,
                    help="sliding-window attention over the full cache (0 = causal; single-sequence workloads)")
    ap.add_argument("--paged", type=int, default=0, help="page size of a paged KV cache (0 = contiguous cache)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-warm", action="store_true", help="skip the back-to-back (warm) figures")
    ap.add_argument("--no-layer-calls", action="store_true", help="skip the one-launch-per-layer figures")
    ap.add_argument("--cpu-budget", type=float, default=10.0, help="seconds of oracle time per workload (about)")
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
    names = list(ORDER) if args.workload == "all" else [args.workload]
    if (args.window or args.rope != "theta" or args.paged) and "batched" in names:
        names = [n for n in names if n != "batched"]
    stream = torch.cuda.current_stream()
    flush = Flush()
    configs = {}
    t_gpu = time.perf_counter()
    for i, name in enumerate(names):
        configs[name] = measure(name, args, flush, stream, first=(i == 0))
        torch.cuda.synchronize()
        torch.cuda.empty_cache()
    t_gpu = time.perf_counter() - t_gpu
    cp = device_copy_gbps()
    sc = stream_copy_gbps(flush)
    for r in configs.values():
        r["splice"]["of_device_copy"] = round(r["splice"]["gbps"] / cp, 4)
        r["splice"]["of_stream_copy"] = round(r["splice"]["gbps"] / sc, 4)
    if not args.no_cpu_baseline:
        for name in names:
            log("timing the CPU oracle:", name)
            configs[name]["cpu_baseline"] = (cpu_baseline_batched(synth.BATCHED, args.cpu_budget) if name == "batched"
                                             else cpu_baseline(synth.WORKLOADS[name], args.cpu_budget))
    head_name = names[-1]
    head = configs[head_name]
    result = {
        "metric": METRIC,
        "value": head["splice"]["gbps"],
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": head["ms_per_step"],
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": head["dtype"],
        "data": "synthetic",
        "config": {"workload": head["workload"], "name": head_name, "splice_bytes": head["splice_bytes"],
                   "attention_flops": head["attention_flops"], "attention_bytes": head["attention_bytes"],
                   "attention_splits": head["attention_splits"], "workspace_bytes": head["workspace_bytes"],
                   "timing": "HIP events per launch, every timed launch after a 1 GiB flush (cold)"},
        "splice": head["splice"],
        "attention": head["attention"],
        "roofline": head["roofline"],
        "roofline_kernels": head["roofline_kernels"],
        "device_copy_gbps": round(cp, 1),
        "stream_copy_gbps": round(sc, 1),
        "gpu_wall_s": round(t_gpu, 2),
        "configs": configs,
    }
    if "cpu_baseline" in head:
        result["cpu_baseline"] = head["cpu_baseline"]
    if "warm" in head:
        result["warm"] = head["warm"]
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
