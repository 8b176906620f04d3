"""Seeded synthetic workloads for reposition+splice and suffix attention.

This module only draws numbers and lays out positions; it holds none of the
method's arithmetic (no rotation, no attention).  Both the HIP path and the
CPU oracle take their inputs from here.

Every draw is N(0, 1) in fp32 from one seeded ``torch.Generator`` per case,
in a fixed order, cast to the storage dtype by torch (round to nearest even
for bf16).  Keys and queries are returned *pre-RoPE*: callers rotate them to
their positions with their own implementation.

Workload shapes follow the models the paper runs (all GQA with per-token KV,
plus DeepSeek-V2-style MLA for the adapter), sized as:
  tiny     1 layer, 4/2 heads, d 64, fp32, 128-token skill 0..127 -> 300..427
           in a 512-slot cache, 16 suffix queries at 512..527
  gqa8b    Llama-3-8B shape: 32 layers, 32/8 heads, d 128, theta 5e5, 4096-token
           skill spliced at 2000 into 8192 slots, 64-token suffix (kv 8256)
  batched  16 sequences x skills of 1024/2048/4096 tokens at random disjoint
           offsets in 8k-12k contexts, 256-token suffix per sequence
  long32k  28 layers, 28/4 heads, d 128, theta 1e6, 32768-token skill moved by
           +16384 into 49152 slots, 1024-token suffix (kv 50176)
  mla      27 layers, 16 heads, rows of 512 latent + 64 k_pe, theta 1e4,
           16384-token skill spliced at 8192 into 32768 slots, 128-token suffix
           (kv 32896), absorbed 576-dim queries, scale 1/sqrt(192)
"""
from __future__ import annotations

import dataclasses
import math
from typing import List, Optional

import numpy as np
import torch

HALF = 0
INTERLEAVED = 1


@dataclasses.dataclass(frozen=True)
class Workload:
    name: str
    n_layers: int
    n_heads: int          # query heads
    n_kv_heads: int       # KV heads (1 for MLA: one shared latent row)
    head_dim: int         # K row / query width (576 for MLA)
    v_dim: int            # V width (512 for MLA: the latent, a prefix of the K row)
    theta: float
    rope_dim: int
    rope_offset: int
    rope_style: int
    dtype: str            # "bf16" | "f32"
    skill_tokens: int
    src_pos0: int
    dst_pos0: int
    ctx_slots: int        # destination context before the suffix
    n_q: int              # suffix tokens, at positions ctx_slots .. ctx_slots+n_q-1
    scale: float
    mla: bool = False

    @property
    def kv_len(self) -> int:
        return self.ctx_slots + self.n_q

    @property
    def group(self) -> int:
        return self.n_heads // self.n_kv_heads

    @property
    def elem_bytes(self) -> int:
        return 2 if self.dtype == "bf16" else 4

    def splice_bytes(self) -> int:
        """Algorithmic bytes of one reposition+splice: skill K/V (or MLA rows) read once, written once."""
        row = self.head_dim + (0 if self.mla else self.v_dim)
        return 2 * self.skill_tokens * self.n_layers * self.n_kv_heads * row * self.elem_bytes

    def attn_flops(self, window: int = 0) -> int:
        """Algorithmic flops: 2*(d_qk + d_v) per (query, head, visible key), all layers
        (window > 0: keys j > q_pos - window only)."""
        vis = 0
        for i in range(self.n_q):
            p = self.ctx_slots + i
            lo = max(0, p - window + 1) if window > 0 else 0
            vis += max(0, min(self.kv_len, p + 1) - lo)
        return 2 * (self.head_dim + self.v_dim) * self.n_heads * vis * self.n_layers

    def attn_bytes(self, window: int = 0) -> int:
        """Algorithmic bytes: K/V over the slots some query sees read once per layer, Q read,
        O written."""
        kv_row = self.head_dim if self.mla else self.head_dim + self.v_dim
        first = max(0, self.ctx_slots - window + 1) if window > 0 else 0
        kv = (self.kv_len - first) * self.n_kv_heads * kv_row
        qo = self.n_q * self.n_heads * (self.head_dim + self.v_dim)
        return (kv + qo) * self.elem_bytes * self.n_layers


TINY = Workload("tiny", 1, 4, 2, 64, 64, 10000.0, 64, 0, HALF, "f32", 128, 0, 300, 512, 16,
                1.0 / math.sqrt(64))
GQA8B = Workload("gqa8b", 32, 32, 8, 128, 128, 500000.0, 128, 0, HALF, "bf16", 4096, 0, 2000, 8192,
                 64, 1.0 / math.sqrt(128))
LONG32K = Workload("long32k", 28, 28, 4, 128, 128, 1000000.0, 128, 0, HALF, "bf16", 32768, 0, 16384,
                   49152, 1024, 1.0 / math.sqrt(128))
MLA = Workload("mla", 27, 16, 1, 576, 512, 10000.0, 64, 512, INTERLEAVED, "bf16", 16384, 0, 8192,
               32768, 128, 1.0 / math.sqrt(192), mla=True)

WORKLOADS = {w.name: w for w in (TINY, GQA8B, LONG32K, MLA)}


def torch_dtype(w: Workload):
    return torch.bfloat16 if w.dtype == "bf16" else torch.float32


class Draws:
    """Sequential N(0,1) draws from one seeded generator on ``device``."""

    def __init__(self, seed: int, device="cpu"):
        self.device = torch.device(device)
        self.gen = torch.Generator(device=self.device)
        self.gen.manual_seed(int(seed))

    def normal(self, shape, dtype=torch.bfloat16) -> torch.Tensor:
        x = torch.randn(tuple(shape), generator=self.gen, dtype=torch.float32, device=self.device)
        return x.to(dtype)

    def integers(self, low: int, high: int, n: int) -> List[int]:
        """n integers uniform in [low, high] inclusive."""
        t = torch.randint(low, high + 1, (n,), generator=self.gen, device=self.device)
        return [int(v) for v in t.cpu().tolist()]


def gqa_case(w: Workload, seed: int = 0, device="cpu", layers: Optional[int] = None):
    """Tensors for one single-sequence workload (GQA or MLA), in draw order.

    Returns a dict with
      ctx_k, ctx_v     destination cache [L][Hkv][kv_len][d] (all slots drawn;
                       the splice and the suffix overwrite their slots)
      skill_k_pre      pre-RoPE skill keys [L][Hkv][n][d]
      skill_v          skill values [L][Hkv][n][dv]
      q_pre            pre-RoPE suffix queries [L][n_q][H][d]
      suf_k_pre, suf_v suffix keys (pre-RoPE) / values [L][Hkv][n_q][*]
      src_pos, dst_pos int32 [n]; q_pos int32 [n_q]; kv_len int
    For MLA the V tensors are absent (the latent is the first v_dim channels
    of each K row)."""
    L = w.n_layers if layers is None else layers
    dt = torch_dtype(w)
    d = Draws(seed, device)
    out = {}
    out["ctx_k"] = d.normal((L, w.n_kv_heads, w.kv_len, w.head_dim), dt)
    if not w.mla:
        out["ctx_v"] = d.normal((L, w.n_kv_heads, w.kv_len, w.v_dim), dt)
    out["skill_k_pre"] = d.normal((L, w.n_kv_heads, w.skill_tokens, w.head_dim), dt)
    if not w.mla:
        out["skill_v"] = d.normal((L, w.n_kv_heads, w.skill_tokens, w.v_dim), dt)
    out["q_pre"] = d.normal((L, w.n_q, w.n_heads, w.head_dim), dt)
    out["suf_k_pre"] = d.normal((L, w.n_kv_heads, w.n_q, w.head_dim), dt)
    if not w.mla:
        out["suf_v"] = d.normal((L, w.n_kv_heads, w.n_q, w.v_dim), dt)
    out["src_pos"] = torch.arange(w.src_pos0, w.src_pos0 + w.skill_tokens, dtype=torch.int32)
    out["dst_pos"] = torch.arange(w.dst_pos0, w.dst_pos0 + w.skill_tokens, dtype=torch.int32)
    out["q_pos"] = torch.arange(w.ctx_slots, w.ctx_slots + w.n_q, dtype=torch.int32)
    out["kv_len"] = w.kv_len
    return out


# ---- batched composition --------------------------------------------------

@dataclasses.dataclass(frozen=True)
class BatchedWorkload:
    name: str = "batched"
    n_seqs: int = 16
    skills: tuple = (1024, 2048, 4096)
    ctx_min: int = 8192
    ctx_max: int = 12288
    src_pos_max: int = 2048
    n_layers: int = 32
    n_heads: int = 32
    n_kv_heads: int = 8
    head_dim: int = 128
    theta: float = 500000.0
    n_q: int = 256
    dtype: str = "bf16"

    @property
    def scale(self) -> float:
        return 1.0 / math.sqrt(self.head_dim)


BATCHED = BatchedWorkload()


def batched_plan(bw: BatchedWorkload, seed: int = 0):
    """Random layout of the batched composition (host-side integers only).

    Per sequence s: context length C_s ~ U{ctx_min..ctx_max}; the skills are
    placed in shuffled order at disjoint offsets by splitting the free space
    C_s - sum(skills) into len(skills)+1 gaps with a uniform random
    composition.  Each skill carries a source position offset
    src_pos0 ~ U{0..src_pos_max} (so delta takes either sign).  The suffix
    occupies positions C_s .. C_s+n_q-1; kv_len = C_s + n_q.  Sequences are
    packed back to back in one slot axis (seq_base).  Skills live back to back
    in one source slot axis (skill_base)."""
    d = Draws(seed + 7919, "cpu")
    n_sk = len(bw.skills)
    skill_base = [0]
    for n in bw.skills[:-1]:
        skill_base.append(skill_base[-1] + n)
    src_pos0 = d.integers(0, bw.src_pos_max, n_sk)
    seqs = []
    seq_base = 0
    for s in range(bw.n_seqs):
        C = d.integers(bw.ctx_min, bw.ctx_max, 1)[0]
        order = torch.randperm(n_sk, generator=d.gen).tolist()
        free = C - sum(bw.skills)
        # uniform random composition of `free` into n_sk+1 non-negative gaps
        cuts = sorted(d.integers(0, free, n_sk))
        gaps = [cuts[0]] + [cuts[i] - cuts[i - 1] for i in range(1, n_sk)] + [free - cuts[-1]]
        pos = gaps[0]
        segs = []
        for j, k in enumerate(order):
            segs.append(dict(skill=k, src_slot0=skill_base[k], n_tokens=bw.skills[k],
                             src_pos0=src_pos0[k], dst_pos0=pos))
            pos += bw.skills[k] + gaps[j + 1]
        seqs.append(dict(ctx=C, kv_len=C + bw.n_q, seq_base=seq_base, segs=segs))
        seq_base += C + bw.n_q
    return dict(skill_base=skill_base, src_pos0=src_pos0, seqs=seqs, total_slots=seq_base,
                skill_slots=sum(bw.skills))


def batched_case(bw: BatchedWorkload, plan, seed: int = 0, device="cpu", layers: Optional[int] = None):
    """Tensors of the batched composition, in draw order.

      ctx_k, ctx_v   packed caches [L][Hkv][total_slots][d]
      skill_k_pre    skill library keys (pre-RoPE) [L][Hkv][sum(skills)][d]
      skill_v        skill library values
      q_pre          packed suffix queries [L][n_seqs*n_q][H][d] (pre-RoPE)
      suf_k_pre, suf_v  [L][Hkv][n_seqs*n_q][d]
    """
    L = bw.n_layers if layers is None else layers
    dt = torch.bfloat16
    d = Draws(seed, device)
    T = plan["total_slots"]
    S = plan["skill_slots"]
    nq = bw.n_q * bw.n_seqs
    out = {}
    out["ctx_k"] = d.normal((L, bw.n_kv_heads, T, bw.head_dim), dt)
    out["ctx_v"] = d.normal((L, bw.n_kv_heads, T, bw.head_dim), dt)
    out["skill_k_pre"] = d.normal((L, bw.n_kv_heads, S, bw.head_dim), dt)
    out["skill_v"] = d.normal((L, bw.n_kv_heads, S, bw.head_dim), dt)
    out["q_pre"] = d.normal((L, nq, bw.n_heads, bw.head_dim), dt)
    out["suf_k_pre"] = d.normal((L, bw.n_kv_heads, nq, bw.head_dim), dt)
    out["suf_v"] = d.normal((L, bw.n_kv_heads, nq, bw.head_dim), dt)
    return out


# ---- rotary frequency tables (model configuration inputs of the splice) ----

def rope_omega(theta: float, rope_dim: int) -> np.ndarray:
    """The plain RoPE schedule theta^(-2i/r), i < r/2."""
    return theta ** (-2.0 * np.arange(rope_dim // 2, dtype=np.float64) / rope_dim)


def mrope_axes(rope_dim: int, sections=(16, 24, 24), layout: str = "sectioned") -> np.ndarray:
    """Axis (0 temporal, 1 height, 2 width) of each rotary pair of an M-RoPE head.

    sectioned: the first sections[0] pairs are temporal, the next sections[1]
    height, the rest width (the Qwen2.5-VL layout).  interleaved: pairs cycle
    temporal, height, width while each axis has pairs left in its section, and
    the remainder goes to the first axis that still has some (the Qwen3-VL
    layout spreads every axis over the whole frequency range)."""
    n = rope_dim // 2
    assert sum(sections) == n
    axes = np.empty(n, dtype=np.int32)
    if layout == "sectioned":
        axes[:] = np.repeat(np.arange(3), sections)
        return axes
    assert layout == "interleaved"
    left = list(sections)
    for i in range(n):
        a = i % 3
        if left[a] == 0:
            a = next(k for k in range(3) if left[k] > 0)
        axes[i] = a
        left[a] -= 1
    return axes


def mrope_temporal_omega(theta: float, rope_dim: int, sections=(16, 24, 24), layout: str = "sectioned"):
    """Frequencies that move an M-RoPE key along the temporal axis only: the plain
    schedule on the temporal pairs, zero on the height and width pairs."""
    return np.where(mrope_axes(rope_dim, sections, layout) == 0, rope_omega(theta, rope_dim), 0.0)


def llama31_omega(theta: float, rope_dim: int, factor: float = 8.0, low_freq_factor: float = 1.0,
                  high_freq_factor: float = 4.0, original_max_position: int = 8192) -> np.ndarray:
    """The Llama-3.1 rescaled schedule: wavelengths shorter than
    original/high_freq_factor keep their frequency, longer than
    original/low_freq_factor are divided by `factor`, and the band between is
    interpolated linearly in original/wavelength."""
    w = rope_omega(theta, rope_dim)
    wavelen = 2.0 * math.pi / w
    low_wl = original_max_position / low_freq_factor
    high_wl = original_max_position / high_freq_factor
    smooth = (original_max_position / wavelen - low_freq_factor) / (high_freq_factor - low_freq_factor)
    mid = (1.0 - smooth) * w / factor + smooth * w
    return np.where(wavelen < high_wl, w, np.where(wavelen > low_wl, w / factor, mid))


def batched_segments(plan):
    """Segment records (pkv_segment fields) of the batched composition: one per
    (sequence, skill), in sequence order."""
    segs = []
    for sq in plan["seqs"]:
        for sg in sq["segs"]:
            segs.append(dict(src_slot0=sg["src_slot0"], dst_seq_base=sq["seq_base"], n_tokens=sg["n_tokens"],
                             src_pos0=sg["src_pos0"], dst_pos0=sg["dst_pos0"], dst_seq_len=sq["kv_len"]))
    return segs


def batched_splice_bytes(bw: BatchedWorkload, plan) -> int:
    """Algorithmic bytes of the batched splice: the library's K and V rows read once (every distinct
    source slot, however many sequences splice it) and every spliced token's K and V rows written once,
    the least HBM traffic the composition needs."""
    src = set()
    for sq in plan["seqs"]:
        for sg in sq["segs"]:
            src.update(range(sg["src_slot0"], sg["src_slot0"] + sg["n_tokens"]))
    written = sum(sg["n_tokens"] for sq in plan["seqs"] for sg in sq["segs"])
    return 2 * (len(src) + written) * bw.n_layers * bw.n_kv_heads * bw.head_dim * 2


def batched_splice_bytes_per_segment(bw: BatchedWorkload, plan) -> int:
    """Bytes of the batched splice with every segment reading its own source (each spliced token's K and
    V rows read once and written once): the work of splicing each sequence on its own."""
    tokens = sum(sg["n_tokens"] for sq in plan["seqs"] for sg in sq["segs"])
    return 2 * 2 * tokens * bw.n_layers * bw.n_kv_heads * bw.head_dim * 2


def batched_attn_flops(bw: BatchedWorkload, plan) -> int:
    """Algorithmic flops of the ragged suffix attention: 4*d per (query, head, visible key)."""
    vis = 0
    for sq in plan["seqs"]:
        C = sq["ctx"]
        vis += sum(min(sq["kv_len"], C + i + 1) for i in range(bw.n_q))
    return 4 * bw.head_dim * bw.n_heads * vis * bw.n_layers


def batched_attn_bytes(bw: BatchedWorkload, plan) -> int:
    """Algorithmic bytes: each sequence's K/V over its kv_len read once per layer, Q read, O written."""
    kv = sum(sq["kv_len"] for sq in plan["seqs"]) * bw.n_kv_heads * 2 * bw.head_dim
    qo = bw.n_seqs * bw.n_q * bw.n_heads * 2 * bw.head_dim
    return (kv + qo) * 2 * bw.n_layers


def to_numpy_bits(t: torch.Tensor) -> np.ndarray:
    """Storage bits of a CPU tensor as numpy: bf16 -> uint16, fp32 -> float32."""
    t = t.detach().cpu().contiguous()
    if t.dtype == torch.bfloat16:
        return t.view(torch.int16).numpy().view(np.uint16)
    if t.dtype == torch.float32:
        return t.numpy()
    if t.dtype == torch.int32:
        return t.numpy()
    raise TypeError(t.dtype)


def from_numpy_bits(a: np.ndarray) -> torch.Tensor:
    """Inverse of :func:`to_numpy_bits`."""
    if a.dtype == np.uint16:
        return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).view(torch.bfloat16)
    return torch.from_numpy(np.ascontiguousarray(a))
