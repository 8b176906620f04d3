"""Shared helpers for the GPU parity tests: storage-bit conversions, the bf16
ulp criterion for re-rotated keys, the attention tolerance, and input
assembly (inputs are drawn by the seeded generators and, where they must be
post-RoPE, rotated by the oracle; nothing here comes from the HIP path)."""
import math
import sys

import numpy as np
import torch

import oracle
from paper_2606_17107_amd import pkv, synth


def log(*args):
    print(*args, flush=True)
    sys.stdout.flush()


def bits_to_f64(b: np.ndarray) -> np.ndarray:
    if b.dtype == np.uint16:
        return (b.astype(np.uint32) << 16).view(np.float32).astype(np.float64)
    return np.asarray(b, dtype=np.float64)


def host_bits(t: torch.Tensor) -> np.ndarray:
    return synth.to_numpy_bits(t)


def dev(a: np.ndarray, device="cuda") -> torch.Tensor:
    return synth.from_numpy_bits(a).to(device)


def bf16_quantum(x: np.ndarray) -> np.ndarray:
    """Spacing of bf16 values in the binade of |x| (x > 0): 2^(floor(log2 x) - 7)."""
    x = np.maximum(np.abs(x), 2.0 ** -126)
    e = np.floor(np.log2(x))
    return np.exp2(e - 7)


def rotary_pair_partner(c: np.ndarray, offset: int, r: int, style: int) -> np.ndarray:
    rel = c - offset
    if style == synth.HALF:
        return np.where(rel < r // 2, c + r // 2, c - r // 2)
    return np.where(rel % 2 == 0, c + 1, c - 1)


FLOOR_FRACTION = 1e-5


def check_rotated_keys(got: np.ndarray, want: np.ndarray, offset: int, r: int, style: int, n_rotated=None):
    """Compare re-rotated bf16 keys (last axis = channels) to the oracle.

    Pass iff |g - o| <= q(max(|o|, |g|, 2^-12 * ||pair||)), where q is the bf16
    spacing at that magnitude and ||pair|| the norm of the element's rotary
    pair: one bf16 ulp, with a floor for values that cancel to near zero.
    The floor may serve at most FLOOR_FRACTION of the re-rotated elements
    (n_rotated; default: every element of the rotary slice in `got`): fp32
    cancellation with exact coefficients needs it for about 1e-6 of them, so a
    larger count means an inaccurate rotation hidden by the floor.  A case with
    fewer than 1e5 rotated elements may still use it once (at a 1e-6 rate one
    such element turns up in a few percent of those cases).
    Returns (number of elements not bit-equal, number that needed the floor)."""
    g = bits_to_f64(got)
    o = bits_to_f64(want)
    d = got.shape[-1]
    c = np.arange(d)
    rot = (c >= offset) & (c < offset + r)
    diff = got != want
    assert not np.any(diff[..., ~rot]), "non-rotary channels must be bit-exact"
    if not diff.any():
        return 0, 0
    idx = np.nonzero(diff)
    ch = idx[-1]
    partner = rotary_pair_partner(ch, offset, r, style)
    pidx = idx[:-1] + (partner,)
    pair_norm = np.hypot(o[idx], o[pidx])
    gv, ov = g[idx], o[idx]
    mag = np.maximum(np.maximum(np.abs(ov), np.abs(gv)), 2.0 ** -12 * pair_norm)
    ok = np.abs(gv - ov) <= bf16_quantum(mag)
    bad = np.count_nonzero(~ok)
    assert bad == 0, "%d re-rotated elements beyond 1 bf16 ulp (e.g. got %r want %r)" % (
        bad, gv[~ok][:4], ov[~ok][:4])
    plain = np.abs(gv - ov) <= bf16_quantum(np.maximum(np.abs(ov), np.abs(gv)))
    n_floor = int(np.count_nonzero(~plain))
    if n_rotated is None:
        n_rotated = int(np.prod(got.shape[:-1])) * r
    assert n_floor <= max(FLOOR_FRACTION * n_rotated, 1), (
        "%d of %d re-rotated elements needed the near-zero floor (bound %.0e of them)"
        % (n_floor, n_rotated, FLOOR_FRACTION))
    return int(diff.sum()), n_floor


def check_attention_close(got: np.ndarray, want: np.ndarray, max_abs=2e-2, mean_abs=2e-3, rel_l2=1e-2):
    """bf16 attention outputs vs the fp64 oracle: max-abs, mean-abs and relative L2."""
    g = bits_to_f64(got) if got.dtype == np.uint16 else got.astype(np.float64)
    err = np.abs(g - want)
    rl2 = np.linalg.norm(g - want) / max(np.linalg.norm(want), 1e-300)
    stats = dict(max_abs=float(err.max()), mean_abs=float(err.mean()), rel_l2=float(rl2))
    assert stats["max_abs"] <= max_abs, stats
    assert stats["mean_abs"] <= mean_abs, stats
    assert stats["rel_l2"] <= rel_l2, stats
    return stats


def rope_cache(k_pre_bits: np.ndarray, positions: np.ndarray, w) -> np.ndarray:
    """Oracle RoPE of pre-RoPE rows [..., slots, d] at per-slot positions."""
    pos = np.broadcast_to(positions.astype(np.int32), k_pre_bits.shape[:-1])
    return oracle.rope_rows(k_pre_bits, pos, w.theta, w.rope_dim, w.rope_offset, w.rope_style)


def rope_queries(q_pre_bits: np.ndarray, q_pos: np.ndarray, w) -> np.ndarray:
    """Oracle RoPE of queries [L][n_q][H][d] at their positions (only the rotary slice)."""
    pos = np.broadcast_to(q_pos.astype(np.int32)[None, :, None], q_pre_bits.shape[:-1])
    return oracle.rope_rows(q_pre_bits, pos, w.theta, w.rope_dim, w.rope_offset, w.rope_style)


def small_workload(name="small", L=2, H=8, Hkv=2, d=128, theta=1e4, style=0, dtype="bf16", skill=200,
                   src0=0, dst0=37, ctx=400, n_q=45, rope_dim=None, rope_offset=0):
    """A Workload of test size spanning several tiles and ragged tails."""
    return synth.Workload(name, L, H, Hkv, d, d, theta, rope_dim or d, rope_offset, style, dtype, skill, src0,
                          dst0, ctx, n_q, 1.0 / math.sqrt(d))


# ---- guard bands around device outputs and workspaces --------------------------
# A kernel that writes outside the tensor it was given would go unnoticed by
# comparisons of the tensor itself; these buffers place the tensor between two
# bands of a sentinel bit pattern and check the bands afterwards.

GUARD = 4096                      # elements (or bytes for a workspace) on each side
_SENTINEL = {torch.bfloat16: (torch.int16, 0x7FC1), torch.float32: (torch.int32, 0x7FC00001),
             torch.uint8: (torch.uint8, 0xA5)}


class Guarded:
    """A contiguous tensor of `shape` inside a buffer with sentinel bands; the
    tensor's own elements start as the sentinel too (so rows a call must not
    write can be checked with `untouched`)."""

    def __init__(self, shape, dtype, device="cuda"):
        self.n = int(np.prod(shape))
        self.buf = torch.empty(GUARD + self.n + GUARD, dtype=dtype, device=device)
        int_t, pattern = _SENTINEL[dtype]
        self.raw = self.buf.view(int_t)
        self.pattern = pattern if int_t != torch.int16 else pattern - (1 << 16) * (pattern >= 1 << 15)
        self.raw.fill_(self.pattern)
        self.t = self.buf[GUARD:GUARD + self.n].view(shape)

    def check(self, what="tensor"):
        r = self.raw.cpu().numpy()
        bad_lo = np.count_nonzero(r[:GUARD] != self.pattern)
        bad_hi = np.count_nonzero(r[GUARD + self.n:] != self.pattern)
        assert bad_lo == 0 and bad_hi == 0, "%s: %d / %d guard elements overwritten before / after it" % (
            what, bad_lo, bad_hi)

    def untouched(self, index):
        """True where the tensor's elements (selected by `index`) still hold the sentinel."""
        r = self.raw[GUARD:GUARD + self.n].view(self.t.shape)
        return bool((r[index] == self.pattern).all().item())


def guarded_attention(q, k_cache, v_cache, q_pos, kv_len, scale, max_kv_len, d_v, **kw):
    """pkv.suffix_attention into a Guarded output with a Guarded workspace; checks both guard bands and
    returns (output Guarded, workspace bytes)."""
    L, rows, H = q.shape[:3]
    out = Guarded((L, rows, H, d_v), q.dtype)
    desc = pkv.make_attn_desc(q, k_cache, v_cache, out.t, max_kv_len,
                              **{k: kw[k] for k in ("n_seqs", "cu_q", "kv_base", "max_q", "variant", "n_splits",
                                                    "window") if k in kw})
    need = pkv.pkv_attention_workspace_size(desc, H, k_cache.shape[1], q.shape[3])
    ws = Guarded((need,), torch.uint8) if need else None
    pkv.suffix_attention(q, k_cache, v_cache, out.t, q_pos, kv_len, scale, max_kv_len,
                         workspace=None if ws is None else ws.t, **kw)
    torch.cuda.synchronize()
    out.check("attention output")
    if ws is not None:
        ws.check("attention workspace")
    return out, need
