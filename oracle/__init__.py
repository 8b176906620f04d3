"""fp64 CPU oracle for RoPE reposition+splice and causal suffix attention.

TEST INFRASTRUCTURE ONLY.  Only ``tests/``, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of ``bench.py`` may import this package.  It shares no
code with the HIP library: the arithmetic lives in ``pkvref.c`` (plain C,
fp64, plain loops, OpenMP only across independent rows), and this module only
marshals numpy arrays into it.

Storage conventions: bf16 tensors are numpy ``uint16`` arrays holding the bf16
bit patterns; fp32 tensors are ``float32`` arrays.  Cache tensors are
``[layers][kv_heads][slots][channels]`` (any element strides; channels
contiguous), queries ``[tokens][heads][channels]``.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "pkvref.c")
_LIB_PATH = os.path.join(_HERE, "libpkvref.so")

BF16 = 0
F32 = 1
HALF = 0
INTERLEAVED = 1

_lib = None


def build(force: bool = True) -> str:
    """Compile ``pkvref.c`` with gcc into ``libpkvref.so`` next to it."""
    if force or not os.path.exists(_LIB_PATH):
        tmp = _LIB_PATH + ".tmp%d" % os.getpid()
        subprocess.check_call(
            ["gcc", "-O2", "-fopenmp", "-fPIC", "-shared", "-std=c11", "-Wall", _SRC, "-o", tmp, "-lm"]
        )
        os.replace(tmp, _LIB_PATH)
    return _LIB_PATH


def _load():
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(_LIB_PATH):
        build(force=False)
    lib = ctypes.CDLL(_LIB_PATH)
    P = ctypes.c_void_p
    i32, i64, f64 = ctypes.c_int32, ctypes.c_int64, ctypes.c_double
    lib.pkvref_round_bf16.restype = ctypes.c_uint16
    lib.pkvref_round_bf16.argtypes = [f64]
    lib.pkvref_rope_omega.restype = f64
    lib.pkvref_rope_omega.argtypes = [f64, ctypes.c_int, ctypes.c_int]
    lib.pkvref_rope_rows.restype = None
    lib.pkvref_rope_rows.argtypes = [ctypes.c_int, P, P, i64, ctypes.c_int, P, f64, ctypes.c_int,
                                     ctypes.c_int, ctypes.c_int, P]
    lib.pkvref_reposition_splice.restype = i64
    lib.pkvref_reposition_splice.argtypes = [
        ctypes.c_int, P, P, P, P, P, P, i64, ctypes.c_int, ctypes.c_int, ctypes.c_int, ctypes.c_int,
        f64, ctypes.c_int, ctypes.c_int, ctypes.c_int, P, P, P, P, i64, P, P]
    lib.pkvref_attention.restype = None
    lib.pkvref_attention.argtypes = [
        ctypes.c_int, P, P, P, P, P, P, i64, i64, ctypes.c_int, ctypes.c_int, ctypes.c_int,
        ctypes.c_int, f64, i64, i64, i64, i64, i64, i64, i64]
    lib.pkvref_max_threads.restype = ctypes.c_int
    lib.pkvref_set_threads.argtypes = [ctypes.c_int]
    _lib = lib
    return lib


def _dtype_code(a: np.ndarray) -> int:
    if a.dtype == np.uint16:
        return BF16
    if a.dtype == np.float32:
        return F32
    raise TypeError("oracle tensors are uint16 (bf16 bits) or float32, got %s" % a.dtype)


def _ptr(a):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


def _estrides(a: np.ndarray):
    return [s // a.itemsize for s in a.strides]


def max_threads() -> int:
    return _load().pkvref_max_threads()


def set_threads(n: int) -> None:
    _load().pkvref_set_threads(int(n))


def round_bf16(x: float) -> int:
    """bf16 bit pattern of fp64 ``x`` rounded once, ties to even."""
    return int(_load().pkvref_round_bf16(float(x)))


def rope_omega(theta: float, r: int, i: int) -> float:
    """Rotary frequency theta^(-2i/r) of pair ``i``."""
    return float(_load().pkvref_rope_omega(float(theta), int(r), int(i)))


def _omega_arg(omega, rope_dim):
    if omega is None:
        return None, None
    w = np.ascontiguousarray(omega, dtype=np.float64)
    assert w.shape == (rope_dim // 2,), "omega needs one frequency per rotary pair"
    return w, _ptr(w)


def rope_rows(x: np.ndarray, pos: np.ndarray, theta: float, rope_dim: int, rope_offset: int = 0,
              style: int = HALF, omega=None) -> np.ndarray:
    """Return R(pos[row]) x[row] for every row of ``x`` (last axis = channels).

    ``pos`` has one int32 position per row (shape ``x.shape[:-1]``).  ``omega``:
    optional per-pair frequencies replacing theta^(-2i/rope_dim)."""
    x = np.ascontiguousarray(x)
    d = x.shape[-1]
    n_rows = x.size // d
    pos = np.ascontiguousarray(np.broadcast_to(pos, x.shape[:-1]), dtype=np.int32).reshape(-1)
    assert pos.size == n_rows
    out = np.empty_like(x)
    w, wp = _omega_arg(omega, rope_dim)
    _load().pkvref_rope_rows(_dtype_code(x), _ptr(x), _ptr(out), n_rows, d, _ptr(pos), float(theta),
                             int(rope_dim), int(rope_offset), int(style), wp)
    return out


def reposition_splice(src_k, src_v, dst_k, dst_v, src_pos, dst_pos, theta, rope_dim, rope_offset=0,
                      style=HALF, dst_capacity=None, omega=None, dst_slot=None) -> int:
    """Splice ``src_k``/``src_v`` ``[L][Hkv][T][*]`` into ``dst_k``/``dst_v`` in place.

    dst_k[l][h][dst_pos[t]] = R(dst_pos[t] - src_pos[t]) src_k[l][h][t]; V copied.
    ``src_v``/``dst_v`` may be None (MLA rows).  Returns the number of tokens
    skipped because dst_pos fell outside [0, dst_capacity)."""
    dt = _dtype_code(src_k)
    assert dst_k.dtype == src_k.dtype and src_k.ndim == 4 and dst_k.ndim == 4
    L, H, T, d = src_k.shape
    v_dim = 0 if src_v is None else src_v.shape[-1]
    src_pos = np.ascontiguousarray(src_pos, dtype=np.int32)
    dst_pos = np.ascontiguousarray(dst_pos, dtype=np.int32)
    assert src_pos.size == T and dst_pos.size == T
    slots = None if dst_slot is None else np.ascontiguousarray(dst_slot, dtype=np.int32)
    assert slots is None or slots.size == T
    cap = dst_k.shape[2] if dst_capacity is None else int(dst_capacity)
    sks = np.array(_estrides(src_k)[:3], dtype=np.int64)
    dks = np.array(_estrides(dst_k)[:3], dtype=np.int64)
    svs = np.array(_estrides(src_v)[:3] if src_v is not None else [0, 0, 0], dtype=np.int64)
    dvs = np.array(_estrides(dst_v)[:3] if dst_v is not None else [0, 0, 0], dtype=np.int64)
    for a in (src_k, dst_k, src_v, dst_v):
        if a is not None:
            assert a.strides[-1] == a.itemsize, "channels must be contiguous"
    return int(_load().pkvref_reposition_splice(
        dt, _ptr(src_k), _ptr(src_v), _ptr(dst_k), _ptr(dst_v), _ptr(src_pos), _ptr(dst_pos), T, L, H,
        d, v_dim, float(theta), int(rope_dim), int(rope_offset), int(style), _ptr(sks), _ptr(svs),
        _ptr(dks), _ptr(dvs), cap, _omega_arg(omega, rope_dim)[1], _ptr(slots)))


def attention(q, k, v, q_pos, kv_len, scale, window=0):
    """Causal attention of one layer and one sequence, fp64 (``window`` > 0:
    slot j is also required to satisfy j > q_pos - window).

    q ``[n_q][H][d_qk]``, k ``[Hkv][slots][d_qk]``, v ``[Hkv][slots][d_v]`` (v may be a
    view into k, e.g. the MLA latent).  Returns ``(out [n_q][H][d_v] fp64,
    lse [n_q][H] fp64)``."""
    dt = _dtype_code(q)
    assert k.dtype == q.dtype and v.dtype == q.dtype
    n_q, H, d_qk = q.shape
    Hkv, slots, d_k = k.shape
    d_v = v.shape[-1]
    assert d_k >= d_qk and H % Hkv == 0 and v.shape[0] == Hkv
    assert kv_len <= slots
    for a in (q, k, v):
        assert a.strides[-1] == a.itemsize
    qs, ks, vs = _estrides(q), _estrides(k), _estrides(v)
    q_pos = np.ascontiguousarray(q_pos, dtype=np.int32)
    assert q_pos.size == n_q
    out = np.zeros((n_q, H, d_v), dtype=np.float64)
    lse = np.zeros((n_q, H), dtype=np.float64)
    _load().pkvref_attention(dt, _ptr(q), _ptr(k), _ptr(v), _ptr(out), _ptr(lse), _ptr(q_pos), n_q,
                             int(kv_len), H, Hkv, d_qk, d_v, float(scale), qs[0], qs[1], ks[0], ks[1],
                             vs[0], vs[1], int(window))
    return out, lse
