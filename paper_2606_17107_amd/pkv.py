"""Thin ctypes binding of libpkv (include/pkv.h), with the same names.

Only argument marshalling happens here: torch tensors contribute their device
pointers and strides, the caller's current HIP stream is passed through, and
every step of the computation runs in the HIP kernels of libpkv.so.  If the
library has not been built this module raises on first use; there is no
fallback implementation.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional, Sequence

import torch

_LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libpkv.so")

PKV_OK = 0
PKV_ERR_NULL = 1
PKV_ERR_SHAPE = 2
PKV_ERR_ALIGN = 3
PKV_ERR_ALIAS = 4
PKV_ERR_UNSUPPORTED = 5
PKV_ERR_DEVICE = 6
STATUS_NAMES = {0: "PKV_OK", 1: "PKV_ERR_NULL", 2: "PKV_ERR_SHAPE", 3: "PKV_ERR_ALIGN",
                4: "PKV_ERR_ALIAS", 5: "PKV_ERR_UNSUPPORTED", 6: "PKV_ERR_DEVICE"}

PKV_BF16 = 0
PKV_F32 = 1
PKV_ROPE_HALF = 0
PKV_ROPE_INTERLEAVED = 1
PKV_ATTN_GQA = 0
PKV_ATTN_MLA = 1

_i64x3 = ctypes.c_int64 * 3


class pkv_layout(ctypes.Structure):
    _fields_ = [
        ("dtype", ctypes.c_int32), ("n_layers", ctypes.c_int32), ("n_kv_heads", ctypes.c_int32),
        ("head_dim", ctypes.c_int32), ("v_dim", ctypes.c_int32), ("n_tokens", ctypes.c_int32),
        ("rope_offset", ctypes.c_int32), ("rope_style", ctypes.c_int32),
        ("dst_capacity", ctypes.c_int32), ("reserved", ctypes.c_int32),
        ("src_k_stride", _i64x3), ("src_v_stride", _i64x3), ("dst_k_stride", _i64x3),
        ("dst_v_stride", _i64x3), ("err_flag", ctypes.c_void_p),
    ]


class pkv_segment(ctypes.Structure):
    _fields_ = [
        ("src_slot0", ctypes.c_int64), ("dst_seq_base", ctypes.c_int64), ("n_tokens", ctypes.c_int32),
        ("src_pos0", ctypes.c_int32), ("dst_pos0", ctypes.c_int32), ("dst_seq_len", ctypes.c_int32),
    ]


class pkv_attn_desc(ctypes.Structure):
    _fields_ = [
        ("dtype", ctypes.c_int32), ("variant", ctypes.c_int32), ("n_layers", ctypes.c_int32),
        ("n_seqs", ctypes.c_int32), ("head_dim_v", ctypes.c_int32), ("total_q", ctypes.c_int32),
        ("max_q", ctypes.c_int32), ("max_kv_len", ctypes.c_int32), ("n_splits", ctypes.c_int32),
        ("window", ctypes.c_int32), ("cu_q", ctypes.c_void_p), ("kv_base", ctypes.c_void_p),
        ("cache_slots", ctypes.c_int64), ("q_stride", _i64x3), ("k_stride", _i64x3),
        ("v_stride", _i64x3), ("o_stride", _i64x3), ("lse_out", ctypes.c_void_p),
    ]


class pkv_paged_cache(ctypes.Structure):
    _fields_ = [
        ("page_size", ctypes.c_int32), ("max_pages", ctypes.c_int32), ("block_table", ctypes.c_void_p),
        ("n_pages", ctypes.c_int64), ("page_stride_k", ctypes.c_int64), ("page_stride_v", ctypes.c_int64),
        ("v_block_table", ctypes.c_void_p),
    ]


SYMBOLS = ("pkv_reposition_splice", "pkv_reposition_splice_freqs", "pkv_reposition_splice_paged",
           "pkv_reposition_splice_batched", "pkv_attention_workspace_size", "pkv_suffix_attention",
           "pkv_suffix_attention_paged", "pkv_suffix_attention_noalloc", "pkv_last_error", "pkv_version")
PKV_NOALLOC_SCRATCH_BYTES = 64 << 20

_lib = None


class PkvError(RuntimeError):
    def __init__(self, status: int, message: str):
        super().__init__("%s: %s" % (STATUS_NAMES.get(status, status), message))
        self.status = status


def lib() -> ctypes.CDLL:
    """Load libpkv.so (raises if it has not been built)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(_LIB_PATH):
        raise RuntimeError("libpkv.so is not built (run python -m paper_2606_17107_amd.build); "
                           "there is no fallback path")
    L = ctypes.CDLL(_LIB_PATH)
    P = ctypes.c_void_p
    L.pkv_reposition_splice.restype = ctypes.c_int
    L.pkv_reposition_splice.argtypes = [P, P, P, P, P, P, ctypes.c_float, ctypes.c_int32,
                                        ctypes.POINTER(pkv_layout), P]
    L.pkv_reposition_splice_freqs.restype = ctypes.c_int
    L.pkv_reposition_splice_freqs.argtypes = [P, P, P, P, P, P, P, ctypes.POINTER(ctypes.c_double),
                                              ctypes.c_int32, ctypes.POINTER(pkv_layout), P]
    L.pkv_reposition_splice_paged.restype = ctypes.c_int
    L.pkv_reposition_splice_paged.argtypes = [P, P, P, P, P, P, ctypes.c_float, ctypes.c_int32,
                                              ctypes.POINTER(pkv_layout), ctypes.POINTER(pkv_paged_cache), P]
    L.pkv_reposition_splice_batched.restype = ctypes.c_int
    L.pkv_reposition_splice_batched.argtypes = [P, P, P, P, P, ctypes.c_int32, ctypes.c_int32,
                                                ctypes.c_float, ctypes.c_int32, ctypes.POINTER(pkv_layout), P]
    L.pkv_attention_workspace_size.restype = ctypes.c_size_t
    L.pkv_attention_workspace_size.argtypes = [ctypes.POINTER(pkv_attn_desc), ctypes.c_int32,
                                               ctypes.c_int32, ctypes.c_int32]
    L.pkv_suffix_attention.restype = ctypes.c_int
    L.pkv_suffix_attention.argtypes = [P, P, P, P, P, P, ctypes.c_int32, ctypes.c_int32, ctypes.c_int32,
                                       ctypes.c_float, ctypes.POINTER(pkv_attn_desc), P, ctypes.c_size_t, P]
    L.pkv_suffix_attention_paged.restype = ctypes.c_int
    L.pkv_suffix_attention_paged.argtypes = [P, P, P, P, P, P, ctypes.c_int32, ctypes.c_int32, ctypes.c_int32,
                                             ctypes.c_float, ctypes.POINTER(pkv_attn_desc),
                                             ctypes.POINTER(pkv_paged_cache), P, ctypes.c_size_t, P]
    L.pkv_suffix_attention_noalloc.restype = ctypes.c_int
    L.pkv_suffix_attention_noalloc.argtypes = [P, P, P, P, P, P, ctypes.c_int32, ctypes.c_int32, ctypes.c_int32,
                                               ctypes.c_float, ctypes.POINTER(pkv_attn_desc), P]
    L.pkv_last_error.restype = ctypes.c_char_p
    L.pkv_last_error.argtypes = []
    L.pkv_version.restype = ctypes.c_int32
    L.pkv_version.argtypes = []
    _lib = L
    return L


def _check(status: int) -> None:
    if status != PKV_OK:
        raise PkvError(status, pkv_last_error())


def _ptr(t) -> Optional[int]:
    if t is None:
        return None
    if isinstance(t, int):
        return t
    return t.data_ptr()


def _keep_until_done(t: Optional[torch.Tensor], stream) -> None:
    """A workspace allocated here is freed when the call returns; when the kernels run on a stream other
    than torch's current one, tell the caching allocator that stream still uses it."""
    if t is None or stream is None:
        return
    if isinstance(stream, int):
        stream = torch.cuda.ExternalStream(stream)
    if stream != torch.cuda.current_stream(t.device):
        t.record_stream(stream)


def _stream(stream) -> Optional[int]:
    if stream is None:
        return torch.cuda.current_stream().cuda_stream if torch.cuda.is_available() else None
    if isinstance(stream, int):
        return stream
    return stream.cuda_stream


# ---- argument checks of the tensor-level calls --------------------------------
# The C entry points take raw device addresses; a host tensor's address handed
# to a kernel would fault the GPU.  The tensor-level calls below check type,
# dtype, size and device of every tensor they pass down (the raw pkv_* calls
# above do not).

def _need(t, name: str, device: torch.device, dtype=None, numel: Optional[int] = None,
          contiguous: bool = False) -> None:
    if t is None:
        return
    if not isinstance(t, torch.Tensor):
        raise TypeError("%s must be a torch.Tensor, got %s" % (name, type(t).__name__))
    if dtype is not None and t.dtype != dtype:
        raise TypeError("%s must be %s, got %s" % (name, dtype, t.dtype))
    if numel is not None and t.numel() < numel:
        raise ValueError("%s holds %d elements, the call reads %d" % (name, t.numel(), numel))
    if contiguous and not t.is_contiguous():
        raise ValueError("%s must be contiguous" % name)
    if t.device != device:
        raise ValueError("%s is on %s, the call runs on %s" % (name, t.device, device))


def _gpu_device(t: torch.Tensor, name: str) -> torch.device:
    if not isinstance(t, torch.Tensor):
        raise TypeError("%s must be a torch.Tensor, got %s" % (name, type(t).__name__))
    if t.device.type != "cuda":
        raise ValueError("libpkv tensors live on the GPU: %s is on %s" % (name, t.device))
    return t.device


def _check_splice_args(src_k, src_v, dst_k, dst_v, src_pos, dst_pos, err_flag, dst_slot=None,
                       n_tokens: Optional[int] = None) -> None:
    dev = _gpu_device(src_k, "src_k")
    n = src_k.shape[2] if n_tokens is None else n_tokens
    for t, name in ((src_v, "src_v"), (dst_k, "dst_k"), (dst_v, "dst_v")):
        _need(t, name, dev, src_k.dtype)
    for t, name in ((src_pos, "src_pos"), (dst_pos, "dst_pos"), (dst_slot, "dst_slot")):
        _need(t, name, dev, torch.int32, n, contiguous=True)
    _need(err_flag, "err_flag", dev, torch.int32, 1)


def _check_attention_args(q, k_cache, v_cache, out, q_pos, kv_len, n_seqs, cu_q, kv_base, lse_out,
                          workspace) -> None:
    dev = _gpu_device(q, "q")
    for t, name in ((k_cache, "k_cache"), (v_cache, "v_cache"), (out, "out")):
        if t is None:
            raise TypeError("%s is required" % name)
        _need(t, name, dev, q.dtype)
    L, rows, H = q.shape[0], q.shape[1], q.shape[2]
    _need(q_pos, "q_pos", dev, torch.int32, rows, contiguous=True)
    _need(kv_len, "kv_len", dev, torch.int32, int(n_seqs), contiguous=True)
    _need(cu_q, "cu_q", dev, torch.int32, int(n_seqs) + 1, contiguous=True)
    _need(kv_base, "kv_base", dev, torch.int64, int(n_seqs), contiguous=True)
    _need(lse_out, "lse_out", dev, torch.float32, L * rows * H, contiguous=True)
    _need(workspace, "workspace", dev, contiguous=True)


# ---- raw C entry points (same names and arguments as pkv.h) -----------------

def pkv_reposition_splice(src_k, src_v, dst_k, dst_v, src_pos, dst_pos, rope_theta, rope_dim, layout,
                          stream=None) -> int:
    return lib().pkv_reposition_splice(_ptr(src_k), _ptr(src_v), _ptr(dst_k), _ptr(dst_v), _ptr(src_pos),
                                       _ptr(dst_pos), float(rope_theta), int(rope_dim),
                                       ctypes.byref(layout) if layout is not None else None, _stream(stream))


def pkv_reposition_splice_freqs(src_k, src_v, dst_k, dst_v, src_pos, dst_pos, dst_slot, omega, rope_dim, layout,
                                stream=None) -> int:
    w = None
    if omega is not None:
        w = (ctypes.c_double * len(omega))(*[float(x) for x in omega])
    return lib().pkv_reposition_splice_freqs(_ptr(src_k), _ptr(src_v), _ptr(dst_k), _ptr(dst_v), _ptr(src_pos),
                                             _ptr(dst_pos), _ptr(dst_slot), w, int(rope_dim),
                                             ctypes.byref(layout) if layout is not None else None, _stream(stream))


def pkv_reposition_splice_paged(src_k, src_v, dst_k, dst_v, src_pos, dst_pos, rope_theta, rope_dim, layout, paging,
                                stream=None) -> int:
    return lib().pkv_reposition_splice_paged(_ptr(src_k), _ptr(src_v), _ptr(dst_k), _ptr(dst_v), _ptr(src_pos),
                                             _ptr(dst_pos), float(rope_theta), int(rope_dim),
                                             ctypes.byref(layout) if layout is not None else None,
                                             ctypes.byref(paging) if paging is not None else None, _stream(stream))


def pkv_reposition_splice_batched(src_k, src_v, dst_k, dst_v, segs, n_segs, max_seg_tokens, rope_theta,
                                  rope_dim, layout, stream=None) -> int:
    return lib().pkv_reposition_splice_batched(
        _ptr(src_k), _ptr(src_v), _ptr(dst_k), _ptr(dst_v), _ptr(segs), int(n_segs), int(max_seg_tokens),
        float(rope_theta), int(rope_dim), ctypes.byref(layout) if layout is not None else None,
        _stream(stream))


def pkv_attention_workspace_size(desc, n_q_heads, n_kv_heads, head_dim) -> int:
    return int(lib().pkv_attention_workspace_size(ctypes.byref(desc) if desc is not None else None,
                                                  int(n_q_heads), int(n_kv_heads), int(head_dim)))


def pkv_suffix_attention(q, k_cache, v_cache, out, q_pos, kv_len, n_q_heads, n_kv_heads, head_dim, scale,
                         desc, workspace, workspace_bytes, stream=None) -> int:
    return lib().pkv_suffix_attention(
        _ptr(q), _ptr(k_cache), _ptr(v_cache), _ptr(out), _ptr(q_pos), _ptr(kv_len), int(n_q_heads),
        int(n_kv_heads), int(head_dim), float(scale), ctypes.byref(desc) if desc is not None else None,
        _ptr(workspace), int(workspace_bytes), _stream(stream))


def pkv_suffix_attention_paged(q, k_pages, v_pages, out, q_pos, kv_len, n_q_heads, n_kv_heads, head_dim, scale,
                               desc, paging, workspace, workspace_bytes, stream=None) -> int:
    return lib().pkv_suffix_attention_paged(
        _ptr(q), _ptr(k_pages), _ptr(v_pages), _ptr(out), _ptr(q_pos), _ptr(kv_len), int(n_q_heads),
        int(n_kv_heads), int(head_dim), float(scale), ctypes.byref(desc) if desc is not None else None,
        ctypes.byref(paging) if paging is not None else None, _ptr(workspace), int(workspace_bytes),
        _stream(stream))


def pkv_suffix_attention_noalloc(q, k_cache, v_cache, out, q_pos, kv_len, n_q_heads, n_kv_heads, head_dim, scale,
                                 desc, stream=None) -> int:
    return lib().pkv_suffix_attention_noalloc(
        _ptr(q), _ptr(k_cache), _ptr(v_cache), _ptr(out), _ptr(q_pos), _ptr(kv_len), int(n_q_heads),
        int(n_kv_heads), int(head_dim), float(scale), ctypes.byref(desc) if desc is not None else None,
        _stream(stream))


def pkv_last_error() -> str:
    return lib().pkv_last_error().decode()


def pkv_version() -> int:
    return int(lib().pkv_version())


# ---- descriptor builders from torch tensors ---------------------------------

def _dtype_code(t: torch.Tensor) -> int:
    if t.dtype == torch.bfloat16:
        return PKV_BF16
    if t.dtype == torch.float32:
        return PKV_F32
    raise TypeError("libpkv tensors are bfloat16 or float32, got %s" % t.dtype)


def _strides3(t: Optional[torch.Tensor]):
    if t is None:
        return _i64x3(0, 0, 0)
    assert t.dim() == 4 and t.stride(3) == 1, "cache tensors are [layer][head][slot][channel], channels contiguous"
    return _i64x3(t.stride(0), t.stride(1), t.stride(2))


def make_layout(src_k: torch.Tensor, src_v: Optional[torch.Tensor], dst_k: torch.Tensor,
                dst_v: Optional[torch.Tensor], rope_offset: int = 0, rope_style: int = PKV_ROPE_HALF,
                n_tokens: Optional[int] = None, err_flag: Optional[torch.Tensor] = None) -> pkv_layout:
    """Layout for [layer][kv_head][slot][channel] tensors (any strides, channels contiguous)."""
    L = pkv_layout()
    L.dtype = _dtype_code(src_k)
    L.n_layers, L.n_kv_heads = src_k.shape[0], src_k.shape[1]
    L.head_dim = src_k.shape[3]
    L.v_dim = 0 if src_v is None else src_v.shape[3]
    L.n_tokens = src_k.shape[2] if n_tokens is None else int(n_tokens)
    L.rope_offset = int(rope_offset)
    L.rope_style = int(rope_style)
    L.dst_capacity = dst_k.shape[2]
    L.reserved = 0
    L.src_k_stride = _strides3(src_k)
    L.src_v_stride = _strides3(src_v)
    L.dst_k_stride = _strides3(dst_k)
    L.dst_v_stride = _strides3(dst_v)
    L.err_flag = None if err_flag is None else err_flag.data_ptr()
    return L


def reposition_splice(src_k, src_v, dst_k, dst_v, src_pos, dst_pos, rope_theta, rope_dim, rope_offset=0,
                      rope_style=PKV_ROPE_HALF, err_flag=None, stream=None) -> None:
    """Tensor-level call of pkv_reposition_splice; raises PkvError on a non-OK status."""
    _check_splice_args(src_k, src_v, dst_k, dst_v, src_pos, dst_pos, err_flag)
    layout = make_layout(src_k, src_v, dst_k, dst_v, rope_offset, rope_style, err_flag=err_flag)
    _check(pkv_reposition_splice(src_k, src_v, dst_k, dst_v, src_pos, dst_pos, rope_theta, rope_dim, layout,
                                 stream))


def reposition_splice_freqs(src_k, src_v, dst_k, dst_v, src_pos, dst_pos, omega, rope_dim, rope_offset=0,
                            rope_style=PKV_ROPE_HALF, dst_slot=None, err_flag=None, stream=None) -> None:
    """Tensor-level call of pkv_reposition_splice_freqs (per-pair frequencies ``omega``; optional
    destination slots, else slot = dst_pos)."""
    _check_splice_args(src_k, src_v, dst_k, dst_v, src_pos, dst_pos, err_flag, dst_slot)
    layout = make_layout(src_k, src_v, dst_k, dst_v, rope_offset, rope_style, err_flag=err_flag)
    _check(pkv_reposition_splice_freqs(src_k, src_v, dst_k, dst_v, src_pos, dst_pos, dst_slot, omega, rope_dim,
                                       layout, stream))


def make_segments(segs: Sequence[dict], device) -> torch.Tensor:
    """Pack segment dicts (src_slot0, dst_seq_base, n_tokens, src_pos0, dst_pos0, dst_seq_len) into a
    device buffer of pkv_segment records."""
    arr = (pkv_segment * max(1, len(segs)))()
    for i, s in enumerate(segs):
        arr[i] = pkv_segment(int(s["src_slot0"]), int(s["dst_seq_base"]), int(s["n_tokens"]),
                             int(s["src_pos0"]), int(s["dst_pos0"]), int(s["dst_seq_len"]))
    raw = torch.frombuffer(bytearray(bytes(arr)), dtype=torch.uint8)
    return raw.to(device)


def reposition_splice_batched(src_k, src_v, dst_k, dst_v, segs_dev: torch.Tensor, n_segs: int,
                              max_seg_tokens: int, rope_theta, rope_dim, rope_offset=0,
                              rope_style=PKV_ROPE_HALF, err_flag=None, stream=None) -> None:
    _check_splice_args(src_k, src_v, dst_k, dst_v, None, None, err_flag)
    _need(segs_dev, "segs_dev", src_k.device, torch.uint8, int(n_segs) * ctypes.sizeof(pkv_segment),
          contiguous=True)
    layout = make_layout(src_k, src_v, dst_k, dst_v, rope_offset, rope_style, err_flag=err_flag)
    _check(pkv_reposition_splice_batched(src_k, src_v, dst_k, dst_v, segs_dev, n_segs, max_seg_tokens,
                                         rope_theta, rope_dim, layout, stream))


def make_attn_desc(q: torch.Tensor, k_cache: torch.Tensor, v_cache: torch.Tensor, out: torch.Tensor,
                   max_kv_len: int, n_seqs: int = 1, cu_q: Optional[torch.Tensor] = None,
                   kv_base: Optional[torch.Tensor] = None, max_q: Optional[int] = None,
                   variant: int = PKV_ATTN_GQA, n_splits: int = 0,
                   lse_out: Optional[torch.Tensor] = None, window: int = 0) -> pkv_attn_desc:
    """Descriptor for q [L][rows][H][d], caches [L][Hkv][slots][*], out [L][rows][H][dv]."""
    d = pkv_attn_desc()
    d.dtype = _dtype_code(q)
    d.variant = int(variant)
    d.n_layers = q.shape[0]
    d.n_seqs = int(n_seqs)
    d.head_dim_v = out.shape[3]
    d.total_q = q.shape[1]
    d.max_q = q.shape[1] if max_q is None else int(max_q)
    d.max_kv_len = int(max_kv_len)
    d.n_splits = int(n_splits)
    d.window = int(window)
    d.cu_q = None if cu_q is None else cu_q.data_ptr()
    d.kv_base = None if kv_base is None else kv_base.data_ptr()
    d.cache_slots = k_cache.shape[2]
    assert q.stride(3) == 1 and out.stride(3) == 1
    d.q_stride = _i64x3(q.stride(0), q.stride(1), q.stride(2))
    d.k_stride = _strides3(k_cache)
    d.v_stride = _strides3(v_cache)
    d.o_stride = _i64x3(out.stride(0), out.stride(1), out.stride(2))
    d.lse_out = None if lse_out is None else lse_out.data_ptr()
    return d


def attention_workspace(desc: pkv_attn_desc, n_q_heads: int, n_kv_heads: int, head_dim: int,
                        device) -> Optional[torch.Tensor]:
    n = pkv_attention_workspace_size(desc, n_q_heads, n_kv_heads, head_dim)
    if n == 0:
        return None
    return torch.empty(n, dtype=torch.uint8, device=device)


def suffix_attention(q, k_cache, v_cache, out, q_pos, kv_len, scale, max_kv_len, n_seqs=1, cu_q=None,
                     kv_base=None, max_q=None, variant=PKV_ATTN_GQA, n_splits=0, lse_out=None,
                     workspace=None, stream=None, window=0) -> None:
    """Tensor-level call of pkv_suffix_attention (allocates the workspace with torch if not given)."""
    _check_attention_args(q, k_cache, v_cache, out, q_pos, kv_len, n_seqs, cu_q, kv_base, lse_out, workspace)
    H = q.shape[2]
    Hkv = k_cache.shape[1]
    D = q.shape[3]
    desc = make_attn_desc(q, k_cache, v_cache, out, max_kv_len, n_seqs, cu_q, kv_base, max_q, variant,
                          n_splits, lse_out, window)
    need = pkv_attention_workspace_size(desc, H, Hkv, D)
    if need and (workspace is None or workspace.numel() * workspace.element_size() < need):
        workspace = torch.empty(need, dtype=torch.uint8, device=q.device)
        _keep_until_done(workspace, stream)
    _check(pkv_suffix_attention(q, k_cache, v_cache, out, q_pos, kv_len, H, Hkv, D, scale, desc,
                                workspace, need, stream))


# ---- paged caches ------------------------------------------------------------
# Pools are [layer][page][in-page slot][kv_head][channel] (any strides, channels
# contiguous); a block table is int32 [n_seqs][max_pages] on the device.

def pool_strides3(pool: Optional[torch.Tensor]):
    """{layer, head, in-page slot} element strides of a 5-D pool."""
    if pool is None:
        return _i64x3(0, 0, 0)
    assert pool.dim() == 5 and pool.stride(4) == 1, "pools are [layer][page][slot][kv_head][channel]"
    return _i64x3(pool.stride(0), pool.stride(3), pool.stride(2))


def make_paging(block_table: torch.Tensor, k_pool: torch.Tensor, v_pool: Optional[torch.Tensor] = None,
                v_block_table: Optional[torch.Tensor] = None) -> pkv_paged_cache:
    assert block_table.dtype == torch.int32 and block_table.dim() == 2 and block_table.is_contiguous()
    if v_block_table is not None:
        assert v_block_table.dtype == torch.int32 and v_block_table.shape == block_table.shape
        assert v_block_table.is_contiguous()
    pg = pkv_paged_cache()
    pg.page_size = k_pool.shape[2]
    pg.max_pages = block_table.shape[1]
    pg.block_table = block_table.data_ptr()
    pg.n_pages = k_pool.shape[1]
    pg.page_stride_k = k_pool.stride(1)
    pg.page_stride_v = 0 if v_pool is None else v_pool.stride(1)
    pg.v_block_table = None if v_block_table is None else v_block_table.data_ptr()
    return pg


def reposition_splice_paged(src_k, src_v, k_pool, v_pool, src_pos, dst_pos, block_table, rope_theta, rope_dim,
                            rope_offset=0, rope_style=PKV_ROPE_HALF, dst_capacity=None, err_flag=None,
                            stream=None, v_block_table=None) -> None:
    """Tensor-level call of pkv_reposition_splice_paged: destination slots are logical slots of the
    sequence whose block-table row is block_table[0]."""
    _check_splice_args(src_k, src_v, k_pool, v_pool, src_pos, dst_pos, err_flag)
    _need(block_table, "block_table", src_k.device, torch.int32, contiguous=True)
    _need(v_block_table, "v_block_table", src_k.device, torch.int32, contiguous=True)
    L = make_layout(src_k, src_v, src_k, src_v, rope_offset, rope_style, err_flag=err_flag)
    L.dst_capacity = (block_table.shape[1] * k_pool.shape[2]) if dst_capacity is None else int(dst_capacity)
    L.dst_k_stride = pool_strides3(k_pool)
    L.dst_v_stride = pool_strides3(v_pool)
    pg = make_paging(block_table, k_pool, v_pool, v_block_table)
    _check(pkv_reposition_splice_paged(src_k, src_v, k_pool, v_pool, src_pos, dst_pos, rope_theta, rope_dim, L, pg,
                                       stream))


def suffix_attention_paged(q, k_pool, v_pool, out, q_pos, kv_len, block_table, scale, max_kv_len, n_seqs=1,
                           cu_q=None, max_q=None, variant=PKV_ATTN_GQA, n_splits=0, lse_out=None, workspace=None,
                           stream=None, window=0, cache_slots=None, v_block_table=None) -> None:
    """Tensor-level call of pkv_suffix_attention_paged (q [L][rows][H][d], pools as above)."""
    _check_attention_args(q, k_pool, v_pool, out, q_pos, kv_len, n_seqs, cu_q, None, lse_out, workspace)
    _need(block_table, "block_table", q.device, torch.int32, contiguous=True)
    _need(v_block_table, "v_block_table", q.device, torch.int32, contiguous=True)
    H = q.shape[2]
    Hkv = k_pool.shape[3]
    D = q.shape[3]
    d = pkv_attn_desc()
    d.dtype = _dtype_code(q)
    d.variant = int(variant)
    d.n_layers = q.shape[0]
    d.n_seqs = int(n_seqs)
    d.head_dim_v = out.shape[3]
    d.total_q = q.shape[1]
    d.max_q = q.shape[1] if max_q is None else int(max_q)
    d.max_kv_len = int(max_kv_len)
    d.n_splits = int(n_splits)
    d.window = int(window)
    d.cu_q = None if cu_q is None else cu_q.data_ptr()
    d.kv_base = None
    d.cache_slots = block_table.shape[1] * k_pool.shape[2] if cache_slots is None else int(cache_slots)
    assert q.stride(3) == 1 and out.stride(3) == 1
    d.q_stride = _i64x3(q.stride(0), q.stride(1), q.stride(2))
    d.k_stride = pool_strides3(k_pool)
    d.v_stride = pool_strides3(v_pool)
    d.o_stride = _i64x3(out.stride(0), out.stride(1), out.stride(2))
    d.lse_out = None if lse_out is None else lse_out.data_ptr()
    pg = make_paging(block_table, k_pool, v_pool, v_block_table)
    need = pkv_attention_workspace_size(d, H, Hkv, D)
    if need and (workspace is None or workspace.numel() * workspace.element_size() < need):
        workspace = torch.empty(need, dtype=torch.uint8, device=q.device)
        _keep_until_done(workspace, stream)
    _check(pkv_suffix_attention_paged(q, k_pool, v_pool, out, q_pos, kv_len, H, Hkv, D, scale, d, pg, workspace,
                                      need, stream))
