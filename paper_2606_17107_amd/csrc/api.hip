// C ABI of libpkv: argument validation, aliasing checks and dispatch to the
// kernel launchers.  The contract of every entry point is documented in
// include/pkv.h.  Nothing here allocates device memory or synchronises.
#include <math.h>
#include <stdarg.h>
#include <stdio.h>
#include <string.h>

#include <mutex>

#include "pkv.h"
#include "pkv_internal.h"

#define PKV_EXPORT extern "C" __attribute__((visibility("default")))

// Split-KV scratch of pkv_suffix_attention_noalloc: a file-scope device array,
// so that entry point never allocates.  Each GPU the library runs on holds its
// own copy (PKV_NOALLOC_SCRATCH_BYTES) until the process ends.  In host code
// `scratch` names a host-side stand-in, not device memory: kernels only ever
// get the per-device address that hipGetSymbolAddress returns for it.
static __device__ __align__(256) unsigned char scratch[PKV_NOALLOC_SCRATCH_BYTES];

namespace {

thread_local char g_err[512] = "";

pkv_status fail(pkv_status st, const char* fmt, ...) {
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(g_err, sizeof g_err, fmt, ap);
    va_end(ap);
    return st;
}

pkv_status ok() {
    g_err[0] = '\0';
    return PKV_OK;
}

bool aligned16(const void* p) { return ((uintptr_t)p & 15u) == 0; }

// Byte range [lo, hi) touched by a tensor with non-negative strides.
struct Range {
    uintptr_t lo = 0, hi = 0;
};

Range extent(const void* p, const int64_t* stride, const int64_t* count, int ndim, int64_t row_elems,
             int elem_bytes) {
    Range r;
    if (!p) return r;
    int64_t last = 0;
    for (int i = 0; i < ndim; ++i) last += (count[i] - 1) * stride[i];
    r.lo = (uintptr_t)p;
    r.hi = r.lo + (uintptr_t)((last + row_elems) * elem_bytes);
    return r;
}

bool overlap(const Range& a, const Range& b) {
    if (a.lo == a.hi || b.lo == b.hi) return false;
    return a.lo < b.hi && b.lo < a.hi;
}

pkv_status device_status(hipError_t e, const char* what) {
    if (e == hipSuccess) return ok();
    return fail(PKV_ERR_DEVICE, "%s: %s", what, hipGetErrorString(e));
}

// Validation of a paged-cache descriptor serving `logical_slots` slots per
// sequence with elements of `eb` bytes; sets *shift to log2(page_size).
pkv_status check_paging(const pkv_paged_cache* pg, int64_t logical_slots, int eb, int* shift) {
    if (!pg) return fail(PKV_ERR_NULL, "paging is NULL");
    if (!pg->block_table) return fail(PKV_ERR_NULL, "paging.block_table is NULL");
    const int32_t b = pg->page_size;
    if (b < 32 || b > (1 << 20) || (b & (b - 1)))
        return fail(PKV_ERR_SHAPE, "page_size %d must be a power of two in [32, 2^20]", b);
    if (pg->max_pages <= 0 || pg->n_pages <= 0 || pg->n_pages > 0x7fffffff)
        return fail(PKV_ERR_SHAPE, "max_pages (%d) and n_pages (%lld) must be positive (n_pages < 2^31)",
                    pg->max_pages, (long long)pg->n_pages);
    if (pg->page_stride_k < 0 || pg->page_stride_v < 0)
        return fail(PKV_ERR_SHAPE, "page strides must be non-negative");
    if ((pg->page_stride_k * eb) % 16 || (pg->page_stride_v * eb) % 16)
        return fail(PKV_ERR_ALIGN, "page strides must be multiples of 16 bytes");
    if (logical_slots > (int64_t)pg->max_pages * b)
        return fail(PKV_ERR_SHAPE, "%lld logical slots exceed max_pages * page_size = %lld",
                    (long long)logical_slots, (long long)pg->max_pages * b);
    int sh = 0;
    while ((1 << sh) < b) ++sh;
    *shift = sh;
    return PKV_OK;
}

// Byte range of a paged pool: {layer, head, page, in-page slot} with strides
// {stride[0], stride[1], page_stride, stride[2]}.
Range paged_extent(const void* p, const int64_t* stride, int64_t page_stride, int64_t n_layers, int64_t n_heads,
                   const pkv_paged_cache* pg, int64_t row_elems, int eb) {
    const int64_t st[4] = {stride[0], stride[1], page_stride, stride[2]};
    const int64_t cnt[4] = {n_layers, n_heads, pg->n_pages, pg->page_size};
    return extent(p, st, cnt, 4, row_elems, eb);
}

// Shared validation of reposition+splice arguments.  Fills `a` on success.
pkv_status check_splice(const void* src_k, const void* src_v, void* dst_k, void* dst_v,
                        float rope_theta, int32_t rope_dim, const pkv_layout* L, bool allow_inplace,
                        pkv::SpliceArgs& a, const pkv_paged_cache* pg = nullptr) {
    if (!L) return fail(PKV_ERR_NULL, "layout is NULL");
    if (!src_k || !dst_k) return fail(PKV_ERR_NULL, "src_k and dst_k are required");
    if (L->dtype != PKV_BF16 && L->dtype != PKV_F32)
        return fail(PKV_ERR_UNSUPPORTED, "dtype %d (expected PKV_BF16 or PKV_F32)", L->dtype);
    if (L->rope_style != PKV_ROPE_HALF && L->rope_style != PKV_ROPE_INTERLEAVED)
        return fail(PKV_ERR_UNSUPPORTED, "rope_style %d", L->rope_style);
    if (L->v_dim > 0 && (!src_v || !dst_v))
        return fail(PKV_ERR_NULL, "v_dim = %d but src_v or dst_v is NULL", L->v_dim);
    if (L->v_dim == 0 && (src_v || dst_v))
        return fail(PKV_ERR_SHAPE, "v_dim = 0 (no V tensors) but src_v or dst_v is given");
    if (L->reserved != 0) return fail(PKV_ERR_SHAPE, "layout.reserved must be 0");
    if (L->n_layers <= 0 || L->n_kv_heads <= 0 || L->head_dim <= 0 || L->v_dim < 0 ||
        L->n_tokens < 0 || L->dst_capacity < 0)
        return fail(PKV_ERR_SHAPE,
                    "sizes must be positive (n_layers %d, n_kv_heads %d, head_dim %d) and "
                    "non-negative (v_dim %d, n_tokens %d, dst_capacity %d)",
                    L->n_layers, L->n_kv_heads, L->head_dim, L->v_dim, L->n_tokens, L->dst_capacity);
    if (rope_dim <= 0 || (rope_dim & 1))
        return fail(PKV_ERR_SHAPE, "rope_dim %d must be positive and even", rope_dim);
    if (rope_dim > 256)
        return fail(PKV_ERR_UNSUPPORTED, "rope_dim %d: rotary slices of at most 256 channels are supported",
                    rope_dim);
    if (L->rope_offset < 0 || (int64_t)L->rope_offset + rope_dim > L->head_dim)
        return fail(PKV_ERR_SHAPE, "rotary slice [%d, %d) lies outside the %d-channel row",
                    L->rope_offset, L->rope_offset + rope_dim, L->head_dim);
    if (!(rope_theta > 0.0f) || !isfinite(rope_theta))
        return fail(PKV_ERR_SHAPE, "rope_theta must be finite and positive");
    for (int i = 0; i < 3; ++i) {
        if (L->src_k_stride[i] < 0 || L->dst_k_stride[i] < 0 || L->src_v_stride[i] < 0 ||
            L->dst_v_stride[i] < 0)
            return fail(PKV_ERR_SHAPE, "strides must be non-negative");
    }
    const int eb = L->dtype == PKV_BF16 ? 2 : 4;
    const int ce = 16 / eb;
    if (L->head_dim % (2 * ce) || L->v_dim % (2 * ce) || L->rope_offset % ce || rope_dim % (2 * ce))
        return fail(PKV_ERR_UNSUPPORTED,
                    "row geometry: head_dim (%d) and v_dim (%d) must be multiples of %d, rope_offset "
                    "(%d) of %d and rope_dim (%d) of %d for this dtype",
                    L->head_dim, L->v_dim, 2 * ce, L->rope_offset, ce, rope_dim, 2 * ce);
    if ((L->head_dim + L->v_dim) / (2 * ce) > 256)
        return fail(PKV_ERR_UNSUPPORTED, "rows wider than %d bytes (K+V) are not supported", 256 * 32);
    if (!aligned16(src_k) || !aligned16(dst_k) || !aligned16(src_v) || !aligned16(dst_v))
        return fail(PKV_ERR_ALIGN, "tensor pointers must be 16-byte aligned");
    for (int i = 0; i < 3; ++i) {
        if ((L->src_k_stride[i] * eb) % 16 || (L->dst_k_stride[i] * eb) % 16 ||
            (L->src_v_stride[i] * eb) % 16 || (L->dst_v_stride[i] * eb) % 16)
            return fail(PKV_ERR_ALIGN, "strides must be multiples of 16 bytes");
    }
    // Aliasing: destination tensors must not overlap sources (except an exact in-place
    // tensor) nor each other.
    const int64_t src_cnt[3] = {L->n_layers, L->n_kv_heads, L->n_tokens > 0 ? L->n_tokens : 1};
    const int64_t dst_cnt[3] = {L->n_layers, L->n_kv_heads, L->dst_capacity > 0 ? L->dst_capacity : 1};
    Range sk = extent(src_k, L->src_k_stride, src_cnt, 3, L->head_dim, eb);
    Range sv = extent(src_v, L->src_v_stride, src_cnt, 3, L->v_dim, eb);
    Range dk = extent(dst_k, L->dst_k_stride, dst_cnt, 3, L->head_dim, eb);
    Range dv = extent(dst_v, L->dst_v_stride, dst_cnt, 3, L->v_dim, eb);
    int page_shift = 0;
    if (pg) {
        pkv_status st = check_paging(pg, L->dst_capacity, eb, &page_shift);
        if (st != PKV_OK) return st;
        dk = paged_extent(dst_k, L->dst_k_stride, pg->page_stride_k, L->n_layers, L->n_kv_heads, pg, L->head_dim, eb);
        dv = paged_extent(dst_v, L->dst_v_stride, pg->page_stride_v, L->n_layers, L->n_kv_heads, pg, L->v_dim, eb);
        allow_inplace = false;
    }
    const bool k_inplace = allow_inplace && src_k == dst_k &&
                           memcmp(L->src_k_stride, L->dst_k_stride, sizeof L->src_k_stride) == 0;
    const bool v_inplace = allow_inplace && src_v && src_v == dst_v &&
                           memcmp(L->src_v_stride, L->dst_v_stride, sizeof L->src_v_stride) == 0;
    if ((!k_inplace && overlap(sk, dk)) || (!v_inplace && overlap(sv, dv)) || overlap(sk, dv) ||
        overlap(sv, dk) || overlap(dk, dv))
        return fail(PKV_ERR_ALIAS, "source and destination tensors overlap (only an exact in-place "
                                   "tensor is allowed)");

    memset(&a, 0, sizeof a);
    a.src_k = (const char*)src_k;
    a.src_v = (const char*)src_v;
    a.dst_k = (char*)dst_k;
    a.dst_v = (char*)dst_v;
    a.elem_bytes = eb;
    a.rope_style = L->rope_style;
    a.n_layers = L->n_layers;
    a.n_kv_heads = L->n_kv_heads;
    a.head_dim = L->head_dim;
    a.v_dim = L->v_dim;
    a.rope_offset = L->rope_offset;
    a.rope_dim = rope_dim;
    a.n_tokens = L->n_tokens;
    a.dst_capacity = L->dst_capacity;
    a.theta = (double)rope_theta;
    for (int i = 0; i < 3; ++i) {
        a.src_k_stride[i] = L->src_k_stride[i];
        a.src_v_stride[i] = L->src_v_stride[i];
        a.dst_k_stride[i] = L->dst_k_stride[i];
        a.dst_v_stride[i] = L->dst_v_stride[i];
    }
    a.err_flag = L->err_flag;
    if (pg) {
        a.dst_pages = pg->block_table;
        a.dst_v_pages = pg->v_block_table;
        a.page_shift = page_shift;
        a.max_pages = pg->max_pages;
        a.n_pages = pg->n_pages;
        a.dst_k_page_stride = pg->page_stride_k;
        a.dst_v_page_stride = pg->page_stride_v;
    }
    return PKV_OK;
}

// Validation of attention arguments; fills `a` (without workspace pointers).
pkv_status check_attention(const void* q, const void* k, const void* v, void* out,
                           const int32_t* q_pos, const int32_t* kv_len, int32_t H, int32_t Hkv,
                           int32_t D, float scale, const pkv_attn_desc* d, bool check_alias,
                           pkv::AttnArgs& a, const pkv_paged_cache* pg = nullptr) {
    if (!d) return fail(PKV_ERR_NULL, "desc is NULL");
    if (!q || !k || !v || !out || !q_pos || !kv_len)
        return fail(PKV_ERR_NULL, "q, k_cache, v_cache, out, q_pos and kv_len are required");
    if (d->dtype != PKV_BF16 && d->dtype != PKV_F32) return fail(PKV_ERR_UNSUPPORTED, "dtype %d", d->dtype);
    if (d->variant != PKV_ATTN_GQA && d->variant != PKV_ATTN_MLA)
        return fail(PKV_ERR_UNSUPPORTED, "variant %d", d->variant);
    if (d->window < 0) return fail(PKV_ERR_SHAPE, "desc.window (%d) must be >= 0", d->window);
    if (H <= 0 || Hkv <= 0 || D <= 0 || H % Hkv)
        return fail(PKV_ERR_SHAPE, "n_q_heads (%d) must be a positive multiple of n_kv_heads (%d)", H, Hkv);
    if (d->n_layers <= 0 || d->n_seqs <= 0 || d->total_q < 0 || d->max_q < 0 || d->max_kv_len < 0 ||
        d->n_splits < 0 || d->cache_slots < 0 || d->head_dim_v <= 0)
        return fail(PKV_ERR_SHAPE, "invalid sizes in desc");
    if (d->max_kv_len > (1 << 30))   // key indices and tile arithmetic stay inside int32
        return fail(PKV_ERR_SHAPE, "max_kv_len (%d) above 2^30", d->max_kv_len);
    if (d->n_seqs > 1 && !d->cu_q) return fail(PKV_ERR_NULL, "cu_q is required when n_seqs > 1");
    if (d->n_seqs == 1 && !d->cu_q && d->max_q < d->total_q)
        return fail(PKV_ERR_SHAPE, "max_q (%d) < total_q (%d)", d->max_q, d->total_q);
    if (!isfinite(scale)) return fail(PKV_ERR_SHAPE, "scale must be finite");
    if (d->variant == PKV_ATTN_GQA) {
        if (D != 64 && D != 128) return fail(PKV_ERR_UNSUPPORTED, "GQA head_dim %d (supported: 64, 128)", D);
        if (d->head_dim_v != D) return fail(PKV_ERR_SHAPE, "GQA needs head_dim_v == head_dim");
    } else {
        if (d->dtype != PKV_BF16) return fail(PKV_ERR_UNSUPPORTED, "MLA attention is bf16 only");
        if (Hkv != 1 || D != 576 || d->head_dim_v != 512)
            return fail(PKV_ERR_SHAPE, "MLA needs n_kv_heads 1, head_dim 576, head_dim_v 512");
        if (v != k || memcmp(d->v_stride, d->k_stride, sizeof d->k_stride) != 0)
            return fail(PKV_ERR_SHAPE, "MLA reads values from the latent channels of k_cache: v_cache must be "
                                       "k_cache with the same strides");
    }
    const int eb = d->dtype == PKV_BF16 ? 2 : 4;
    if (!aligned16(q) || !aligned16(k) || !aligned16(v) || !aligned16(out))
        return fail(PKV_ERR_ALIGN, "q, k_cache, v_cache and out must be 16-byte aligned");
    for (int i = 0; i < 3; ++i) {
        if (d->q_stride[i] < 0 || d->k_stride[i] < 0 || d->v_stride[i] < 0 || d->o_stride[i] < 0)
            return fail(PKV_ERR_SHAPE, "strides must be non-negative");
        if ((d->q_stride[i] * eb) % 16 || (d->k_stride[i] * eb) % 16 || (d->v_stride[i] * eb) % 16 ||
            (d->o_stride[i] * eb) % 16)
            return fail(PKV_ERR_ALIGN, "strides must be multiples of 16 bytes");
    }
    // The kernels address the keys of one tile (up to 32 slots) by 32-bit byte
    // offsets from its first key.
    constexpr int64_t kMaxSlotBytes = (int64_t)1 << 26;
    if (d->k_stride[2] > kMaxSlotBytes / eb || d->v_stride[2] > kMaxSlotBytes / eb)
        return fail(PKV_ERR_SHAPE, "slot strides k_stride[2] / v_stride[2] (%lld / %lld elements) exceed 64 MiB",
                    (long long)d->k_stride[2], (long long)d->v_stride[2]);
    int page_shift = 0;
    if (pg) {
        if (d->dtype != PKV_BF16) return fail(PKV_ERR_UNSUPPORTED, "paged attention is bf16 only");
        if (d->kv_base) return fail(PKV_ERR_SHAPE, "desc.kv_base must be NULL for a paged cache");
        pkv_status st = check_paging(pg, d->cache_slots, eb, &page_shift);
        if (st != PKV_OK) return st;
        if (d->variant == PKV_ATTN_MLA && (pg->page_stride_v != pg->page_stride_k || pg->v_block_table))
            return fail(PKV_ERR_SHAPE, "MLA reads values from the latent channels: page_stride_v must equal "
                                       "page_stride_k and there is no separate v_block_table");
    }
    // out must not overlap any input
    if (check_alias && d->total_q > 0) {
        const int64_t oc[3] = {d->n_layers, d->total_q, H};
        const int64_t qc[3] = {d->n_layers, d->total_q, H};
        const int64_t slots = d->cache_slots > 0 ? d->cache_slots : 1;
        const int64_t kc[3] = {d->n_layers, Hkv, slots};
        Range ro = extent(out, d->o_stride, oc, 3, d->head_dim_v, eb);
        Range rq = extent(q, d->q_stride, qc, 3, D, eb);
        Range rk = extent(k, d->k_stride, kc, 3, D, eb);
        Range rv = extent(v, d->v_stride, kc, 3, d->head_dim_v, eb);
        if (pg) {
            rk = paged_extent(k, d->k_stride, pg->page_stride_k, d->n_layers, Hkv, pg, D, eb);
            rv = paged_extent(v, d->v_stride, pg->page_stride_v, d->n_layers, Hkv, pg, d->head_dim_v, eb);
        }
        if (overlap(ro, rq) || overlap(ro, rk) || overlap(ro, rv))
            return fail(PKV_ERR_ALIAS, "out overlaps an input tensor");
    }
    memset(&a, 0, sizeof a);
    a.q = q;
    a.k = k;
    a.v = v;
    a.out = out;
    a.q_pos = q_pos;
    a.kv_len = kv_len;
    a.cu_q = d->cu_q;
    a.kv_base = d->kv_base;
    a.lse_out = d->lse_out;
    a.dtype = d->dtype;
    a.variant = d->variant;
    a.n_layers = d->n_layers;
    a.n_seqs = d->n_seqs;
    a.n_heads = H;
    a.n_kv_heads = Hkv;
    a.head_dim = D;
    a.head_dim_v = d->head_dim_v;
    a.total_q = d->total_q;
    a.max_q = d->cu_q ? d->max_q : d->total_q;
    a.max_kv_len = d->max_kv_len;
    a.n_splits = d->n_splits;
    a.window = d->window;
    a.cache_slots = d->cache_slots;
    a.scale = scale;
    for (int i = 0; i < 3; ++i) {
        a.q_stride[i] = d->q_stride[i];
        a.k_stride[i] = d->k_stride[i];
        a.v_stride[i] = d->v_stride[i];
        a.o_stride[i] = d->o_stride[i];
    }
    if (pg) {
        a.block_table = pg->block_table;
        a.v_block_table = pg->v_block_table;
        a.page_shift = page_shift;
        a.max_pages = pg->max_pages;
        a.n_pages = pg->n_pages;
        a.k_page_stride = pg->page_stride_k;
        a.v_page_stride = pg->page_stride_v;
    }
    return PKV_OK;
}

}  // namespace

PKV_EXPORT pkv_status pkv_reposition_splice(const void* src_k, const void* src_v, void* dst_k,
                                            void* dst_v, const int32_t* src_pos, const int32_t* dst_pos,
                                            float rope_theta, int32_t rope_dim,
                                            const pkv_layout* layout, void* stream) {
    pkv::SpliceArgs a;
    pkv_status st = check_splice(src_k, src_v, dst_k, dst_v, rope_theta, rope_dim, layout, true, a);
    if (st != PKV_OK) return st;
    if (!src_pos || !dst_pos) return fail(PKV_ERR_NULL, "src_pos and dst_pos are required");
    a.src_pos = src_pos;
    a.dst_pos = dst_pos;
    if (a.n_tokens == 0) return ok();
    return device_status(pkv::launch_splice(a, (hipStream_t)stream), "reposition_splice launch");
}

PKV_EXPORT pkv_status pkv_reposition_splice_freqs(const void* src_k, const void* src_v, void* dst_k,
                                                  void* dst_v, const int32_t* src_pos, const int32_t* dst_pos,
                                                  const int32_t* dst_slot, const double* omega, int32_t rope_dim,
                                                  const pkv_layout* layout, void* stream) {
    pkv::SpliceArgs a;
    pkv_status st = check_splice(src_k, src_v, dst_k, dst_v, 1.0f, rope_dim, layout, true, a);
    if (st != PKV_OK) return st;
    if (!src_pos || !dst_pos) return fail(PKV_ERR_NULL, "src_pos and dst_pos are required");
    if (!omega) return fail(PKV_ERR_NULL, "omega is required");
    for (int i = 0; i < rope_dim / 2; ++i)
        if (!isfinite(omega[i])) return fail(PKV_ERR_SHAPE, "omega[%d] is not finite", i);
    a.src_pos = src_pos;
    a.dst_pos = dst_pos;
    a.dst_slot = dst_slot;
    a.omega = omega;
    if (a.n_tokens == 0) return ok();
    return device_status(pkv::launch_splice(a, (hipStream_t)stream), "reposition_splice_freqs launch");
}

PKV_EXPORT pkv_status pkv_reposition_splice_paged(const void* src_k, const void* src_v, void* dst_k,
                                                  void* dst_v, const int32_t* src_pos, const int32_t* dst_pos,
                                                  float rope_theta, int32_t rope_dim, const pkv_layout* layout,
                                                  const pkv_paged_cache* paging, void* stream) {
    pkv::SpliceArgs a;
    if (!paging) return fail(PKV_ERR_NULL, "paging is NULL");
    pkv_status st = check_splice(src_k, src_v, dst_k, dst_v, rope_theta, rope_dim, layout, false, a, paging);
    if (st != PKV_OK) return st;
    if (!src_pos || !dst_pos) return fail(PKV_ERR_NULL, "src_pos and dst_pos are required");
    a.src_pos = src_pos;
    a.dst_pos = dst_pos;
    if (a.n_tokens == 0) return ok();
    return device_status(pkv::launch_splice(a, (hipStream_t)stream), "reposition_splice_paged launch");
}

PKV_EXPORT pkv_status pkv_reposition_splice_batched(const void* src_k, const void* src_v, void* dst_k,
                                                    void* dst_v, const pkv_segment* segs, int32_t n_segs,
                                                    int32_t max_seg_tokens, float rope_theta,
                                                    int32_t rope_dim, const pkv_layout* layout,
                                                    void* stream) {
    static_assert(sizeof(pkv_segment) == sizeof(pkv::SpliceSegment), "segment layout");
    pkv::SpliceArgs a;
    pkv_status st = check_splice(src_k, src_v, dst_k, dst_v, rope_theta, rope_dim, layout, false, a);
    if (st != PKV_OK) return st;
    if (n_segs < 0 || max_seg_tokens < 0)
        return fail(PKV_ERR_SHAPE, "n_segs (%d) and max_seg_tokens (%d) must be non-negative", n_segs,
                    max_seg_tokens);
    if (n_segs > 65535) return fail(PKV_ERR_UNSUPPORTED, "at most 65535 segments per call");
    if (n_segs > 0 && !segs) return fail(PKV_ERR_NULL, "segs is NULL");
    if (!aligned16(segs)) return fail(PKV_ERR_ALIGN, "segs must be 16-byte aligned");
    if (n_segs == 0 || max_seg_tokens == 0) return ok();
    a.segs = (const pkv::SpliceSegment*)segs;
    a.n_segs = n_segs;
    a.max_seg_tokens = max_seg_tokens;
    return device_status(pkv::launch_splice(a, (hipStream_t)stream), "reposition_splice_batched launch");
}

PKV_EXPORT size_t pkv_attention_workspace_size(const pkv_attn_desc* desc, int32_t n_q_heads,
                                               int32_t n_kv_heads, int32_t head_dim) {
    if (!desc) return 0;
    // Geometry checks only; pointers are not needed to size the workspace.
    static const char dummy[16] __attribute__((aligned(16))) = {0};
    static const int32_t idummy[4] __attribute__((aligned(16))) = {0};
    pkv::AttnArgs a;
    char saved[sizeof g_err];
    memcpy(saved, g_err, sizeof g_err);
    pkv_status st = check_attention(dummy, dummy, dummy, (void*)dummy, idummy, idummy, n_q_heads,
                                    n_kv_heads, head_dim, 1.0f, desc, false, a);
    memcpy(g_err, saved, sizeof g_err);
    if (st != PKV_OK) return 0;
    return pkv::attention_workspace_bytes(a, pkv::attention_splits(a));
}

namespace {

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_dev[kMaxDevices] = {};   // device address of `scratch`, per device

// Device address of `scratch` on the current device, looked up once per device
// (with that device current: each GPU holds the array at its own address).
pkv_status scratch_on_current_device(void** out) {
    int dev = -1;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return fail(PKV_ERR_DEVICE, "hipGetDevice: %s", hipGetErrorString(e));
    if (dev < 0 || dev >= kMaxDevices)
        return fail(PKV_ERR_UNSUPPORTED, "device %d: the allocation-free entry point serves devices 0..%d", dev,
                    kMaxDevices - 1);
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (!g_scratch_dev[dev]) {
        void* p = nullptr;
        e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess || !p)
            return fail(PKV_ERR_DEVICE, "hipGetSymbolAddress(scratch) on device %d: %s", dev, hipGetErrorString(e));
        g_scratch_dev[dev] = p;
    }
    *out = g_scratch_dev[dev];
    return PKV_OK;
}

// Workspace layout shared by both attention entry points:
// [split][layer][row][head][d_v] partial outputs, then [split][layer][row][head] LSEs.
void set_workspace(pkv::AttnArgs& a, void* workspace) {
    const size_t rows = (size_t)a.n_splits * a.n_layers * a.total_q * a.n_heads;
    a.ws_o = (float*)workspace;
    a.ws_lse = a.ws_o + rows * a.head_dim_v;
}

pkv_status run_attention(const void* q, const void* k_cache, const void* v_cache, void* out, const int32_t* q_pos,
                         const int32_t* kv_len, int32_t n_q_heads, int32_t n_kv_heads, int32_t head_dim, float scale,
                         const pkv_attn_desc* desc, const pkv_paged_cache* paging, void* workspace,
                         size_t workspace_bytes, void* stream) {
    pkv::AttnArgs a;
    pkv_status st = check_attention(q, k_cache, v_cache, out, q_pos, kv_len, n_q_heads, n_kv_heads,
                                    head_dim, scale, desc, true, a, paging);
    if (st != PKV_OK) return st;
    const int splits = pkv::attention_splits(a);
    const size_t need = pkv::attention_workspace_bytes(a, splits);
    if (need > 0) {
        if (!workspace) return fail(PKV_ERR_NULL, "workspace of %zu bytes is required", need);
        if (workspace_bytes < need)
            return fail(PKV_ERR_SHAPE, "workspace_bytes %zu < required %zu", workspace_bytes, need);
        if (!aligned16(workspace)) return fail(PKV_ERR_ALIGN, "workspace must be 16-byte aligned");
    }
    a.n_splits = splits;
    if (need > 0) set_workspace(a, workspace);
    if (a.total_q == 0) return ok();
    return device_status(pkv::launch_attention(a, (hipStream_t)stream), "suffix_attention launch");
}

}  // namespace

PKV_EXPORT pkv_status pkv_suffix_attention(const void* q, const void* k_cache, const void* v_cache,
                                           void* out, const int32_t* q_pos, const int32_t* kv_len,
                                           int32_t n_q_heads, int32_t n_kv_heads, int32_t head_dim,
                                           float scale, const pkv_attn_desc* desc, void* workspace,
                                           size_t workspace_bytes, void* stream) {
    return run_attention(q, k_cache, v_cache, out, q_pos, kv_len, n_q_heads, n_kv_heads, head_dim, scale, desc,
                         nullptr, workspace, workspace_bytes, stream);
}

PKV_EXPORT pkv_status pkv_suffix_attention_paged(const void* q, const void* k_pages, const void* v_pages,
                                                 void* out, const int32_t* q_pos, const int32_t* kv_len,
                                                 int32_t n_q_heads, int32_t n_kv_heads, int32_t head_dim,
                                                 float scale, const pkv_attn_desc* desc,
                                                 const pkv_paged_cache* paging, void* workspace,
                                                 size_t workspace_bytes, void* stream) {
    if (!paging) return fail(PKV_ERR_NULL, "paging is NULL");
    return run_attention(q, k_pages, v_pages, out, q_pos, kv_len, n_q_heads, n_kv_heads, head_dim, scale, desc,
                         paging, workspace, workspace_bytes, stream);
}

PKV_EXPORT pkv_status pkv_suffix_attention_noalloc(const void* q, const void* k_cache, const void* v_cache,
                                                   void* out, const int32_t* q_pos, const int32_t* kv_len,
                                                   int32_t n_q_heads, int32_t n_kv_heads, int32_t head_dim,
                                                   float scale, const pkv_attn_desc* desc, void* stream) {
    pkv::AttnArgs a;
    pkv_status st = check_attention(q, k_cache, v_cache, out, q_pos, kv_len, n_q_heads, n_kv_heads, head_dim,
                                    scale, desc, true, a);
    if (st != PKV_OK) return st;
    int splits = pkv::attention_splits(a);
    size_t need = pkv::attention_workspace_bytes(a, splits);
    if (need > PKV_NOALLOC_SCRATCH_BYTES) {
        if (desc->n_splits > 0)
            return fail(PKV_ERR_SHAPE,
                        "%d splits need %zu bytes of partials, more than the %zu-byte scratch of the "
                        "allocation-free entry point (use fewer splits, n_splits = 0, or pkv_suffix_attention "
                        "with a workspace)",
                        splits, need, (size_t)PKV_NOALLOC_SCRATCH_BYTES);
        while (splits > 1 && pkv::attention_workspace_bytes(a, splits) > PKV_NOALLOC_SCRATCH_BYTES) --splits;
        need = pkv::attention_workspace_bytes(a, splits);
    }
    a.n_splits = splits;
    if (need > 0) {
        void* sp = nullptr;
        st = scratch_on_current_device(&sp);
        if (st != PKV_OK) return st;
        set_workspace(a, sp);
    }
    if (a.total_q == 0) return ok();
    return device_status(pkv::launch_attention(a, (hipStream_t)stream), "suffix_attention_noalloc launch");
}

PKV_EXPORT const char* pkv_last_error(void) { return g_err; }

PKV_EXPORT int32_t pkv_version(void) { return PKV_VERSION; }
