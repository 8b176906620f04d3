// Reposition + splice: rotate a chunk's cached post-RoPE keys by
// delta = dst_pos - src_pos and write them, with the values copied bit-exact,
// into the destination cache slots given by the destination positions.
// (Paper Sec. 5 "From mechanism to prediction"; Fig. "Two cache operations"
// (b); Sec. 8 MLA adapter: only the decoupled k_pe slice of a latent row
// rotates.)
//
// Design (HBM-bound stream, about 1.5 flop/byte):
//   * A row of K (head_dim channels) or V (v_dim channels) is cut into 16-byte
//     chunks.  Every thread ("lane") owns two chunks of one token's row and
//     keeps that assignment for every (layer, kv_head) row it visits, so the
//     cos/sin of its pairs are formed once and reused from registers.
//       - rotary lane l:     chunks rope_c0+l and rope_c0+rope_nc/2+l.  With
//         HALF pairing these hold the two partners of the same 8 (bf16) or
//         4 (fp32) pairs; with INTERLEAVED pairing each chunk holds whole
//         pairs.  Either way a lane rotates 16/elem_bytes pairs.
//       - other K lanes:     two non-rotary chunks, copied.
//       - V lanes:           chunks m and m+n_vc/2, copied.
//     Lanes of consecutive tokens are consecutive threads, so each load or
//     store instruction of a wave covers whole 128-byte lines of
//     token-contiguous caches.
//   * The angle delta*omega_i and its cos/sin are computed in fp64 once per
//     thread and rounded to fp32; the rotation itself is fp32 with one
//     round-to-nearest-even to bf16.  delta == 0 copies bit-exact.
//   * The block grid is (token tiles, row chunks[, segments]); every thread
//     walks rows_per_block (layer, kv_head) rows, issuing the loads of
//     kUnroll rows before using them to keep bytes in flight.
#include <math.h>

#include "pkv_internal.h"

namespace pkv {
namespace {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

// Launch-shape constants (tuned on MI355X; overridable at build time).
#ifndef PKV_SPLICE_UNROLL
#define PKV_SPLICE_UNROLL 4        // rows whose loads are issued before any is used
#endif
#ifndef PKV_SPLICE_TARGET_BLOCKS
#define PKV_SPLICE_TARGET_BLOCKS 8192
#endif
#ifndef PKV_SPLICE_MIN_ROWS
#define PKV_SPLICE_MIN_ROWS 8      // rows per thread at least (amortises the cos/sin)
#endif
#ifndef PKV_SPLICE_NONTEMPORAL
#define PKV_SPLICE_NONTEMPORAL 1   // streaming loads/stores: the data is touched once
#endif
constexpr int kUnroll = PKV_SPLICE_UNROLL;
constexpr int kHalf = 0;

__device__ inline u32x4 ld16(const char* p) {
#if PKV_SPLICE_NONTEMPORAL
    return __builtin_nontemporal_load((const u32x4*)p);
#else
    return *(const u32x4*)p;
#endif
}
__device__ inline void st16(char* p, u32x4 v) {
#if PKV_SPLICE_NONTEMPORAL
    __builtin_nontemporal_store(v, (u32x4*)p);
#else
    *(u32x4*)p = v;
#endif
}

struct Geo {
    int lanes_k, lanes_v, lanes, tok_per_block, rows_per_block;
    int rope_c0, rope_nc, n_kc, n_vc, n_rows;
};

__device__ inline float bf_lo(uint32_t u) { return __uint_as_float(u << 16); }
__device__ inline float bf_hi(uint32_t u) { return __uint_as_float(u & 0xffff0000u); }

// fp32 -> bf16, round to nearest even (finite inputs).
__device__ inline uint32_t bf_rne(float f) {
    uint32_t u = __float_as_uint(f);
    u += 0x7fffu + ((u >> 16) & 1u);
    return u >> 16;
}
__device__ inline uint32_t bf_pack(float lo, float hi) { return bf_rne(lo) | (bf_rne(hi) << 16); }

__device__ inline void rot(float a, float b, float c, float s, float& ra, float& rb) {
    ra = fmaf(a, c, -(b * s));
    rb = fmaf(a, s, b * c);
}

// Rotate the pairs held by chunks x (first) and y (second) of a rotary lane.
template <int EB, int STYLE>
__device__ inline void rotate_chunks(u32x4& x, u32x4& y, const float* c, const float* s) {
    if constexpr (EB == 2) {
        if constexpr (STYLE == kHalf) {
            // element e of x pairs with element e of y; coefficient e
#pragma unroll
            for (int w = 0; w < 4; ++w) {
                float a0, b0, a1, b1;
                rot(bf_lo(x[w]), bf_lo(y[w]), c[2 * w], s[2 * w], a0, b0);
                rot(bf_hi(x[w]), bf_hi(y[w]), c[2 * w + 1], s[2 * w + 1], a1, b1);
                x[w] = bf_pack(a0, a1);
                y[w] = bf_pack(b0, b1);
            }
        } else {
            // each 32-bit word is one (even, odd) pair; x uses coefficients 0..3, y 4..7
#pragma unroll
            for (int w = 0; w < 4; ++w) {
                float a, b;
                rot(bf_lo(x[w]), bf_hi(x[w]), c[w], s[w], a, b);
                x[w] = bf_pack(a, b);
                rot(bf_lo(y[w]), bf_hi(y[w]), c[4 + w], s[4 + w], a, b);
                y[w] = bf_pack(a, b);
            }
        }
    } else {
        if constexpr (STYLE == kHalf) {
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                float a, b;
                rot(__uint_as_float(x[e]), __uint_as_float(y[e]), c[e], s[e], a, b);
                x[e] = __float_as_uint(a);
                y[e] = __float_as_uint(b);
            }
        } else {
#pragma unroll
            for (int p = 0; p < 2; ++p) {
                float a, b;
                rot(__uint_as_float(x[2 * p]), __uint_as_float(x[2 * p + 1]), c[p], s[p], a, b);
                x[2 * p] = __float_as_uint(a);
                x[2 * p + 1] = __float_as_uint(b);
                rot(__uint_as_float(y[2 * p]), __uint_as_float(y[2 * p + 1]), c[2 + p], s[2 + p], a, b);
                y[2 * p] = __float_as_uint(a);
                y[2 * p + 1] = __float_as_uint(b);
            }
        }
    }
}

template <int EB, int STYLE, bool SEG>
__global__ __launch_bounds__(256) void splice_kernel(SpliceArgs a, Geo g) {
    constexpr int CE = 16 / EB;   // elements per 16-byte chunk = pairs per rotary lane
    const int tid = threadIdx.x;
    const int tl = tid / g.lanes;
    const int lane = tid - tl * g.lanes;
    if (tl >= g.tok_per_block) return;
    const int64_t t = (int64_t)blockIdx.x * g.tok_per_block + tl;

    int64_t src_slot, dst_slot, delta;
    bool valid;
    if constexpr (SEG) {
        const SpliceSegment sg = a.segs[blockIdx.z];
        if (t >= sg.n_tokens) return;
        src_slot = sg.src_slot0 + t;
        const int64_t p = (int64_t)sg.dst_pos0 + t;
        dst_slot = sg.dst_seq_base + p;
        delta = (int64_t)sg.dst_pos0 - (int64_t)sg.src_pos0;
        valid = src_slot >= 0 && src_slot < a.n_tokens && p >= 0 && p < sg.dst_seq_len &&
                dst_slot >= 0 && dst_slot < a.dst_capacity;
    } else {
        if (t >= a.n_tokens) return;
        src_slot = t;
        const int32_t dp = a.dst_pos[t];
        dst_slot = dp;
        delta = (int64_t)dp - (int64_t)a.src_pos[t];
        valid = dst_slot >= 0 && dst_slot < a.dst_capacity;
    }
    if (!valid) {
        if (lane == 0 && blockIdx.y == 0 && a.err_flag) atomicOr(a.err_flag, 1);
        return;
    }

    // This lane's two chunks and whether they rotate.
    const bool is_k = lane < g.lanes_k;
    const int half_r = g.rope_nc >> 1;
    int ca, cb;
    bool rope = false;
    if (is_k) {
        if (lane < half_r) {
            rope = true;
            ca = g.rope_c0 + lane;
            cb = ca + half_r;
        } else {
            const int m = lane - half_r;
            const int hn = (g.n_kc - g.rope_nc) >> 1;
            const int i0 = m, i1 = m + hn;
            ca = i0 < g.rope_c0 ? i0 : i0 + g.rope_nc;
            cb = i1 < g.rope_c0 ? i1 : i1 + g.rope_nc;
        }
    } else {
        const int m = lane - g.lanes_k;
        ca = m;
        cb = m + (g.n_vc >> 1);
    }
    rope = rope && delta != 0;

    float cs[CE], sn[CE];
    if (rope) {
        const double inv_r = 1.0 / (double)a.rope_dim;
#pragma unroll
        for (int j = 0; j < CE; ++j) {
            int pair;
            if constexpr (STYLE == kHalf)
                pair = lane * CE + j;
            else
                pair = j < CE / 2 ? lane * (CE / 2) + j : (half_r + lane) * (CE / 2) + (j - CE / 2);
            const double w = pow(a.theta, -2.0 * (double)pair * inv_r);
            double sd, cd;
            sincos((double)delta * w, &sd, &cd);
            cs[j] = (float)cd;
            sn[j] = (float)sd;
        }
    }

    const int64_t s0 = is_k ? a.src_k_stride[0] : a.src_v_stride[0];
    const int64_t s1 = is_k ? a.src_k_stride[1] : a.src_v_stride[1];
    const int64_t s2 = is_k ? a.src_k_stride[2] : a.src_v_stride[2];
    const int64_t d0 = is_k ? a.dst_k_stride[0] : a.dst_v_stride[0];
    const int64_t d1 = is_k ? a.dst_k_stride[1] : a.dst_v_stride[1];
    const int64_t d2 = is_k ? a.dst_k_stride[2] : a.dst_v_stride[2];
    const char* sbase = (is_k ? a.src_k : a.src_v) + src_slot * s2 * EB;
    char* dbase = (is_k ? a.dst_k : a.dst_v) + dst_slot * d2 * EB;
    const int oa = ca * 16, ob = cb * 16;

    const int r0 = blockIdx.y * g.rows_per_block;
    const int r1 = min(r0 + g.rows_per_block, g.n_rows);
    for (int r = r0; r < r1; r += kUnroll) {
        u32x4 va[kUnroll], vb[kUnroll];
        int64_t doff[kUnroll];
#pragma unroll
        for (int u = 0; u < kUnroll; ++u) {
            const int rr = r + u;
            if (rr < r1) {
                const int layer = rr / a.n_kv_heads;
                const int head = rr - layer * a.n_kv_heads;
                const int64_t so = ((int64_t)layer * s0 + (int64_t)head * s1) * EB;
                doff[u] = ((int64_t)layer * d0 + (int64_t)head * d1) * EB;
                va[u] = ld16(sbase + so + oa);
                vb[u] = ld16(sbase + so + ob);
            }
        }
#pragma unroll
        for (int u = 0; u < kUnroll; ++u) {
            if (r + u < r1) {
                if (rope) rotate_chunks<EB, STYLE>(va[u], vb[u], cs, sn);
                st16(dbase + doff[u] + oa, va[u]);
                st16(dbase + doff[u] + ob, vb[u]);
            }
        }
    }
}

template <int EB, int STYLE>
hipError_t launch_typed(const SpliceArgs& a, const Geo& g, dim3 grid, dim3 block, hipStream_t st) {
    if (a.segs)
        hipLaunchKernelGGL((splice_kernel<EB, STYLE, true>), grid, block, 0, st, a, g);
    else
        hipLaunchKernelGGL((splice_kernel<EB, STYLE, false>), grid, block, 0, st, a, g);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_splice(const SpliceArgs& a, hipStream_t stream) {
    const int ce = 16 / a.elem_bytes;
    Geo g;
    g.n_kc = a.head_dim / ce;
    g.n_vc = a.v_dim / ce;
    g.rope_c0 = a.rope_offset / ce;
    g.rope_nc = a.rope_dim / ce;
    g.lanes_k = g.n_kc / 2;
    g.lanes_v = g.n_vc / 2;
    g.lanes = g.lanes_k + g.lanes_v;
    g.tok_per_block = g.lanes >= 256 ? 1 : 256 / g.lanes;
    g.n_rows = a.n_layers * a.n_kv_heads;

    const bool seg = a.segs != nullptr;
    // Every index array the kernel dereferences must be present.
    if (!a.src_k || !a.dst_k || (g.lanes_v > 0 && (!a.src_v || !a.dst_v)) ||
        (!seg && (!a.src_pos || !a.dst_pos)))
        return hipErrorInvalidValue;
    const int64_t tokens = seg ? a.max_seg_tokens : a.n_tokens;
    const int64_t nz = seg ? a.n_segs : 1;
    if (tokens <= 0 || nz <= 0 || g.n_rows <= 0) return hipSuccess;

    const int64_t gx = (tokens + g.tok_per_block - 1) / g.tok_per_block;
    // Enough blocks to fill 256 CUs several times over, while every thread
    // still visits several rows so its cos/sin are reused.
    int64_t want_y = (PKV_SPLICE_TARGET_BLOCKS + gx * nz - 1) / (gx * nz);
    if (want_y < 1) want_y = 1;
    int rows = (int)((g.n_rows + want_y - 1) / want_y);
    rows = rows < PKV_SPLICE_MIN_ROWS ? (g.n_rows < PKV_SPLICE_MIN_ROWS ? g.n_rows : PKV_SPLICE_MIN_ROWS) : rows;
    g.rows_per_block = rows;
    const int gy = (g.n_rows + rows - 1) / rows;

    dim3 grid((unsigned)gx, (unsigned)gy, (unsigned)nz);
    dim3 block((unsigned)(g.tok_per_block * g.lanes));
    if (a.elem_bytes == 2)
        return a.rope_style == kHalf ? launch_typed<2, 0>(a, g, grid, block, stream)
                                     : launch_typed<2, 1>(a, g, grid, block, stream);
    return a.rope_style == kHalf ? launch_typed<4, 0>(a, g, grid, block, stream)
                                 : launch_typed<4, 1>(a, g, grid, block, stream);
}

}  // namespace pkv
