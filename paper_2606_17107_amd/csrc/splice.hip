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
//     cos/sin of its pairs are formed once and reused from registers.  When
//     the whole wave shares one delta, each lane forms one pair's cos/sin and
//     the rotary lanes gather theirs by shuffle.
//       - rotary lane l:     chunks rope_c0+l and rope_c0+rope_nc/2+l.  With
//         HALF pairing these hold the two partners of the same 8 (bf16) or
//         4 (fp32) pairs; with INTERLEAVED pairing each chunk holds whole
//         pairs.  Either way a lane rotates 16/elem_bytes pairs.
//       - other K lanes:     two non-rotary chunks, copied.
//       - V lanes:           chunks m and m+n_vc/2, copied.
//     Lanes of consecutive tokens are consecutive threads, so each load or
//     store instruction of a wave covers whole 128-byte lines of
//     token-contiguous caches.
//   * omega_i = theta^(-2i/r) is formed in fp64 from seven powers of theta
//     the host passes in the kernel arguments (relative error about 1e-15
//     from the products).  Each thread forms delta*omega_i in fp64 and
//     reduces it by pi/2 with a two-part pi/2.  For the supported
//     |delta| < 2^24 and omega_i <= 1 the angle is below 2^24, so the error
//     of the reduced angle is dominated by omega_i's relative error times the
//     angle (below about 2e-8) plus the rounding of the fp64 product (below
//     2^24 * 2^-53 = 2^-29): below the fp32 rounding of the sin/cos that
//     follows, and far below the bf16 spacing (2^-8 relative) of the result.
//     sin and cos of the reduced angle in [-pi/4, pi/4] are their Taylor
//     series in fp32 (truncation error below 2e-9).  The rotation itself is fp32 with one round-to-nearest-even
//     to bf16.  delta == 0 copies bit-exact.
//   * A block covers a tile of tokens and a few (layer, kv_head) rows: many
//     small blocks keep the rows in flight at any moment close together in
//     memory.  The grid is (token tiles, row groups, segments); token tiles are
//     renumbered so that each XCD streams one contiguous range.  The K/V loads
//     of the first rows are issued before the positions are read and the
//     coefficients formed.
#include <math.h>

#include "pkv_internal.h"

namespace pkv {
namespace {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

// Launch shape (measured on MI355X).
constexpr int kUnroll = 1;         // rows whose loads are issued before any is used
constexpr int kRowsPerBlock = 1;   // (layer, kv_head) rows per block
constexpr int kBlock = 256;        // threads per block
constexpr int kSegTiles = 32;      // segment mode: token-tile blocks per (row group, segment)
constexpr int kSegAhead = 6;       // segment mode: tiles whose loads are issued before the first store
constexpr int kHalf = 0;
constexpr int kWave = 64;
constexpr int kXcds = 8;

// Streaming (non-temporal) loads and stores: a single chunk is touched once.
__device__ inline u32x4 ld16(const char* p) { return __builtin_nontemporal_load((const u32x4*)p); }
// Cached load: segment mode, where several segments may read one source chunk.
__device__ inline u32x4 ld16_cached(const char* p) { return *(const u32x4*)p; }
__device__ inline void st16(char* p, u32x4 v) { __builtin_nontemporal_store(v, (u32x4*)p); }

struct Geo {
    int lanes_k, lanes_v, lanes, tok_per_block, rows_per_block;
    int rope_c0, rope_nc, n_kc, n_vc, n_rows, n_pairs;
    int xcd_tiles;          // tiles per XCD when the tile count divides by 8, else 0
    int seg_xcd_rows;       // segment mode, 1-D grid: row groups per XCD (0: 3-D grid)
    int seg_n, seg_tile_blocks;   // segment mode, 1-D grid: segments, tile blocks
    uint32_t lanes_magic;   // ceil(2^32 / lanes)
    double rho[7];          // theta^(-2*2^b/rope_dim), b = 0..6
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

// Frequencies omega_i = theta^(-2i/r) for pairs i < 128 (rotary slices up to
// 256 channels), formed in fp64 from the seven powers rho_b = theta^(-2*2^b/r)
// the host passes in: omega_i is the product of rho_b over the set bits b of
// i (relative error below 1e-15; no memory access).
constexpr int kPairBits = 7;

// cos and sin of delta*omega.  The argument is formed and reduced by pi/2 in
// fp64; sin and cos of the reduced angle r (|r| <= pi/4) are the Taylor series
//   sin r = r - r^3/3! + r^5/5! - r^7/7! + r^9/9!
//   cos r = 1 - r^2/2! + r^4/4! - r^6/6! + r^8/8! - r^10/10!
// evaluated by Horner's rule in fp32; the quadrant picks signs and swaps.
__device__ inline void delta_sincos(int64_t delta, double omega, float& c, float& s) {
    const double x = (double)delta * omega;
    const double k = rint(x * 0.63661977236758134308);            // 2/pi
    double r = fma(-k, 1.5707963267948966192, x);                // pi/2, leading part
    r = fma(-k, 6.123233995736766036e-17, r);                    // pi/2, trailing part
    const float f = (float)r;
    const float z = f * f;
    float ps = fmaf(z, 2.75573192e-6f, -1.98412698e-4f);          // 1/9!, -1/7!
    ps = fmaf(z, ps, 8.33333333e-3f);                             // 1/5!
    ps = fmaf(z, ps, -0.166666667f);                              // -1/3!
    const float sr = fmaf(f * z, ps, f);
    float pc = fmaf(z, -2.75573192e-7f, 2.48015873e-5f);          // -1/10!, 1/8!
    pc = fmaf(z, pc, -1.38888889e-3f);                            // -1/6!
    pc = fmaf(z, pc, 4.16666667e-2f);                             // 1/4!
    pc = fmaf(z, pc, -0.5f);                                      // -1/2!
    const float cr = fmaf(z, pc, 1.0f);
    const int q = (int)((int64_t)k & 3);
    const float sa = (q & 1) ? cr : sr;
    const float ca = (q & 1) ? sr : cr;
    s = (q & 2) ? -sa : sa;
    c = ((q + 1) & 2) ? -ca : ca;
}

// Explicit per-pair frequencies (scaled RoPE, or M-RoPE with the spatial pairs
// at zero); an empty argument when the theta schedule is used.
template <bool TAB>
struct FreqArg {};
template <>
struct FreqArg<true> {
    double w[1 << kPairBits];
};

__device__ inline double pair_omega(int pair, const Geo& g) {
    double w = 1.0;
#pragma unroll
    for (int b = 0; b < kPairBits; ++b)
        if ((pair >> b) & 1) w *= g.rho[b];
    return w;
}

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

// Pair index of coefficient j of rotary lane l (HALF: the lane's chunk holds CE
// consecutive pairs; INTERLEAVED: each of its two chunks holds CE/2 pairs).
template <int CE, int STYLE>
__device__ inline int lane_pair(int l, int j, int half_r) {
    if constexpr (STYLE == kHalf)
        return l * CE + j;
    else
        return j < CE / 2 ? l * (CE / 2) + j : (half_r + l) * (CE / 2) + (j - CE / 2);
}

template <int EB, int STYLE, bool SEG, bool TAB, bool PAGED>
__global__ __launch_bounds__(kBlock) void splice_kernel(SpliceArgs a, Geo g, FreqArg<TAB> ft) {
    static_assert(!(PAGED && SEG), "paged destinations are per-token mode only");
    constexpr int CE = 16 / EB;   // elements per 16-byte chunk = pairs per rotary lane
    // Explicit frequencies: lane l holds those of pairs l and 64 + l, loaded
    // before anything else so that waiting for them leaves the later loads in
    // flight; other lanes' pairs are gathered by shuffle.
    double w_lo = 0.0, w_hi = 0.0;
    if constexpr (TAB) {
        w_lo = ft.w[__lane_id()];
        w_hi = ft.w[kWave + __lane_id()];
    }
    // Grid: token mode (tiles, row groups); segment mode (segments, tile
    // blocks, row groups) with the segment the fastest axis, so the blocks of
    // all segments at one (tile block, row) are dispatched together and
    // segments that read the same source chunk (a shared skill) find it in the
    // caches.  When the row groups divide evenly over the XCDs, segment mode
    // runs on a 1-D grid whose ids are dealt to the XCDs round-robin: XCD x
    // takes row groups x*seg_xcd_rows .. one at a time, so every read of one
    // source chunk goes through one XCD's L2 and only the first reaches
    // memory; within a row the tile blocks of one segment are consecutive, so
    // the blocks in flight write into few destination ranges (a row's source
    // chunks, a few MB, stay in that L2 meanwhile).
    int grp = blockIdx.y, seg_i = 0, tile_blk = 0, tile_blocks = 1;
    if constexpr (SEG) {
        if (g.seg_xcd_rows) {
            const uint32_t id = blockIdx.x;
            const uint32_t slot = id / kXcds;
            tile_blk = (int)(slot % (uint32_t)g.seg_tile_blocks);
            const uint32_t rest = slot / (uint32_t)g.seg_tile_blocks;
            seg_i = (int)(rest % (uint32_t)g.seg_n);
            grp = (int)(id % kXcds) * g.seg_xcd_rows + (int)(rest / (uint32_t)g.seg_n);
            tile_blocks = g.seg_tile_blocks;
        } else {
            seg_i = blockIdx.x;
            tile_blk = blockIdx.y;
            tile_blocks = gridDim.y;
            grp = blockIdx.z;
        }
    }
    const uint32_t tid = threadIdx.x;
    const uint32_t tl = g.lanes == 1 ? tid : __umulhi(tid, g.lanes_magic);   // tid / lanes, exact here
    const int lane = (int)(tid - tl * (uint32_t)g.lanes);
    const bool in_tile = (int)tl < g.tok_per_block;

    // Segment mode: the whole block works on one segment, whose delta is
    // uniform; its tiles are shared out round-robin over the blocks of the
    // x axis, which is sized for the longest segment (capped), so short
    // segments leave few blocks idle.
    SpliceSegment sg{};
    int64_t n_tok = a.n_tokens;
    if constexpr (SEG) {
        sg = a.segs[seg_i];
        n_tok = sg.n_tokens;
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
    const int64_t s0 = is_k ? a.src_k_stride[0] : a.src_v_stride[0];
    const int64_t s1 = is_k ? a.src_k_stride[1] : a.src_v_stride[1];
    const int64_t s2 = is_k ? a.src_k_stride[2] : a.src_v_stride[2];
    const int64_t d0 = is_k ? a.dst_k_stride[0] : a.dst_v_stride[0];
    const int64_t d1 = is_k ? a.dst_k_stride[1] : a.dst_v_stride[1];
    const int64_t d2 = is_k ? a.dst_k_stride[2] : a.dst_v_stride[2];
    const int64_t dpg = PAGED ? (is_k ? a.dst_k_page_stride : a.dst_v_page_stride) : 0;
    const char* const src_t = (is_k ? a.src_k : a.src_v) + ca * 16;
    char* const dst_t = (is_k ? a.dst_k : a.dst_v) + ca * 16;
    const int ob = (cb - ca) * 16;

    // Rows r0..r1 of this block, walked as (layer, head) without division;
    // rows past r1 in the last unrolled step load row r1 - 1 again.
    const int r0 = grp * g.rows_per_block;
    const int r1 = min(r0 + g.rows_per_block, g.n_rows);
    const int layer0 = r0 / a.n_kv_heads;
    const int head0 = r0 - layer0 * a.n_kv_heads;
    const int last_layer = (r1 - 1) / a.n_kv_heads;
    const int last_head = (r1 - 1) - last_layer * a.n_kv_heads;

    float cs[CE], sn[CE];
    // Rotation coefficients of this lane's CE pairs for the lane's delta.
    // When every working lane of the wave has the same delta (always so in
    // segment mode; so for a contiguous chunk in token mode), lane j
    // evaluates pair j once and rotary lanes gather theirs by shuffle;
    // otherwise each rotary lane evaluates its own CE pairs.  Every lane of
    // the wave calls this (the shuffles need them all).
    auto coefficients = [&](int64_t delta, bool work) __attribute__((always_inline)) {
        const int32_t d_ref = __shfl((int32_t)delta, 0);
        const bool uniform = __all(!work || delta == (int64_t)d_ref) && g.n_pairs <= kWave;
        if (uniform) {
            if (d_ref != 0) {
                float c1 = 1.0f, s1v = 0.0f;
                const int j = __lane_id();
                if (j < g.n_pairs) delta_sincos(d_ref, TAB ? w_lo : pair_omega(j, g), c1, s1v);
#pragma unroll
                for (int e = 0; e < CE; ++e) {
                    const int src = rope ? lane_pair<CE, STYLE>(lane, e, half_r) : 0;
                    cs[e] = __shfl(c1, src);
                    sn[e] = __shfl(s1v, src);
                }
            }
        } else if constexpr (TAB) {
            // every lane takes part in the shuffles (the branch is wave-uniform)
            double wp[CE];
#pragma unroll
            for (int e = 0; e < CE; ++e) {
                const int pr = rope ? lane_pair<CE, STYLE>(lane, e, half_r) : 0;
                const double lo = __shfl(w_lo, pr & (kWave - 1)), hi = __shfl(w_hi, pr & (kWave - 1));
                wp[e] = pr < kWave ? lo : hi;
            }
            if (rope && delta != 0) {
#pragma unroll
                for (int e = 0; e < CE; ++e) delta_sincos(delta, wp[e], cs[e], sn[e]);
            }
        } else if (rope && delta != 0) {
#pragma unroll
            for (int e = 0; e < CE; ++e)
                delta_sincos(delta, pair_omega(lane_pair<CE, STYLE>(lane, e, half_r), g), cs[e], sn[e]);
        }
    };

    if constexpr (SEG) {
        // Segment mode: one (layer, head) row per block and one delta per
        // segment, so the coefficients are formed once.  The block's tiles
        // (tile_blk, tile_blk + tile_blocks, ...) go kSegAhead at a time:
        // the loads of all of them are issued before the first store, so each
        // wave keeps kSegAhead tiles of loads in flight.  Lanes without a
        // readable source row load nothing.
        static_assert(kRowsPerBlock == 1, "segment mode handles one row per block");
        const char* const srow = src_t + ((int64_t)layer0 * s0 + (int64_t)head0 * s1) * EB;
        char* const drow = dst_t + ((int64_t)layer0 * d0 + (int64_t)head0 * d1) * EB;
        const int64_t delta = (int64_t)sg.dst_pos0 - (int64_t)sg.src_pos0;
        coefficients(delta, true);
        const bool rot = rope && delta != 0;
        for (uint32_t step = 0;; step += kSegAhead) {
            if ((int64_t)(tile_blk + step * tile_blocks) * g.tok_per_block >= n_tok) break;   // uniform
            u32x4 va[kSegAhead], vb[kSegAhead];
            int64_t dst_row[kSegAhead];
            bool present[kSegAhead], work[kSegAhead];
#pragma unroll
            for (int u = 0; u < kSegAhead; ++u) {
                const int64_t t = (int64_t)(tile_blk + (step + u) * tile_blocks) * g.tok_per_block + tl;
                present[u] = in_tile && t < n_tok;
                const int64_t src_slot = sg.src_slot0 + t;
                const bool active = present[u] && src_slot >= 0 && src_slot < a.n_tokens;
                const int64_t p = (int64_t)sg.dst_pos0 + t;
                const int64_t dst_slot = p >= 0 && p < sg.dst_seq_len ? sg.dst_seq_base + p : -1;
                work[u] = active && dst_slot >= 0 && dst_slot < a.dst_capacity;
                dst_row[u] = dst_slot * d2;
                va[u] = vb[u] = u32x4{0u, 0u, 0u, 0u};
                if (active) {
                    const char* sp = srow + src_slot * s2 * EB;
                    va[u] = ld16_cached(sp);
                    vb[u] = ld16_cached(sp + ob);
                }
            }
#pragma unroll
            for (int u = 0; u < kSegAhead; ++u) {
                if (work[u]) {
                    if (rot) rotate_chunks<EB, STYLE>(va[u], vb[u], cs, sn);
                    char* dp = drow + dst_row[u] * EB;
                    st16(dp, va[u]);
                    st16(dp + ob, vb[u]);
                }
                if (present[u] && !work[u] && lane == 0 && grp == 0 && a.err_flag) atomicOr(a.err_flag, 1);
            }
        }
        return;
    }

    // Token mode: one tile per block.  Workgroups are dealt to the XCDs
    // round-robin, so when the tile count divides evenly the tiles are
    // renumbered to give each XCD one contiguous range of tokens.
    uint32_t tile = blockIdx.x;
    if (g.xcd_tiles) tile = (tile % kXcds) * g.xcd_tiles + tile / kXcds;
    const int64_t t = (int64_t)tile * g.tok_per_block + tl;

    // Loads go out in the order their results are needed: positions, then
    // the K/V rows.  Memory counters retire in order, so waiting for the
    // positions (and the frequencies) leaves the K/V loads in flight while
    // the coefficients are formed.  Lanes and rows without work load from a
    // clamped, in-range address and store nothing; they stay to the end
    // because the wave shares its coefficients through shuffles.
    const bool present = in_tile && t < n_tok;   // a token of the chunk
    const bool active = present;
    const int64_t src_slot = active ? t : a.n_tokens - 1;
    const int32_t dp = a.dst_pos[src_slot];
    const int32_t spos = a.src_pos[src_slot];
    const int32_t dslot = a.dst_slot ? a.dst_slot[src_slot] : 0;
    const char* sbase = src_t + src_slot * s2 * EB;

    int layer = layer0, head = head0;
    u32x4 va[kUnroll], vb[kUnroll];
    int64_t doff[kUnroll];
    auto load_rows = [&](int r) __attribute__((always_inline)) {
#pragma unroll
        for (int u = 0; u < kUnroll; ++u) {
            const bool in = r + u < r1;
            const int l = in ? layer : last_layer, h = in ? head : last_head;
            doff[u] = ((int64_t)l * d0 + (int64_t)h * d1) * EB;
            const char* sp = sbase + ((int64_t)l * s0 + (int64_t)h * s1) * EB;
            va[u] = ld16(sp);
            vb[u] = ld16(sp + ob);
            if (++head == a.n_kv_heads) {
                head = 0;
                ++layer;
            }
        }
    };
    load_rows(r0);

    const int64_t dst_slot = a.dst_slot ? dslot : dp;   // slots follow positions unless given
    const int64_t delta = (int64_t)dp - (int64_t)spos;
    const bool valid = dst_slot >= 0 && dst_slot < a.dst_capacity;
    const bool work = active && valid;
    // Paged destination: the slot's page id is read from an in-range entry
    // for every lane (no branch, so the wait for it stays with the K/V
    // wait before the stores); a page outside the pool skips the token.
    int64_t dst_row = dst_slot;
    bool page_ok = true;
    if constexpr (PAGED) {
        const int64_t pidx = work ? dst_slot >> a.page_shift : 0;
        const int32_t* table = !is_k && a.dst_v_pages ? a.dst_v_pages : a.dst_pages;
        const int32_t page = table[pidx];
        page_ok = page >= 0 && page < a.n_pages;
        dst_row = (int64_t)page * dpg + (dst_slot & ((1 << a.page_shift) - 1)) * d2;
    } else {
        dst_row = dst_slot * d2;
    }

    coefficients(delta, work);
    const bool rot = rope && delta != 0;

    if (work && page_ok) {
        char* dbase = dst_t + dst_row * EB;
        for (int r = r0;;) {
#pragma unroll
            for (int u = 0; u < kUnroll; ++u) {
                if (r + u < r1) {
                    if (rot) rotate_chunks<EB, STYLE>(va[u], vb[u], cs, sn);
                    st16(dbase + doff[u], va[u]);
                    st16(dbase + doff[u] + ob, vb[u]);
                }
            }
            r += kUnroll;
            if (r >= r1) break;
            load_rows(r);
        }
    }
    if (present && !(work && page_ok) && lane == 0 && grp == 0 && a.err_flag) atomicOr(a.err_flag, 1);
}

template <int EB, int STYLE>
hipError_t launch_typed(const SpliceArgs& a, const Geo& g, dim3 grid, dim3 block, hipStream_t st) {
    if (a.dst_pages) {   // paged destination: per-token mode, theta schedule
        if (a.segs || a.omega) return hipErrorInvalidValue;
        const FreqArg<false> ft;
        hipLaunchKernelGGL((splice_kernel<EB, STYLE, false, false, true>), grid, block, 0, st, a, g, ft);
    } else if (a.omega) {   // explicit frequencies: per-token mode
        if (a.segs) return hipErrorInvalidValue;
        FreqArg<true> ft;
        for (int i = 0; i < (1 << kPairBits); ++i) ft.w[i] = i < g.n_pairs ? a.omega[i] : 0.0;
        hipLaunchKernelGGL((splice_kernel<EB, STYLE, false, true, false>), grid, block, 0, st, a, g, ft);
    } else {
        const FreqArg<false> ft;
        if (a.segs)
            hipLaunchKernelGGL((splice_kernel<EB, STYLE, true, false, false>), grid, block, 0, st, a, g, ft);
        else
            hipLaunchKernelGGL((splice_kernel<EB, STYLE, false, false, false>), grid, block, 0, st, a, g, ft);
    }
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
    g.n_pairs = a.rope_dim / 2;
    g.lanes_k = g.n_kc / 2;
    g.lanes_v = g.n_vc / 2;
    g.lanes = g.lanes_k + g.lanes_v;
    g.tok_per_block = g.lanes >= kBlock ? 1 : kBlock / g.lanes;
    g.n_rows = a.n_layers * a.n_kv_heads;

    const bool seg = a.segs != nullptr;
    // Every index array the kernel dereferences must be present.
    if (!a.src_k || !a.dst_k || (g.lanes_v > 0 && (!a.src_v || !a.dst_v)) ||
        (!seg && (!a.src_pos || !a.dst_pos)))
        return hipErrorInvalidValue;
    if (a.dst_pages && (a.page_shift < 5 || a.page_shift > 20 || a.n_pages <= 0 ||
                        a.dst_capacity > ((int64_t)a.max_pages << a.page_shift)))
        return hipErrorInvalidValue;
    const int64_t tokens = seg ? a.max_seg_tokens : a.n_tokens;
    const int64_t nz = seg ? a.n_segs : 1;
    if (tokens <= 0 || nz <= 0 || g.n_rows <= 0) return hipSuccess;

    if (g.n_pairs > (1 << kPairBits)) return hipErrorInvalidValue;
    g.rows_per_block = g.n_rows < kRowsPerBlock ? g.n_rows : kRowsPerBlock;
    int64_t n_tiles = (tokens + g.tok_per_block - 1) / g.tok_per_block;
    if (seg && n_tiles > kSegTiles) n_tiles = kSegTiles;   // blocks loop over a segment's tiles
    const int64_t n_groups = (g.n_rows + g.rows_per_block - 1) / g.rows_per_block;
    if (n_tiles > 0x7fffffff || n_groups > 65535 || nz > 65535) return hipErrorInvalidConfiguration;
    // Segment mode sizes the tile axis for the longest segment, so a shorter
    // segment's tiles would all fall on the first XCDs: keep round-robin order.
    g.xcd_tiles = !seg && n_tiles % kXcds == 0 ? (int)(n_tiles / kXcds) : 0;
    g.lanes_magic = g.lanes > 1 ? (uint32_t)((0x100000000ull + g.lanes - 1) / g.lanes) : 0;   // ceil(2^32/lanes)

    for (int b = 0; b < kPairBits; ++b) g.rho[b] = pow(a.theta, -2.0 * (double)(1 << b) / (double)a.rope_dim);

    // Segment mode with row groups divisible by the XCD count: 1-D grid
    // (decoded in the kernel so that each XCD owns whole row groups).
    const int64_t seg_1d = nz * n_tiles * n_groups;
    g.seg_xcd_rows = seg && n_groups % kXcds == 0 && seg_1d <= 0x7fffffff ? (int)(n_groups / kXcds) : 0;
    g.seg_n = (int)nz;
    g.seg_tile_blocks = (int)n_tiles;
    dim3 grid = seg ? (g.seg_xcd_rows ? dim3((unsigned)seg_1d, 1u, 1u)
                                      : dim3((unsigned)nz, (unsigned)n_tiles, (unsigned)n_groups))
                    : dim3((unsigned)n_tiles, (unsigned)n_groups, 1u);
    dim3 block((unsigned)kBlock);
    if (a.elem_bytes == 2)
        return a.rope_style == kHalf ? launch_typed<2, 0>(a, g, grid, block, stream)
                                     : launch_typed<2, 1>(a, g, grid, block, stream);
    return a.rope_style == kHalf ? launch_typed<4, 0>(a, g, grid, block, stream)
                                 : launch_typed<4, 1>(a, g, grid, block, stream);
}

}  // namespace pkv
