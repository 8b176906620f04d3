// bf16 GQA suffix attention for gfx950: causal attention of the suffix /
// erratum queries over the spliced cache (paper Sec. 5 "Linear-time TTFT";
// Sec. 4 erratum; Sec. 6 delta prefill).
//
// Work decomposition
//   * MFMA 32x32x16 bf16 -> fp32.  The N axis carries (query, head-in-group)
//     rows of one KV head: row m <-> query m / G, head kv_head*G + m % G, so a
//     K/V byte staged in LDS serves every row of the workgroup (QB 32-row
//     blocks per wave, NW waves).
//   * Scores are formed transposed, S^T = K Q^T: a lane holds 16 keys of ONE
//     row, so the running max needs one cross-lane step and the running sum
//     none until the end, and the probabilities P^T already sit in the lane
//     layout of the B operand of O^T = V^T P^T (no LDS round trip for P).
//   * K and V tiles of 64 keys stream HBM -> LDS with LDS-DMA loads
//     (global_load_lds, 16 bytes per lane) through NS stages, so NS-1 tiles
//     are in flight while one is consumed.  16-byte chunks of a row are
//     XOR-swizzled by swz(key) (below) to spread LDS banks.
//   * V stays row-major ([key][channel]) in LDS; the transposed A operand of
//     the PV product comes from ds_read_b64_tr_b16, with the keys of each
//     16-key step ordered as the P^T accumulator holds them.
#include <type_traits>

#include "attn_common.h"

namespace pkv {
namespace {

constexpr int BN = 64;   // keys per tile

// XOR swizzle of a row's 16-byte chunk index by its key (3 bits).  K operand
// reads take one logical chunk from 8 consecutive keys: swz maps keys 0..7
// to 0,2,4,6,1,3,5,7, all distinct, so they hit 8 distinct bank groups.  The
// transposed V reads take two adjacent chunks (c, c+1; c even) from 4
// consecutive keys 4m..4m+3: swz gives 2r (+1), so the four rows land on four
// distinct chunk pairs.
__device__ inline int swz(int key) { return ((key & 3) << 1) | ((key >> 2) & 1); }

// Scheduling pattern for the overlapped region (QK^T of the next tile next
// to the probabilities of this one): per K-operand read, its two MFMAs
// (32 cycles each) with about eight VALU instructions in their shadow.
#ifndef PKV_ATTN_PINGPONG
#define PKV_ATTN_PINGPONG 1
#endif
#ifndef PKV_ATTN_INTERLEAVE
#define PKV_ATTN_INTERLEAVE 1
#endif
template <int KS>
__device__ inline void interleave_region() {
    if (!PKV_ATTN_INTERLEAVE) return;
#pragma unroll
    for (int i = 0; i < 2 * KS; ++i) {
        if (i % 2 == 0) __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);   // DS read
        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);                   // MFMA
        __builtin_amdgcn_sched_group_barrier(0x002, 8, 0);                   // VALU
    }
}

template <int D, int QB, int NW, int NS, bool PIPE>
__global__ __launch_bounds__(NW * 64, NW == 4 && NS == 2 ? 2 : 1) void attn_gqa_bf16_kernel(AttnArgs a, Plan p) {
    constexpr int CH = D / 8;              // 16-byte chunks per row
    constexpr int PER = 2 * CH / NW;       // LDS-DMA loads per wave per tile (K and V)
    constexpr int KS = D / 16;             // MFMA k-steps over channels
    constexpr int DB = D / 32;             // 32-channel output blocks
    constexpr int TE = BN * D;             // elements of one K or V tile
    static_assert(2 * CH % NW == 0, "tile loads must split evenly over the waves");
    static_assert(NS >= 2 && NS <= 4, "2..4 stages");

    // K stages, then V stages: same-kind stages sit within 48 KB of each other,
    // so one address register per operand serves every stage through the
    // 16-bit immediate offset of the LDS read.
    __shared__ __attribute__((aligned(16))) uint16_t k0[TE], k1[TE], k2[NS > 2 ? TE : 8], k3[NS > 3 ? TE : 8];
    __shared__ __attribute__((aligned(16))) uint16_t v0[TE], v1[TE], v2[NS > 2 ? TE : 8], v3[NS > 3 ? TE : 8];
    __shared__ int red[NW];
    // Stage selectors; every call site passes a constant after unrolling, so
    // each LDS access names one array and the compiler can tell in-flight
    // LDS-DMA writes to one stage from reads of another.
    auto kst = [&](int st) -> uint16_t* { return st == 0 ? k0 : st == 1 ? k1 : st == 2 ? k2 : k3; };
    auto vst = [&](int st) -> uint16_t* { return st == 0 ? v0 : st == 1 ? v1 : st == 2 ? v2 : v3; };

    int group, rb;
    if (!decode(p, group, rb)) return;
    const int split = group % p.splits;
    int rest = group / p.splits;
    const int kvh = rest % a.n_kv_heads;
    rest /= a.n_kv_heads;
    const int layer = rest % a.n_layers;
    const int seq = rest / a.n_layers;
    const SeqInfo si = seq_info(a, seq);
    const int M = si.nq * p.G;
    const int m0 = rb * (NW * 32 * QB);
    if (m0 >= M) return;

    const int tid = threadIdx.x;
    const int wave = tid >> 6;
    const int lane = tid & 63;
    const int j = lane & 31;
    const int hl = lane >> 5;

    // Rows of this lane (one per 32-row block) and their visible key ranges.
    int qi[QB], head[QB], row_end[QB];
    bool row_ok[QB];
    int rmax = 0, rmin = 0x7fffffff;
#pragma unroll
    for (int qb = 0; qb < QB; ++qb) {
        const int m = m0 + (wave * QB + qb) * 32 + j;
        row_ok[qb] = m < M;
        qi[qb] = row_ok[qb] ? m / p.G : 0;
        head[qb] = kvh * p.G + (row_ok[qb] ? m - qi[qb] * p.G : 0);
        const int qpos = row_ok[qb] ? a.q_pos[si.q0 + qi[qb]] : -1;
        row_end[qb] = row_ok[qb] ? max(0, min(si.kvl, qpos + 1)) : 0;
        rmax = max(rmax, row_end[qb]);
        if (row_ok[qb]) rmin = min(rmin, row_end[qb]);
    }
    const int wmin = wave_min_i(rmin);
    const int wmax = wave_max_i(rmax);
    if (lane == 0) red[wave] = wmax;
    __syncthreads();
    int e_max = 0;
#pragma unroll
    for (int w = 0; w < NW; ++w) e_max = max(e_max, red[w]);

    const int k_begin = split * p.chunk;
    const int loop_end = min(min(si.kvl, k_begin + p.chunk), e_max);
    const int n_tiles = loop_end > k_begin ? (loop_end - k_begin + BN - 1) / BN : 0;

    // Q^T B operands: 8 channels of the row per k-step.
    bf16x8 qf[QB][KS];
#pragma unroll
    for (int qb = 0; qb < QB; ++qb) {
        const uint16_t* qrow = (const uint16_t*)a.q + (int64_t)layer * a.q_stride[0] +
                               (int64_t)(si.q0 + qi[qb]) * a.q_stride[1] + (int64_t)head[qb] * a.q_stride[2];
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) {
            u32x4 v = {0u, 0u, 0u, 0u};
            if (row_ok[qb]) v = *(const u32x4*)(qrow + ks * 16 + hl * 8);
            qf[qb][ks] = __builtin_bit_cast(bf16x8, v);
        }
    }

    const uint16_t* kbase = (const uint16_t*)a.k + (int64_t)layer * a.k_stride[0] +
                            (int64_t)kvh * a.k_stride[1] + si.base * a.k_stride[2];
    const uint16_t* vbase = (const uint16_t*)a.v + (int64_t)layer * a.v_stride[0] +
                            (int64_t)kvh * a.v_stride[1] + si.base * a.v_stride[2];
    const int64_t kss = a.k_stride[2], vss = a.v_stride[2];
    const int last_key = loop_end - 1;

    // Per-lane source offsets (bytes, relative to the tile's first key) of the
    // PER 16-byte chunks this lane moves per tile; lane l of block b fills LDS
    // chunk slot b*64 + l, i.e. key slot/CH, physical chunk slot%CH, which
    // holds logical chunk (phys ^ swz(key)) of that key's row.
    int32_t src_off[PER];
    int key_of[PER];
#pragma unroll
    for (int i = 0; i < PER; ++i) {
        const int q = wave * PER + i;
        const bool isv = q >= CH;
        const int slot = (isv ? q - CH : q) * 64 + lane;
        key_of[i] = slot / CH;
        const int logical = (slot % CH) ^ swz(key_of[i]);
        src_off[i] = (int32_t)((int64_t)key_of[i] * (isv ? vss : kss) * 2 + logical * 16);
    }
    // Stage the tile starting at key t0.  A tile that runs past the last
    // visible key re-reads that key for the missing rows (masked later).
    auto issue = [&](int t0, uint16_t* ks_dst, uint16_t* vs_dst) {
        const bool full = t0 + BN <= loop_end;
        const char* kt = (const char*)(kbase + (int64_t)t0 * kss);
        const char* vt = (const char*)(vbase + (int64_t)t0 * vss);
#pragma unroll
        for (int i = 0; i < PER; ++i) {
            const int q = wave * PER + i;            // wave-uniform
            const bool isv = q >= CH;
            const int blk = isv ? q - CH : q;
            int32_t off = src_off[i];
            if (!full) {
                const int over = t0 + key_of[i] - last_key;
                if (over > 0) off -= over * (int32_t)((isv ? vss : kss) * 2);
            }
            const char* src = (isv ? vt : kt) + off;
            uint16_t* dst = (isv ? vs_dst : ks_dst) + blk * 64 * 8;
            __builtin_amdgcn_global_load_lds((const void*)src, PKV_LDS(void, dst), 16, 0, 0);
        }
    };

    f32x16 o[DB][QB];
#pragma unroll
    for (int db = 0; db < DB; ++db)
#pragma unroll
        for (int qb = 0; qb < QB; ++qb) o[db][qb] = f32x16{};
    float m_run[QB], l_run[QB];
#pragma unroll
    for (int qb = 0; qb < QB; ++qb) {
        m_run[qb] = -INFINITY;
        l_run[qb] = 0.f;
    }
    const float sc2 = a.scale * kLog2e;

    // Raw scores S^T = K Q^T of the tile held in K stage ks_src.
    auto qk = [&](const uint16_t* ks_src, f32x16 (&s)[2][QB]) {
#pragma unroll
        for (int kb = 0; kb < 2; ++kb)
#pragma unroll
            for (int qb = 0; qb < QB; ++qb) s[kb][qb] = f32x16{};
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) {
#pragma unroll
            for (int kb = 0; kb < 2; ++kb) {
                const int key = kb * 32 + j;
                const int phys = (ks * 2 + hl) ^ swz(key);
                const u32x4 kv = *(const u32x4*)(ks_src + key * D + phys * 8);
                const bf16x8 kf = __builtin_bit_cast(bf16x8, kv);
#pragma unroll
                for (int qb = 0; qb < QB; ++qb)
                    s[kb][qb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf, qf[qb][ks], s[kb][qb], 0, 0, 0);
            }
        }
        // Keep the K-operand reads one or two MFMAs ahead instead of all at once.
        sched_reads_mfma<2 * KS, 1, QB>();
    };

    // Softmax, part 1 (branchy, before the overlapped region): mask the raw
    // scores of the tile at key t0 if needed, take each row's maximum and
    // move the reference maximum lazily.  The reference only moves when the
    // scaled tile maximum exceeds it by more than kLazy, so most tiles skip
    // rescaling O; probabilities then stay below 2^kLazy, well inside fp32 and
    // bf16 range, and the final O/l is unchanged.
    constexpr float kLazy = 8.0f;
    auto row_max = [&](int t0, f32x16 (&s)[2][QB], auto mask_tag) {
        constexpr bool MASK = decltype(mask_tag)::value;
#pragma unroll
        for (int qb = 0; qb < QB; ++qb) {
            if (MASK) {
#pragma unroll
                for (int kb = 0; kb < 2; ++kb)
#pragma unroll
                    for (int r = 0; r < 16; ++r) {
                        const int key = t0 + kb * 32 + (r >> 2) * 8 + hl * 4 + (r & 3);
                        if (key >= row_end[qb]) s[kb][qb][r] = sc2 >= 0.f ? -INFINITY : INFINITY;
                    }
            }
            float mx;
            if (sc2 >= 0.f) {
                mx = -INFINITY;
#pragma unroll
                for (int kb = 0; kb < 2; ++kb)
#pragma unroll
                    for (int r = 0; r < 16; ++r) mx = fmaxf(mx, s[kb][qb][r]);
                mx = fmaxf(mx, __shfl_xor(mx, 32));
            } else {
                mx = INFINITY;
#pragma unroll
                for (int kb = 0; kb < 2; ++kb)
#pragma unroll
                    for (int r = 0; r < 16; ++r) mx = fminf(mx, s[kb][qb][r]);
                mx = fminf(mx, __shfl_xor(mx, 32));
            }
            const float msc = mx * sc2;       // this tile's maximum of the scaled scores
            const bool up = msc > m_run[qb] + kLazy;
            if (__builtin_amdgcn_ballot_w64(up) != 0) {
                const float m_new = up ? msc : m_run[qb];
                const float alpha = m_run[qb] == -INFINITY ? 0.f : __builtin_amdgcn_exp2f(m_run[qb] - m_new);
                l_run[qb] *= alpha;
#pragma unroll
                for (int db = 0; db < DB; ++db) o[db][qb] *= alpha;
                m_run[qb] = m_new;
            }
        }
    };

    // Softmax, part 2 (branch-free): probabilities, row sums and the bf16
    // P^T operands.  Masked scores are +-inf here; their probability is
    // forced to 0 (also when the scale is 0).
    auto probs = [&](int t0, f32x16 (&s)[2][QB], bf16x8 (&pb)[QB][4], auto mask_tag) {
        constexpr bool MASK = decltype(mask_tag)::value;
#pragma unroll
        for (int qb = 0; qb < QB; ++qb) {
            const float neg_m = m_run[qb] == -INFINITY ? 0.f : -m_run[qb];
            float lsum = 0.f;
#pragma unroll
            for (int kb = 0; kb < 2; ++kb) {
#pragma unroll
                for (int r = 0; r < 16; ++r) {
                    float e = __builtin_amdgcn_exp2f(fmaf(s[kb][qb][r], sc2, neg_m));
                    if (MASK) {
                        const int key = t0 + kb * 32 + (r >> 2) * 8 + hl * 4 + (r & 3);
                        if (key >= row_end[qb]) e = 0.f;
                    }
                    s[kb][qb][r] = e;
                    lsum += e;
                }
            }
            l_run[qb] += lsum;
#pragma unroll
            for (int st = 0; st < 4; ++st) {
                f32x8 pv;
#pragma unroll
                for (int e = 0; e < 8; ++e) pv[e] = s[st >> 1][qb][(st & 1) * 8 + e];
                pb[qb][st] = __builtin_convertvector(pv, bf16x8);
            }
        }
    };

    // O^T += V^T P^T for the tile held in V stage vs_src.
    auto pv = [&](const uint16_t* vs_src, const bf16x8 (&pb)[QB][4]) {
        // O^T += V^T P^T.  Lane group g (16 lanes) reads channels
        // 32db + 16(g&1) .. +15 for keys {16st + 8b + 4(g>>1) + 0..3}, b = 0, 1.
        const int g = lane >> 4, sl = lane & 15;
        const int hh = g >> 1;
#pragma unroll
        for (int st = 0; st < 4; ++st) {
#pragma unroll
            for (int db = 0; db < DB; ++db) {
                s16x4 part[2];
#pragma unroll
                for (int b = 0; b < 2; ++b) {
                    const int key = st * 16 + b * 8 + hh * 4 + (sl >> 2);
                    const int col = db * 32 + (g & 1) * 16 + (sl & 3) * 4;
                    const int phys = (col >> 3) ^ swz(key);
                    const uint16_t* ptr = vs_src + key * D + phys * 8 + (col & 7);
                    part[b] = __builtin_amdgcn_ds_read_tr16_b64_v4i16(PKV_LDS(s16x4, ptr));
                }
                const s16x4 p0 = part[0], p1 = part[1];
                const bf16x8 vf = __builtin_bit_cast(
                    bf16x8, (short __attribute__((ext_vector_type(8)))){p0[0], p0[1], p0[2], p0[3], p1[0], p1[1],
                                                                          p1[2], p1[3]});
#pragma unroll
                for (int qb = 0; qb < QB; ++qb)
                    o[db][qb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vf, pb[qb][st], o[db][qb], 0, 0, 0);
            }
        }
        sched_reads_mfma<4 * DB, 2, QB>();
    };

    // Software pipeline over key tiles.  Stage i % NS holds tile i; tile i is
    // issued NS-1 iterations ahead.  Iteration i runs QK^T of tile i+1 (MFMA)
    // next to the softmax of tile i (VALU), then PV of tile i, so the two
    // units overlap within a wave.  Tile i's K is read in iteration i-1 and its
    // V in iteration i; the barrier closing iteration i-1 frees its stage for
    // tile i+NS-1 and publishes tile i+1 (waited for by every wave before it).
    static_assert(!PIPE || NS == 4, "the ping-pong schedule uses four LDS stages");
    auto wait_outstanding = [&](int tiles_after) {
        if (NS > 3 && tiles_after >= 3) wait_vmcnt<(NS > 3 ? 3 : 1) * PER>();
        else if (NS > 2 && tiles_after >= 2) wait_vmcnt<(NS > 2 ? 2 : 1) * PER>();
        else if (tiles_after == 1) wait_vmcnt<PER>();
        else wait_vmcnt<0>();
    };
#pragma unroll
    for (int s = 0; s < (PIPE ? 1 : NS - 1); ++s)
        if (s < n_tiles) issue(k_begin + s * BN, kst(s), vst(s));
    if constexpr (!PIPE) {
        // Plain order: tile i is waited for, then QK^T, softmax and PV run back
        // to back.  The barrier that publishes tile i also proves every wave
        // finished tile i-1, so tile i-1's stage is refilled right after it.
        for (int t = 0; t < n_tiles; t += NS) {
#pragma unroll
            for (int s = 0; s < NS; ++s) {
                const int i = t + s;
                if (i < n_tiles) {
                    wait_outstanding(min(i + NS - 2, n_tiles - 1) - i);
                    __builtin_amdgcn_s_waitcnt(15 | (7 << 4) | (0 << 8) | (3 << 14));
                    bare_barrier();
                    const int ahead = i + NS - 1;
                    if (ahead < n_tiles)
                        issue(k_begin + ahead * BN, kst((s + NS - 1) % NS), vst((s + NS - 1) % NS));
                    f32x16 sc[2][QB];
                    qk(kst(s), sc);
                    bf16x8 pb[QB][4];
                    const int t0 = k_begin + i * BN;
                    if (t0 + BN > wmin) {
                        row_max(t0, sc, std::true_type{});
                        probs(t0, sc, pb, std::true_type{});
                    } else {
                        row_max(t0, sc, std::false_type{});
                        probs(t0, sc, pb, std::false_type{});
                    }
                    pv(vst(s), pb);
                }
            }
        }
    } else {
        // Ping-pong schedule.  The 8 waves form two groups of 4 (waves w and
        // w+4 share a SIMD); group 1 runs one half-step behind group 0.  A wave
        // alternates an MFMA phase (PV of its previous tile, then QK^T of its
        // next tile) with a VALU phase (softmax of that tile), so at every
        // half-step each SIMD holds one wave in each phase and the matrix core
        // and the VALU work at the same time.  Tile t is read in half-steps
        // 2t .. 2t+3; it is issued at half-step 2t-4 into the stage that tile
        // t-4 left, and every wave waits for it before the barrier that opens
        // half-step 2t.
        static_assert(NW == 8, "two groups of four waves");
        const int gp = wave >> 2;
        f32x16 sc[2][QB];
        bf16x8 pb[QB][4];
        auto mfma_phase = [&](int t, const uint16_t* vs_prev, const uint16_t* ks_cur) {
            if (t >= 1 && t - 1 < n_tiles) pv(vs_prev, pb);
            if (t < n_tiles) qk(ks_cur, sc);
        };
        auto valu_phase = [&](int t) {
            if (t < 0 || t >= n_tiles) return;
            const int t0 = k_begin + t * BN;
            if (t0 + BN > wmin) {
                row_max(t0, sc, std::true_type{});
                probs(t0, sc, pb, std::true_type{});
            } else {
                row_max(t0, sc, std::false_type{});
                probs(t0, sc, pb, std::false_type{});
            }
        };
        if (n_tiles > 1) issue(k_begin + BN, kst(1), vst(1));   // tile 0 went out above
        if (n_tiles > 0) {
            wait_outstanding(n_tiles > 1 ? 1 : 0);
            bare_barrier();
        }
        const int H = 2 * n_tiles + 2;
        for (int h0 = 0; h0 < H; h0 += 8) {
#pragma unroll
            for (int e = 0; e < 8; ++e) {
                const int h = h0 + e;
                if (h < H) {
                    const int m = h >> 1;
                    const int sm = e >> 1;   // == m % 4
                    if ((e & 1) == 0) {
                        if (m + 2 < n_tiles) issue(k_begin + (m + 2) * BN, kst((sm + 2) % 4), vst((sm + 2) % 4));
                        if (gp == 0) mfma_phase(m, vst((sm + 3) % 4), kst(sm));
                        else valu_phase(m - 1);
                    } else {
                        if (gp == 0) valu_phase(m);
                        else mfma_phase(m, vst((sm + 3) % 4), kst(sm));
                        if (m + 1 < n_tiles) wait_outstanding(min(m + 2, n_tiles - 1) - (m + 1));
                    }
                    __builtin_amdgcn_s_waitcnt(15 | (7 << 4) | (0 << 8) | (3 << 14));
                    bare_barrier();
                }
            }
        }
    }

    // Finish each row: the two lanes of a column hold disjoint partial sums.
#pragma unroll
    for (int qb = 0; qb < QB; ++qb) {
        const float l_tot = l_run[qb] + __shfl_xor(l_run[qb], 32);
        if (!row_ok[qb]) continue;
        const float inv = l_tot > 0.f ? 1.f / l_tot : 0.f;
        const float lse2 = l_tot > 0.f ? m_run[qb] + __log2f(l_tot) : -INFINITY;
        const int64_t row = si.q0 + qi[qb];
        if (p.splits == 1) {
            uint16_t* orow = (uint16_t*)a.out + (int64_t)layer * a.o_stride[0] + row * a.o_stride[1] +
                             (int64_t)head[qb] * a.o_stride[2];
#pragma unroll
            for (int db = 0; db < DB; ++db) {
#pragma unroll
                for (int b = 0; b < 4; ++b) {
                    u32x2 w;
                    w[0] = bf_rne(o[db][qb][4 * b] * inv) | (bf_rne(o[db][qb][4 * b + 1] * inv) << 16);
                    w[1] = bf_rne(o[db][qb][4 * b + 2] * inv) | (bf_rne(o[db][qb][4 * b + 3] * inv) << 16);
                    *(u32x2*)(orow + db * 32 + b * 8 + hl * 4) = w;
                }
            }
            if (a.lse_out && hl == 0)
                a.lse_out[((int64_t)layer * a.total_q + row) * a.n_heads + head[qb]] = lse2 * kLn2;
        } else {
            const int64_t item =
                (((int64_t)split * a.n_layers + layer) * a.total_q + row) * a.n_heads + head[qb];
            float* wo = a.ws_o + item * D;
#pragma unroll
            for (int db = 0; db < DB; ++db) {
#pragma unroll
                for (int b = 0; b < 4; ++b) {
                    f32x4 w = {o[db][qb][4 * b] * inv, o[db][qb][4 * b + 1] * inv, o[db][qb][4 * b + 2] * inv,
                               o[db][qb][4 * b + 3] * inv};
                    *(f32x4*)(wo + db * 32 + b * 8 + hl * 4) = w;
                }
            }
            if (hl == 0) a.ws_lse[item] = lse2;
        }
    }
}

template <int D, int QB, int NW>
hipError_t launch_shape(const AttnArgs& a, const Plan& p, dim3 grid, hipStream_t stream) {
    if constexpr (NW == 8) {   // two wave groups per SIMD: ping-pong schedule
        hipLaunchKernelGGL((attn_gqa_bf16_kernel<D, QB, NW, 4, PKV_ATTN_PINGPONG != 0>), grid, dim3(NW * 64), 0,
                           stream, a, p);
    } else if (p.ns == 2) {    // two independent workgroups per CU
        hipLaunchKernelGGL((attn_gqa_bf16_kernel<D, QB, NW, 2, false>), grid, dim3(NW * 64), 0, stream, a, p);
    } else {
        hipLaunchKernelGGL((attn_gqa_bf16_kernel<D, QB, NW, 3, false>), grid, dim3(NW * 64), 0, stream, a, p);
    }
    return hipGetLastError();
}

template <int D>
hipError_t launch_d(const AttnArgs& a, const Plan& p, dim3 grid, hipStream_t stream) {
    if (p.nw == 8) return launch_shape<D, 1, 8>(a, p, grid, stream);
    return launch_shape<D, 1, 4>(a, p, grid, stream);
}

}  // namespace

hipError_t launch_attn_gqa_bf16(const AttnArgs& a, const Plan& p, dim3 grid, hipStream_t stream) {
    if (a.head_dim == 64) return launch_d<64>(a, p, grid, stream);
    return launch_d<128>(a, p, grid, stream);
}

}  // namespace pkv
