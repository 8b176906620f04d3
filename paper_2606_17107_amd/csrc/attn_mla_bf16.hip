// bf16 MLA suffix attention (absorbed form) for gfx950.
//
// The MLA cache keeps, per token, one latent row [c_kv (512) | k_pe (64)]
// shared by every head (paper Sec. 8, MLA adapter: a position-free latent
// plus a small decoupled-RoPE sub-vector).  With absorbed queries
// q = [q_latent (512) | q_pe (64)] per head, the scores run over all 576
// channels and the values are the 512 latent channels of the same row:
//     o_h = sum_j softmax_j(scale <q_h, row_j>) row_j[0:512]
//
// Work decomposition (one KV "head", so every query head is a row):
//   * MFMA 32x32x16 bf16 -> fp32; row m <-> query m / H, head m % H.  Two
//     waves share each block of 32 rows.  Each forms the partial scores over
//     one half of the 576 channels (its Q^T half, 72 VGPRs, in registers),
//     the two partials are exchanged through LDS and added (fp32), both waves
//     run the same online softmax, and each accumulates one 256-channel half
//     of O^T (128 values per lane).
//   * S^T = K Q^T (36 k-steps), online softmax in-lane as in the GQA kernel,
//     O^T += V^T P^T where V^T comes from the same LDS tile through
//     ds_read_b64_tr_b16 (channels 0..511).
//   * Tiles of 32 keys (36 KB) stream HBM -> LDS by LDS-DMA through NS
//     stages; chunks XOR-swizzled by the key as in the GQA kernel.
//   * Four waves (two pairs, 64 rows) per workgroup and two LDS stages
//     (eight waves, two per SIMD, and three stages were measured no faster).
//   * One wave per SIMD, so every stall is exposed: the operand reads of each
//     MFMA chain are issued in fenced groups a fixed distance ahead (the
//     compiler's own order left each MFMA waiting on its read), the second
//     half of the probabilities is formed between the PV MFMAs that consume
//     the first, and the row maximum crosses the two wave halves with a
//     permlane swap.  The 128 output accumulators live in VGPRs (a per-file
//     compiler option): left in AGPRs, every tile copied them out and back
//     for the rarely taken rescale.
//   * Rows wholly owned by one wave (all 576 score and 512 value channels, no
//     exchange) would need 144 + 256 registers for Q^T and O and do not fit.
#include <type_traits>

#include "attn_common.h"

namespace pkv {
namespace {

constexpr int kMlaWaves = 4;    // two wave pairs, 64 rows
constexpr int kMlaStages = 2;   // LDS stages of 32-key tiles
constexpr int kMlaAhead = 2;    // LDS operand reads issued this many operands ahead of their MFMA

constexpr int MBN = 32;        // keys per tile
constexpr int DQK = 576;       // score channels
constexpr int DV = 512;        // value (latent) channels
constexpr int MCH = DQK / 8;   // 16-byte chunks per row: 72

// XOR swizzle of the low three bits of a row's 16-byte chunk index by its key.
// A row is 72 chunks, so consecutive keys start in alternate halves of the 16
// bank groups (16 bytes each).  K operand reads take one chunk from each of 16
// consecutive keys: for either key parity the swizzle is a bijection of
// (key >> 1) & 7, so the 16 reads hit 16 groups.  Transposed V reads take a
// 4-chunk aligned window from each of 4 consecutive keys: keys 4q and 4q+2
// (and 4q+1, 4q+3) differ in bit 2 of the swizzle, which moves the window to
// the other half of its 8-chunk group.
__device__ inline int mswz(int key) { return (((key >> 1) & 1) << 2) | ((key >> 2) & 3); }

template <bool PAGED>
__global__ __launch_bounds__(kMlaWaves * 64, 1) void attn_mla_bf16_kernel(AttnArgs a, Plan p) {
    constexpr int NS = kMlaStages, NW = kMlaWaves;
    constexpr int NBLK = MBN * MCH / 64;       // 64-lane LDS-DMA blocks per tile: 36
    constexpr int PER = (NBLK + NW - 1) / NW;  // blocks of the busiest wave per tile
    constexpr int KS = DQK / 16 / 2;           // k-steps per wave (its half of the channels): 18
    constexpr int DB = DV / 64;                // 32-channel blocks per wave (its half of DV): 8
    constexpr int RPW = NW / 2 * 32;           // rows per workgroup
    constexpr int TE = MBN * DQK;              // elements per tile
    static_assert(NW % 2 == 0, "pairs of waves share 32 rows");
    static_assert(NS == 2, "two LDS stages");

    __shared__ __attribute__((aligned(16))) uint16_t t0_[TE], t1_[TE];
    __shared__ int red[NW], red_start[NW];
    // Partial-score exchange: [wave][4 chunks][64 lanes] x 16 bytes.
    __shared__ __attribute__((aligned(16))) float xch[NW * 4 * 64 * 4];
    auto stage = [&](int st) -> uint16_t* { return st == 0 ? t0_ : t1_; };

    int group, rb;
    if (!decode(p, group, rb)) return;
    const int split = group % p.splits;
    int rest = group / p.splits;   // one KV head
    const int layer = rest % a.n_layers;
    const int seq = rest / a.n_layers;
    const SeqInfo si = seq_info(a, seq);
    const int H = a.n_heads;
    const int M = si.nq * H;
    const int m0 = rb * RPW;
    const int vhalf = (threadIdx.x >> 6) & 1;   // which 256-channel half of O this wave owns
    if (m0 >= M) return;

    const int tid = threadIdx.x;
    const int wave = tid >> 6;
    const int lane = tid & 63;
    const int j = lane & 31;
    const int hl = lane >> 5;

    const int m = m0 + (wave >> 1) * 32 + j;
    const bool row_ok = m < M;
    const int qi = row_ok ? m / H : 0;
    const int head = row_ok ? m - qi * H : 0;
    // Q^T operands first: they do not depend on the positions, so their
    // latency overlaps the key-range set-up.
    bf16x8 qf[KS];
    {
        const uint16_t* qrow = (const uint16_t*)a.q + (int64_t)layer * a.q_stride[0] +
                               (int64_t)(si.q0 + qi) * a.q_stride[1] + (int64_t)head * a.q_stride[2];
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) {
            u32x4 v = {0u, 0u, 0u, 0u};
            if (row_ok) v = *(const u32x4*)(qrow + (vhalf * KS + ks) * 16 + hl * 8);
            qf[ks] = __builtin_bit_cast(bf16x8, v);
        }
    }

    const int qpos = row_ok ? a.q_pos[si.q0 + qi] : -1;
    // Visible keys [row_start, row_end): causal, and with a sliding window
    // also row_start = q_pos - window + 1.
    const int row_end = row_ok ? max(0, min(si.kvl, qpos + 1)) : 0;
    const int row_start = a.window > 0 && row_ok ? max(0, qpos - a.window + 1) : 0;
    const int wmin = wave_min_i(row_ok ? row_end : 0x7fffffff);
    const int wmax = wave_max_i(row_end);
    const int wsmin = wave_min_i(row_ok ? row_start : 0x7fffffff);
    const int wsmax = wave_max_i(row_start);   // tiles below this need the window mask
    if (lane == 0) {
        red[wave] = wmax;
        red_start[wave] = wsmin;
    }
    __syncthreads();
    int e_max = 0, s_min = 0x7fffffff;
#pragma unroll
    for (int w = 0; w < NW; ++w) {
        e_max = max(e_max, red[w]);
        s_min = min(s_min, red_start[w]);
    }
    // Tiles wholly before every row's window start are skipped.
    const int split_begin = split * p.chunk;
    const int k_begin = max(split_begin, s_min == 0x7fffffff ? 0 : s_min / MBN * MBN);
    const int loop_end = min(min(si.kvl, split_begin + p.chunk), e_max);
    const int n_tiles = loop_end > k_begin ? (loop_end - k_begin + MBN - 1) / MBN : 0;

    const uint16_t* kbase = (const uint16_t*)a.k + (int64_t)layer * a.k_stride[0] + si.base * a.k_stride[2];
    const int64_t kss = a.k_stride[2];
    const int last_key = loop_end - 1;
    // Wave w moves blocks w, w + NW, ... of each tile (NBLK / NW or one more):
    // lane l of block b fills LDS chunk slot 64b + l (key slot / 72, physical
    // chunk slot % 72, holding logical chunk phys ^ mswz(key)).
    const int n_mine = (NBLK - wave + NW - 1) / NW;   // wave-uniform
    int32_t src_off[PER];
    int key_of[PER];
#pragma unroll
    for (int i = 0; i < PER; ++i) {
        const int b = i < n_mine ? wave + i * NW : wave;   // idle slots mirror block `wave` (never issued)
        const int slot = b * 64 + lane;
        key_of[i] = slot / MCH;
        const int logical = (slot % MCH) ^ mswz(key_of[i]);
        src_off[i] = (int32_t)((int64_t)key_of[i] * kss * 2 + logical * 16);
    }
    // Paged cache: a 32-key tile lies in one page (page sizes are multiples of 32).
    PageWindow pw;
    if constexpr (PAGED) pw.init(a.block_table, a, seq, k_begin >> a.page_shift);
    auto issue = [&](int t0, uint16_t* dst_stage) {
        const char* kt;
        if constexpr (PAGED)
            kt = (const char*)(kbase + pw.offset(a, t0, a.k_page_stride, kss));
        else
            kt = (const char*)(kbase + (int64_t)t0 * kss);
        const uint32_t lds0 = lds_addr_of(dst_stage + wave * 64 * 8);
        if (t0 + MBN <= loop_end) {   // full tile: no per-lane adjustment
#pragma unroll
            for (int i = 0; i < PER; ++i)
                if (i < n_mine) lds_dma16(lds0 + i * NW * 1024, kt, (uint32_t)src_off[i]);
        } else {
#pragma unroll
            for (int i = 0; i < PER; ++i) {
                if (i < n_mine) {
                    const int over = t0 + key_of[i] - last_key;
                    const uint32_t back = over > 0 ? (uint32_t)(over * (int32_t)(kss * 2)) : 0u;
                    lds_dma16(lds0 + i * NW * 1024, kt, (uint32_t)src_off[i] - back);
                }
            }
        }
    };

    // Per-lane LDS element offsets of the MFMA operands within a stage.  The
    // swizzle only permutes the low three bits of a chunk index, so:
    //   K (A of S^T = K Q^T), k-step ks: logical chunk c0 + 2ks of key j
    //     (c0 = 36 vhalf + hl) sits at kofs[ks & 3] + (ks >> 2) * 64;
    //   V^T (A of O^T = V^T P^T), 16-key step st, half b, channel block db:
    //     lane group g = lane >> 4 reads channels 256 vhalf + 32db + 16(g&1) +
    //     4(sl&3)..+3 of key 16st + 8b + 4(g>>1) + (sl>>2), sl = lane & 15 (the
    //     key order of the P^T accumulator); the swizzle of that key depends
    //     only on its low four bits, so the read is at
    //     vofs[db & 1][b] + 16st * 576 + (db >> 1) * 64.
    int kofs[4], vofs[2][2];
    {
        const int sk = mswz(j);
        const int c0 = vhalf * KS * 2 + hl;
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            const int c = c0 + 2 * q;
            kofs[q] = j * DQK + ((c & ~7) | ((c & 7) ^ sk)) * 8;
        }
        const int g = lane >> 4, sl = lane & 15;
        const int vkey = (g >> 1) * 4 + (sl >> 2);
#pragma unroll
        for (int par = 0; par < 2; ++par)
#pragma unroll
            for (int b = 0; b < 2; ++b) {
                const int key = b * 8 + vkey;
                const int c7 = par * 4 + (g & 1) * 2 + ((sl & 3) >> 1);
                vofs[par][b] = key * DQK + (vhalf * 32 + (c7 ^ mswz(key))) * 8 + (sl & 1) * 4;
            }
    }

    f32x16 o[DB];
#pragma unroll
    for (int db = 0; db < DB; ++db) o[db] = f32x16{};
    float m_run = -INFINITY, l_run = 0.f;
    const float sc2 = a.scale * kLog2e;
    constexpr float kLazy = 8.0f;

    auto compute = [&](int t0, const uint16_t* ts, auto mask_tag) {
        constexpr bool MASK = decltype(mask_tag)::value;
        // Partial S^T = K Q^T over this wave's 288 channels, 32 keys (one
        // accumulation chain: dependent MFMAs on the same accumulator issue
        // back to back).
        // Fenced groups: MFMA ks, then the read of the operand A steps ahead,
        // so A LDS round trips stay in flight across the chain.
        constexpr int A = kMlaAhead < KS ? kMlaAhead : KS;
        auto k_operand = [&](int ks) __attribute__((always_inline)) {
            return __builtin_bit_cast(bf16x8, *(const u32x4*)(ts + kofs[ks & 3] + (ks >> 2) * 64));
        };
        bf16x8 kop[KS];
#pragma unroll
        for (int ks = 0; ks < A; ++ks) kop[ks] = k_operand(ks);
        __builtin_amdgcn_sched_barrier(0);
        f32x16 s = f32x16{};
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) {
            s = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kop[ks], qf[ks], s, 0, 0, 0);
            if (ks + A < KS) kop[ks + A] = k_operand(ks + A);
            __builtin_amdgcn_sched_barrier(0);
        }
        // Exchange the partial scores with the other wave of the pair (the
        // lanes of both waves hold the same (key, row) elements).
        float* mine = xch + wave * 1024;
        const float* other = xch + (wave ^ 1) * 1024;
#pragma unroll
        for (int c = 0; c < 4; ++c)
            *(f32x4*)(mine + (c * 64 + lane) * 4) = f32x4{s[4 * c], s[4 * c + 1], s[4 * c + 2], s[4 * c + 3]};
        __builtin_amdgcn_s_waitcnt(15 | (7 << 4) | (0 << 8) | (3 << 14));
        bare_barrier();
#pragma unroll
        for (int c = 0; c < 4; ++c) {
            const f32x4 x = *(const f32x4*)(other + (c * 64 + lane) * 4);
            s[4 * c] += x[0];
            s[4 * c + 1] += x[1];
            s[4 * c + 2] += x[2];
            s[4 * c + 3] += x[3];
        }
        if (MASK) {
#pragma unroll
            for (int r = 0; r < 16; ++r) {
                const int kk = t0 + (r >> 2) * 8 + hl * 4 + (r & 3);
                if (kk >= row_end || kk < row_start) s[r] = sc2 >= 0.f ? -INFINITY : INFINITY;
            }
        }
        float mx;
        if (sc2 >= 0.f) {
            mx = -INFINITY;
#pragma unroll
            for (int r = 0; r < 16; ++r) mx = fmaxf(mx, s[r]);
            // lanes l and l + 32 hold the two 16-key halves of a row; a
            // permlane swap pairs them without a trip through LDS
            const auto sw = __builtin_amdgcn_permlane32_swap(__float_as_uint(mx), __float_as_uint(mx), false, false);
            mx = fmaxf(__uint_as_float(sw[0]), __uint_as_float(sw[1]));
        } else {
            mx = INFINITY;
#pragma unroll
            for (int r = 0; r < 16; ++r) mx = fminf(mx, s[r]);
            const auto sw = __builtin_amdgcn_permlane32_swap(__float_as_uint(mx), __float_as_uint(mx), false, false);
            mx = fminf(__uint_as_float(sw[0]), __uint_as_float(sw[1]));
        }
        const float msc = mx * sc2;
        const bool up = msc > m_run + kLazy;
        if (__builtin_amdgcn_ballot_w64(up) != 0) {
            const float m_new = up ? msc : m_run;
            const float alpha = m_run == -INFINITY ? 0.f : __builtin_amdgcn_exp2f(m_run - m_new);
            l_run *= alpha;
#pragma unroll
            for (int db = 0; db < DB; ++db) o[db] *= alpha;
            m_run = m_new;
        }
        const float neg_m = m_run == -INFINITY ? 0.f : -m_run;
        float lsum = 0.f;
        auto prob = [&](int r) __attribute__((always_inline)) {
            float e = __builtin_amdgcn_exp2f(fmaf(s[r], sc2, neg_m));
            if (MASK) {
                const int kk = t0 + (r >> 2) * 8 + hl * 4 + (r & 3);
                if (kk >= row_end || kk < row_start) e = 0.f;
            }
            s[r] = e;
            lsum += e;
        };
        auto pack = [&](int st) __attribute__((always_inline)) {
            f32x8 pv;
#pragma unroll
            for (int e = 0; e < 8; ++e) pv[e] = s[st * 8 + e];
            return __builtin_convertvector(pv, bf16x8);
        };
        // Probabilities of the first 16 keys now; those of the second 16 are
        // formed between the MFMAs that consume the first (one per MFMA).
        bf16x8 pb[2];
#pragma unroll
        for (int r = 0; r < 8; ++r) prob(r);
        pb[0] = pack(0);
        // O^T += V^T P^T: V is channels 0..511 of the same tile; operand
        // q = (16-key step q / DB, channel block q % DB), read A steps ahead.
        constexpr int NQ = 2 * DB;
        constexpr int AV = kMlaAhead < NQ ? kMlaAhead : NQ;
        static_assert(DB == 8, "one second-half probability per first-half MFMA");
        auto v_operand = [&](int q) __attribute__((always_inline)) {
            const int st = q / DB, db = q % DB;
            s16x4 part[2];
#pragma unroll
            for (int b = 0; b < 2; ++b)
                part[b] = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
                    PKV_LDS(s16x4, ts + vofs[db & 1][b] + st * 16 * DQK + (db >> 1) * 64));
            const s16x4 p0 = part[0], p1 = part[1];
            return __builtin_bit_cast(bf16x8, (short __attribute__((ext_vector_type(8)))){
                                                  p0[0], p0[1], p0[2], p0[3], p1[0], p1[1], p1[2], p1[3]});
        };
        bf16x8 vop[NQ];
#pragma unroll
        for (int q = 0; q < AV; ++q) vop[q] = v_operand(q);
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int q = 0; q < NQ; ++q) {
            o[q % DB] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vop[q], pb[q / DB], o[q % DB], 0, 0, 0);
            if (q < 8) prob(8 + q);
            if (q == 7) pb[1] = pack(1);
            if (q + AV < NQ) vop[q + AV] = v_operand(q + AV);
            __builtin_amdgcn_sched_barrier(0);
        }
        l_run += lsum;
    };

    // Each wave waits for its own loads: n_mine per tile (PER or PER - 1).
    auto wait_tiles = [&](int tiles_after, auto per_tag) {
        constexpr int Q = decltype(per_tag)::value;
        if (NS > 3 && tiles_after >= 3) wait_vmcnt<(NS > 3 ? 3 : 1) * Q>();
        else if (NS > 2 && tiles_after >= 2) wait_vmcnt<(NS > 2 ? 2 : 1) * Q>();
        else if (tiles_after == 1) wait_vmcnt<Q>();
        else wait_vmcnt<0>();
    };
    auto wait_outstanding = [&](int tiles_after) {
        if (n_mine == PER) wait_tiles(tiles_after, std::integral_constant<int, PER>{});
        else wait_tiles(tiles_after, std::integral_constant<int, (PER > 1 ? PER - 1 : 1)>{});
    };
#pragma unroll
    for (int s = 0; s < NS - 1; ++s)
        if (s < n_tiles) issue(k_begin + s * MBN, stage(s));   // tiles 0 .. NS-2
    // Stage i % NS holds tile i.  Each iteration waits for tile i, then (after
    // the barrier, when every wave has finished tile i-1) refills tile i-1's
    // stage with tile i+NS-1.
    for (int t = 0; t < n_tiles; t += NS) {
#pragma unroll
        for (int s = 0; s < NS; ++s) {
            const int i = t + s;
            if (i < n_tiles) {
                const int issued = min(i + NS - 2, n_tiles - 1);   // last tile already in flight
                wait_outstanding(issued - i);
                __builtin_amdgcn_s_waitcnt(15 | (7 << 4) | (0 << 8) | (3 << 14));
                bare_barrier();
                const int ahead = i + NS - 1;
                if (ahead < n_tiles) issue(k_begin + ahead * MBN, stage((s + NS - 1) % NS));
                const int t0 = k_begin + i * MBN;
                if (t0 + MBN > wmin || t0 < wsmax)
                    compute(t0, stage(s), std::true_type{});
                else
                    compute(t0, stage(s), std::false_type{});
            }
        }
    }

    const float l_tot = l_run + __shfl_xor(l_run, 32);
    if (!row_ok) return;
    const float inv = l_tot > 0.f ? 1.f / l_tot : 0.f;
    const float lse2 = l_tot > 0.f ? m_run + __log2f(l_tot) : -INFINITY;
    const int64_t row = si.q0 + qi;
    if (p.splits == 1) {
        uint16_t* orow = (uint16_t*)a.out + (int64_t)layer * a.o_stride[0] + row * a.o_stride[1] +
                         (int64_t)head * a.o_stride[2];
#pragma unroll
        for (int db = 0; db < DB; ++db) {
#pragma unroll
            for (int b = 0; b < 4; ++b) {
                u32x2 w;
                w[0] = bf_rne(o[db][4 * b] * inv) | (bf_rne(o[db][4 * b + 1] * inv) << 16);
                w[1] = bf_rne(o[db][4 * b + 2] * inv) | (bf_rne(o[db][4 * b + 3] * inv) << 16);
                *(u32x2*)(orow + vhalf * 256 + db * 32 + b * 8 + hl * 4) = w;
            }
        }
        if (a.lse_out && hl == 0 && vhalf == 0) a.lse_out[((int64_t)layer * a.total_q + row) * H + head] = lse2 * kLn2;
    } else {
        const int64_t item = (((int64_t)split * a.n_layers + layer) * a.total_q + row) * H + head;
        float* wo = a.ws_o + item * DV;
#pragma unroll
        for (int db = 0; db < DB; ++db) {
#pragma unroll
            for (int b = 0; b < 4; ++b) {
                f32x4 w = {o[db][4 * b] * inv, o[db][4 * b + 1] * inv, o[db][4 * b + 2] * inv,
                           o[db][4 * b + 3] * inv};
                *(f32x4*)(wo + vhalf * 256 + db * 32 + b * 8 + hl * 4) = w;
            }
        }
        if (hl == 0 && vhalf == 0) a.ws_lse[item] = lse2;
    }
}

}  // namespace

hipError_t launch_attn_mla_bf16(const AttnArgs& a, const Plan& p, dim3 grid, hipStream_t stream) {
    if (p.nw != kMlaWaves || p.ns != kMlaStages || p.BM != kMlaWaves / 2 * 32) return hipErrorInvalidValue;
    if (a.block_table)
        hipLaunchKernelGGL((attn_mla_bf16_kernel<true>), grid, dim3(kMlaWaves * 64), 0, stream, a, p);
    else
        hipLaunchKernelGGL((attn_mla_bf16_kernel<false>), grid, dim3(kMlaWaves * 64), 0, stream, a, p);
    return hipGetLastError();
}

}  // namespace pkv
