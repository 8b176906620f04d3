// bf16 MLA suffix attention (absorbed form) for gfx950.
//
// The MLA cache keeps, per token, one latent row [c_kv (512) | k_pe (64)]
// shared by every head (paper Sec. 8, MLA adapter: no rotation is applied to
// c_kv; only the 64 k_pe channels are rotated by position).  With absorbed
// queries q = [q_latent (512) | q_pe (64)] per head, the scores run over all
// 576 channels and the values are the 512 latent channels of the same row:
//     o_h = sum_j softmax_j(scale <q_h, row_j>) row_j[0:512]
//
// Work decomposition (one KV "head", so every query head is a row):
//   * MFMA 32x32x16 bf16 -> fp32; row m <-> query m / H, head m % H.  Each
//     wave owns 32 rows outright: their Q^T over all 576 channels (36 k-step
//     operands, 144 VGPRs) and their O^T over all 512 value channels (16
//     blocks, 256 accumulators in the AGPR file).  Four waves share every K/V
//     tile in LDS, so one workgroup covers 128 rows and a tile byte serves all
//     of them.
//   * S^T = K Q^T (36 MFMAs, one accumulation chain), online softmax in-lane
//     (a lane holds 16 keys of one row; the two halves of a row pair up with
//     a permlane swap), O^T += V^T P^T (32 MFMAs) where V^T comes from the
//     same LDS tile through ds_read_b64_tr_b16 (channels 0..511).  Every MFMA
//     reads one 1 KB operand from LDS; the LDS-DMA fill adds 36 KB per tile
//     for the workgroup, about 1.13 KB of LDS traffic per MFMA in all.
//   * Tiles of 32 keys (36 KB) stream HBM -> LDS by LDS-DMA through 2 stages
//     (one tile in flight while one is consumed); 16-byte chunks are
//     XOR-swizzled by key against bank conflicts.
//   * One wave per SIMD: the 256 output accumulators fill the AGPR file and
//     Q^T with the working set fills the VGPRs.  The compiler chooses one
//     register file for all MFMA accumulators of a function, so the score
//     MFMAs are builtins accumulating in VGPRs (a per-file compiler option)
//     and the PV MFMAs are inline assembly accumulating in AGPRs ("+a"
//     operands); nothing else touches the accumulators until the epilogue,
//     which first waits out the MFMA write latency.  The wave hides its own
//     latencies: the LDS operand reads of each MFMA chain are issued in fenced
//     groups a fixed distance ahead, and the second half of the
//     probabilities is formed between the PV MFMAs that consume the first.
//   * The accumulators are never rescaled.  Each row's reference maximum is
//     the maximum of its first tile with a visible key; later probabilities
//     2^(s - ref) may exceed 1, which costs no relative precision in fp32 and
//     bf16, up to 2^32.  A tile whose maximum exceeds the reference by more
//     than that (a score spike far above everything before it) marks the
//     workgroup, which then runs its key range a second time with every
//     row's exact maximum, known from the first pass, as the reference.
#include <type_traits>

#include "attn_common.h"

namespace pkv {
namespace {

constexpr int kMlaWaves = 4;    // 32 rows per wave, 128 per workgroup
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
    constexpr int PER = NBLK / NW;             // blocks per wave per tile: 9
    constexpr int KS = DQK / 16;               // k-steps over the score channels: 36
    constexpr int DB = DV / 32;                // 32-channel output blocks: 16
    constexpr int RPW = NW * 32;               // rows per workgroup
    constexpr int TE = MBN * DQK;              // elements per tile
    static_assert(NBLK % NW == 0, "tile loads must split evenly over the waves");
    static_assert(NS >= 2 && NS <= 4 && (NS - 2) * PER < 64, "2..4 stages within the vmcnt range");

    __shared__ __attribute__((aligned(16))) uint16_t stage_lds[NS * TE];
    __shared__ int red[NW], red_start[NW];
    auto stage = [&](int st) __attribute__((always_inline)) -> uint16_t* { return stage_lds + st * TE; };

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
    if (m0 >= M) return;

    const int tid = threadIdx.x;
    const int wave = tid >> 6;
    const int lane = tid & 63;
    const int j = lane & 31;
    const int hl = lane >> 5;

    const int m = m0 + wave * 32 + j;
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
            if (row_ok) v = *(const u32x4*)(qrow + ks * 16 + hl * 8);
            qf[ks] = __builtin_bit_cast(bf16x8, v);
        }
    }

    const int qpos = row_ok ? a.q_pos[si.q0 + qi] : -1;
    // Visible keys [row_start, row_end): causal, and with a sliding window
    // also row_start = q_pos - window + 1.
    int row_start, row_end;
    visible_range(qpos, si.kvl, a.window, row_start, row_end);   // (0, 0) for rows past M
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
    // Keys [lo, hi) hold every key a row of the workgroup sees (whole tiles
    // from the first window start); the splits share them in equal runs of
    // whole tiles.
    const int lo = s_min == 0x7fffffff ? 0 : s_min / MBN * MBN;
    const int hi = min(si.kvl, e_max);
    const int run = hi > lo ? ((hi - lo + p.splits - 1) / p.splits + MBN - 1) / MBN * MBN : 0;
    const int k_begin = lo + split * run;
    const int loop_end = min(hi, k_begin + run);
    const int n_tiles = loop_end > k_begin ? (loop_end - k_begin + MBN - 1) / MBN : 0;

    const uint16_t* kbase = (const uint16_t*)a.k + (int64_t)layer * a.k_stride[0] + si.base * a.k_stride[2];
    const int64_t kss = a.k_stride[2];
    const int last_key = loop_end - 1;
    // Wave w moves blocks w, w + NW, ... of each tile: lane l of block b fills
    // LDS chunk slot 64b + l (key slot / 72, physical chunk slot % 72, holding
    // logical chunk phys ^ mswz(key)).
    int32_t src_off[PER];
    int key_of[PER];
#pragma unroll
    for (int i = 0; i < PER; ++i) {
        const int slot = (wave + i * NW) * 64 + lane;
        key_of[i] = slot / MCH;
        const int logical = (slot % MCH) ^ mswz(key_of[i]);
        src_off[i] = (int32_t)((int64_t)key_of[i] * kss * 2 + logical * 16);
    }
    // Paged cache: a 32-key tile lies in one page (page sizes are multiples of 32).
    PageWindow pw;
    if constexpr (PAGED) pw.init(a.block_table, a, seq, k_begin >> a.page_shift);
    auto issue = [&](int t0, uint16_t* dst_stage) __attribute__((always_inline)) {
        const char* kt;
        if constexpr (PAGED)
            kt = (const char*)(kbase + pw.offset(a, t0, a.k_page_stride, kss));
        else
            kt = (const char*)(kbase + (int64_t)t0 * kss);
        const uint32_t lds0 = lds_addr_of(dst_stage + wave * 64 * 8);
        if (t0 + MBN <= loop_end) {   // full tile: no per-lane adjustment
#pragma unroll
            for (int i = 0; i < PER; ++i) lds_dma16(lds0 + i * NW * 1024, kt, (uint32_t)src_off[i]);
        } else {
            // A tile that runs past the last visible key re-reads that key for
            // the missing rows (masked later).
#pragma unroll
            for (int i = 0; i < PER; ++i) {
                const int over = t0 + key_of[i] - last_key;
                const uint32_t back = over > 0 ? (uint32_t)(over * (int32_t)(kss * 2)) : 0u;
                lds_dma16(lds0 + i * NW * 1024, kt, (uint32_t)src_off[i] - back);
            }
        }
    };

    // Per-lane LDS element offsets of the MFMA operands within a stage.  The
    // swizzle only permutes the low three bits of a chunk index, so:
    //   K (A of S^T = K Q^T), k-step ks: logical chunk 2ks + hl of key j sits
    //     at kofs[ks & 3] + (ks >> 2) * 64;
    //   V^T (A of O^T = V^T P^T), 16-key step st, half b, channel block db:
    //     lane group g = lane >> 4 reads channels 32db + 16(g&1) + 4(sl&3)..+3
    //     of key 16st + 8b + 4(g>>1) + (sl>>2), sl = lane & 15 (the key order
    //     of the P^T accumulator); the swizzle of that key depends only on its
    //     low four bits, so the read is at vofs[db & 1][b] + 16st * 576 +
    //     (db >> 1) * 64.
    int kofs[4], vofs[2][2];
    {
        const int sk = mswz(j);
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            const int c = hl + 2 * q;
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
                vofs[par][b] = key * DQK + (c7 ^ mswz(key)) * 8 + (sl & 1) * 4;
            }
    }

    // O^T accumulators, zeroed by an MFMA of zero operands (an assignment
    // would let the compiler keep them in VGPRs).  The zero operand is often
    // written by VALU just before: two wait states before the MFMA reads it.
    f32x16 o[DB];
    const bf16x8 zero8 = {};
    auto zero_o = [&]() __attribute__((always_inline)) {
#pragma unroll
        for (int db = 0; db < DB; ++db)
            asm volatile("s_nop 1\n\tv_mfma_f32_32x32x16_bf16 %0, %1, %1, 0" : "=a"(o[db]) : "v"(zero8));
    };
    zero_o();
    float m_run = -INFINITY;   // reference maximum (log2 units, scaled), fixed once set
    float m_seen = -INFINITY;  // largest scaled score seen
    float l_run = 0.f;
    bool spike = false;        // some score exceeded the reference by more than kSpan
    const float sc2 = a.scale * kLog2e;
    constexpr float kSpan = 32.0f;

    auto compute = [&](int t0, const uint16_t* ts, auto mask_tag) __attribute__((always_inline)) {
        constexpr bool MASK = decltype(mask_tag)::value;
        // S^T = K Q^T over the 576 channels, 32 keys: one accumulation chain.
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
        const float msc = mx * sc2;   // this tile's maximum of the scaled scores
        m_seen = fmaxf(m_seen, msc);
        // The row's first tile with a visible key sets the reference (a tile
        // with none has msc = -inf, or NaN when the scale is 0).
        if (m_run == -INFINITY && msc > -INFINITY) m_run = msc;
        spike |= msc > m_run + kSpan;
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
            // The first MFMA reads pb[0], written by VALU just before: two
            // wait states (the compiler does not see into the statement).
            if (q == 0)
                asm volatile("s_nop 1\n\tv_mfma_f32_32x32x16_bf16 %0, %1, %2, %0"
                             : "+a"(o[q % DB]) : "v"(vop[q]), "v"(pb[q / DB]));
            else
                asm volatile("v_mfma_f32_32x32x16_bf16 %0, %1, %2, %0"
                             : "+a"(o[q % DB]) : "v"(vop[q]), "v"(pb[q / DB]));
            if (q < 8) prob(8 + q);
            if (q == 7) pb[1] = pack(1);
            if (q + AV < NQ) vop[q + AV] = v_operand(q + AV);
            __builtin_amdgcn_sched_barrier(0);
        }
        l_run += lsum;
    };

    // Stage i % NS holds tile i.  Each iteration waits for tile i (at most
    // NS-2 later tiles stay in flight), then, after the barrier (every wave
    // has finished tile i-1), refills tile i-1's stage with tile i+NS-1.
    auto wait_outstanding = [&](int tiles_after) __attribute__((always_inline)) {
        if (tiles_after >= NS - 2) {
            wait_vmcnt<(NS - 2) * PER>();
        } else {
            static_for<0, NS - 2>([&](auto k_tag) {
                constexpr int K = decltype(k_tag)::value;
                if (tiles_after == K) wait_vmcnt<K * PER>();
            });
        }
    };
    auto run_tiles = [&]() __attribute__((always_inline)) {
#pragma unroll
    for (int s = 0; s < NS - 1; ++s)
        if (s < n_tiles) issue(k_begin + s * MBN, stage(s));
    for (int t = 0; t < n_tiles; t += NS) {
        static_for<0, NS>([&](auto s_tag) {
            constexpr int S = decltype(s_tag)::value;
            const int i = t + S;
            if (i < n_tiles) {
                wait_outstanding(min(i + NS - 2, n_tiles - 1) - i);
                __builtin_amdgcn_s_waitcnt(15 | (7 << 4) | (0 << 8) | (3 << 14));   // this wave's LDS reads done
                bare_barrier();
                const int ahead = i + NS - 1;
                if (ahead < n_tiles) issue(k_begin + ahead * MBN, stage((S + NS - 1) % NS));
                const int t0 = k_begin + i * MBN;
                if (t0 + MBN > wmin || t0 < wsmax)
                    compute(t0, stage(S), std::true_type{});
                else
                    compute(t0, stage(S), std::false_type{});
            }
        });
    }
    };
    run_tiles();
    // A spike anywhere in the workgroup: run the key range again with the
    // exact maxima as references (they bound every score, so the second
    // pass cannot spike).  Every wave has consumed every tile it waited for.
    const bool wave_spike = __builtin_amdgcn_ballot_w64(spike) != 0;   // every lane votes
    if (lane == 0) red[wave] = wave_spike;
    __syncthreads();
    bool again = false;
#pragma unroll
    for (int w = 0; w < NW; ++w) again |= red[w] != 0;
    __syncthreads();
    if (again) {
        zero_o();
        l_run = 0.f;
        m_run = m_seen;
        run_tiles();
    }

    // The epilogue reads the accumulators: wait out the MFMA write latency
    // first (the statements also keep those reads after the wait).
    asm volatile("s_nop 7\n\ts_nop 7\n\ts_nop 7" : "+a"(o[0]), "+a"(o[1]), "+a"(o[2]), "+a"(o[3]), "+a"(o[4]),
                 "+a"(o[5]), "+a"(o[6]), "+a"(o[7]));
    asm volatile("" : "+a"(o[8]), "+a"(o[9]), "+a"(o[10]), "+a"(o[11]), "+a"(o[12]), "+a"(o[13]), "+a"(o[14]),
                 "+a"(o[15]));

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
                *(u32x2*)(orow + db * 32 + b * 8 + hl * 4) = w;
            }
        }
        if (a.lse_out && hl == 0) a.lse_out[((int64_t)layer * a.total_q + row) * H + head] = lse2 * kLn2;
    } else {
        const int64_t item = (((int64_t)split * a.n_layers + layer) * a.total_q + row) * H + head;
        float* wo = a.ws_o + item * DV;
#pragma unroll
        for (int db = 0; db < DB; ++db) {
#pragma unroll
            for (int b = 0; b < 4; ++b) {
                f32x4 w = {o[db][4 * b] * inv, o[db][4 * b + 1] * inv, o[db][4 * b + 2] * inv,
                           o[db][4 * b + 3] * inv};
                *(f32x4*)(wo + db * 32 + b * 8 + hl * 4) = w;
            }
        }
        if (hl == 0) a.ws_lse[item] = lse2;
    }
}

}  // namespace

hipError_t launch_attn_mla_bf16(const AttnArgs& a, const Plan& p, dim3 grid, hipStream_t stream) {
    if (p.nw != kMlaWaves || p.ns != kMlaStages || p.BM != kMlaWaves * 32) return hipErrorInvalidValue;
    if (a.block_table)
        hipLaunchKernelGGL((attn_mla_bf16_kernel<true>), grid, dim3(kMlaWaves * 64), 0, stream, a, p);
    else
        hipLaunchKernelGGL((attn_mla_bf16_kernel<false>), grid, dim3(kMlaWaves * 64), 0, stream, a, p);
    return hipGetLastError();
}

}  // namespace pkv
