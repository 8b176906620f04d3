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
//   * K and V tiles of 32 keys stream HBM -> LDS with LDS-DMA loads
//     (global_load_lds, 16 bytes per lane) through 4 stages, so 3 tiles are
//     in flight while one is consumed.  16-byte chunks of a row are
//     XOR-swizzled by key (swz_k / swz_v below) to spread LDS banks.
//   * V stays row-major ([key][channel]) in LDS; the transposed A operand of
//     the PV product comes from ds_read_b64_tr_b16, with the keys of each
//     16-key step ordered as the P^T accumulator holds them.
#include <type_traits>

#include "attn_common.h"

namespace pkv {
namespace {


// Kernel shape: 4 waves of 32 rows (one 32-row block each), two workgroups
// per CU, 32-key tiles through 4 LDS stages (64 KB), software-pipelined.
constexpr int kQB = 1;       // 32-row blocks per wave
constexpr int kWaves = 4;
constexpr int kStages = 4;
constexpr int kAhead = 3;    // LDS operand reads issued this many operands ahead of their MFMA

// XOR swizzles of a row's 16-byte chunk index by its key.  LDS has 64 banks
// of 4 bytes (256 bytes per cycle); the rows one read touches must spread
// over the 16 bank groups of 16 bytes.
//   D = 128 (16 chunks per row, every row starting at bank 0):
//     K tiles: an operand read takes one logical chunk from 16 consecutive
//     keys, so the swizzle is a bijection of key & 15.
//     V tiles: a transposed read takes a 4-chunk window from 4 consecutive
//     keys, so bits 2..3 follow key & 3; depending on key & 7 only, it is the
//     same for keys 8 apart, which keeps their reads one immediate apart.
//     (Measured: K reads conflict free; V reads at the transposed-read rate.)
//   D = 64 (8 chunks per row, rows alternating between bank halves): keys of
//     one parity share a half, 3 bits suffice for both.
template <int D>
__device__ inline int swz_k(int key) {
    if constexpr (D == 128) return ((key & 3) << 2) | ((key >> 2) & 3);
    else return ((key & 3) << 1) | ((key >> 2) & 1);
}
template <int D>
__device__ inline int swz_v(int key) {
    if constexpr (D == 128) return (key & 3) << 2;
    else return ((key & 3) << 1) | ((key >> 2) & 1);
}

template <int D, bool PAGED>
__global__ __launch_bounds__(kWaves * 64, 2) void attn_gqa_bf16_kernel(AttnArgs a, Plan p) {
    constexpr int QB = kQB, NW = kWaves, NS = kStages;
    constexpr int CH = D / 8;              // 16-byte chunks per row
    constexpr int BN = 32;                 // keys per tile
    constexpr int NKB = BN / 32;           // 32-key blocks per tile
    constexpr int KBLK = BN * CH / 64;     // 64-lane LDS-DMA blocks per K (or V) tile
    constexpr int PER = 2 * KBLK / NW;     // LDS-DMA loads per wave per tile (K and V)
    constexpr int KS = D / 16;             // MFMA k-steps over channels
    constexpr int DB = D / 32;             // 32-channel output blocks
    constexpr int TE = BN * D;             // elements of one K or V tile
    static_assert(2 * KBLK % NW == 0, "tile loads must split evenly over the waves");
    static_assert(NS >= 2 && NS <= 10 && (NS - 2) * PER < 64, "2..10 stages within the vmcnt range");

    // One LDS block: NS K stages, then NS V stages.  Stage offsets are
    // compile-time constants after unrolling, so one address register per
    // operand serves every stage through the 16-bit immediate offset of the
    // LDS read (K stages within 48 KB of the block, V stages of the V half).
    __shared__ __attribute__((aligned(16))) uint16_t stage_lds[2 * NS * TE];
    __shared__ int red[NW], red_min[NW], red_start[NW], red_smax[NW];
    auto kst = [&](int st) __attribute__((always_inline)) -> uint16_t* { return stage_lds + st * TE; };
    auto vst = [&](int st) __attribute__((always_inline)) -> uint16_t* { return stage_lds + (NS + st) * TE; };

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

    // Rows of this lane (one per 32-row block) and their visible key ranges
    // [row_start, row_end): causal, and with a sliding window also
    // row_start = q_pos - window + 1.
    int qi[QB], head[QB], row_end[QB], row_start[QB];
    bool row_ok[QB];
#pragma unroll
    for (int qb = 0; qb < QB; ++qb) {
        const int m = m0 + (wave * QB + qb) * 32 + j;
        row_ok[qb] = m < M;
        qi[qb] = row_ok[qb] ? m / p.G : 0;
        head[qb] = kvh * p.G + (row_ok[qb] ? m - qi[qb] * p.G : 0);
    }
    // Q^T B operands: 8 channels of the row per k-step (loaded first: they do not
    // depend on the positions, so their latency overlaps the key-range set-up).
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

    int rmax = 0, rmin = 0x7fffffff, smin = 0x7fffffff, smax = 0;
#pragma unroll
    for (int qb = 0; qb < QB; ++qb) {
        const int qpos = row_ok[qb] ? a.q_pos[si.q0 + qi[qb]] : -1;
        visible_range(qpos, si.kvl, a.window, row_start[qb], row_end[qb]);   // (0, 0) for rows past M
        rmax = max(rmax, row_end[qb]);
        if (row_ok[qb]) {
            rmin = min(rmin, row_end[qb]);
            smin = min(smin, row_start[qb]);
            smax = max(smax, row_start[qb]);
        }
    }
    const int wmin = wave_min_i(rmin);
    const int wmax = wave_max_i(rmax);
    const int wsmin = wave_min_i(smin);
    const int wsmax = wave_max_i(smax);   // tiles below this need the window mask
    if (lane == 0) {
        red[wave] = wmax;
        red_min[wave] = wmin;
        red_start[wave] = wsmin;
        red_smax[wave] = wsmax;
    }
    __syncthreads();
    int e_max = 0, e_min = 0x7fffffff, s_min = 0x7fffffff, s_max = 0;
#pragma unroll
    for (int w = 0; w < NW; ++w) {
        e_max = max(e_max, red[w]);
        e_min = min(e_min, red_min[w]);
        s_min = min(s_min, red_start[w]);
        s_max = max(s_max, red_smax[w]);
    }

    // Keys [lo, hi) hold every key a row of the workgroup sees (whole tiles
    // from the first window start; tiles wholly before every window are
    // skipped); the splits share them in equal runs of whole tiles.
    const int lo = s_min == 0x7fffffff ? 0 : s_min / BN * BN;
    const int hi = min(si.kvl, e_max);
    const int run = hi > lo ? ((hi - lo + p.splits - 1) / p.splits + BN - 1) / BN * BN : 0;
    const int k_begin = lo + split * run;
    const int loop_end = min(hi, k_begin + run);
    const int n_tiles = loop_end > k_begin ? (loop_end - k_begin + BN - 1) / BN : 0;

    const uint16_t* kbase = (const uint16_t*)a.k + (int64_t)layer * a.k_stride[0] +
                            (int64_t)kvh * a.k_stride[1] + si.base * a.k_stride[2];
    const uint16_t* vbase = (const uint16_t*)a.v + (int64_t)layer * a.v_stride[0] +
                            (int64_t)kvh * a.v_stride[1] + si.base * a.v_stride[2];
    const int64_t kss = a.k_stride[2], vss = a.v_stride[2];
    const int last_key = loop_end - 1;

    // LDS-DMA: every tile is KBLK 64-lane blocks of K, then KBLK of V; wave w
    // moves blocks w*PER .. w*PER+PER-1 (all K or all V).  Lane l of block b
    // fills LDS chunk slot b*64 + l, i.e. key slot/CH, physical chunk slot%CH,
    // which holds logical chunk (phys ^ swizzle(key)) of that key's row.
    static_assert(KBLK % PER == 0, "a wave's blocks must be all K or all V");
    const bool wave_v = wave * PER >= KBLK;
    const int blk0 = (wave * PER) % KBLK;
    const char* const tens = (const char*)(wave_v ? vbase : kbase);
    const int64_t trow = (wave_v ? vss : kss) * 2;   // bytes between keys
    auto dma_key = [&](int i) __attribute__((always_inline)) { return ((blk0 + i) * 64 + lane) / CH; };
    uint32_t src_off[PER];   // bytes from the tile's first key
#pragma unroll
    for (int i = 0; i < PER; ++i) {
        const int key = dma_key(i);
        const int logical = (lane % CH) ^ (wave_v ? swz_v<D>(key) : swz_k<D>(key));
        src_off[i] = (uint32_t)(key * trow + logical * 16);
    }
    // Stage the tile starting at key t0.  A tile that runs past the last
    // visible key re-reads that key for the missing rows (masked later).
    // Paged cache: tiles start on a multiple of BN, which divides the page
    // size, so each tile lies in one page.
    PageWindow pw;
    // Waves that move V blocks read V's own block table when there is one.
    if constexpr (PAGED)
        pw.init(wave_v && a.v_block_table ? a.v_block_table : a.block_table, a, seq, k_begin >> a.page_shift);
    const int64_t tpage = (wave_v ? a.v_page_stride : a.k_page_stride) * 2;   // bytes between pages
    auto issue = [&](int t0, uint16_t* ks_dst, uint16_t* vs_dst) __attribute__((always_inline)) {
        const char* tile;
        if constexpr (PAGED)
            tile = tens + pw.offset(a, t0, tpage, trow);
        else
            tile = tens + (int64_t)t0 * trow;
        const uint32_t lds0 = lds_addr_of((wave_v ? vs_dst : ks_dst) + blk0 * 64 * 8);
        if (t0 + BN <= loop_end) {
#pragma unroll
            for (int i = 0; i < PER; ++i) lds_dma16(lds0 + i * 1024, tile, src_off[i]);
        } else {
#pragma unroll
            for (int i = 0; i < PER; ++i) {
                const int over = t0 + dma_key(i) - last_key;
                lds_dma16(lds0 + i * 1024, tile, src_off[i] - (over > 0 ? (uint32_t)(over * trow) : 0u));
            }
        }
    };

    // Per-lane LDS element offsets of the MFMA operands within a stage.  The
    // K swizzle depends only on key & 15 and the V swizzle on key & 7, the same
    // for a lane's K reads of every key block and its V reads of every 8 keys,
    // so those strides are immediates:
    //   K (A of S^T = K Q^T), k-step ks, key block kb: kofs[ks] + kb * 32 * D
    //   V^T (A of O^T = V^T P^T), 16-key step st, half b, channel block db:
    //       vofs[db] + (st * 16 + b * 8) * D
    int kofs[KS], vofs[DB];
    {
        const int sk = swz_k<D>(j);
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) kofs[ks] = j * D + (((ks * 2 + hl) ^ sk) << 3);
        const int g = lane >> 4, sl = lane & 15;
        const int vkey = (g >> 1) * 4 + (sl >> 2);   // key within its group of 8
        const int sv = swz_v<D>(vkey);
#pragma unroll
        for (int db = 0; db < DB; ++db)
            vofs[db] = vkey * D + (((db * 4 + (g & 1) * 2 + ((sl & 3) >> 1)) ^ sv) << 3) + (sl & 1) * 4;
    }
    auto k_operand = [&](const uint16_t* ks_src, int ks, int kb) __attribute__((always_inline)) {
        return __builtin_bit_cast(bf16x8, *(const u32x4*)(ks_src + kofs[ks] + kb * 32 * D));
    };
    auto v_operand = [&](const uint16_t* vs_src, int st, int db) __attribute__((always_inline)) {
        const uint16_t* base = vs_src + vofs[db] + st * 16 * D;
        const s16x4 p0 = __builtin_amdgcn_ds_read_tr16_b64_v4i16(PKV_LDS(s16x4, base));
        const s16x4 p1 = __builtin_amdgcn_ds_read_tr16_b64_v4i16(PKV_LDS(s16x4, base + 8 * D));
        return __builtin_bit_cast(bf16x8, (short __attribute__((ext_vector_type(8)))){p0[0], p0[1], p0[2], p0[3],
                                                                                       p1[0], p1[1], p1[2], p1[3]});
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
    auto qk = [&](const uint16_t* ks_src, f32x16 (&s)[NKB][QB]) __attribute__((always_inline)) {
#pragma unroll
        for (int kb = 0; kb < NKB; ++kb)
#pragma unroll
            for (int qb = 0; qb < QB; ++qb) s[kb][qb] = f32x16{};
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) {
#pragma unroll
            for (int kb = 0; kb < NKB; ++kb) {
                const bf16x8 kf = k_operand(ks_src, ks, kb);
#pragma unroll
                for (int qb = 0; qb < QB; ++qb)
                    s[kb][qb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf, qf[qb][ks], s[kb][qb], 0, 0, 0);
            }
        }
        // Keep the K-operand reads one or two MFMAs ahead instead of all at once.
        sched_reads_mfma<NKB * KS, 1, QB>();
    };

    // Softmax, part 1 (branchy, before the overlapped region): mask the raw
    // scores of the tile at key t0 if needed, take each row's maximum and
    // move the reference maximum lazily.  The reference only moves when the
    // scaled tile maximum exceeds it by more than kLazy, so most tiles skip
    // rescaling O; probabilities then stay below 2^kLazy, well inside fp32 and
    // bf16 range, and the final O/l is unchanged.
    constexpr float kLazy = 8.0f;
    auto row_max = [&](int t0, f32x16 (&s)[NKB][QB], auto mask_tag) __attribute__((always_inline)) {
        constexpr bool MASK = decltype(mask_tag)::value;
#pragma unroll
        for (int qb = 0; qb < QB; ++qb) {
            if (MASK) {
#pragma unroll
                for (int kb = 0; kb < NKB; ++kb)
#pragma unroll
                    for (int r = 0; r < 16; ++r) {
                        const int key = t0 + kb * 32 + (r >> 2) * 8 + hl * 4 + (r & 3);
                        if (key >= row_end[qb] || key < row_start[qb]) s[kb][qb][r] = sc2 >= 0.f ? -INFINITY : INFINITY;
                    }
            }
            float mx;
            if (sc2 >= 0.f) {
                mx = -INFINITY;
#pragma unroll
                for (int kb = 0; kb < NKB; ++kb)
#pragma unroll
                    for (int r = 0; r < 16; ++r) mx = fmaxf(mx, s[kb][qb][r]);
                mx = fmaxf(mx, __shfl_xor(mx, 32));
            } else {
                mx = INFINITY;
#pragma unroll
                for (int kb = 0; kb < NKB; ++kb)
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
    auto probs = [&](int t0, f32x16 (&s)[NKB][QB], bf16x8 (&pb)[QB][2 * NKB], auto mask_tag) __attribute__((always_inline)) {
        constexpr bool MASK = decltype(mask_tag)::value;
#pragma unroll
        for (int qb = 0; qb < QB; ++qb) {
            const float neg_m = m_run[qb] == -INFINITY ? 0.f : -m_run[qb];
            float lsum = 0.f;
#pragma unroll
            for (int kb = 0; kb < NKB; ++kb) {
#pragma unroll
                for (int r = 0; r < 16; ++r) {
                    float e = __builtin_amdgcn_exp2f(fmaf(s[kb][qb][r], sc2, neg_m));
                    if (MASK) {
                        const int key = t0 + kb * 32 + (r >> 2) * 8 + hl * 4 + (r & 3);
                        if (key >= row_end[qb] || key < row_start[qb]) e = 0.f;
                    }
                    s[kb][qb][r] = e;
                    lsum += e;
                }
            }
            l_run[qb] += lsum;
#pragma unroll
            for (int st = 0; st < 2 * NKB; ++st) {
                f32x8 pv;
#pragma unroll
                for (int e = 0; e < 8; ++e) pv[e] = s[st >> 1][qb][(st & 1) * 8 + e];
                pb[qb][st] = __builtin_convertvector(pv, bf16x8);
            }
        }
    };

    // O^T += V^T P^T for the tile held in V stage vs_src.
    auto pv = [&](const uint16_t* vs_src, const bf16x8 (&pb)[QB][2 * NKB]) __attribute__((always_inline)) {
        // Lane group g (16 lanes) reads channels 32db + 16(g&1) .. +15 for
        // keys {16st + 8b + 4(g>>1) + 0..3}, b = 0, 1: the key order of the
        // P^T accumulator rows.
#pragma unroll
        for (int st = 0; st < 2 * NKB; ++st) {
#pragma unroll
            for (int db = 0; db < DB; ++db) {
                const bf16x8 vf = v_operand(vs_src, st, db);
#pragma unroll
                for (int qb = 0; qb < QB; ++qb)
                    o[db][qb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vf, pb[qb][st], o[db][qb], 0, 0, 0);
            }
        }
        sched_reads_mfma<2 * NKB * DB, 2, QB>();
    };

    // Processing order.  The pipelined schedule takes the F tiles that need
    // no mask for any row of the workgroup (key range [s_max, e_min): past
    // every row's window start, before every row's end) first; the n_lead
    // tiles before s_max and the tail after them follow in plain order with
    // masks.  Online softmax does not depend on the order of the tiles.
    // Without a window n_lead is 0 and the order is ascending.
    const int n_lead = a.window > 0 ? min(n_tiles, max(0, (s_max - k_begin + BN - 1) / BN)) : 0;
    const int F = sc2 > 0.f ? max(0, min(n_tiles - n_lead, (e_min - (k_begin + n_lead * BN)) / BN)) : 0;
    auto key_of = [&](int i) __attribute__((always_inline)) {
        const int t = i < F ? i + n_lead : (i < F + n_lead ? i - F : i);
        return k_begin + t * BN;
    };

    // Tiles are staged through NS LDS stages: tile i lives in stage i % NS
    // and is issued NS-1 tiles ahead of its use.  Wait until at most
    // tiles_after later tiles (at most NS-2) are still in flight.
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
    auto lds_reads_done = []() __attribute__((always_inline)) { __builtin_amdgcn_s_waitcnt(15 | (7 << 4) | (0 << 8) | (3 << 14)); };

    // One tile in plain order: wait for it, then QK^T, softmax and PV back to
    // back.  The barrier that publishes tile i also proves every wave finished
    // tile i-1, so tile i-1's stage is refilled with tile i+NS-1 right after.
    auto plain_tile = [&](int i, auto stage_tag) __attribute__((always_inline)) {
        constexpr int S = decltype(stage_tag)::value;
        wait_outstanding(min(i + NS - 2, n_tiles - 1) - i);
        lds_reads_done();
        bare_barrier();
        const int ahead = i + NS - 1;
        if (ahead < n_tiles) issue(key_of(ahead), kst((S + NS - 1) % NS), vst((S + NS - 1) % NS));
        f32x16 sc[NKB][QB];
        qk(kst(S), sc);
        bf16x8 pb[QB][2 * NKB];
        const int t0 = key_of(i);
        if (t0 + BN > wmin || t0 < wsmax) {
            row_max(t0, sc, std::true_type{});
            probs(t0, sc, pb, std::true_type{});
        } else {
            row_max(t0, sc, std::false_type{});
            probs(t0, sc, pb, std::false_type{});
        }
        pv(vst(S), pb);
    };
    auto plain_from = [&](int first) __attribute__((always_inline)) {
        for (int t = first - first % NS; t < n_tiles; t += NS) {
            static_for<0, NS>([&](auto s_tag) {
                const int i = t + decltype(s_tag)::value;
                if (i >= first && i < n_tiles) plain_tile(i, s_tag);
            });
        }
    };

#pragma unroll
    for (int s = 0; s < NS - 1; ++s)
        if (s < n_tiles) issue(key_of(s), kst(s), vst(s));

    {
        // Intra-wave software pipeline over the leading tiles that need no
        // mask (F of them, the same for every wave); tiles are 32 keys (one
        // key block).  With S(t) the raw scores of tile t, iteration t runs
        //   segment 1: S(t+1) = K Q^T (MFMA) interleaved with the
        //              probabilities of tile t (exp2, VALU);
        //   segment 2: O += V^T P(t) (MFMA) interleaved with the row maxima of
        //              S(t+1) and the row sums of P(t) (VALU);
        // then moves the reference maximum if needed.  A wave that alternates
        // its own MFMA and VALU instructions keeps both units busy; an
        // MFMA-only and a VALU-only wave sharing a SIMD overlap far less.  Two
        // workgroups of four waves share each CU, so the two waves on a SIMD
        // never wait at each other's barriers.  Iteration t reads K of tile
        // t+1 and V of tile t; tile t+3 is issued after the barrier opening
        // it, into the stage that tile t-1 left.  A wave raises its priority
        // for segment 2, so of the two waves on a SIMD the one streaming the
        // PV MFMAs issues first and the other fills in with segment 1's VALU
        // work (measured 5% on the 8B workload, 1% on the 32k one).
        static_assert(NS >= 4 && NS % 2 == 0 && NKB == 1,
                      "the pipelined schedule uses an even number (>= 4) of LDS stages of 32-key tiles");

        const bf16x2 ones = {(__bf16)1.0f, (__bf16)1.0f};

        // Segment 1: nxt = raw scores of key block kbn of the K stage; the
        // probabilities of cur into pb (two 16-key operands per row block).
        // Written as fenced groups of one K operand's MFMAs, their share of
        // the VALU work and the operand read kAhead steps ahead, so
        // the LDS reads stay in flight across MFMAs.
        auto seg1 = [&](const uint16_t* ks_src, int kbn, f32x16 (&cur)[QB], f32x16 (&nxt)[QB],
                        bf16x8 (&pb)[QB][2]) __attribute__((always_inline)) {
            constexpr int A = kAhead < KS ? kAhead : KS;
            constexpr int PER_K = 16 / KS;   // probabilities per k-step and row block
            bf16x8 kop[KS];
#pragma unroll
            for (int q = 0; q < A; ++q) kop[q] = k_operand(ks_src, q, kbn);
            __builtin_amdgcn_sched_barrier(0);
#pragma unroll
            for (int q = 0; q < KS; ++q) {
#pragma unroll
                for (int qb = 0; qb < QB; ++qb) {
                    nxt[qb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kop[q], qf[qb][q], q == 0 ? f32x16{} : nxt[qb],
                                                                     0, 0, 0);
                    const float neg_m = -m_run[qb];
#pragma unroll
                    for (int r = q * PER_K; r < (q + 1) * PER_K; ++r)
                        cur[qb][r] = __builtin_amdgcn_exp2f(fmaf(cur[qb][r], sc2, neg_m));
#pragma unroll
                    for (int h = 0; h < 2; ++h) {
                        if ((q + 1) * PER_K == 8 * (h + 1)) {
                            f32x8 pv8;
#pragma unroll
                            for (int e = 0; e < 8; ++e) pv8[e] = cur[qb][h * 8 + e];
                            pb[qb][h] = __builtin_convertvector(pv8, bf16x8);
                        }
                    }
                }
                if (q + A < KS) kop[q + A] = k_operand(ks_src, q + A, kbn);
                __builtin_amdgcn_sched_barrier(0);
            }
        };

        // Segment 2: O^T += V^T P^T for key block kbc of the V stage; the row
        // maxima of nxt (over both lanes of a row, into mx) and the row sums
        // of pb alongside, in fenced groups as in segment 1.
        auto seg2 = [&](const uint16_t* vs_src, int kbc, const bf16x8 (&pb)[QB][2], const f32x16 (&nxt)[QB],
                        float (&mx)[QB]) __attribute__((always_inline)) {
            constexpr int NQ = 2 * DB;                 // V operands: two 16-key steps x DB channel blocks
            constexpr int A = kAhead < NQ ? kAhead : NQ;
            constexpr int PER_M = 16 / NQ;             // maxima per operand and row block
            constexpr int PER_D = 8 / NQ > 0 ? 8 / NQ : 1;   // sum steps per operand and row block
            bf16x8 vop[NQ];
#pragma unroll
            for (int q = 0; q < A; ++q) vop[q] = v_operand(vs_src, 2 * kbc + q / DB, q % DB);
            __builtin_amdgcn_sched_barrier(0);
            float m0[QB], m1[QB], l0[QB], l1[QB];
#pragma unroll
            for (int qb = 0; qb < QB; ++qb) {
                m0[qb] = -INFINITY;
                m1[qb] = -INFINITY;
                l0[qb] = 0.f;
                l1[qb] = 0.f;
            }
#pragma unroll
            for (int q = 0; q < NQ; ++q) {
                const int h = q / DB, db = q % DB;
#pragma unroll
                for (int qb = 0; qb < QB; ++qb) {
                    o[db][qb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vop[q], pb[qb][h], o[db][qb], 0, 0, 0);
#pragma unroll
                    for (int r = q * PER_M; r < (q + 1) * PER_M; r += 2) {
                        m0[qb] = fmaxf(m0[qb], nxt[qb][r]);
                        m1[qb] = fmaxf(m1[qb], nxt[qb][r + 1]);
                    }
#pragma unroll
                    for (int d = q * PER_D; d < (q + 1) * PER_D && d < 8; ++d) {
                        const bf16x8 pp = pb[qb][d >> 2];
                        const int e = (d & 3) * 2;
                        if (d & 1) l1[qb] = __builtin_amdgcn_fdot2_f32_bf16((bf16x2){pp[e], pp[e + 1]}, ones, l1[qb], false);
                        else l0[qb] = __builtin_amdgcn_fdot2_f32_bf16((bf16x2){pp[e], pp[e + 1]}, ones, l0[qb], false);
                    }
                }
                if (q + A < NQ) vop[q + A] = v_operand(vs_src, 2 * kbc + (q + A) / DB, (q + A) % DB);
                __builtin_amdgcn_sched_barrier(0);
            }
#pragma unroll
            for (int qb = 0; qb < QB; ++qb) {
                l_run[qb] += l0[qb] + l1[qb];
                // lanes l and l+32 hold the two 16-key halves of the same row
                const float m = fmaxf(m0[qb], m1[qb]);
                const auto sw = __builtin_amdgcn_permlane32_swap(__float_as_uint(m), __float_as_uint(m), false, false);
                mx[qb] = fmaxf(__uint_as_float(sw[0]), __uint_as_float(sw[1]));
            }
        };

        // Move the reference maxima after the tile's PV (lazily, as row_max).
        auto move_max = [&](const float (&mx)[QB]) __attribute__((always_inline)) {
#pragma unroll
            for (int qb = 0; qb < QB; ++qb) {
                const float msc = mx[qb] * sc2;
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

        // One step: scores of the next tile from ks_next, the current tile's
        // probabilities and PV from vs_cur.
        auto half_step = [&](const uint16_t* ks_next, int kbn, const uint16_t* vs_cur, int kbc, f32x16 (&cur)[QB],
                             f32x16 (&nxt)[QB]) __attribute__((always_inline)) {
            bf16x8 pb[QB][2];
            float mx[QB];
            seg1(ks_next, kbn, cur, nxt, pb);
            __builtin_amdgcn_s_setprio(1);
            seg2(vs_cur, kbc, pb, nxt, mx);
            __builtin_amdgcn_s_setprio(0);
            move_max(mx);
        };

        auto iteration = [&](int i, auto u_tag, f32x16 (&cur)[QB], f32x16 (&nxt)[QB]) __attribute__((always_inline)) {
            constexpr int U = decltype(u_tag)::value;
            wait_outstanding(min(i + NS - 2, n_tiles - 1) - (i + 1));   // tile i+1 has landed
            lds_reads_done();
            bare_barrier();
            if (i + NS - 1 < n_tiles)
                issue(key_of(i + NS - 1), kst((U + NS - 1) % NS), vst((U + NS - 1) % NS));
            half_step(kst((U + 1) % NS), 0, vst(U), 0, cur, nxt);
        };

        // Last pipelined tile: probabilities and PV without overlap; issues
        // the tile that plain order would issue at this point.
        auto drain = [&](int i, auto u_tag, f32x16 (&cur)[QB]) __attribute__((always_inline)) {
            constexpr int U = decltype(u_tag)::value;
            lds_reads_done();
            bare_barrier();
            if (i + NS - 1 < n_tiles)
                issue(key_of(i + NS - 1), kst((U + NS - 1) % NS), vst((U + NS - 1) % NS));
            bf16x8 pb[QB][2];
#pragma unroll
            for (int qb = 0; qb < QB; ++qb) {
                const float neg_m = -m_run[qb];
                float lsum = 0.f;
#pragma unroll
                for (int r = 0; r < 16; ++r) {
                    cur[qb][r] = __builtin_amdgcn_exp2f(fmaf(cur[qb][r], sc2, neg_m));
                    lsum += cur[qb][r];
                }
                l_run[qb] += lsum;
#pragma unroll
                for (int h = 0; h < 2; ++h) {
                    f32x8 pv8;
#pragma unroll
                    for (int e = 0; e < 8; ++e) pv8[e] = cur[qb][h * 8 + e];
                    pb[qb][h] = __builtin_convertvector(pv8, bf16x8);
                }
            }
#pragma unroll
            for (int h = 0; h < 2; ++h)
#pragma unroll
                for (int db = 0; db < DB; ++db) {
                    const bf16x8 vf = v_operand(vst(U), h, db);
#pragma unroll
                    for (int qb = 0; qb < QB; ++qb)
                        o[db][qb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vf, pb[qb][h], o[db][qb], 0, 0, 0);
                }
        };

        if (F >= 2) {
            f32x16 sA[QB], sB[QB];
            wait_outstanding(min(NS - 2, n_tiles - 1));
            lds_reads_done();
            bare_barrier();
            // scores of tile 0 and their maxima
#pragma unroll
            for (int qb = 0; qb < QB; ++qb) sA[qb] = f32x16{};
#pragma unroll
            for (int ks = 0; ks < KS; ++ks) {
                const bf16x8 kf = k_operand(kst(0), ks, 0);
#pragma unroll
                for (int qb = 0; qb < QB; ++qb)
                    sA[qb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf, qf[qb][ks], sA[qb], 0, 0, 0);
            }
            {
                float mx[QB];
#pragma unroll
                for (int qb = 0; qb < QB; ++qb) {
                    float m = sA[qb][0];
#pragma unroll
                    for (int r = 1; r < 16; ++r) m = fmaxf(m, sA[qb][r]);
                    const auto sw =
                        __builtin_amdgcn_permlane32_swap(__float_as_uint(m), __float_as_uint(m), false, false);
                    mx[qb] = fmaxf(__uint_as_float(sw[0]), __uint_as_float(sw[1]));
                }
                move_max(mx);
            }
            for (int t = 0; t + 1 < F; t += NS) {
                static_for<0, NS>([&](auto u_tag) {
                    constexpr int u = decltype(u_tag)::value;
                    const int i = t + u;
                    if (i + 1 < F) {
                        if constexpr (u % 2 == 0) iteration(i, u_tag, sA, sB);
                        else iteration(i, u_tag, sB, sA);
                    }
                });
            }
            const int last = F - 1;
            static_for<0, NS>([&](auto u_tag) {
                constexpr int u = decltype(u_tag)::value;
                if (last % NS == u) {
                    if constexpr (u % 2 == 0) drain(last, u_tag, sA);
                    else drain(last, u_tag, sB);
                }
            });
        }
        plain_from(F >= 2 ? F : 0);
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

template <int D, bool PAGED>
hipError_t launch_d(const AttnArgs& a, const Plan& p, dim3 grid, hipStream_t stream) {
    if (p.nw != kWaves || p.qb != kQB || p.ns != kStages) return hipErrorInvalidValue;
    hipLaunchKernelGGL((attn_gqa_bf16_kernel<D, PAGED>), grid, dim3(kWaves * 64), 0, stream, a, p);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_attn_gqa_bf16(const AttnArgs& a, const Plan& p, dim3 grid, hipStream_t stream) {
    if (a.block_table) {
        if (a.head_dim == 64) return launch_d<64, true>(a, p, grid, stream);
        return launch_d<128, true>(a, p, grid, stream);
    }
    if (a.head_dim == 64) return launch_d<64, false>(a, p, grid, stream);
    return launch_d<128, false>(a, p, grid, stream);
}

}  // namespace pkv
