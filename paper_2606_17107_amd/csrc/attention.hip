// Suffix attention: plan, fp32 kernel, split-KV combine and dispatch.
// (Paper Sec. 5 "Linear-time TTFT": the transplant costs a re-rotation pass
// plus the causal attention of the suffix over the spliced cache.)
// The bf16 GQA kernel lives in attn_gqa_bf16.hip.
#include "attn_common.h"

namespace pkv {

hipError_t launch_attn_gqa_bf16(const AttnArgs& a, const Plan& p, dim3 grid, hipStream_t stream);
hipError_t launch_attn_mla_bf16(const AttnArgs& a, const Plan& p, dim3 grid, hipStream_t stream);

namespace {

constexpr int kCUs = 256;   // compute units of an MI355X

// fp32 GQA kernel on fp32 matrix cores (v_mfma_f32_32x32x2_f32).  Each of the
// two waves owns 32 rows (query, head-in-group) of one KV head.  As in the
// bf16 kernel the scores are formed transposed, S^T = K Q^T, so a lane holds 16
// keys of one row and its probabilities are already the B operand of
// O^T = V^T P^T: a 2-key step pairs key 8jj + rr (held by lanes 0-31) with key
// 8jj + 4 + rr (lanes 32-63), both in accumulator register 4jj + rr.  K/V tiles
// of 32 keys move through registers into LDS (the next tile's loads are in
// flight while one is consumed): K transposed ([channel][key], a half-wave's 32
// reads of one score step are 32 consecutive words), V row-major ([key][channel],
// likewise for the PV operand).  fp32 online softmax with an exact rescale per
// tile, in log2 units.
template <int D>
__global__ __launch_bounds__(128) void attn_gqa_f32(AttnArgs a, Plan p) {
    constexpr int BN = 32;                 // keys per tile
    constexpr int NW = 2;                  // waves, 32 rows each
    constexpr int KSF = D / 2;             // score steps (2 channels each)
    constexpr int DB = D / 32;             // 32-channel output blocks
    constexpr int NL = BN * D / 4 / (NW * 64);   // 16-byte loads per thread per tensor and tile
    __shared__ __attribute__((aligned(16))) float kt_lds[D * BN];   // [channel][key]
    __shared__ __attribute__((aligned(16))) float v_lds[BN * D];    // [key][channel]
    __shared__ int red[NW], red_min[NW], red_start[NW], red_smax[NW];

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
    const int m0 = rb * (NW * 32);
    if (m0 >= M) return;

    const int tid = threadIdx.x;
    const int wave = tid >> 6;
    const int lane = tid & 63;
    const int j = lane & 31;
    const int hl = lane >> 5;
    const int m = m0 + wave * 32 + j;
    const bool row_ok = m < M;
    const int qi = row_ok ? m / p.G : 0;
    const int head = kvh * p.G + (row_ok ? m - qi * p.G : 0);

    // Q^T B operand: channel 2s + hl of the lane's row for step s, scaled.
    float qf[KSF];
    {
        const float* qrow = (const float*)a.q + (int64_t)layer * a.q_stride[0] +
                            (int64_t)(si.q0 + qi) * a.q_stride[1] + (int64_t)head * a.q_stride[2];
#pragma unroll
        for (int s = 0; s < KSF; ++s) qf[s] = row_ok ? qrow[2 * s + hl] * a.scale : 0.f;
    }
    const int qpos = row_ok ? a.q_pos[si.q0 + qi] : -1;
    int row_start, row_end;
    visible_range(qpos, si.kvl, a.window, row_start, row_end);   // (0, 0) for rows past M
    const int wmin = wave_min_i(row_ok ? row_end : 0x7fffffff);
    const int wmax = wave_max_i(row_end);
    const int wsmin = wave_min_i(row_ok ? row_start : 0x7fffffff);
    const int wsmax = wave_max_i(row_start);
    if (lane == 0) {
        red[wave] = wmax;
        red_min[wave] = wmin;
        red_start[wave] = wsmin;
        red_smax[wave] = wsmax;
    }
    __syncthreads();
    const int e_max = max(red[0], red[1]);
    const int s_min = min(red_start[0], red_start[1]);
    // Keys [lo, hi) hold every key a row of the workgroup sees (whole tiles
    // from the first window start); the splits share them in equal runs of
    // whole tiles.
    const int lo = s_min == 0x7fffffff ? 0 : s_min / BN * BN;
    const int hi = min(si.kvl, e_max);
    const int run = hi > lo ? ((hi - lo + p.splits - 1) / p.splits + BN - 1) / BN * BN : 0;
    const int k_begin = lo + split * run;
    const int k_end = min(hi, k_begin + run);

    const float* kbase = (const float*)a.k + (int64_t)layer * a.k_stride[0] + (int64_t)kvh * a.k_stride[1] +
                         si.base * a.k_stride[2];
    const float* vbase = (const float*)a.v + (int64_t)layer * a.v_stride[0] + (int64_t)kvh * a.v_stride[1] +
                         si.base * a.v_stride[2];
    // Thread tid moves 16-byte pieces tid + 128 i of each tensor's tile.  K:
    // key (tid + 128 i) % 32, channels 4 ((tid + 128 i) / 32) .. +3 (consecutive
    // threads write consecutive words of the transposed tile); V: key
    // (tid + 128 i) / (D/4), channels 4 ((tid + 128 i) % (D/4)) .. +3.  Keys
    // past k_end load zeros (their scores are masked, and 0 * 0 adds nothing).
    f32x4 pk[NL], pv[NL];
    auto load_tile = [&](int t0) __attribute__((always_inline)) {
#pragma unroll
        for (int i = 0; i < NL; ++i) {
            const int id = tid + i * (NW * 64);
            const int kk = id % BN, kc = id / BN, vk = id / (D / 4), vc = id % (D / 4);
            pk[i] = t0 + kk < k_end ? *(const f32x4*)(kbase + (int64_t)(t0 + kk) * a.k_stride[2] + kc * 4)
                                    : f32x4{0.f, 0.f, 0.f, 0.f};
            pv[i] = t0 + vk < k_end ? *(const f32x4*)(vbase + (int64_t)(t0 + vk) * a.v_stride[2] + vc * 4)
                                    : f32x4{0.f, 0.f, 0.f, 0.f};
        }
    };

    f32x16 o[DB];
#pragma unroll
    for (int db = 0; db < DB; ++db) o[db] = f32x16{};
    float m_run = -INFINITY, l_run = 0.f;   // running maximum (log2 units) and sum
    if (k_begin < k_end) load_tile(k_begin);
    for (int t0 = k_begin; t0 < k_end; t0 += BN) {
        __syncthreads();   // every wave is done with the previous tile
#pragma unroll
        for (int i = 0; i < NL; ++i) {
            const int id = tid + i * (NW * 64);
            const int kk = id % BN, kc = id / BN, vk = id / (D / 4), vc = id % (D / 4);
#pragma unroll
            for (int e = 0; e < 4; ++e) kt_lds[(kc * 4 + e) * BN + kk] = pk[i][e];
            *(f32x4*)(v_lds + vk * D + vc * 4) = pv[i];
        }
        __syncthreads();
        if (t0 + BN < k_end) load_tile(t0 + BN);

        // S^T = K Q^T: step s takes channels 2s (lanes 0-31) and 2s + 1 (lanes 32-63).
        f32x16 sc = f32x16{};
#pragma unroll
        for (int s = 0; s < KSF; ++s)
            sc = __builtin_amdgcn_mfma_f32_32x32x2f32(kt_lds[(2 * s + hl) * BN + j], qf[s], sc, 0, 0, 0);
        // Element r of the lane holds key t0 + 8 (r / 4) + 4 hl + r % 4 of row j.
        float mx = -INFINITY;
#pragma unroll
        for (int r = 0; r < 16; ++r) {
            const int key = t0 + (r >> 2) * 8 + hl * 4 + (r & 3);
            const float v = key < row_end && key >= row_start && key < k_end ? sc[r] * kLog2e : -INFINITY;
            sc[r] = v;
            mx = fmaxf(mx, v);
        }
        mx = fmaxf(mx, __shfl_xor(mx, 32));
        // Branch-free (the MFMAs below run for the whole wave): a row that has
        // seen no visible key keeps o = 0 and l = 0 (alpha 0, probabilities 0).
        const float m_new = fmaxf(m_run, mx);
        const float alpha = m_run == -INFINITY ? 0.f : __builtin_amdgcn_exp2f(m_run - m_new);
        float lsum = 0.f;
#pragma unroll
        for (int r = 0; r < 16; ++r) {
            const float e = sc[r] == -INFINITY ? 0.f : __builtin_amdgcn_exp2f(sc[r] - m_new);
            sc[r] = e;
            lsum += e;
        }
        l_run = l_run * alpha + lsum;
        m_run = m_new;
#pragma unroll
        for (int db = 0; db < DB; ++db) {
            o[db] *= alpha;
#pragma unroll
            for (int jj = 0; jj < 4; ++jj)
#pragma unroll
                for (int rr = 0; rr < 4; ++rr)
                    o[db] = __builtin_amdgcn_mfma_f32_32x32x2f32(v_lds[(8 * jj + 4 * hl + rr) * D + db * 32 + j],
                                                                 sc[4 * jj + rr], o[db], 0, 0, 0);
        }
    }

    // The two halves of a row hold disjoint keys.
    const float l_tot = l_run + __shfl_xor(l_run, 32);
    if (!row_ok) return;
    const float inv = l_tot > 0.f ? 1.f / l_tot : 0.f;
    const float lse2 = l_tot > 0.f ? m_run + __log2f(l_tot) : -INFINITY;
    const int64_t row = si.q0 + qi;
    // Element 4 jj + rr of block db holds channel 32 db + 8 jj + 4 hl + rr of the row.
    float* dst;
    if (p.splits == 1) {
        dst = (float*)a.out + (int64_t)layer * a.o_stride[0] + row * a.o_stride[1] + (int64_t)head * a.o_stride[2];
        if (a.lse_out && hl == 0)
            a.lse_out[((int64_t)layer * a.total_q + row) * a.n_heads + head] = lse2 * kLn2;
    } else {
        // split partial: normalised output and its log2-sum-exp (the combine's domain)
        const int64_t item = (((int64_t)split * a.n_layers + layer) * a.total_q + row) * a.n_heads + head;
        dst = a.ws_o + item * D;
        if (hl == 0) a.ws_lse[item] = lse2;
    }
#pragma unroll
    for (int db = 0; db < DB; ++db)
#pragma unroll
        for (int jj = 0; jj < 4; ++jj)
            *(f32x4*)(dst + db * 32 + jj * 8 + hl * 4) =
                f32x4{o[db][4 * jj] * inv, o[db][4 * jj + 1] * inv, o[db][4 * jj + 2] * inv, o[db][4 * jj + 3] * inv};
}

// Merge split-KV partials: out = sum_s w_s O_s / sum_s w_s with
// w_s = 2^(lse_s - max lse).  Grid (row tiles, sequences from seq0, layers);
// a thread takes kCombineCV 16-byte chunks of one (query, head) output row,
// so its index arithmetic (32-bit) and log-sum-exp loads serve several
// chunks.  Rows that no sequence owns (outside every cu_q range) are left
// untouched, as the one-pass kernels leave them.
constexpr int kCombineCV = 2;   // 16-byte output chunks per thread
constexpr int kCombineCB = 8;   // splits whose partials are loaded in one batch
__global__ __launch_bounds__(256) void attn_combine(AttnArgs a, int seq0) {
    constexpr int CV = kCombineCV, CB = kCombineCB;
    const int dv = a.head_dim_v;
    const int64_t items = (int64_t)a.n_layers * a.total_q * a.n_heads;   // partial records per split
    const uint32_t per_item = (uint32_t)dv / (4 * CV);                  // threads per (query, head)
    const uint32_t idx = blockIdx.x * 256u + threadIdx.x;
    const uint32_t rh = idx / per_item;
    const int c0 = (int)(idx - rh * per_item) * CV;                      // first chunk of this thread
    const uint32_t qi = rh / (uint32_t)a.n_heads;
    const int head = (int)(rh - qi * (uint32_t)a.n_heads);
    if (qi >= (uint32_t)a.max_q) return;
    const int seq = seq0 + (int)blockIdx.y;
    const int layer = (int)blockIdx.z;
    int q0 = 0, nq = a.total_q;
    if (a.cu_q) {
        q0 = a.cu_q[seq];
        nq = a.cu_q[seq + 1] - q0;
    }
    if (q0 < 0 || nq < 0 || (int64_t)q0 + nq > a.total_q) nq = 0;   // as seq_info
    if ((int)qi >= nq) return;
    const int64_t row = q0 + (int)qi;
    const int64_t item = ((int64_t)layer * a.total_q + row) * a.n_heads + head;
    // The log-sum-exps and partial outputs of up to CB splits are loaded in
    // one batch (independent loads: one memory round trip), then weighted by
    // w_s = 2^(lse_s - max) and summed in split order; a later batch (more
    // than CB splits) rescales the sums to its larger maximum.
    const int ns = a.n_splits;
    float mx = -INFINITY, wsum = 0.f;
    f32x4 acc[CV];
#pragma unroll
    for (int k = 0; k < CV; ++k) acc[k] = f32x4{0.f, 0.f, 0.f, 0.f};
    for (int s0 = 0; s0 < ns; s0 += CB) {
        float l[CB];
        f32x4 v[CB][CV];
#pragma unroll
        for (int j = 0; j < CB; ++j) {
            const bool in = s0 + j < ns;
            l[j] = in ? a.ws_lse[(int64_t)(s0 + j) * items + item] : -INFINITY;
            const float* src = a.ws_o + ((int64_t)(s0 + j) * items + item) * dv + c0 * 4;
#pragma unroll
            for (int k = 0; k < CV; ++k) v[j][k] = in ? *(const f32x4*)(src + k * 4) : f32x4{0.f, 0.f, 0.f, 0.f};
        }
        float bm = -INFINITY;
#pragma unroll
        for (int j = 0; j < CB; ++j) bm = fmaxf(bm, l[j]);
        if (bm == -INFINITY) continue;
        if (bm > mx) {
            if (mx != -INFINITY) {
                const float r = __builtin_amdgcn_exp2f(mx - bm);
#pragma unroll
                for (int k = 0; k < CV; ++k) acc[k] *= r;
                wsum *= r;
            }
            mx = bm;
        }
#pragma unroll
        for (int j = 0; j < CB; ++j) {
            if (l[j] == -INFINITY) continue;
            const float w = __builtin_amdgcn_exp2f(l[j] - mx);
#pragma unroll
            for (int k = 0; k < CV; ++k) acc[k] += w * v[j][k];
            wsum += w;
        }
    }
    const float inv = wsum > 0.f ? 1.f / wsum : 0.f;
    const int64_t oofs = (int64_t)layer * a.o_stride[0] + row * a.o_stride[1] + (int64_t)head * a.o_stride[2] + c0 * 4;
#pragma unroll
    for (int k = 0; k < CV; ++k) {
        if (a.dtype == 1) {
            *(f32x4*)((float*)a.out + oofs + k * 4) =
                f32x4{acc[k][0] * inv, acc[k][1] * inv, acc[k][2] * inv, acc[k][3] * inv};
        } else {
            u32x2 w;
            w[0] = bf_rne(acc[k][0] * inv) | (bf_rne(acc[k][1] * inv) << 16);
            w[1] = bf_rne(acc[k][2] * inv) | (bf_rne(acc[k][3] * inv) << 16);
            *(u32x2*)((uint16_t*)a.out + oofs + k * 4) = w;
        }
    }
    if (a.lse_out && c0 == 0)
        a.lse_out[item] = wsum > 0.f ? (mx + __log2f(wsum)) * kLn2 : -INFINITY;
}

Plan make_plan(const AttnArgs& a, int splits) {
    Plan p;
    p.G = a.n_heads / a.n_kv_heads;
    const int64_t m_rows = (int64_t)a.max_q * p.G;
    if (a.variant == 1) {
        // MLA: four waves of 32 whole rows; 32-key tiles in 2 LDS stages.
        p.qb = 1;
        p.nw = 4;
        p.ns = 2;
    } else {
        // bf16 GQA: 4 waves x 32 rows, two workgroups per CU, pipelined over
        // 32-key tiles in 4 LDS stages.  (The fp32 kernel also uses 32-key
        // tiles.)
        p.qb = 1;
        p.nw = 4;
        p.ns = 4;
    }
    p.BM = a.dtype == 1 ? 64 : p.nw * 32 * p.qb;
    p.rbs = (int)((m_rows + p.BM - 1) / p.BM);
    if (p.rbs < 1) p.rbs = 1;
    p.splits = splits;
    p.n_groups = a.n_layers * a.n_kv_heads * a.n_seqs * splits;
    return p;
}

// Workgroups that fit on one CU at once (LDS and register bound).
int wgs_per_cu(const AttnArgs& a, const Plan& p) {
    if (a.variant == 1) return 1;                     // MLA: two 36 KB stages, one wave per SIMD
    const int tile = 32;                              // keys per K/V tile
    const int lds = p.ns * 2 * tile * a.head_dim * 2;
    const int n = (160 * 1024) / lds;
    return n < 1 ? 1 : (n > 2 ? 2 : n);               // two waves per SIMD at most (registers)
}

}  // namespace

int attention_splits(const AttnArgs& a) {
    if (a.n_splits > 0) {
        int s = a.n_splits;
        const int max_s = (a.max_kv_len + 63) / 64;
        if (s > max_s) s = max_s < 1 ? 1 : max_s;
        return s;
    }
    // Pick the split count that minimises the estimated time: the workgroup
    // rounds over the CUs times the duration of one workgroup (a fixed cost
    // for its start-up, first loads and partial write, plus 1/s of the keys),
    // plus, for s > 1, the split partials written and read back by the
    // combine pass.  Nominal rates (measured on MI355X): the bf16 kernels
    // sustain about 1.0 PFLOP/s (GQA) and 1.1 PFLOP/s (MLA), a workgroup's
    // fixed cost is about 20 us, the combine streams at about 5 TB/s.  At
    // least 512 keys per split, at most 32 splits.
    const Plan p = make_plan(a, 1);
    const int64_t wgs = (int64_t)p.n_groups * p.rbs;   // workgroups per split
    // Keys one workgroup's rows see: with a sliding window, about the window
    // plus the span of the queries (contiguous suffix positions).
    const int64_t kv = a.window > 0 && (int64_t)a.window + a.max_q < a.max_kv_len ? (int64_t)a.window + a.max_q
                                                                                  : a.max_kv_len;
    if (a.dtype == 1) {
        // fp32 path (small problems): one workgroup per CU, at least 64 keys
        // per split, at most 32 splits.
        int64_t s = (kCUs + wgs - 1) / wgs;
        const int64_t max_s = kv / 64;
        if (s > max_s) s = max_s;
        if (s > 32) s = 32;
        return s < 1 ? 1 : (int)s;
    }
    const int64_t slots = kCUs * (int64_t)wgs_per_cu(a, p);
    const double rate = a.variant == 1 ? 1.1e15 : 1.0e15;
    const double slot_rate = rate / (double)slots;
    const double wg_flops = (double)p.BM * kv * (a.head_dim + a.head_dim_v) * 2.0;
    const double comb_bytes = (double)a.n_layers * a.total_q * a.n_heads * (a.head_dim_v + 1) * 4.0 * 2.0;
    int best = 1;
    double best_t = 1e30;
    for (int s = 1; s <= 32; ++s) {
        if (s > 1 && kv / s < 512) break;
        const double rounds = (double)((wgs * s + slots - 1) / slots);
        const double t = rounds * (20e-6 + (wg_flops / s) / slot_rate) + (s > 1 ? s * comb_bytes / 5e12 + 5e-6 : 0.0);
        if (t < best_t * (1.0 - 1e-9)) {
            best_t = t;
            best = s;
        }
    }
    return best;
}

size_t attention_workspace_bytes(const AttnArgs& a, int n_splits) {
    if (n_splits <= 1) return 0;
    const size_t rows = (size_t)n_splits * a.n_layers * a.total_q * a.n_heads;
    return rows * a.head_dim_v * sizeof(float) + rows * sizeof(float);
}

hipError_t launch_attention(const AttnArgs& a, hipStream_t stream) {
    const Plan p = make_plan(a, a.n_splits < 1 ? 1 : a.n_splits);
    const int64_t groups_padded = ((int64_t)p.n_groups + kXcds - 1) / kXcds * kXcds;
    const int64_t n_wg = groups_padded * p.rbs;
    if (n_wg <= 0) return hipSuccess;
    if (n_wg > 0x7fffffff) return hipErrorInvalidValue;
    dim3 grid((unsigned)n_wg), block(256);   // the bf16 launchers set their own block size
    hipError_t e;
    if (a.dtype == 1) {
        if (a.head_dim == 64)
            hipLaunchKernelGGL((attn_gqa_f32<64>), grid, dim3(128), 0, stream, a, p);
        else
            hipLaunchKernelGGL((attn_gqa_f32<128>), grid, dim3(128), 0, stream, a, p);
        e = hipGetLastError();
    } else {
        e = a.variant == 1 ? launch_attn_mla_bf16(a, p, grid, stream) : launch_attn_gqa_bf16(a, p, grid, stream);
    }
    if (e != hipSuccess || p.splits == 1) return e;
    // One (row tiles, sequences, layers) grid per 65535 sequences.
    const int64_t threads = (int64_t)a.max_q * a.n_heads * (a.head_dim_v / (4 * kCombineCV));
    if (threads == 0 || a.n_layers == 0 || a.n_seqs == 0) return hipSuccess;
    if (a.head_dim_v % (4 * kCombineCV) || threads > 0xffffffffLL || a.n_layers > 65535) return hipErrorInvalidValue;
    for (int seq0 = 0; seq0 < a.n_seqs; seq0 += 65535) {
        const int nseq = a.n_seqs - seq0 < 65535 ? a.n_seqs - seq0 : 65535;
        dim3 cgrid((unsigned)((threads + 255) / 256), (unsigned)nseq, (unsigned)a.n_layers);
        hipLaunchKernelGGL(attn_combine, cgrid, block, 0, stream, a, seq0);
        e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    return hipSuccess;
}

}  // namespace pkv
