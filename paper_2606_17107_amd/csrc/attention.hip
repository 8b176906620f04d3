// Causal attention of suffix / erratum queries over a spliced KV cache
// (paper Sec. 5 "Linear-time TTFT": the transplant costs a re-rotation pass
// plus the suffix; Sec. 6: the agent prefills only the delta).
//
// bf16 GQA kernel (gfx950, wave64, MFMA 32x32x16 bf16 -> fp32):
//   * Rows of the MFMA "N" dimension are (query, head-in-group) pairs of one
//     KV head: row m <-> query m / G, head kv_head*G + m % G, so every K/V byte
//     staged in LDS serves BM rows.  A workgroup is 4 waves x 32 rows.
//   * Scores are computed transposed, S^T = K Q^T (keys on the MFMA M axis).
//     A lane then holds 16 keys of ONE query row, so the row max needs one
//     cross-lane step (the two lanes sharing a column) and the row sum none
//     until the end.  The fp32 probabilities P^T sit in the accumulator in
//     exactly the lane layout the next MFMA wants for its B operand, so
//     O^T = V^T P^T runs with no LDS round trip for P.
//   * V is staged in LDS transposed ([channel][key]) with the keys of every
//     16-key step permuted so that a lane's eight A-operand keys are
//     contiguous (one 16-byte LDS read).
//   * Split-KV: a workgroup covers one key range of one (layer, kv head,
//     sequence, row block); partial (O, log-sum-exp) go to the workspace and a
//     combine kernel merges them.
//   * XCD-aware order: all row blocks that read the same K/V range are given
//     workgroup ids with the same residue mod 8, so they run on one XCD and
//     share its L2.
#include <math.h>

#include "pkv_internal.h"

namespace pkv {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

constexpr int kXcds = 8;
constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;

struct Plan {
    int G;          // query heads per KV head
    int BM;         // rows per workgroup
    int rbs;        // row blocks per group
    int n_groups;   // layers x kv heads x sequences x splits
    int splits;
    int chunk;      // keys per split (multiple of the key tile)
};

// Decode a workgroup id into (group, row block) so that the row blocks of a
// group share an XCD.
__device__ inline bool decode(const Plan& p, int& group, int& rb) {
    const int id = blockIdx.x;
    const int xcd = id % kXcds;
    const int slot = id / kXcds;
    rb = slot % p.rbs;
    group = (slot / p.rbs) * kXcds + xcd;
    return group < p.n_groups;
}

struct SeqInfo {
    int q0, nq, kvl;
    int64_t base;
};

__device__ inline SeqInfo seq_info(const AttnArgs& a, int seq) {
    SeqInfo s;
    if (a.cu_q) {
        s.q0 = a.cu_q[seq];
        s.nq = a.cu_q[seq + 1] - s.q0;
    } else {
        s.q0 = 0;
        s.nq = a.total_q;
    }
    // Keep every row and slot index inside the tensors the caller described.
    if (s.q0 < 0 || s.nq < 0 || (int64_t)s.q0 + s.nq > a.total_q) s.nq = 0;
    s.base = a.kv_base ? a.kv_base[seq] : 0;
    int64_t kvl = a.kv_len[seq];
    if (s.base < 0) kvl = 0;
    if (kvl > a.max_kv_len) kvl = a.max_kv_len;
    if (kvl > a.cache_slots - s.base) kvl = a.cache_slots - s.base;
    if (kvl < 0) kvl = 0;
    s.kvl = (int)kvl;
    return s;
}

__device__ inline float wave_max(float v) {
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) v = fmaxf(v, __shfl_xor(v, o));
    return v;
}
__device__ inline int wave_max_i(int v) {
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) v = max(v, __shfl_xor(v, o));
    return v;
}
__device__ inline int wave_min_i(int v) {
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) v = min(v, __shfl_xor(v, o));
    return v;
}

__device__ inline uint32_t bf_rne(float f) {
    uint32_t u = __float_as_uint(f);
    u += 0x7fffu + ((u >> 16) & 1u);
    return u >> 16;
}

// Position of key k (0..63) of a tile inside its LDS V^T row: within each
// 16-key step, lane-half h reads 8 contiguous slots holding keys
// {4h..4h+3, 8+4h..8+4h+3} — the keys its P^T accumulator entries belong to.
__device__ inline int vt_slot(int k) {
    const int st = k >> 4, kk = k & 15;
    const int b = kk >> 3, h = (kk >> 2) & 1, c = kk & 3;
    return (st << 4) + (h << 3) + (b << 2) + c;
}

template <int D>
__global__ __launch_bounds__(256, 2) void attn_gqa_bf16(AttnArgs a, Plan p) {
    constexpr int BN = 64;            // keys per tile
    constexpr int KST = D + 8;        // LDS row stride of K (elements), 16-byte multiple + 16
    constexpr int VST = BN + 8;       // LDS row stride of V^T
    constexpr int KS = D / 16;        // MFMA k-steps over channels
    constexpr int DB = D / 32;        // 32-channel output blocks
    __shared__ __attribute__((aligned(16))) uint16_t k_lds[BN * KST];
    __shared__ __attribute__((aligned(16))) uint16_t v_lds[D * VST];
    __shared__ int red[8];

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
    const int m0 = rb * p.BM;
    if (m0 >= M) return;

    const int tid = threadIdx.x;
    const int wave = tid >> 6;
    const int lane = tid & 63;
    const int j = lane & 31;
    const int hl = lane >> 5;

    // This lane's query row.
    const int m = m0 + wave * 32 + j;
    const bool row_ok = m < M;
    const int qi = row_ok ? m / p.G : 0;
    const int head = kvh * p.G + (row_ok ? m - qi * p.G : 0);
    const int qpos = row_ok ? a.q_pos[si.q0 + qi] : -1;
    const int row_end = row_ok ? max(0, min(si.kvl, qpos + 1)) : 0;   // visible keys [0, row_end)

    const int k_begin = split * p.chunk;
    const int k_end = min(si.kvl, k_begin + p.chunk);
    // Workgroup-wide last visible key and per-wave first masked key.
    const int wmax = wave_max_i(row_end);
    const int wmin = wave_min_i(row_ok ? row_end : 0x7fffffff);
    if (lane == 0) red[wave] = wmax;
    __syncthreads();
    const int e_max = max(max(red[0], red[1]), max(red[2], red[3]));
    const int loop_end = min(k_end, e_max);

    // Q^T operand: 8 channels per k-step.
    const uint16_t* qrow = (const uint16_t*)a.q + (int64_t)layer * a.q_stride[0] +
                           (int64_t)(si.q0 + qi) * a.q_stride[1] + (int64_t)head * a.q_stride[2];
    bf16x8 qf[KS];
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
        u32x4 v = {0u, 0u, 0u, 0u};
        if (row_ok) v = *(const u32x4*)(qrow + ks * 16 + hl * 8);
        qf[ks] = __builtin_bit_cast(bf16x8, v);
    }

    f32x16 o[DB];
#pragma unroll
    for (int db = 0; db < DB; ++db) o[db] = f32x16{};
    float m_run = -INFINITY, l_run = 0.f;
    const float sc2 = a.scale * kLog2e;

    const uint16_t* kbase = (const uint16_t*)a.k + (int64_t)layer * a.k_stride[0] +
                            (int64_t)kvh * a.k_stride[1] + si.base * a.k_stride[2];
    const uint16_t* vbase = (const uint16_t*)a.v + (int64_t)layer * a.v_stride[0] +
                            (int64_t)kvh * a.v_stride[1] + si.base * a.v_stride[2];

    for (int t0 = k_begin; t0 < loop_end; t0 += BN) {
        __syncthreads();
        // K tile -> LDS, row-major with padding.
        constexpr int KCH = D / 8;   // 16-byte chunks per row
#pragma unroll
        for (int i = 0; i < BN * KCH / 256; ++i) {
            const int id = tid + i * 256;
            const int key = id / KCH, c = id % KCH;
            u32x4 v = {0u, 0u, 0u, 0u};
            if (t0 + key < loop_end) v = *(const u32x4*)(kbase + (int64_t)(t0 + key) * a.k_stride[2] + c * 8);
            *(u32x4*)(k_lds + key * KST + c * 8) = v;
        }
        // V tile -> LDS transposed; each thread moves two adjacent keys so it can
        // write packed pairs.
#pragma unroll
        for (int i = 0; i < (BN / 2) * KCH / 256; ++i) {
            const int id = tid + i * 256;
            const int pr = id % (BN / 2), c = id / (BN / 2);
            const int k0 = 2 * pr;
            u32x4 v0 = {0u, 0u, 0u, 0u}, v1 = {0u, 0u, 0u, 0u};
            if (t0 + k0 < loop_end) v0 = *(const u32x4*)(vbase + (int64_t)(t0 + k0) * a.v_stride[2] + c * 8);
            if (t0 + k0 + 1 < loop_end)
                v1 = *(const u32x4*)(vbase + (int64_t)(t0 + k0 + 1) * a.v_stride[2] + c * 8);
            const int slot = vt_slot(k0);
#pragma unroll
            for (int w = 0; w < 4; ++w) {
                // channels 8c+2w (low halves) and 8c+2w+1 (high halves)
                const uint32_t lo = (v0[w] & 0xffffu) | (v1[w] << 16);
                const uint32_t hi = (v0[w] >> 16) | (v1[w] & 0xffff0000u);
                *(uint32_t*)(v_lds + (c * 8 + 2 * w) * VST + slot) = lo;
                *(uint32_t*)(v_lds + (c * 8 + 2 * w + 1) * VST + slot) = hi;
            }
        }
        __syncthreads();

        // S^T = K Q^T for two 32-key blocks.
        f32x16 s[2];
#pragma unroll
        for (int kb = 0; kb < 2; ++kb) {
            s[kb] = f32x16{};
#pragma unroll
            for (int ks = 0; ks < KS; ++ks) {
                const u32x4 kv = *(const u32x4*)(k_lds + (kb * 32 + j) * KST + ks * 16 + hl * 8);
                s[kb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, kv), qf[ks],
                                                                 s[kb], 0, 0, 0);
            }
        }
        // Scale to log2 units and mask keys this row cannot see.
        const bool need_mask = t0 + BN > wmin;
        float mx = -INFINITY;
#pragma unroll
        for (int kb = 0; kb < 2; ++kb) {
#pragma unroll
            for (int r = 0; r < 16; ++r) {
                float v = s[kb][r] * sc2;
                if (need_mask) {
                    const int key = t0 + kb * 32 + (r >> 2) * 8 + hl * 4 + (r & 3);
                    if (key >= row_end) v = -INFINITY;
                }
                s[kb][r] = v;
                mx = fmaxf(mx, v);
            }
        }
        mx = fmaxf(mx, __shfl_xor(mx, 32));
        const float m_new = fmaxf(m_run, mx);
        const float m_use = m_new == -INFINITY ? 0.f : m_new;
        const float alpha = __builtin_amdgcn_exp2f(m_run - m_use);
        float lsum = 0.f;
#pragma unroll
        for (int kb = 0; kb < 2; ++kb) {
#pragma unroll
            for (int r = 0; r < 16; ++r) {
                const float e = __builtin_amdgcn_exp2f(s[kb][r] - m_use);
                s[kb][r] = e;
                lsum += e;
            }
        }
        l_run = l_run * alpha + lsum;
        m_run = m_new;
#pragma unroll
        for (int db = 0; db < DB; ++db) o[db] *= alpha;

        // O^T += V^T P^T over four 16-key steps.
#pragma unroll
        for (int st = 0; st < BN / 16; ++st) {
            const int kb = st >> 1, sub = st & 1;
            u32x4 pw;
#pragma unroll
            for (int w = 0; w < 4; ++w)
                pw[w] = bf_rne(s[kb][sub * 8 + 2 * w]) | (bf_rne(s[kb][sub * 8 + 2 * w + 1]) << 16);
            const bf16x8 pb = __builtin_bit_cast(bf16x8, pw);
#pragma unroll
            for (int db = 0; db < DB; ++db) {
                const u32x4 vv = *(const u32x4*)(v_lds + (db * 32 + j) * VST + st * 16 + hl * 8);
                o[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, vv), pb, o[db],
                                                                 0, 0, 0);
            }
        }
    }

    // Finish the row: the two lanes of a column hold disjoint partial sums.
    const float l_tot = l_run + __shfl_xor(l_run, 32);
    if (!row_ok) return;
    const float inv = l_tot > 0.f ? 1.f / l_tot : 0.f;
    const float lse2 = l_tot > 0.f ? m_run + __log2f(l_tot) : -INFINITY;   // log2 units
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
        if (a.lse_out && hl == 0)
            a.lse_out[((int64_t)layer * a.total_q + row) * a.n_heads + head] = lse2 * kLn2;
    } else {
        const int64_t item = (((int64_t)split * a.n_layers + layer) * a.total_q + row) * a.n_heads + head;
        float* wo = a.ws_o + item * D;
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

// fp32 GQA kernel: four lanes per row, each holding D/4 channels of q and o;
// K/V tiles staged in LDS; exact fp32 online softmax per key.
template <int D>
__global__ __launch_bounds__(256) void attn_gqa_f32(AttnArgs a, Plan p) {
    constexpr int BN = 32;
    constexpr int DQ = D / 4;
    __shared__ float k_lds[BN * D];
    __shared__ float v_lds[BN * D];
    __shared__ int red[4];

    int group, rb;
    if (!decode(p, group, rb)) return;
    int rest = group;   // one split
    const int kvh = rest % a.n_kv_heads;
    rest /= a.n_kv_heads;
    const int layer = rest % a.n_layers;
    const int seq = rest / a.n_layers;
    const SeqInfo si = seq_info(a, seq);
    const int M = si.nq * p.G;
    const int m0 = rb * 64;
    if (m0 >= M) return;

    const int tid = threadIdx.x;
    const int r = tid >> 2, part = tid & 3;
    const int m = m0 + r;
    const bool row_ok = m < M;
    const int qi = row_ok ? m / p.G : 0;
    const int head = kvh * p.G + (row_ok ? m - qi * p.G : 0);
    const int qpos = row_ok ? a.q_pos[si.q0 + qi] : -1;
    const int row_end = row_ok ? max(0, min(si.kvl, qpos + 1)) : 0;
    const int wmax = wave_max_i(row_end);
    if ((tid & 63) == 0) red[tid >> 6] = wmax;
    __syncthreads();
    const int loop_end = max(max(red[0], red[1]), max(red[2], red[3]));

    const float* qrow = (const float*)a.q + (int64_t)layer * a.q_stride[0] +
                        (int64_t)(si.q0 + qi) * a.q_stride[1] + (int64_t)head * a.q_stride[2] + part * DQ;
    float qv[DQ], ov[DQ];
#pragma unroll
    for (int c = 0; c < DQ; ++c) {
        qv[c] = row_ok ? qrow[c] * a.scale : 0.f;
        ov[c] = 0.f;
    }
    float m_run = -INFINITY, l_run = 0.f;
    const float* kbase = (const float*)a.k + (int64_t)layer * a.k_stride[0] + (int64_t)kvh * a.k_stride[1] +
                         si.base * a.k_stride[2];
    const float* vbase = (const float*)a.v + (int64_t)layer * a.v_stride[0] + (int64_t)kvh * a.v_stride[1] +
                         si.base * a.v_stride[2];
    for (int t0 = 0; t0 < loop_end; t0 += BN) {
        __syncthreads();
        for (int id = tid; id < BN * D / 4; id += 256) {
            const int key = id / (D / 4), c = id % (D / 4);
            f32x4 kv = {0.f, 0.f, 0.f, 0.f}, vv = {0.f, 0.f, 0.f, 0.f};
            if (t0 + key < loop_end) {
                kv = *(const f32x4*)(kbase + (int64_t)(t0 + key) * a.k_stride[2] + c * 4);
                vv = *(const f32x4*)(vbase + (int64_t)(t0 + key) * a.v_stride[2] + c * 4);
            }
            *(f32x4*)(k_lds + key * D + c * 4) = kv;
            *(f32x4*)(v_lds + key * D + c * 4) = vv;
        }
        __syncthreads();
        const int n = min(BN, loop_end - t0);
        for (int kk = 0; kk < n; ++kk) {
            float s = 0.f;
#pragma unroll
            for (int c = 0; c < DQ; ++c) s = fmaf(qv[c], k_lds[kk * D + part * DQ + c], s);
            s += __shfl_xor(s, 1);
            s += __shfl_xor(s, 2);
            if (t0 + kk >= row_end) continue;   // invisible to this row (uniform over its 4 lanes)
            const float m_new = fmaxf(m_run, s);
            const float alpha = expf(m_run - m_new);
            const float pe = expf(s - m_new);
            l_run = l_run * alpha + pe;
#pragma unroll
            for (int c = 0; c < DQ; ++c) ov[c] = fmaf(ov[c], alpha, pe * v_lds[kk * D + part * DQ + c]);
            m_run = m_new;
        }
    }
    if (!row_ok) return;
    const float inv = l_run > 0.f ? 1.f / l_run : 0.f;
    const int64_t row = si.q0 + qi;
    float* orow = (float*)a.out + (int64_t)layer * a.o_stride[0] + row * a.o_stride[1] +
                  (int64_t)head * a.o_stride[2] + part * DQ;
#pragma unroll
    for (int c = 0; c < DQ; ++c) orow[c] = ov[c] * inv;
    if (a.lse_out && part == 0)
        a.lse_out[((int64_t)layer * a.total_q + row) * a.n_heads + head] =
            l_run > 0.f ? m_run + logf(l_run) : -INFINITY;
}

// Merge split-KV partials: out = sum_s w_s O_s / sum_s w_s with
// w_s = 2^(lse_s - max lse).  One thread per 4 output channels.
__global__ __launch_bounds__(256) void attn_combine(AttnArgs a) {
    const int dv = a.head_dim_v;
    const int chunks = dv / 4;
    const int64_t items = (int64_t)a.n_layers * a.total_q * a.n_heads;
    const int64_t gid = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    const int64_t item = gid / chunks;
    const int c = (int)(gid % chunks);
    if (item >= items) return;
    const int head = (int)(item % a.n_heads);
    const int64_t lr = item / a.n_heads;
    const int64_t row = lr % a.total_q;
    const int layer = (int)(lr / a.total_q);
    float mx = -INFINITY;
    for (int s = 0; s < a.n_splits; ++s) mx = fmaxf(mx, a.ws_lse[(int64_t)s * items + item]);
    f32x4 acc = {0.f, 0.f, 0.f, 0.f};
    float wsum = 0.f;
    if (mx != -INFINITY) {
        for (int s = 0; s < a.n_splits; ++s) {
            const float l = a.ws_lse[(int64_t)s * items + item];
            if (l == -INFINITY) continue;
            const float w = __builtin_amdgcn_exp2f(l - mx);
            const f32x4 v = *(const f32x4*)(a.ws_o + ((int64_t)s * items + item) * dv + c * 4);
            acc += w * v;
            wsum += w;
        }
    }
    const float inv = wsum > 0.f ? 1.f / wsum : 0.f;
    uint16_t* orow = (uint16_t*)a.out + (int64_t)layer * a.o_stride[0] + row * a.o_stride[1] +
                     (int64_t)head * a.o_stride[2] + c * 4;
    u32x2 w;
    w[0] = bf_rne(acc[0] * inv) | (bf_rne(acc[1] * inv) << 16);
    w[1] = bf_rne(acc[2] * inv) | (bf_rne(acc[3] * inv) << 16);
    *(u32x2*)orow = w;
    if (a.lse_out && c == 0)
        a.lse_out[item] = wsum > 0.f ? (mx + __log2f(wsum)) * kLn2 : -INFINITY;
}

Plan make_plan(const AttnArgs& a, int splits) {
    Plan p;
    p.G = a.n_heads / a.n_kv_heads;
    p.BM = a.dtype == 1 ? 64 : 128;
    const int64_t rows = (int64_t)a.max_q * p.G;
    p.rbs = (int)((rows + p.BM - 1) / p.BM);
    if (p.rbs < 1) p.rbs = 1;
    p.splits = splits;
    p.n_groups = a.n_layers * a.n_kv_heads * a.n_seqs * splits;
    const int tile = 64;
    int chunk = (a.max_kv_len + splits - 1) / splits;
    chunk = (chunk + tile - 1) / tile * tile;
    p.chunk = chunk < tile ? tile : chunk;
    return p;
}

}  // namespace

int attention_splits(const AttnArgs& a) {
    if (a.dtype == 1) return 1;   // fp32 path: one pass over the keys
    if (a.n_splits > 0) {
        int s = a.n_splits;
        const int max_s = (a.max_kv_len + 63) / 64;
        if (s > max_s) s = max_s < 1 ? 1 : max_s;
        return s;
    }
    // Aim for about four workgroups per CU on 256 CUs, with at least 256 keys
    // per split.
    const Plan p = make_plan(a, 1);
    const int64_t wgs = (int64_t)p.n_groups * p.rbs;
    int s = (int)((1024 + wgs - 1) / wgs);
    const int max_s = a.max_kv_len / 256;
    if (s > max_s) s = max_s;
    if (s > 16) s = 16;
    if (s < 1) s = 1;
    return s;
}

size_t attention_workspace_bytes(const AttnArgs& a, int n_splits) {
    if (n_splits <= 1) return 0;
    const size_t rows = (size_t)n_splits * a.n_layers * a.total_q * a.n_heads;
    return rows * a.head_dim_v * sizeof(float) + rows * sizeof(float);
}

hipError_t launch_attention(const AttnArgs& a, hipStream_t stream) {
    if (a.variant != 0) return hipErrorNotSupported;
    const Plan p = make_plan(a, a.n_splits < 1 ? 1 : a.n_splits);
    const int64_t groups_padded = ((int64_t)p.n_groups + kXcds - 1) / kXcds * kXcds;
    const int64_t n_wg = groups_padded * p.rbs;
    if (n_wg <= 0) return hipSuccess;
    if (n_wg > 0x7fffffff) return hipErrorInvalidValue;
    dim3 grid((unsigned)n_wg), block(256);
    if (a.dtype == 1) {
        if (a.head_dim == 64)
            hipLaunchKernelGGL((attn_gqa_f32<64>), grid, block, 0, stream, a, p);
        else
            hipLaunchKernelGGL((attn_gqa_f32<128>), grid, block, 0, stream, a, p);
        return hipGetLastError();
    }
    if (a.head_dim == 64)
        hipLaunchKernelGGL((attn_gqa_bf16<64>), grid, block, 0, stream, a, p);
    else
        hipLaunchKernelGGL((attn_gqa_bf16<128>), grid, block, 0, stream, a, p);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess || p.splits == 1) return e;
    const int64_t threads = (int64_t)a.n_layers * a.total_q * a.n_heads * (a.head_dim_v / 4);
    dim3 cgrid((unsigned)((threads + 255) / 256));
    hipLaunchKernelGGL(attn_combine, cgrid, block, 0, stream, a);
    return hipGetLastError();
}

}  // namespace pkv
