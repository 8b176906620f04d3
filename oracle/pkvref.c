/*
 * pkvref — plain, slow fp64 CPU oracle for RoPE reposition+splice and causal
 * suffix attention over a spliced KV cache.
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing in the product library includes, links or
 * calls this file; only the test suite, the smoke check and the CPU-baseline
 * leg of the benchmark use it.  It shares no code, header or constant with the
 * HIP path.
 *
 * What it computes (the plain definitions, written out in fp64):
 *   - RoPE (paper, Related work: repositioning relies on rotary position
 *     embeddings).  The paper does not spell out the pairing or the frequency
 *     schedule; this oracle takes the standard reading
 *         omega_i = theta^(-2i/r),  i in [0, r/2)
 *     and a pair (a, b) at position p maps to
 *         (a cos(p omega_i) - b sin(p omega_i),  a sin(p omega_i) + b cos(p omega_i)).
 *     HALF pairing: (a, b) = (x[o+i], x[o+i+r/2]); INTERLEAVED: (x[o+2i], x[o+2i+1]).
 *     Channels outside [o, o+r) are untouched.
 *     An explicit per-pair table omega[i] may replace the theta schedule: the
 *     paper's repositioning also covers the RoPE extensions (Related work:
 *     rotary embeddings and their extensions), i.e. rescaled frequencies, and
 *     M-RoPE, whose rotary pairs belong to temporal / height / width axes
 *     (Sec. 8 "Multimodal"; Fig. "attention-variant adapters" (b)): moving an
 *     image along the trajectory re-rotates only the temporal pairs, which is
 *     the table with omega[i] = 0 on the spatial pairs.
 *   - Reposition + splice (Sec. 5, "From mechanism to prediction"; Fig. "Two
 *     cache operations" (b); App. B skill example): the cached keys are
 *     post-RoPE, so a chunk cached at source positions is moved to target
 *     positions by rotating each key by delta = dst_pos - src_pos and writing it
 *     to the destination slot dst_pos; values carry no position and are copied
 *     unchanged.  MLA adapter (Sec. 8 and Fig. "attention-variant adapters"
 *     (a)): only the decoupled k_pe slice rotates, the latent is copied as-is.
 *   - Causal attention of the suffix/erratum queries over the spliced cache
 *     (Sec. 5 "Linear-time TTFT": a re-rotation pass plus the suffix):
 *         o = sum_j softmax_j(scale <q, k_j>) v_j over visible slots
 *         j < kv_len and j <= q_pos.
 *
 * Arithmetic: every stored input is read exactly (bf16 and fp32 both embed in
 * fp64), all arithmetic is fp64 with libm cos/sin/exp/pow, and a stored
 * output is rounded once, round-to-nearest-even, directly from fp64.
 * Attention outputs are returned unrounded in fp64.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#define REF_BF16 0
#define REF_F32 1
#define REF_HALF 0
#define REF_INTERLEAVED 1

/* ---- storage formats --------------------------------------------------- */

static double ref_load(const void* base, int dtype, int64_t i) {
    if (dtype == REF_BF16) {
        uint16_t h = ((const uint16_t*)base)[i];
        uint32_t u = (uint32_t)h << 16;
        float f;
        memcpy(&f, &u, sizeof f);
        return (double)f;
    }
    return (double)((const float*)base)[i];
}

/* fp64 -> bf16 bits, one rounding, ties to even.  bf16 keeps 8 significant
 * bits and the fp32 exponent range (normal exponents -126..127). */
uint16_t pkvref_round_bf16(double x) {
    if (isnan(x)) return 0x7fc0;
    uint16_t sign = signbit(x) ? 0x8000 : 0x0000;
    double a = fabs(x);
    if (a == 0.0) return sign;
    int e;
    frexp(a, &e);          /* a = f * 2^e, f in [0.5, 1) => 2^(e-1) <= a < 2^e */
    int ue = e - 1;        /* exponent of the leading bit */
    if (ue < -126) ue = -126;               /* subnormal range: fixed quantum */
    double quantum = ldexp(1.0, ue - 7);    /* spacing of bf16 values here */
    double q = a / quantum;                 /* exact: power-of-two scaling */
    double r = nearbyint(q);                /* default rounding mode: ties to even */
    double v = r * quantum;                 /* exact */
    if (v >= ldexp(1.0, 128)) return (uint16_t)(sign | 0x7f80);   /* overflow to inf */
    float f = (float)v;                      /* exact: v has at most 8 significant bits */
    uint32_t u;
    memcpy(&u, &f, sizeof u);
    return (uint16_t)(sign | ((u >> 16) & 0x7fff));
}

static void ref_store(void* base, int dtype, int64_t i, double v) {
    if (dtype == REF_BF16)
        ((uint16_t*)base)[i] = pkvref_round_bf16(v);
    else
        ((float*)base)[i] = (float)v;   /* one IEEE rounding, ties to even */
}

static void ref_copy_elem(void* dst, const void* src, int dtype, int64_t di, int64_t si) {
    if (dtype == REF_BF16)
        ((uint16_t*)dst)[di] = ((const uint16_t*)src)[si];
    else
        memcpy((char*)dst + 4 * di, (const char*)src + 4 * si, 4);   /* bit pattern */
}

/* ---- RoPE --------------------------------------------------------------- */

/* Rotary frequency of pair i for rotary width r. */
double pkvref_rope_omega(double theta, int r, int i) {
    return pow(theta, -2.0 * (double)i / (double)r);
}

/* Channel indices of pair i inside the rotary slice [o, o+r). */
static void ref_pair_index(int style, int o, int r, int i, int* ia, int* ib) {
    if (style == REF_HALF) {
        *ia = o + i;
        *ib = o + i + r / 2;
    } else {
        *ia = o + 2 * i;
        *ib = o + 2 * i + 1;
    }
}

/* Rotate one row of d channels by position multiple p:
 * out = R(p) in, channels outside the rotary slice copied bit-exact.
 * in and out may be different arrays; in_off/out_off are element offsets. */
static void ref_rotate_row(int dtype, const void* in, int64_t in_off, void* out, int64_t out_off,
                           int d, double p, double theta, int r, int o, int style, const double* omega) {
    for (int c = 0; c < d; ++c)
        if (c < o || c >= o + r) ref_copy_elem(out, in, dtype, out_off + c, in_off + c);
    for (int i = 0; i < r / 2; ++i) {
        int ia, ib;
        ref_pair_index(style, o, r, i, &ia, &ib);
        double ang = p * (omega ? omega[i] : pkvref_rope_omega(theta, r, i));
        double cs = cos(ang), sn = sin(ang);
        double a = ref_load(in, dtype, in_off + ia);
        double b = ref_load(in, dtype, in_off + ib);
        ref_store(out, dtype, out_off + ia, a * cs - b * sn);
        ref_store(out, dtype, out_off + ib, a * sn + b * cs);
    }
}

/* RoPE at per-row positions: out[row] = R(pos[row]) in[row] for rows laid out
 * contiguously with n_rows x d elements.  Used to build post-RoPE keys and
 * queries from pre-RoPE draws.  omega: NULL (theta schedule) or rope_dim/2
 * per-pair frequencies. */
void pkvref_rope_rows(int dtype, const void* in, void* out, int64_t n_rows, int d,
                      const int32_t* pos, double theta, int rope_dim, int rope_offset, int style,
                      const double* omega) {
#pragma omp parallel for schedule(static)
    for (int64_t row = 0; row < n_rows; ++row)
        ref_rotate_row(dtype, in, row * d, out, row * d, d, (double)pos[row], theta, rope_dim,
                       rope_offset, style, omega);
}

/* Reposition + splice.  For every layer l, KV head h and skill token t:
 *     dst_k[l][h][dst_pos[t]] = R(dst_pos[t] - src_pos[t]) src_k[l][h][t]
 *     dst_v[l][h][dst_pos[t]] = src_v[l][h][t]              (bit-exact)
 * Strides are in elements: {layer, head, token}; channels are contiguous.
 * v_dim == 0 means no V tensor (MLA: the latent lives in the K row and is the
 * non-rotary part of it).  A token whose dst_pos falls outside
 * [0, dst_capacity) is skipped; the return value counts skipped tokens.
 * omega: NULL (theta schedule) or rope_dim/2 per-pair frequencies.
 * dst_slot: NULL (the destination slot is dst_pos[t]) or the slot of each
 * token, for layouts where positions and cache slots differ (M-RoPE images,
 * whose tokens share one temporal position). */
int64_t pkvref_reposition_splice(int dtype, const void* src_k, const void* src_v, void* dst_k,
                                 void* dst_v, const int32_t* src_pos, const int32_t* dst_pos,
                                 int64_t n_tokens, int n_layers, int n_kv_heads, int head_dim,
                                 int v_dim, double theta, int rope_dim, int rope_offset, int style,
                                 const int64_t* src_k_stride, const int64_t* src_v_stride,
                                 const int64_t* dst_k_stride, const int64_t* dst_v_stride,
                                 int64_t dst_capacity, const double* omega, const int32_t* dst_slot) {
    int64_t skipped = 0;
    for (int64_t t = 0; t < n_tokens; ++t) {
        int64_t slot = dst_slot ? dst_slot[t] : dst_pos[t];
        if (slot < 0 || slot >= dst_capacity) ++skipped;
    }
#pragma omp parallel for collapse(2) schedule(static)
    for (int l = 0; l < n_layers; ++l) {
        for (int h = 0; h < n_kv_heads; ++h) {
            for (int64_t t = 0; t < n_tokens; ++t) {
                int64_t slot = dst_slot ? dst_slot[t] : dst_pos[t];
                if (slot < 0 || slot >= dst_capacity) continue;
                double delta = (double)dst_pos[t] - (double)src_pos[t];
                int64_t sk = l * src_k_stride[0] + h * src_k_stride[1] + t * src_k_stride[2];
                int64_t dk = l * dst_k_stride[0] + h * dst_k_stride[1] + slot * dst_k_stride[2];
                ref_rotate_row(dtype, src_k, sk, dst_k, dk, head_dim, delta, theta, rope_dim,
                               rope_offset, style, omega);
                if (v_dim > 0) {
                    int64_t sv = l * src_v_stride[0] + h * src_v_stride[1] + t * src_v_stride[2];
                    int64_t dv = l * dst_v_stride[0] + h * dst_v_stride[1] + slot * dst_v_stride[2];
                    for (int c = 0; c < v_dim; ++c) ref_copy_elem(dst_v, src_v, dtype, dv + c, sv + c);
                }
            }
        }
    }
    return skipped;
}

/* Causal attention of n_q queries of one sequence and one layer over a cache.
 *   q:   element (i, h, c) at q[i*q_tok + h*q_head + c], c < d_qk
 *   k:   element (g, j, c) at k[g*k_head + j*k_tok + c],  c < d_qk
 *   v:   element (g, j, c) at v[g*v_head + j*v_tok + c],  c < d_v
 *   out: fp64, element (i, h, c) at out[(i*n_heads + h)*d_v + c]
 *   lse: fp64 [n_q*n_heads] (optional), natural-log sum-exp of scaled scores
 * Query head h reads KV head h / (n_heads / n_kv_heads).  Slot j is visible to
 * query i iff j < kv_len and j <= q_pos[i], and, for window > 0, also
 * j > q_pos[i] - window: the sliding-window layers keep the full per-token
 * cache and the mask alone enforces the window (Sec. 8, the sliding-window
 * configuration fix; Fig. "attention-variant adapters" (c)).  A row with no
 * visible slot gets out = 0 and lse = -inf. */
void pkvref_attention(int dtype, const void* q, const void* k, const void* v, double* out,
                      double* lse, const int32_t* q_pos, int64_t n_q, int64_t kv_len, int n_heads,
                      int n_kv_heads, int d_qk, int d_v, double scale, int64_t q_tok,
                      int64_t q_head, int64_t k_head, int64_t k_tok, int64_t v_head,
                      int64_t v_tok, int64_t window) {
    int group = n_heads / n_kv_heads;
#pragma omp parallel for collapse(2) schedule(dynamic, 1)
    for (int64_t i = 0; i < n_q; ++i) {
        for (int h = 0; h < n_heads; ++h) {
            int g = h / group;
            /* visible slots lo .. hi-1 */
            int64_t hi = kv_len;
            if ((int64_t)q_pos[i] + 1 < hi) hi = (int64_t)q_pos[i] + 1;
            int64_t lo = 0;
            if (window > 0 && (int64_t)q_pos[i] - window + 1 > lo) lo = (int64_t)q_pos[i] - window + 1;
            int64_t n_vis = hi - lo;
            if (n_vis < 0) n_vis = 0;
            double* o = out + (i * n_heads + h) * d_v;
            for (int c = 0; c < d_v; ++c) o[c] = 0.0;
            if (n_vis == 0) {
                if (lse) lse[i * n_heads + h] = -INFINITY;
                continue;
            }
            /* scaled scores over the visible slots and their maximum */
            double* sc = (double*)malloc((size_t)n_vis * sizeof(double));
            double m = -INFINITY;
            for (int64_t j = 0; j < n_vis; ++j) {
                double s = 0.0;
                for (int c = 0; c < d_qk; ++c)
                    s += ref_load(q, dtype, i * q_tok + h * q_head + c) *
                         ref_load(k, dtype, g * k_head + (lo + j) * k_tok + c);
                sc[j] = s * scale;
                if (sc[j] > m) m = sc[j];
            }
            /* softmax weights (shifted by the maximum) and the weighted sum of values */
            double sum = 0.0;
            for (int64_t j = 0; j < n_vis; ++j) {
                double w = exp(sc[j] - m);
                sum += w;
                for (int c = 0; c < d_v; ++c) o[c] += w * ref_load(v, dtype, g * v_head + (lo + j) * v_tok + c);
            }
            free(sc);
            for (int c = 0; c < d_v; ++c) o[c] /= sum;
            if (lse) lse[i * n_heads + h] = m + log(sum);
        }
    }
}

int pkvref_max_threads(void) {
#ifdef _OPENMP
    extern int omp_get_max_threads(void);
    return omp_get_max_threads();
#else
    return 1;
#endif
}

void pkvref_set_threads(int n) {
#ifdef _OPENMP
    extern void omp_set_num_threads(int);
    omp_set_num_threads(n);
#else
    (void)n;
#endif
}
