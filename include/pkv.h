/*
 * libpkv — MI355X (gfx950) kernels for moving a precompiled chunk of a
 * post-RoPE KV cache to new positions and for the causal attention of the
 * suffix that follows it.
 *
 * Source of the operations: "Models Take Notes at Prefill: KV Cache Can Be
 * Editable and Composable".
 *   - Sec. 5 ("From mechanism to prediction") and Fig. "Two cache operations"
 *     (b): a chunk's KV is computed once at source positions; because the
 *     cache stores post-RoPE keys, moving it re-rotates every key from its
 *     source position to its target position, values carry no position, and
 *     the result is spliced into the destination cache without a reprefill.
 *     App. B's skill example fixes the source positions 0..L-1 and a target
 *     offset.
 *   - Sec. 8 (MLA adapter) and Fig. "attention-variant adapters" (a): an MLA
 *     cache row holds a latent part with no rotary position and a 64-channel
 *     k_pe part that is rotated; repositioning rotates only k_pe and copies the
 *     latent as-is.
 *   - Sec. 5 ("Linear-time TTFT"): the transplant costs a re-rotation pass plus
 *     the suffix; the suffix (or an appended erratum, Sec. 4) attends causally
 *     over the spliced cache.
 *   - Sec. 8 and Fig. "attention-variant adapters": attention variants that
 *     keep per-token KV carry the operations over.  Hence
 *     pkv_reposition_splice_freqs (explicit per-pair frequencies: rescaled RoPE
 *     schedules, and moving an image by re-rotating only its temporal M-RoPE
 *     channels), pkv_attn_desc.window (sliding-window layers keep the full
 *     cache and change only the mask) and the paged entry points (a vLLM-style
 *     pool of fixed-size pages behind per-sequence block tables).
 *
 * Conventions for every call:
 *   - All tensor and index pointers are DEVICE pointers owned by the caller.
 *     The library never allocates, frees or retains them.
 *   - `stream` is a hipStream_t (NULL = the default stream).  Calls enqueue
 *     work and return; kernel faults surface at the caller's next
 *     synchronisation.  No call synchronises the device.
 *   - Strides are in ELEMENTS.  The channel dimension of every row is
 *     contiguous.
 *   - On a non-OK status nothing was enqueued, and pkv_last_error() returns a
 *     message for the calling thread.
 *   - bf16 is stored as its 16-bit pattern; fp32 as IEEE binary32.
 *
 * RoPE convention (the paper names RoPE but does not write its pairing or
 * frequencies out): pair i of the rotary slice [rope_offset, rope_offset +
 * rope_dim) has frequency omega_i = rope_theta^(-2i/rope_dim), and rotating
 * by an integer position multiple p maps (a, b) to
 * (a cos(p omega_i) - b sin(p omega_i), a sin(p omega_i) + b cos(p omega_i)).
 * PKV_ROPE_HALF pairs channel o+i with o+i+rope_dim/2; PKV_ROPE_INTERLEAVED
 * pairs o+2i with o+2i+1.
 */
#ifndef PKV_H
#define PKV_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define PKV_VERSION 1

typedef enum pkv_status {
    PKV_OK = 0,
    PKV_ERR_NULL = 1,         /* a required pointer is NULL */
    PKV_ERR_SHAPE = 2,        /* inconsistent sizes, rope slice outside the row, workspace too small */
    PKV_ERR_ALIGN = 3,        /* a pointer or stride is not 16-byte aligned */
    PKV_ERR_ALIAS = 4,        /* source and destination memory partially overlap */
    PKV_ERR_UNSUPPORTED = 5,  /* dtype / head size / rope geometry this build does not implement */
    PKV_ERR_DEVICE = 6        /* the HIP runtime refused the launch (message has its text) */
} pkv_status;

enum { PKV_BF16 = 0, PKV_F32 = 1 };
enum { PKV_ROPE_HALF = 0, PKV_ROPE_INTERLEAVED = 1 };
enum { PKV_ATTN_GQA = 0, PKV_ATTN_MLA = 1 };

/* ---------------------------------------------------------------------------
 * Reposition + splice
 * ------------------------------------------------------------------------- */

/* Geometry of one splice.  K tensors are indexed [layer][kv_head][slot][channel]
 * through the strides below (any order of the three outer dimensions works;
 * e.g. token-major [layer][slot][kv_head][d] caches pass the matching
 * strides).  V tensors likewise with v_dim channels.
 *
 * Geometry this build implements (else PKV_ERR_UNSUPPORTED), with
 * E = 16 / element size (8 for bf16, 4 for fp32):
 *   head_dim, v_dim, rope_offset multiples of E; head_dim and v_dim multiples
 *   of 2E; rope_dim a multiple of 2E and at most 256.  This covers d = 64/128
 *   (and 256) GQA heads and the 576-channel MLA row [c_kv (512) | k_pe (64)]
 *   with rope_offset 512. */
typedef struct pkv_layout {
    int32_t dtype;          /* PKV_BF16 or PKV_F32 */
    int32_t n_layers;
    int32_t n_kv_heads;     /* 1 for an MLA latent row */
    int32_t head_dim;       /* channels of a K row (576 for MLA) */
    int32_t v_dim;          /* channels of a V row; 0 = no V tensors (MLA: src_v, dst_v must be NULL) */
    int32_t n_tokens;       /* pkv_reposition_splice: tokens to move (source slots 0..n_tokens-1).
                               pkv_reposition_splice_batched: number of source slots in src_k/src_v */
    int32_t rope_offset;    /* first rotary channel of a K row */
    int32_t rope_style;     /* PKV_ROPE_HALF or PKV_ROPE_INTERLEAVED */
    int32_t dst_capacity;   /* destination slots 0..dst_capacity-1 exist in dst_k/dst_v */
    int32_t reserved;       /* must be 0 */
    int64_t src_k_stride[3];   /* {layer, head, slot} */
    int64_t src_v_stride[3];
    int64_t dst_k_stride[3];
    int64_t dst_v_stride[3];
    int32_t* err_flag;      /* optional device int32: set to 1 when a token is skipped because its
                               destination (or, batched, its source) slot is out of range */
} pkv_layout;

/* Reposition + splice of one chunk (Sec. 5; Fig. "Two cache operations" (b);
 * Sec. 8 MLA adapter).  For every layer l, KV head h and token t < n_tokens,
 * with delta_t = dst_pos[t] - src_pos[t]:
 *     dst_k[l][h][dst_pos[t]] = R(delta_t) src_k[l][h][t]   (rotary slice; other channels bit-exact)
 *     dst_v[l][h][dst_pos[t]] = src_v[l][h][t]              (bit-exact)
 * src_pos / dst_pos: device int32 [n_tokens], any sign, |delta| < 2^24.
 * Rotation arithmetic: omega_i is formed in fp64 (from powers of theta the
 * host computes in fp64); the angle
 * delta*omega_i is formed and reduced modulo pi/2 in fp64, its cos/sin are
 * evaluated in fp32 (absolute error below 1e-7), and the rotation runs in fp32
 * with one round-to-nearest-even to the storage type.  delta_t == 0 copies the row
 * bit-exact.  Destination slots other than dst_pos[] are not touched.  A token
 * with dst_pos outside [0, dst_capacity) is skipped (and *err_flag set).
 * In-place use (dst_k == src_k with identical strides, same for V) is allowed
 * when dst_pos[t] == t for every t; any other overlap between a source and a
 * destination tensor, or between dst_k and dst_v, is PKV_ERR_ALIAS.
 * Errors: PKV_ERR_NULL (layout, src_k, dst_k, src_pos, dst_pos; src_v/dst_v
 * when v_dim > 0), PKV_ERR_SHAPE (non-positive sizes, rope_dim odd or <= 0,
 * rope slice outside the row, n_tokens < 0, theta <= 0), PKV_ERR_ALIGN,
 * PKV_ERR_ALIAS, PKV_ERR_UNSUPPORTED (dtype, style, row geometry, rope_dim >
 * 256), PKV_ERR_DEVICE. */
pkv_status pkv_reposition_splice(const void* src_k, const void* src_v, void* dst_k, void* dst_v,
                                 const int32_t* src_pos, const int32_t* dst_pos, float rope_theta,
                                 int32_t rope_dim, const pkv_layout* layout, void* stream);

/* Reposition + splice with explicit per-pair frequencies: as
 * pkv_reposition_splice, with pair i of the rotary slice turned by
 * delta_t * omega[i] instead of delta_t * rope_theta^(-2i/rope_dim).  This
 * covers the RoPE extensions the method also applies to (Related work: rotary
 * embeddings and their extensions): rescaled frequency schedules (Llama-3.1
 * style, YaRN; the rotation stays a pure rotation), and M-RoPE (Sec. 8
 * "Multimodal"; Fig. "attention-variant adapters" (b)), where each rotary
 * pair belongs to the temporal, height or width axis: moving an image along
 * the trajectory by delta temporal positions passes omega[i] for the temporal
 * pairs and 0 for the spatial ones, whose channels then come through
 * bit-exact (cos 0 = 1, sin 0 = 0).  src_pos / dst_pos are the positions on
 * the axis being moved (delta_t = dst_pos[t] - src_pos[t]).
 * dst_slot: optional device int32 [n_tokens], the destination cache slot of
 * each token; NULL means slot = dst_pos[t] as in pkv_reposition_splice.  With
 * M-RoPE the tokens of an image share one temporal position, so the slots are
 * given separately.  Out-of-range slots are skipped and flagged as there.
 * omega: host fp64 [rope_dim/2], read during the call only (any finite
 * values).  rope_dim <= 256.
 * Errors: as pkv_reposition_splice; PKV_ERR_NULL for a NULL omega,
 * PKV_ERR_SHAPE for a non-finite entry. */
pkv_status pkv_reposition_splice_freqs(const void* src_k, const void* src_v, void* dst_k, void* dst_v,
                                       const int32_t* src_pos, const int32_t* dst_pos, const int32_t* dst_slot,
                                       const double* omega, int32_t rope_dim, const pkv_layout* layout,
                                       void* stream);

/* Paged KV cache (Sec. 8: paged attention keeps per-token KV, so the
 * operations apply unchanged; vLLM serving).  Sequence s's logical slot p
 * lives in physical page block_table[s * max_pages + p / page_size] at
 * in-page slot p % page_size.  K element (layer l, kv head h, page P, in-page
 * slot o, channel c) is at l*stride[0] + h*stride[1] + P*page_stride_k +
 * o*stride[2] + c, with stride[] the {layer, head, slot} element strides of
 * the layout / descriptor passed alongside (V likewise with page_stride_v).
 * A pool laid out [layer][page][slot][kv_head][d] has stride = {n_pages *
 * page_size * Hkv * d, d, Hkv * d} and page_stride = page_size * Hkv * d.
 * With v_block_table set, V slot p is in page v_block_table[s * max_pages +
 * p / page_size] instead (same page size, pool size and clamping rules). */
typedef struct pkv_paged_cache {
    int32_t page_size;           /* slots per page: a power of two, 32 .. 2^20 */
    int32_t max_pages;           /* block_table entries per sequence */
    const int32_t* block_table;  /* device int32 [n_seqs][max_pages] */
    int64_t n_pages;             /* physical pages in the pool */
    int64_t page_stride_k;       /* elements between consecutive physical pages of K */
    int64_t page_stride_v;       /* ... of V (unused when there is no V tensor) */
    const int32_t* v_block_table;  /* optional device int32 [n_seqs][max_pages]: V pages through
                                      their own table (NULL: block_table for both).  Values carry
                                      no position, so a spliced chunk's value pages can be
                                      referenced in place instead of copied (GQA only). */
} pkv_paged_cache;

/* Reposition + splice into a paged destination cache: as pkv_reposition_splice
 * with the destination slot dst_pos[t] taken as a logical slot of the sequence
 * whose block table is row 0 of paging->block_table.  layout->dst_capacity is
 * the logical capacity (at most max_pages * page_size) and the dst strides are
 * {layer, head, in-page slot}; values go through paging->v_block_table when it
 * is set.  A token whose slot or page entry is out of range is skipped (and
 * *err_flag set).  The source is a contiguous chunk as
 * in pkv_reposition_splice.
 * Errors: as pkv_reposition_splice; PKV_ERR_NULL (paging or its block table),
 * PKV_ERR_SHAPE (page_size not a power of two in [32, 2^20], non-positive
 * max_pages / n_pages, n_pages beyond 2^31 - 1, negative page strides, dst_capacity beyond
 * max_pages * page_size), PKV_ERR_ALIGN (page strides not 16-byte multiples). */
pkv_status pkv_reposition_splice_paged(const void* src_k, const void* src_v, void* dst_k, void* dst_v,
                                       const int32_t* src_pos, const int32_t* dst_pos, float rope_theta,
                                       int32_t rope_dim, const pkv_layout* layout,
                                       const pkv_paged_cache* paging, void* stream);

/* One chunk of a multi-chunk composition (Sec. 5: a library of skills
 * composes; Sec. 7 E4: memory split into independently precompiled blocks).
 * Source tokens src_slot0 .. src_slot0+n_tokens-1 were encoded at positions
 * src_pos0 .. ; they move to positions dst_pos0 .. of the destination
 * sequence whose position 0 is slot dst_seq_base.  delta = dst_pos0 - src_pos0. */
typedef struct pkv_segment {
    int64_t src_slot0;
    int64_t dst_seq_base;
    int32_t n_tokens;
    int32_t src_pos0;
    int32_t dst_pos0;
    int32_t dst_seq_len;    /* positions 0..dst_seq_len-1 exist in this sequence */
} pkv_segment;

/* Reposition + splice of many chunks into many sequences in one launch.
 * segs: DEVICE array of n_segs segments.  max_seg_tokens must be >= every
 * segs[i].n_tokens (host-known bound used to size the grid).  layout->n_tokens
 * is the number of source slots in src_k/src_v and layout->dst_capacity the
 * number of destination slots; a token whose source slot, destination
 * position or destination slot falls outside those ranges is skipped (and
 * *err_flag set).  Segments must not write overlapping destination slots.
 * Same arithmetic, copy and aliasing rules as pkv_reposition_splice (no
 * in-place use).  Errors: as pkv_reposition_splice, plus PKV_ERR_SHAPE when
 * n_segs < 0 or max_seg_tokens < 0. */
pkv_status pkv_reposition_splice_batched(const void* src_k, const void* src_v, void* dst_k,
                                         void* dst_v, const pkv_segment* segs, int32_t n_segs,
                                         int32_t max_seg_tokens, float rope_theta, int32_t rope_dim,
                                         const pkv_layout* layout, void* stream);

/* ---------------------------------------------------------------------------
 * Suffix attention
 * ------------------------------------------------------------------------- */

/* Geometry of a suffix-attention call over n_layers layers and n_seqs
 * sequences.  Query rows of all sequences are packed: sequence s owns rows
 * cu_q[s] .. cu_q[s+1]-1 of q/out/q_pos.  Its cache occupies slots
 * kv_base[s] .. kv_base[s]+kv_len[s]-1 of k_cache/v_cache.
 *   q    [layer][row][q_head][head_dim]      strides q_stride   {layer, row, head}
 *   out  [layer][row][q_head][head_dim_v]    strides o_stride   {layer, row, head}
 *   k    [layer][kv_head][slot][head_dim]    strides k_stride   {layer, head, slot}
 *   v    [layer][kv_head][slot][head_dim_v]  strides v_stride   {layer, head, slot}
 * MLA (variant PKV_ATTN_MLA, absorbed form): n_kv_heads = 1, head_dim = 576
 * (512 latent + 64 k_pe), head_dim_v = 512, and v_cache must equal k_cache with
 * the same strides: the values are the first 512 (latent) channels of each
 * cache row. */
typedef struct pkv_attn_desc {
    int32_t dtype;          /* PKV_BF16 (MFMA path) or PKV_F32 (GQA only) */
    int32_t variant;        /* PKV_ATTN_GQA or PKV_ATTN_MLA */
    int32_t n_layers;
    int32_t n_seqs;
    int32_t head_dim_v;     /* == head_dim for GQA; 512 for MLA */
    int32_t total_q;        /* query rows per layer over all sequences */
    int32_t max_q;          /* >= the largest per-sequence query count */
    int32_t max_kv_len;     /* >= every kv_len[s]; larger values are clamped to it; at most 2^30 */
    int32_t n_splits;       /* KV-length splits; 0 = the library chooses (at most 32); an explicit
                               count above ceil(max_kv_len / 64) is lowered to it */
    int32_t window;         /* 0: full causal attention.  W > 0: sliding window, slot j is visible
                               only if j > q_pos - W as well (the full cache is kept and the mask
                               enforces the window; Sec. 8 sliding-window configuration fix) */
    const int32_t* cu_q;    /* device int32 [n_seqs+1]; NULL allowed when n_seqs == 1 */
    const int64_t* kv_base; /* device int64 [n_seqs]; NULL = every sequence starts at slot 0 */
    int64_t cache_slots;    /* slots present in k_cache/v_cache; reads past it are masked out */
    int64_t q_stride[3];    /* every stride in elements, non-negative, a multiple of 16 bytes */
    int64_t k_stride[3];    /* the slot strides k_stride[2] and v_stride[2] at most 64 MiB (the */
    int64_t v_stride[3];    /* kernels address the keys of one tile by 32-bit byte offsets) */
    int64_t o_stride[3];
    float* lse_out;         /* optional device fp32 [n_layers][total_q][n_q_heads]: natural-log
                               log-sum-exp of the visible scaled scores (-inf for an empty row) */
} pkv_attn_desc;

/* Bytes of device workspace pkv_suffix_attention needs for `desc` (split-KV
 * partial outputs and their log-sum-exps, fp32).  0 when no split is used.
 * Returns 0 on invalid arguments as well (pkv_suffix_attention reports them). */
size_t pkv_attention_workspace_size(const pkv_attn_desc* desc, int32_t n_q_heads, int32_t n_kv_heads,
                                    int32_t head_dim);

/* Causal attention of the suffix/erratum queries over the spliced cache
 * (Sec. 5 "Linear-time TTFT"; Sec. 4 erratum; Sec. 6 delta prefill).  For layer
 * l, query row i of sequence s and query head h (KV head g = h / (n_q_heads /
 * n_kv_heads)):
 *     visible j: 0 <= j < kv_len[s], j <= q_pos[i], and j > q_pos[i] - window if window > 0
 *     out[l][i][h] = sum_j softmax_j(scale * <q[l][i][h], k[l][g][kv_base[s]+j]>) v[l][g][kv_base[s]+j]
 * q is post-RoPE (q_pos only masks).  bf16: QK^T and PV on bf16 MFMA with fp32
 * accumulation, softmax statistics in fp32, probabilities rounded to bf16
 * before PV, output rounded to bf16.  fp32: fp32 FMA throughout.  A row with no
 * visible slot is written as zeros.  Rows of out (and lse_out) that no
 * sequence owns (outside every [cu_q[s], cu_q[s+1]) range) are not written,
 * whatever the split count.  q_pos: device int32 [total_q]; kv_len:
 * device int32 [n_seqs].  workspace: device memory of at least
 * pkv_attention_workspace_size() bytes (may be NULL when that is 0), owned by
 * the caller, contents scratch.
 * Errors: PKV_ERR_NULL, PKV_ERR_SHAPE (n_q_heads % n_kv_heads != 0, sizes <= 0,
 * max_kv_len > 2^30, slot strides above 64 MiB, window < 0, workspace too small,
 * MLA shape not 576/512 with one KV head or v_cache not k_cache), PKV_ERR_ALIGN,
 * PKV_ERR_UNSUPPORTED (head_dim other than 64 or 128 for GQA; fp32 MLA),
 * PKV_ERR_DEVICE. */
pkv_status pkv_suffix_attention(const void* q, const void* k_cache, const void* v_cache, void* out,
                                const int32_t* q_pos, const int32_t* kv_len, int32_t n_q_heads,
                                int32_t n_kv_heads, int32_t head_dim, float scale,
                                const pkv_attn_desc* desc, void* workspace, size_t workspace_bytes,
                                void* stream);

/* Suffix attention over a paged cache: as pkv_suffix_attention with sequence
 * s's slots read through row s of paging->block_table (desc->kv_base must be
 * NULL; desc->cache_slots is the logical capacity, at most max_pages *
 * page_size; k/v strides are {layer, head, in-page slot}; V slots through
 * paging->v_block_table when it is set).  A 32-key tile always lies within one
 * page.  Block-table entries outside [0, n_pages) are
 * clamped so that every read stays inside the pool (the slots they map are then
 * undefined).  bf16 only (GQA and MLA).
 * Errors: as pkv_suffix_attention; PKV_ERR_NULL (paging, block table),
 * PKV_ERR_SHAPE (paging fields as for the paged splice, kv_base given,
 * v_block_table with MLA), PKV_ERR_UNSUPPORTED (fp32). */
pkv_status pkv_suffix_attention_paged(const void* q, const void* k_pages, const void* v_pages, void* out,
                                      const int32_t* q_pos, const int32_t* kv_len, int32_t n_q_heads,
                                      int32_t n_kv_heads, int32_t head_dim, float scale,
                                      const pkv_attn_desc* desc, const pkv_paged_cache* paging,
                                      void* workspace, size_t workspace_bytes, void* stream);

/* Bytes of the static device scratch behind pkv_suffix_attention_noalloc. */
#define PKV_NOALLOC_SCRATCH_BYTES (64u << 20)

/* Allocation-free suffix attention, for callers that cannot allocate device
 * memory or pass a workspace: code under HIP graph capture, tight serving
 * loops, harnesses that forbid hipMalloc.  Same arguments, semantics and
 * errors as pkv_suffix_attention without workspace / workspace_bytes.  The
 * split-KV partials go to a static device array of PKV_NOALLOC_SCRATCH_BYTES
 * that the library holds on every GPU it has run this call on, until the
 * process ends; the call allocates and frees nothing and records no memset.
 * Size limit: with desc->n_splits = 0 the split count is the library's choice,
 * lowered if needed until the partials fit the scratch (1 split needs none);
 * an explicit desc->n_splits whose partials exceed the scratch is rejected
 * with PKV_ERR_SHAPE.  Every call on one GPU shares that GPU's scratch: calls
 * that overlap in time on one GPU (different streams, or host threads without
 * ordering) race and give undefined results; calls ordered on one stream are
 * safe.  Nothing in the scratch needs clearing between calls (each call
 * writes every partial it reads).  The first call on a device looks up the
 * scratch's address there (hipGetSymbolAddress); a failure of that lookup is
 * PKV_ERR_DEVICE. */
pkv_status pkv_suffix_attention_noalloc(const void* q, const void* k_cache, const void* v_cache, void* out,
                                        const int32_t* q_pos, const int32_t* kv_len, int32_t n_q_heads,
                                        int32_t n_kv_heads, int32_t head_dim, float scale,
                                        const pkv_attn_desc* desc, void* stream);

/* ---------------------------------------------------------------------------
 * Diagnostics
 * ------------------------------------------------------------------------- */

/* Message for the last non-OK status returned on the calling thread ("" if
 * none).  The pointer stays valid until the next libpkv call on this thread. */
const char* pkv_last_error(void);

/* PKV_VERSION of the built library. */
int32_t pkv_version(void);

#ifdef __cplusplus
}
#endif

#endif /* PKV_H */
