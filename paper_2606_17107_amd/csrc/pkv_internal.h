// Internal interface between the C ABI (api.hip) and the kernel launchers.
// Nothing here is exported from libpkv.so.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace pkv {

// ---- reposition + splice ---------------------------------------------------

struct SpliceSegment {   // same layout as pkv_segment in pkv.h
    int64_t src_slot0;
    int64_t dst_seq_base;
    int32_t n_tokens;
    int32_t src_pos0;
    int32_t dst_pos0;
    int32_t dst_seq_len;
};

struct SpliceArgs {
    const char* src_k;
    const char* src_v;
    char* dst_k;
    char* dst_v;
    // per-token mode
    const int32_t* src_pos;
    const int32_t* dst_pos;
    const int32_t* dst_slot;  // destination slots, or null (slot = dst_pos)
    // segment mode
    const SpliceSegment* segs;
    int32_t n_segs;
    int32_t max_seg_tokens;

    int32_t elem_bytes;      // 2 (bf16) or 4 (fp32)
    int32_t rope_style;
    int32_t n_layers;
    int32_t n_kv_heads;
    int32_t head_dim;
    int32_t v_dim;
    int32_t rope_offset;
    int32_t rope_dim;
    int64_t n_tokens;        // per-token mode: tokens; segment mode: source slots
    int64_t dst_capacity;
    double theta;
    const double* omega;      // host, rope_dim/2 per-pair frequencies, or null (theta schedule)
    int64_t src_k_stride[3];  // elements
    int64_t src_v_stride[3];
    int64_t dst_k_stride[3];
    int64_t dst_v_stride[3];
    int32_t* err_flag;
    // paged destination (per-token mode): logical slot p -> page
    // dst_pages[p >> page_shift], in-page slot p & (page_size - 1)
    const int32_t* dst_pages;  // null: contiguous destination
    const int32_t* dst_v_pages;  // V through its own table, or null (dst_pages)
    int32_t page_shift;
    int32_t max_pages;
    int64_t n_pages;
    int64_t dst_k_page_stride;  // elements
    int64_t dst_v_page_stride;
};

hipError_t launch_splice(const SpliceArgs& a, hipStream_t stream);

// ---- suffix attention --------------------------------------------------------

struct AttnArgs {
    const void* q;
    const void* k;
    const void* v;
    void* out;
    const int32_t* q_pos;
    const int32_t* kv_len;
    const int32_t* cu_q;      // may be null (one sequence)
    const int64_t* kv_base;   // may be null
    float* lse_out;           // may be null
    float* ws_o;              // split partial outputs (fp32) or null
    float* ws_lse;            // split partial log-sum-exp (fp32) or null
    int32_t dtype;            // 0 bf16, 1 fp32
    int32_t variant;          // 0 GQA, 1 MLA
    int32_t n_layers;
    int32_t n_seqs;
    int32_t n_heads;
    int32_t n_kv_heads;
    int32_t head_dim;
    int32_t head_dim_v;
    int32_t total_q;
    int32_t max_q;
    int32_t max_kv_len;
    int32_t n_splits;
    int32_t window;           // 0: full causal; W > 0: slots j > q_pos - W only
    int64_t cache_slots;
    float scale;
    int64_t q_stride[3];
    int64_t k_stride[3];
    int64_t v_stride[3];
    int64_t o_stride[3];
    // paged cache: sequence s's slot p is in page block_table[s * max_pages +
    // (p >> page_shift)], in-page slot p & (page_size - 1)
    const int32_t* block_table;  // null: contiguous cache
    const int32_t* v_block_table;  // V through its own table, or null (block_table)
    int32_t page_shift;
    int32_t max_pages;
    int64_t n_pages;
    int64_t k_page_stride;       // elements
    int64_t v_page_stride;
};

// Split plan shared by the workspace query and the launcher.
int attention_splits(const AttnArgs& a);
size_t attention_workspace_bytes(const AttnArgs& a, int n_splits);
hipError_t launch_attention(const AttnArgs& a, hipStream_t stream);

}  // namespace pkv
