// Device-side pieces shared by the suffix-attention kernels: the work plan,
// the XCD-aware workgroup decode, per-sequence bounds and small wave helpers.
#pragma once

#include <math.h>

#include <type_traits>

#include "pkv_internal.h"

namespace pkv {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
typedef short s16x4 __attribute__((ext_vector_type(4)));

#ifndef PKV_LDS
#define PKV_LDS(T, p) ((__attribute__((address_space(3))) T*)(p))
#endif

constexpr int kXcds = 8;
constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;

struct Plan {
    int G;          // query heads per KV head
    int BM;         // rows per workgroup
    int rbs;        // row blocks per group
    int n_groups;   // layers x kv heads x sequences x splits
    int splits;     // each workgroup's key range is shared by this many splits in equal runs of whole tiles
    int qb, nw, ns; // bf16 GQA kernel shape: 32-row blocks per wave, waves, LDS stages
};

// Workgroup id -> (group, row block).  Workgroups are dispatched round-robin
// over the 8 XCDs by id; giving every row block of a group (which all read the
// same K/V range) an id with the same residue mod 8 keeps them on one XCD, at
// consecutive dispatch slots, so they share that XCD's L2.
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

// Paged caches: the block-table row of one sequence seen through a window of
// 256 consecutive entries held by the wave, four registers of 64 lanes (lane
// l of register r holds entry w0 + 64 r + l).  Tiles are visited in ascending
// order, so the window moves forward a whole window at a time; each entry is
// clamped into the pool when loaded, so every tile read stays inside it.
struct PageWindow {
    const int32_t* row;   // the sequence's row of the block table
    int n_entries;        // max_pages
    int last_page;        // n_pages - 1
    int w0;               // first entry in the window
    int id0, id1, id2, id3;   // four registers, not an array: no indexed private memory

    __device__ __forceinline__ int entry(int e) const {
        const int v = e < n_entries ? row[e] : 0;
        return min(max(v, 0), last_page);
    }
    __device__ __forceinline__ void load(int first) {
        w0 = first;
        const int l = first + (int)__lane_id();
        id0 = entry(l);
        id1 = entry(l + 64);
        id2 = entry(l + 128);
        id3 = entry(l + 192);
    }
    __device__ __forceinline__ void init(const int32_t* table, const AttnArgs& a, int seq, int first_entry) {
        row = table + (int64_t)seq * a.max_pages;
        n_entries = a.max_pages;
        last_page = (int)(a.n_pages - 1);
        load(first_entry);
    }
    // Element offset of logical slot t0 (the first key of a tile, which lies
    // in one page) from the pool's (layer, head) origin.
    __device__ __forceinline__ int64_t offset(const AttnArgs& a, int t0, int64_t page_stride, int64_t slot_stride) {
        const int e = t0 >> a.page_shift;
        if ((unsigned)(e - w0) >= 256u) load(e);
        const int rel = e - w0;
        // Read the lane from each register and select among the scalars: a
        // select among the registers would be folded into an indexed access of
        // the struct, which then cannot live in registers.
        const int r = rel >> 6, l = rel & 63;
        const int p0 = __builtin_amdgcn_readlane(id0, l), p1 = __builtin_amdgcn_readlane(id1, l);
        const int p2 = __builtin_amdgcn_readlane(id2, l), p3 = __builtin_amdgcn_readlane(id3, l);
        const int page = r == 0 ? p0 : r == 1 ? p1 : r == 2 ? p2 : p3;
        return (int64_t)page * page_stride + (int64_t)(t0 & ((1 << a.page_shift) - 1)) * slot_stride;
    }
};

// Visible keys [start, end) of a row at position qpos over a cache of kvl
// keys: causal (keys up to qpos) and, with a window W > 0, keys above
// qpos - W.  Both bounds lie in [0, kvl] and are formed without overflow for
// every int32 position and window; a row before the cache (qpos < 0) sees
// nothing.
__device__ inline void visible_range(int qpos, int kvl, int window, int& start, int& end) {
    end = qpos < kvl ? max(0, qpos + 1) : kvl;
    start = window > 0 && qpos >= window ? min(qpos - window + 1, kvl) : 0;
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

// A wave-uniform 64-bit value in scalar registers.  readfirstlane returns a
// signed int: each half is taken as uint32_t before widening.
__device__ inline uint64_t uniform_u64(uint64_t v) {
    const uint32_t lo = (uint32_t)__builtin_amdgcn_readfirstlane((uint32_t)v);
    const uint32_t hi = (uint32_t)__builtin_amdgcn_readfirstlane((uint32_t)(v >> 32));
    return ((uint64_t)hi << 32) | lo;
}

// LDS byte address of a pointer into a __shared__ array (the low 32 bits of
// its flat address).
__device__ inline uint32_t lds_addr_of(const void* p) { return (uint32_t)(uintptr_t)p; }

// One 16-byte LDS-DMA load per lane (global_load_lds_dwordx4, saddr form):
// lane l's 16 bytes at sbase + voff[l] land at LDS byte address lds_addr +
// 16*l; lds_addr (M0) and sbase are wave-uniform.  Written as inline assembly
// so that the compiler does not see an LDS write in flight: with the builtin
// it would wait for every outstanding LDS read (lgkmcnt 0) wherever it needs
// any one of them.  Completion is tracked by the kernels themselves with
// explicit vmcnt waits before the barrier that publishes a stage; the memory
// clobber keeps LDS accesses on their side.  M0 is an input operand of the
// statement ("{m0}" constraint): the compiler writes it right before the
// load and knows it holds the LDS address, so none of its own uses of M0 can
// be disturbed.  The s_nop gives the one wait state between that M0 write
// and the load that reads it.
__device__ inline void lds_dma_asm(uint32_t m0, uint64_t sbase, uint32_t voff) {
    asm volatile("s_nop 0\n\tglobal_load_lds_dwordx4 %0, %1" ::"v"(voff), "s"(sbase), "{m0}"(m0) : "memory");
}

__device__ inline void lds_dma16(uint32_t lds_addr, const void* sbase, uint32_t voff) {
    lds_dma_asm((uint32_t)__builtin_amdgcn_readfirstlane(lds_addr), uniform_u64((uint64_t)(uintptr_t)sbase), voff);
}

// Compile-time loop: f(std::integral_constant<int, I>) for I = B .. E-1.
template <int B, int E, typename F>
__device__ __forceinline__ void static_for(F&& f) {
    if constexpr (B < E) {
        f(std::integral_constant<int, B>{});
        static_for<B + 1, E>(f);
    }
}

// Wait until at most N vector-memory operations of this wave are outstanding
// (gfx9 s_waitcnt encoding: vmcnt split over bits 3:0 and 15:14; expcnt and
// lgkmcnt left at their "no wait" maxima).
template <int N>
__device__ inline void wait_vmcnt() {
    static_assert(N >= 0 && N < 64, "vmcnt range");
    __builtin_amdgcn_s_waitcnt((N & 15) | (7 << 4) | (15 << 8) | ((N >> 4) << 14));
}

// Workgroup barrier without the release/acquire fences of __syncthreads():
// the fences would force the wave to drain every in-flight LDS-DMA load,
// which is exactly what the staged pipeline must not do.  Ordering of the
// LDS traffic around it is established by explicit s_waitcnt.
__device__ inline void bare_barrier() {
    __builtin_amdgcn_s_barrier();
    asm volatile("" ::: "memory");
}

// Scheduling pattern for a run of N operand loads from LDS, R reads per
// operand, each operand feeding Q MFMAs: the first A operands' reads go first,
// then every MFMA group is followed by the reads of the operand A steps ahead.
// This bounds the registers held by prefetched operands while keeping A LDS
// round trips in flight.
template <int N, int R, int Q, int A = 2>
__device__ inline void sched_reads_mfma() {
    constexpr int A0 = A < N ? A : N;
    __builtin_amdgcn_sched_group_barrier(0x100, A0 * R, 0);
#pragma unroll
    for (int i = 0; i < N; ++i) {
        __builtin_amdgcn_sched_group_barrier(0x008, Q, 0);
        if (i + A0 < N) __builtin_amdgcn_sched_group_barrier(0x100, R, 0);
    }
}

}  // namespace pkv
