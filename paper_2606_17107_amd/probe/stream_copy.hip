// A plain device copy with the access pattern of the single-chunk splice:
// 8 KB per 256-thread block, each thread moving two 16-byte chunks with
// non-temporal loads and stores, blocks renumbered so that each XCD streams
// one contiguous range.  It does no arithmetic, so its rate is the practical
// ceiling of the splice's memory traffic on this GPU; the benchmark times it
// beside the splice.  Built into its own library (not part of libpkv).
#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
constexpr int kBlock = 256;
constexpr int kXcds = 8;
constexpr size_t kBlockBytes = 2 * kBlock * 16;

__global__ __launch_bounds__(kBlock) void stream_copy_kernel(u32x4* dst, const u32x4* src, uint32_t n_blocks,
                                                             uint32_t per_xcd) {
    uint32_t b = blockIdx.x;
    if (per_xcd) b = (b % kXcds) * per_xcd + b / kXcds;
    if (b >= n_blocks) return;
    const size_t i = (size_t)b * (2 * kBlock) + threadIdx.x;
    const u32x4 x = __builtin_nontemporal_load(src + i);
    const u32x4 y = __builtin_nontemporal_load(src + i + kBlock);
    __builtin_nontemporal_store(x, dst + i);
    __builtin_nontemporal_store(y, dst + i + kBlock);
}

}  // namespace

// Copies `bytes` from src to dst (device pointers, 16-byte aligned, not
// overlapping) on `stream` (a hipStream_t, or null).  bytes must be a multiple
// of 8192.  Returns 0 on success, 1 for a bad argument, 2 for a launch error.
extern "C" __attribute__((visibility("default"))) int pkv_stream_copy(void* dst, const void* src, size_t bytes,
                                                                      void* stream) {
    if (!dst || !src || bytes % kBlockBytes || ((uintptr_t)dst | (uintptr_t)src) % 16) return 1;
    const size_t n = bytes / kBlockBytes;
    if (n == 0) return 0;
    if (n > 0x7fffffffu) return 1;
    const uint32_t per_xcd = n % kXcds == 0 ? (uint32_t)(n / kXcds) : 0;
    hipLaunchKernelGGL(stream_copy_kernel, dim3((unsigned)n), dim3(kBlock), 0, (hipStream_t)stream, (u32x4*)dst,
                       (const u32x4*)src, (uint32_t)n, per_xcd);
    return hipGetLastError() == hipSuccess ? 0 : 2;
}
