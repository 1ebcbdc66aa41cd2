// Bandwidth probes for the roofline: plain HBM copy, read and write kernels shaped like the
// row kernel's traffic (one 1024-thread workgroup per row, 16-byte buffer accesses, every
// vector of a row in flight at once, non-temporal, rows taken from a queue as the fused pass
// takes them). They measure what this device achieves for pure reads, pure writes and an equal
// mix; they are not part of the loss.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "../../include/cis_probe.h"

namespace {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
constexpr int kBlock = 1024;
constexpr int kSlots = 19;
constexpr int kRsrcWord3 = 0x00020000;
constexpr int kAuxNT = 2;

__device__ __forceinline__ __amdgpu_buffer_rsrc_t rsrc(const void* base, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), 0, (int)bytes, kRsrcWord3);
}

// mode 0: copy, 1: read only, 2: write only. A workgroup's first row is blockIdx.x; thread 0
// draws the next one from the counter at sink[kSinkWords] while the row is in flight, and the
// other waves read it after the row's barrier (double-buffered: one barrier per row).
constexpr int kSinkWords = 1024;
template <int MODE>
__global__ __launch_bounds__(kBlock) void probe_kernel(const void* src, void* dst, int64_t rows,
                                                       uint32_t row_bytes, uint32_t* sink) {
  __shared__ unsigned long long next[2];
  unsigned long long* const queue = reinterpret_cast<unsigned long long*>(sink + kSinkWords);
  uint32_t acc = 0;
  int buf = 0;
  for (int64_t r = blockIdx.x; r < rows;) {
    unsigned long long tk = 0ull;
    if (threadIdx.x == 0) tk = atomicAdd(queue, 1ull);
    const __amdgpu_buffer_rsrc_t rs = rsrc((const char*)src + r * row_bytes, row_bytes);
    const __amdgpu_buffer_rsrc_t ws = rsrc((char*)dst + r * row_bytes, row_bytes);
    u32x4 v[kSlots];
#pragma unroll
    for (int k = 0; k < kSlots; ++k) {
      const uint32_t o = (threadIdx.x + k * kBlock) * 16u;
      v[k] = MODE == 2 ? u32x4{o, o, o, o} : __builtin_amdgcn_raw_buffer_load_b128(rs, o, 0, kAuxNT);
    }
#pragma unroll
    for (int k = 0; k < kSlots; ++k) {
      const uint32_t o = (threadIdx.x + k * kBlock) * 16u;
      if (MODE == 1)
        acc ^= v[k].x ^ v[k].y ^ v[k].z ^ v[k].w;
      else
        __builtin_amdgcn_raw_buffer_store_b128(v[k], ws, o, 0, kAuxNT);
    }
    if (threadIdx.x == 0) next[buf] = tk;
    __syncthreads();
    r = (int64_t)gridDim.x + (int64_t)next[buf];
    buf ^= 1;
  }
  if (MODE == 1 && acc == 0x9E3779B9u) sink[threadIdx.x] = acc;  // keeps the loads alive
}

__global__ __launch_bounds__(64) void probe_queue_reset(uint32_t* sink) {
  if (threadIdx.x == 0) *reinterpret_cast<unsigned long long*>(sink + kSinkWords) = 0ull;
}

// Mode 3: the fastest equal read/write stream found on this part. Short-lived 128-thread
// workgroups each copy 4 KiB (two 16-byte non-temporal vectors per thread), so the CUs hold
// many independent small copies at different phases.
constexpr int kSmallBlock = 128;
__global__ __launch_bounds__(kSmallBlock) void probe_small_copy(const u32x4* src, u32x4* dst,
                                                               int64_t nvec) {
  const int64_t base = (int64_t)blockIdx.x * kSmallBlock * 2 + threadIdx.x;
  u32x4 v[2];
#pragma unroll
  for (int i = 0; i < 2; ++i) {
    const int64_t j = base + (int64_t)i * kSmallBlock;
    if (j < nvec) v[i] = __builtin_nontemporal_load(src + j);
  }
#pragma unroll
  for (int i = 0; i < 2; ++i) {
    const int64_t j = base + (int64_t)i * kSmallBlock;
    if (j < nvec) __builtin_nontemporal_store(v[i], dst + j);
  }
}

// Mode 4: the read-only counterpart of mode 3 (short-lived 128-thread workgroups, 4 KiB each,
// non-temporal loads), the fastest read stream found on this part.
__global__ __launch_bounds__(kSmallBlock) void probe_small_read(const u32x4* src, int64_t nvec,
                                                                uint32_t* sink) {
  const int64_t base = (int64_t)blockIdx.x * kSmallBlock * 2 + threadIdx.x;
  uint32_t acc = 0;
#pragma unroll
  for (int i = 0; i < 2; ++i) {
    const int64_t j = base + (int64_t)i * kSmallBlock;
    if (j < nvec) {
      const u32x4 v = __builtin_nontemporal_load(src + j);
      acc ^= v.x ^ v.y ^ v.z ^ v.w;
    }
  }
  if (acc == 0x9E3779B9u) sink[threadIdx.x] = acc;  // keeps the loads alive
}

}  // namespace

extern "C" int cis_probe_bandwidth(int mode, const void* src, void* dst, int64_t rows,
                                   int64_t row_bytes, int grid, uint32_t* sink,
                                   hipStream_t stream) {
  if (mode == 3 || mode == 4) {  // contiguous small blocks over rows*row_bytes; grid unused
    if (rows < 0 || row_bytes <= 0 || row_bytes % 16 != 0) return -2;
    if (!src || (mode == 3 && !dst) || (mode == 4 && !sink)) return -1;
    const int64_t nvec = rows * (row_bytes / 16);
    if (nvec == 0) return 0;
    const int64_t blocks = (nvec + 2 * kSmallBlock - 1) / (2 * kSmallBlock);
    if (blocks > INT32_MAX) return -2;
    const u32x4* s4 = (const u32x4*)src;
    u32x4* d4 = (u32x4*)dst;
    if (mode == 4) {
      void* args4[] = {&s4, (void*)&nvec, &sink};
      return hipLaunchKernel((const void*)&probe_small_read, dim3((unsigned)blocks),
                             dim3(kSmallBlock), args4, 0, stream) == hipSuccess ? 0 : -6;
    }
    void* args3[] = {&s4, &d4, (void*)&nvec};
    return hipLaunchKernel((const void*)&probe_small_copy, dim3((unsigned)blocks), dim3(kSmallBlock),
                           args3, 0, stream) == hipSuccess ? 0 : -6;
  }
  if (mode < 0 || mode > 2 || rows < 0 || grid < 1) return -4;
  if (row_bytes <= 0 || row_bytes % 16 != 0 || row_bytes > (int64_t)kSlots * kBlock * 16)
    return -2;
  if ((mode != 2 && !src) || (mode != 1 && !dst) || !sink) return -1;
  if (reinterpret_cast<uintptr_t>(sink) % 8 != 0) return -2;
  void* qargs[] = {&sink};
  if (hipLaunchKernel((const void*)&probe_queue_reset, dim3(1), dim3(64), qargs, 0, stream) !=
      hipSuccess)
    return -6;
  void* args[] = {&src, &dst, &rows, &row_bytes, &sink};
  uint32_t rb = (uint32_t)row_bytes;
  args[3] = &rb;
  const void* fn = mode == 0 ? (const void*)&probe_kernel<0>
                 : mode == 1 ? (const void*)&probe_kernel<1> : (const void*)&probe_kernel<2>;
  return hipLaunchKernel(fn, dim3(grid), dim3(kBlock), args, 0, stream) == hipSuccess ? 0 : -6;
}
