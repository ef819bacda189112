// Measurement probe (not part of libdcp): a device copy whose reads take the
// same path as the attention kernels' tile loads, global_load_lds_dwordx4
// (global memory straight into LDS, 16 bytes per lane), followed by 16-byte
// LDS reads and plain global stores.  Its size is known exactly, so what
// the HBM byte counters (FETCH_SIZE, WRITE_SIZE) report for it calibrates
// them for the kernels' direct-to-LDS reads.
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace {

constexpr int kThreads = 256;
constexpr int kChunk = kThreads * 16;  // bytes one workgroup moves per step

__global__ __launch_bounds__(kThreads) void dma_copy_kernel(const uint8_t* __restrict__ src, uint8_t* __restrict__ dst,
                                                            int64_t n_chunks) {
  __shared__ __attribute__((aligned(16))) uint8_t buf[kChunk];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  for (int64_t c = blockIdx.x; c < n_chunks; c += gridDim.x) {
    const uint8_t* g = src + c * kChunk + wave * 1024 + lane * 16;
    const uint32_t m0 =
        __builtin_amdgcn_readfirstlane(static_cast<uint32_t>(reinterpret_cast<uintptr_t>(buf + wave * 1024)));
    asm volatile("s_mov_b32 m0, %0\n\tglobal_load_lds_dwordx4 %1, off\n\ts_waitcnt vmcnt(0)"
                 :
                 : "s"(m0), "v"(reinterpret_cast<uint64_t>(g))
                 : "memory");
    // (each wavefront reads back only the 1 KB its own copy wrote)
    const uint4 x = *reinterpret_cast<const uint4*>(buf + wave * 1024 + lane * 16);
    *reinterpret_cast<uint4*>(dst + c * kChunk + wave * 1024 + lane * 16) = x;
    __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "workgroup");
    __builtin_amdgcn_wave_barrier();
  }
}

}  // namespace

// Copies `bytes` (a multiple of 4096) from src to dst on `stream`.
// Returns 0, or -1 for a bad size, or the launch error code.
extern "C" int dcp_probe_dma_copy(const void* src, void* dst, int64_t bytes, void* stream) {
  if (bytes <= 0 || bytes % kChunk) return -1;
  const int64_t n = bytes / kChunk;
  const unsigned grid = unsigned(n < 256 * 64 ? n : 256 * 64);
  hipLaunchKernelGGL(dma_copy_kernel, dim3(grid), dim3(kThreads), 0, static_cast<hipStream_t>(stream),
                     static_cast<const uint8_t*>(src), static_cast<uint8_t*>(dst), n);
  return int(hipGetLastError());
}
