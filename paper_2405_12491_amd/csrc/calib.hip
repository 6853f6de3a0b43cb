// calib.hip -- microbenchmarks that measure the per-level bandwidths of the Eq. 1 model on the
// device at hand (BandWidth_l of Table 6): the per-lane LDS gather rate, which bounds the
// traversal kernels, and the HBM copy rate.  Built into its own library (libbridger_calib.so);
// nothing in the prediction library calls it.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "bridger_calib.h"

namespace bridger_calib {

constexpr int kThreads = 256;             // four waves per workgroup
constexpr int kLdsBytes = 16384;          // per workgroup: ten fit a CU's LDS
constexpr int kReadsPerIter = 16;         // independent reads per lane per iteration
constexpr int kBlocksPerCU = 8;           // 32 resident waves per CU
constexpr int kWarmLaunches = 10;         // untimed launches before the timed ones

// Every lane reads W bytes at kReadsPerIter addresses per iteration, read k of lane l at byte
// lane_addr[64 k + l] (each below 1024 (k + 1), a multiple of W): per-lane values held in
// registers, as the traversal kernels' gathers are, and one register per read, so that the
// compiler cannot pair reads into two-address instructions.  With a table that puts the 32
// lanes of each half-wave on 32 different dwords the gather is free of bank conflicts; with
// random addresses it is not; with `distinct` < 64 the lanes share that many addresses
// (lane l reads the (l mod distinct)-th of the conflict-free addresses), as the lanes of a wave
// share the few node records of a tree's upper levels.  The empty asm with a memory clobber keeps the compiler from
// hoisting the (loop-invariant) reads out of the loop.
template <int W>
__global__ __launch_bounds__(kThreads) void lds_gather_kernel(const uint32_t *lane_addr, int iters,
                                                              uint32_t *sink) {
  __shared__ __attribute__((aligned(16))) uint32_t lds[kLdsBytes / 4];
  for (int i = threadIdx.x; i < kLdsBytes / 4; i += kThreads) lds[i] = (uint32_t)i * 2654435761u;
  __syncthreads();
  uint32_t addr[kReadsPerIter];
#pragma unroll
  for (int k = 0; k < kReadsPerIter; ++k) addr[k] = lane_addr[64 * k + (threadIdx.x & 63)];
  const uint8_t *p = reinterpret_cast<const uint8_t *>(lds);
  uint32_t acc = 0;
  for (int it = 0; it < iters; ++it) {
    asm volatile("" ::: "memory");
#pragma unroll
    for (int k = 0; k < kReadsPerIter; ++k) {
      const uint8_t *q = p + addr[k];
      if constexpr (W == 4) {
        acc ^= *reinterpret_cast<const uint32_t *>(q);
      } else if constexpr (W == 8) {
        const uint2 v = *reinterpret_cast<const uint2 *>(q);
        acc ^= v.x ^ v.y;
      } else {
        const uint4 v = *reinterpret_cast<const uint4 *>(q);
        acc ^= v.x ^ v.y ^ v.z ^ v.w;
      }
    }
  }
  if (acc == 0x9e3779b9u) sink[blockIdx.x] = acc;  // keeps the reads alive; practically never taken
}

// Per-lane global-memory gathers of W bytes from an L2-resident buffer of mask + 1 bytes: every
// lane issues kReadsPerIter independent loads per iteration at byte (lane_addr[64 k + l] +
// it * kGlobalStride) & mask, so each iteration touches new cache lines (the L1 holds few of
// them) while the buffer stays in L2, as the node records of the global-node kernels do.
// lane_addr entries are multiples of 128 plus a multiple of W below 128 - W + 1, so no load
// crosses a line; with `distinct` < 64 lanes share that many lines.
constexpr uint32_t kGlobalStride = 128u * 4099u;  // an odd number of lines per iteration
template <int W>
__global__ __launch_bounds__(kThreads) void global_gather_kernel(const uint8_t *__restrict__ buf,
                                                                 uint32_t mask,
                                                                 const uint32_t *lane_addr,
                                                                 int iters, uint32_t *sink) {
  uint32_t addr[kReadsPerIter];
#pragma unroll
  for (int k = 0; k < kReadsPerIter; ++k) addr[k] = lane_addr[64 * k + (threadIdx.x & 63)];
  uint32_t acc = 0;
  for (int it = 0; it < iters; ++it) {
    const uint32_t shift = (uint32_t)it * kGlobalStride;
#pragma unroll
    for (int k = 0; k < kReadsPerIter; ++k) {
      const uint8_t *q = buf + ((addr[k] + shift) & mask);
      if constexpr (W == 4) {
        acc ^= *reinterpret_cast<const uint32_t *>(q);
      } else if constexpr (W == 8) {
        const uint2 v = *reinterpret_cast<const uint2 *>(q);
        acc ^= v.x ^ v.y;
      } else {
        const uint4 v = *reinterpret_cast<const uint4 *>(q);
        acc ^= v.x ^ v.y ^ v.z ^ v.w;
      }
    }
  }
  if (acc == 0x9e3779b9u) sink[blockIdx.x] = acc;  // keeps the loads alive; practically never taken
}

__global__ __launch_bounds__(kThreads) void copy_kernel(const uint4 *__restrict__ src,
                                                        uint4 *__restrict__ dst, int64_t n) {
  const int64_t stride = (int64_t)gridDim.x * kThreads;
  for (int64_t i = (int64_t)blockIdx.x * kThreads + threadIdx.x; i < n; i += stride) dst[i] = src[i];
}

template <class Launch>
static hipError_t time_ms(Launch launch, int reps, double *ms) {
  hipEvent_t e0 = nullptr, e1 = nullptr;
  hipError_t e = hipEventCreate(&e0);
  if (e == hipSuccess) e = hipEventCreate(&e1);
  if (e == hipSuccess) {
    for (int w = 0; w < kWarmLaunches; ++w) launch();  // first-launch costs and the clock ramp
    e = hipGetLastError();
  }
  if (e == hipSuccess) e = hipEventRecord(e0, nullptr);
  for (int r = 0; r < reps && e == hipSuccess; ++r) {
    launch();
    e = hipGetLastError();
  }
  if (e == hipSuccess) e = hipEventRecord(e1, nullptr);
  if (e == hipSuccess) e = hipEventSynchronize(e1);
  float t = 0.0f;
  if (e == hipSuccess) e = hipEventElapsedTime(&t, e0, e1);
  if (e == hipSuccess) *ms = t / reps;
  if (e0) (void)hipEventDestroy(e0);
  if (e1) (void)hipEventDestroy(e1);
  return e;
}

}  // namespace bridger_calib

using namespace bridger_calib;

extern "C" {

int bridger_calib_device(int32_t *n_cu, int32_t *max_clock_khz, int32_t *lds_bytes_per_cu) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  hipDeviceProp_t p;
  if (e == hipSuccess) e = hipGetDeviceProperties(&p, dev);
  if (e != hipSuccess) return (int)e;
  if (n_cu) *n_cu = p.multiProcessorCount;
  if (max_clock_khz) *max_clock_khz = p.clockRate;
  if (lds_bytes_per_cu) *lds_bytes_per_cu = (int32_t)p.maxSharedMemoryPerMultiProcessor;
  return 0;
}

int bridger_calib_lds_gather(int32_t width_bytes, int32_t distinct, int32_t reps,
                             double *ms_per_launch, double *wave_reads_per_s) {
  if (!(width_bytes == 4 || width_bytes == 8 || width_bytes == 16) || reps < 1 || distinct < 0 ||
      distinct > 64 || (distinct & (distinct - 1)) != 0)
    return (int)hipErrorInvalidValue;
  int32_t n_cu = 0;
  int e0 = bridger_calib_device(&n_cu, nullptr, nullptr);
  if (e0 != 0) return e0;
  // Lane addresses (bytes).  Conflict-free (distinct = 64): the 32 lanes of a half-wave take 32
  // different elements of W bytes, in a permuted order (so the addresses are not simply
  // lane-ordered), the two half-waves two consecutive spans of 32 elements.  distinct = d < 64:
  // lane l takes the address of lane (l mod d).  Random (distinct = 0): elements drawn with a
  // fixed linear congruential sequence from the 1024 / W elements of the read's 1 KB window.
  uint32_t host[64 * kReadsPerIter];
  uint32_t s = 12345u;
  const uint32_t w = (uint32_t)width_bytes;
  for (int k = 0; k < kReadsPerIter; ++k) {
    for (int l = 0; l < 64; ++l) {
      s = s * 1664525u + 1013904223u;
      const int src = distinct ? l % distinct : l;
      // 13 is odd: (l * 13 + k) mod 32 is a permutation of 0..31 for every k
      const uint32_t j = (uint32_t)(((src & 31) * 13 + k) % 32);
      host[64 * k + l] = 1024u * (uint32_t)k +
                         (distinct ? (uint32_t)((src >> 5) * 32 + j) * w
                                   : ((s >> 8) % (1024u / w)) * w);
    }
  }
  uint32_t *d_base = nullptr, *d_sink = nullptr;
  const int blocks = n_cu * kBlocksPerCU;
  hipError_t e = hipMalloc(&d_base, sizeof(host));
  if (e == hipSuccess) e = hipMalloc(&d_sink, sizeof(uint32_t) * (size_t)blocks);
  if (e == hipSuccess) e = hipMemcpy(d_base, host, sizeof(host), hipMemcpyHostToDevice);
  const int iters = 1024;
  double ms = 0.0;
  if (e == hipSuccess) {
    auto launch = [&]() {
      if (width_bytes == 4)
        hipLaunchKernelGGL(lds_gather_kernel<4>, dim3(blocks), dim3(kThreads), 0, nullptr, d_base,
                           iters, d_sink);
      else if (width_bytes == 8)
        hipLaunchKernelGGL(lds_gather_kernel<8>, dim3(blocks), dim3(kThreads), 0, nullptr, d_base,
                           iters, d_sink);
      else
        hipLaunchKernelGGL(lds_gather_kernel<16>, dim3(blocks), dim3(kThreads), 0, nullptr,
                           d_base, iters, d_sink);
    };
    e = time_ms(launch, reps, &ms);
  }
  if (d_base) (void)hipFree(d_base);
  if (d_sink) (void)hipFree(d_sink);
  if (e != hipSuccess) return (int)e;
  const double wave_reads = (double)blocks * (kThreads / 64) * iters * kReadsPerIter;
  if (ms_per_launch) *ms_per_launch = ms;
  if (wave_reads_per_s) *wave_reads_per_s = wave_reads / (ms * 1e-3);
  return 0;
}

int bridger_calib_global_gather(int32_t width_bytes, int32_t distinct, int32_t buffer_log2,
                                int32_t reps, double *ms_per_launch, double *wave_loads_per_s) {
  if (!(width_bytes == 4 || width_bytes == 8 || width_bytes == 16) || reps < 1 ||
      distinct < 1 || distinct > 64 || (distinct & (distinct - 1)) != 0 || buffer_log2 < 16 ||
      buffer_log2 > 30)
    return (int)hipErrorInvalidValue;
  int32_t n_cu = 0;
  int e0 = bridger_calib_device(&n_cu, nullptr, nullptr);
  if (e0 != 0) return e0;
  const uint32_t bytes = 1u << buffer_log2;
  // lane l, read k: line ((l mod distinct) * 16 + k) * 37 (mod the buffer's lines), at a
  // position inside the line that is a multiple of W
  uint32_t host[64 * kReadsPerIter];
  const uint32_t w = (uint32_t)width_bytes, lines = bytes / 128u;
  for (int k = 0; k < kReadsPerIter; ++k)
    for (int l = 0; l < 64; ++l) {
      const uint32_t src = (uint32_t)(l % distinct);
      const uint32_t line = ((src * 16u + (uint32_t)k) * 37u) % lines;
      host[64 * k + l] = line * 128u + ((src * w) % 128u);
    }
  uint8_t *d_buf = nullptr;
  uint32_t *d_addr = nullptr, *d_sink = nullptr;
  const int blocks = n_cu * kBlocksPerCU;
  hipError_t e = hipMalloc(&d_buf, bytes);
  if (e == hipSuccess) e = hipMalloc(&d_addr, sizeof(host));
  if (e == hipSuccess) e = hipMalloc(&d_sink, sizeof(uint32_t) * (size_t)blocks);
  if (e == hipSuccess) e = hipMemset(d_buf, 3, bytes);
  if (e == hipSuccess) e = hipMemcpy(d_addr, host, sizeof(host), hipMemcpyHostToDevice);
  const int iters = 256;
  double ms = 0.0;
  if (e == hipSuccess) {
    const uint32_t mask = bytes - 1u;
    auto launch = [&]() {
      if (width_bytes == 4)
        hipLaunchKernelGGL(global_gather_kernel<4>, dim3(blocks), dim3(kThreads), 0, nullptr,
                           d_buf, mask, d_addr, iters, d_sink);
      else if (width_bytes == 8)
        hipLaunchKernelGGL(global_gather_kernel<8>, dim3(blocks), dim3(kThreads), 0, nullptr,
                           d_buf, mask, d_addr, iters, d_sink);
      else
        hipLaunchKernelGGL(global_gather_kernel<16>, dim3(blocks), dim3(kThreads), 0, nullptr,
                           d_buf, mask, d_addr, iters, d_sink);
    };
    e = time_ms(launch, reps, &ms);
  }
  if (d_buf) (void)hipFree(d_buf);
  if (d_addr) (void)hipFree(d_addr);
  if (d_sink) (void)hipFree(d_sink);
  if (e != hipSuccess) return (int)e;
  const double wave_loads = (double)blocks * (kThreads / 64) * iters * kReadsPerIter;
  if (ms_per_launch) *ms_per_launch = ms;
  if (wave_loads_per_s) *wave_loads_per_s = wave_loads / (ms * 1e-3);
  return 0;
}

int bridger_calib_copy(int64_t bytes, int32_t reps, double *ms_per_copy, double *bytes_per_s) {
  if (bytes < 16 || reps < 1) return (int)hipErrorInvalidValue;
  const int64_t n = bytes / 16;
  int32_t n_cu = 0;
  int e0 = bridger_calib_device(&n_cu, nullptr, nullptr);
  if (e0 != 0) return e0;
  uint4 *a = nullptr, *b = nullptr;
  hipError_t e = hipMalloc(&a, (size_t)n * 16);
  if (e == hipSuccess) e = hipMalloc(&b, (size_t)n * 16);
  if (e == hipSuccess) e = hipMemset(a, 1, (size_t)n * 16);
  double ms = 0.0;
  if (e == hipSuccess) {
    const int blocks = n_cu * 16;
    auto launch = [&]() {
      hipLaunchKernelGGL(copy_kernel, dim3(blocks), dim3(kThreads), 0, nullptr, a, b, n);
    };
    e = time_ms(launch, reps, &ms);
  }
  if (a) (void)hipFree(a);
  if (b) (void)hipFree(b);
  if (e != hipSuccess) return (int)e;
  if (ms_per_copy) *ms_per_copy = ms;
  if (bytes_per_s) *bytes_per_s = 2.0 * (double)n * 16 / (ms * 1e-3);  // read + write
  return 0;
}

}  // extern "C"
