// normalize.hip -- gfx950 row-norm pass for the fused Normalizer (unit L2 rows).
#include "kernel_common.h"

#include <mutex>

namespace bridger {

// ================================================================== ROW NORMS
// s = sum of double(x_f)^2, one multiply and one add at a time in the row's order (feature
// order for dense rows, stored order for CSR rows, skipping indices outside [0, F)), then
// norm = sqrt(s), or 1 for an all-zero row.  The squares of floats are exact in double and the
// sum cannot overflow; contraction into fused multiply-adds is disabled so the order of
// roundings is exactly the one stated.  The fused kernels then divide each feature by the
// row's norm in double and round to float.
//
// Dense rows: a one-wave block owns 64 rows and walks the features in slices of 32.  Each slice
// is loaded with 32 independent loads per lane (two rows' 32-feature segments per instruction;
// indices clamped into the rows and the slice, so no load is guarded and all of them are in
// flight at once) into an LDS tile with a row stride of 33 words, so that afterwards every lane
// reads its own row's slice from 32 different banks and carries its row's running sum on.
// Clamped loads only fill tile entries that no lane reads (columns past the slice) or that
// belong to rows past the end (whose norms are not written).
constexpr int kNormRows = 64;
constexpr int kNormSlice = 32, kNormStride = kNormSlice + 1;

__global__ __launch_bounds__(kNormRows) void row_norm_kernel(LaunchArgs a, double *norm) {
#pragma clang fp contract(off)
  __shared__ float tile[kNormRows * kNormStride];
  const int lane = threadIdx.x;
  const int64_t r0 = (int64_t)blockIdx.x * kNormRows;
  const int64_t row = r0 + lane;
  double s = 0.0;
  if (a.csr) {
    if (row >= a.n_rows) return;
    const int64_t p0 = a.csr_indptr[row], p1 = a.csr_indptr[row + 1];
    for (int64_t e = p0; e < p1; ++e) {
      const int f = a.csr_indices[e];
      if (f >= 0 && f < a.F) {
        const double v = (double)a.X[e];
        s = s + v * v;
      }
    }
  } else {
    const int F = a.F;
    const int cc = lane & (kNormSlice - 1), rsub = lane / kNormSlice;  // 2 rows per load
    const int64_t last = a.n_rows - 1;
    for (int f0 = 0; f0 < F; f0 += kNormSlice) {
      const int fc = (F - f0 < kNormSlice) ? F - f0 : kNormSlice;
      const int col = f0 + (cc < fc ? cc : fc - 1);
      float v[kNormRows / 2];
#pragma unroll
      for (int k = 0; k < kNormRows / 2; ++k) {
        const int64_t rw = r0 + 2 * k + rsub;
        v[k] = a.X[(rw < last ? rw : last) * (int64_t)F + col];
      }
#pragma unroll
      for (int k = 0; k < kNormRows / 2; ++k) tile[(2 * k + rsub) * kNormStride + cc] = v[k];
      __syncthreads();
      for (int c = 0; c < fc; ++c) {
        const double x = (double)tile[lane * kNormStride + c];
        s = s + x * x;
      }
      __syncthreads();
    }
    if (row >= a.n_rows) return;
  }
  norm[row] = (s == 0.0) ? 1.0 : __builtin_sqrt(s);
}

int launch_row_norm(const LaunchArgs &a, double *norm, void *stream) {
  const int64_t blocks = (a.n_rows + kNormRows - 1) / kNormRows;
  hipLaunchKernelGGL(row_norm_kernel, dim3((uint32_t)blocks), dim3(kNormRows), 0,
                     (hipStream_t)stream, a, norm);
  return (int)hipGetLastError();
}

// ================================================= scratch of the allocation-free predict
// The row norms of bridger_forest_predict_noalloc live in this file-scope device array (every
// GPU the library runs on holds its own copy until the process ends), so that call allocates
// nothing.  Host code never passes the array's name to a kernel: in host code that name is a
// host-side stand-in, not a device address.  The device address comes from hipGetSymbolAddress,
// taken once per device with that device current, and is passed to the row-norm kernel like
// the stream-ordered buffer of bridger_forest_predict.  The norms are written for every row
// before any kernel reads them, so nothing needs clearing between calls; calls that overlap on
// one GPU (other streams, other handles) share the array and race.
static __device__ __align__(256) double scratch[kNoAllocMaxRows];

int noalloc_norm_scratch(double **ptr) {
  constexpr int kMaxDevices = 64;
  static std::mutex mu;
  static double *addr[kMaxDevices] = {};
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return (int)e;
  if (dev < 0 || dev >= kMaxDevices) return (int)hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(mu);
  if (!addr[dev]) {
    void *p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess || !p) return e != hipSuccess ? (int)e : (int)hipErrorInvalidSymbol;
    addr[dev] = (double *)p;
  }
  *ptr = addr[dev];
  return 0;
}

}  // namespace bridger
