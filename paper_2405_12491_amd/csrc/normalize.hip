// normalize.hip -- gfx950 row-norm pass for the fused Normalizer (unit L2 rows).
#include "kernel_common.h"

namespace bridger {

// ================================================================== ROW NORMS
// One lane per row: s = sum of double(x_f)^2, one multiply and one add at a time in the row's
// order (feature order for dense rows, stored order for CSR rows, skipping indices outside
// [0, F)), then norm = sqrt(s), or 1 for an all-zero row.  The squares of floats are exact in
// double and the sum cannot overflow; contraction into fused multiply-adds is disabled so the
// order of roundings is exactly the one stated.  The fused kernels then divide each feature by
// the row's norm in double and round to float.
__global__ __launch_bounds__(256) void row_norm_kernel(LaunchArgs a, double *norm) {
#pragma clang fp contract(off)
  const int64_t row = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (row >= a.n_rows) return;
  double s = 0.0;
  auto add = [&](float x) {
    const double v = (double)x;
    s = s + v * v;
  };
  if (a.csr) {
    const int64_t p0 = a.csr_indptr[row], p1 = a.csr_indptr[row + 1];
    for (int64_t e = p0; e < p1; ++e) {
      const int f = a.csr_indices[e];
      if (f >= 0 && f < a.F) add(a.X[e]);
    }
  } else if (a.x_vec4) {
    const float4 *x4 = reinterpret_cast<const float4 *>(a.X + row * (int64_t)a.F);
    for (int i = 0; i < (a.F >> 2); ++i) {
      const float4 v = x4[i];
      add(v.x);
      add(v.y);
      add(v.z);
      add(v.w);
    }
  } else {
    const float *xr = a.X + row * (int64_t)a.F;
    for (int f = 0; f < a.F; ++f) add(xr[f]);
  }
  norm[row] = (s == 0.0) ? 1.0 : __builtin_sqrt(s);
}

int launch_row_norm(const LaunchArgs &a, double *norm, void *stream) {
  const int64_t blocks = (a.n_rows + 255) / 256;
  hipLaunchKernelGGL(row_norm_kernel, dim3((uint32_t)blocks), dim3(256), 0, (hipStream_t)stream,
                     a, norm);
  return (int)hipGetLastError();
}

}  // namespace bridger
