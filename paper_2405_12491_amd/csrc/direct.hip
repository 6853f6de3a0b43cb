// direct.hip -- gfx950 fallback kernel: nodes and features read from global memory.
#include "vector_leaves.h"

namespace bridger {

// ======================================================================== DIRECT
// Fallback for any forest: one row per lane, nodes and features read from global memory.
// VK: 0 scalar leaves; 4 or 8 (K <= VK) or 64 vector leaves (class sums in registers / LDS).
template <bool LEAVES, int VK = 0>
__global__ __launch_bounds__(256) void direct_kernel(LaunchArgs a) {
  extern __shared__ __attribute__((aligned(16))) uint8_t smem[];
  constexpr bool VK_REG = VK == 4 || VK == 8;  // vector leaves, class sums in registers
  constexpr int VR = VK_REG ? VK : 4;
  const int64_t row = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const bool row_ok = row < a.n_rows;
  const int64_t rr = row_ok ? row : 0;
  const float *xr = a.X + rr * (int64_t)a.F;
  const int4 *recs = reinterpret_cast<const int4 *>(a.nodes);
  const int T = a.n_trees;
  double *acc_lds = reinterpret_cast<double *>(smem) + threadIdx.x;
  const int slot_stride = blockDim.x;
  ClassAcc ca;
  ca.k = 0;
  ca.acc = class_init(a, 0, true);
  ca.next_b = a.class_begin[1];
  double vacc[VR];
  if (VK_REG) vec_init_reg(a, vacc, true);
  if (VK == 64) vec_init(a, acc_lds, slot_stride, true);
  for (int t = 0; t < T; ++t) {
    int n = a.tree_start[t];
    int4 rc = recs[n];
    while (rc.y >= 0) {
      const float xv = a.pre_kind ? preprocess(a, rc.y, rr, xr[rc.y]) : xr[rc.y];
      n = (xv <= __int_as_float(rc.x)) ? rc.z : rc.w;
      rc = recs[n];
    }
    if (LEAVES) {
      if (row_ok) a.out_leaf[row * (int64_t)T + a.tree_order[t]] = a.leaf_map[n];
    } else if (VK) {
      const int64_t leaf[1] = {n};
      if (VK_REG) vec_add_reg(a, vacc, leaf);
      else vec_add(a, acc_lds, slot_stride, leaf);
    } else {
      class_advance(a, ca, t, acc_lds, slot_stride, true);
      ca.acc += (double)__int_as_float(rc.x);
    }
  }
  if (LEAVES) return;
  if (VK_REG) {
    vec_store_reg(a, vacc, acc_lds, slot_stride);
  } else if (!VK) {
    class_flush_all(a, ca, acc_lds, slot_stride, true);
  }
  if (row_ok) finalize_store(a, reinterpret_cast<double *>(smem) + threadIdx.x, slot_stride, row);
}

// ---------------------------------------------------------------------- launchers
int launch_direct(const LaunchArgs &a, int64_t n_wg, void *stream) {
  const int lds = a.out_leaf ? 0 : 256 * 8 * a.K;
  if (a.out_leaf) return launch_common(direct_kernel<true>, 256, n_wg, lds, stream, a);
  if (a.vec && a.K <= 4)
    return launch_common(direct_kernel<false, 4>, 256, n_wg, lds, stream, a);
  if (a.vec && a.K <= 8)
    return launch_common(direct_kernel<false, 8>, 256, n_wg, lds, stream, a);
  if (a.vec) return launch_common(direct_kernel<false, 64>, 256, n_wg, lds, stream, a);
  return launch_common(direct_kernel<false>, 256, n_wg, lds, stream, a);
}

}  // namespace bridger
