// perfect_walk.h -- the per-lane walk of perfect trees shared by the PERFECT kernels.
#pragma once
#include "kernel_common.h"

namespace bridger {

// ======================================================================= PERFECT
// Trees are perfect of depth D (layout in internal.h).  The kernel reads the traversal copy
// of the layout, whose records hold {threshold, byte offset of the feature's row in the LDS
// tile} so that the feature gather needs one add.  A lane's state per tree is its 1-based heap
// slot m (root 1, children 2m and 2m + 1); each lane walks U trees at once, so U independent
// LDS reads are in flight per lane.  One level of one tree:
//   rec = LDS[base + 8m]  (64-bit gather),  x = LDS[rec.offset + lane's row]  (32-bit gather),
//   m   = 2m + (x <= rec.threshold ? 0 : 1).
// With only finite thresholds (FIN) the step is computed as the sign bit of threshold - x
// shifted into m by one funnel shift, which needs no compare mask: for finite t and x != NaN
// the IEEE difference t - x is +0 when x == t and otherwise nonzero with the sign of t - x
// (denormals are kept; ties and -0 are handled by storing thresholds of zero as +0), it is
// -inf for x = +inf and +inf for x = -inf, and a NaN feature is stored as +inf, which every
// finite threshold sends right as the compare would.  After D levels m - 2^D is the leaf.
// One level for one tree: record {w, offset} and the lane's feature value (element size XB).
// Bins (XB = 2, 1): w is the threshold's rank k and x <= t_k iff bin <= k, so the step is the
// sign bit of k - bin (both below 2^16).
template <bool FIN, int XB>
__device__ __forceinline__ uint32_t gather_x(const uint8_t *smem, uint32_t addr) {
  if constexpr (XB == 4) return __float_as_uint(lds_f32(smem, addr));
  else if constexpr (XB == 2) return lds_u16(smem, addr);
  else return lds_u8(smem, addr);
}
template <bool FIN, int XB>
__device__ __forceinline__ uint32_t step_slot(uint32_t m, uint32_t w, uint32_t x) {
  if constexpr (XB != 4) {
    return __builtin_amdgcn_alignbit(m, w - x, 31);
  } else if constexpr (FIN) {
    const float diff = __uint_as_float(w) - __uint_as_float(x);
    return __builtin_amdgcn_alignbit(m, __float_as_uint(diff), 31);
  } else {
    return 2u * m + ((__uint_as_float(x) <= __uint_as_float(w)) ? 0u : 1u);
  }
}

template <int D, int U, bool FIN, int XB = 4>
__device__ __forceinline__ void walk_trees(const uint8_t *smem, uint32_t b0, uint32_t tb,
                                           uint32_t lane_off, uint32_t (&m)[U]) {
#pragma unroll
  for (int u = 0; u < U; ++u) m[u] = 1u;
#pragma unroll
  for (int d = 0; d < D; ++d) {
    uint2 rec[U];
    uint32_t xv[U];
#pragma unroll
    for (int u = 0; u < U; ++u) rec[u] = lds_u64(smem, (m[u] << 3) + b0 + (uint32_t)u * tb);
#pragma unroll
    for (int u = 0; u < U; ++u) xv[u] = gather_x<FIN, XB>(smem, rec[u].y + lane_off);
#pragma unroll
    for (int u = 0; u < U; ++u) m[u] = step_slot<FIN, XB>(m[u], rec[u].x, xv[u]);
  }
}

// Same walk with the root records given as wave-uniform values (scalar registers): level 0
// then needs only the feature gather.  Finite thresholds (fp32) or bins (XB = 2, 1).
template <int D, int U, int XB = 4>
__device__ __forceinline__ void walk_trees_root(const uint8_t *smem, uint32_t b0, uint32_t tb,
                                                uint32_t lane_off, const uint2 *root,
                                                uint32_t (&m)[U]) {
  {
    uint32_t xv[U];
#pragma unroll
    for (int u = 0; u < U; ++u) xv[u] = gather_x<true, XB>(smem, root[u].y + lane_off);
#pragma unroll
    for (int u = 0; u < U; ++u) m[u] = step_slot<true, XB>(1u, root[u].x, xv[u]);
  }
#pragma unroll
  for (int d = 1; d < D; ++d) {
    uint2 rec[U];
    uint32_t xv[U];
#pragma unroll
    for (int u = 0; u < U; ++u) rec[u] = lds_u64(smem, (m[u] << 3) + b0 + (uint32_t)u * tb);
#pragma unroll
    for (int u = 0; u < U; ++u) xv[u] = gather_x<true, XB>(smem, rec[u].y + lane_off);
#pragma unroll
    for (int u = 0; u < U; ++u) m[u] = step_slot<true, XB>(m[u], rec[u].x, xv[u]);
  }
}

// The same walk over records read from global memory (L1/L2) instead of an LDS chunk: tree
// u's block starts at byte t0_off + u * tb of `nodes`; the feature values still come from the
// LDS tile.
template <int D, int U, bool FIN, int XB = 4>
__device__ __forceinline__ void walk_trees_global(const uint8_t *smem, const uint8_t *nodes,
                                                  size_t t0_off, uint32_t tb, uint32_t lane_off,
                                                  uint32_t (&m)[U]) {
#pragma unroll
  for (int u = 0; u < U; ++u) m[u] = 1u;
#pragma unroll
  for (int d = 0; d < D; ++d) {
    uint2 rec[U];
    uint32_t xv[U];
#pragma unroll
    for (int u = 0; u < U; ++u)
      rec[u] = *reinterpret_cast<const uint2 *>(nodes + t0_off + (size_t)u * tb + (m[u] << 3));
#pragma unroll
    for (int u = 0; u < U; ++u) xv[u] = gather_x<FIN, XB>(smem, rec[u].y + lane_off);
#pragma unroll
    for (int u = 0; u < U; ++u) m[u] = step_slot<FIN, XB>(m[u], rec[u].x, xv[u]);
  }
}

}  // namespace bridger
