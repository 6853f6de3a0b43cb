// vector_leaves.h -- class sums for forests whose leaves hold K class values (tree classifiers).
#pragma once
#include "kernel_common.h"

namespace bridger {

// Vector leaves: each tree adds its leaf's K class values to all K class sums, which live in
// LDS (slot k * slot_stride) from the start.  vec_add takes the leaves of N consecutive trees
// (the family's leaf indices into a.leaf_vec, whose rows are padded to whole 16-byte groups)
// and adds them class by class in tree order: 16-byte loads (one cache line per lane and
// group of four classes) and one LDS read and write per class for the N trees.
__device__ __forceinline__ void vec_init(const LaunchArgs &a, double *acc_lds, int slot_stride,
                                         bool first_group) {
  for (int k = 0; k < a.K; ++k) acc_lds[k * slot_stride] = class_init(a, k, first_group);
}

template <int N>
__device__ __forceinline__ void vec_add(const LaunchArgs &a, double *acc_lds, int slot_stride,
                                        const int64_t (&leaf)[N]) {
  const int K = a.K, groups = vec_stride(K) >> 2;
  const float4 *v[N];
#pragma unroll
  for (int u = 0; u < N; ++u)
    v[u] = reinterpret_cast<const float4 *>(a.leaf_vec) + leaf[u] * groups;
  for (int k4 = 0; k4 < groups; ++k4) {
    float4 w[N];
#pragma unroll
    for (int u = 0; u < N; ++u) w[u] = v[u][k4];
#pragma unroll
    for (int c = 0; c < 4; ++c) {
      const int k = 4 * k4 + c;
      if (k < K) {
        double s = acc_lds[k * slot_stride];
#pragma unroll
        for (int u = 0; u < N; ++u) s += (double)(c == 0 ? w[u].x : c == 1 ? w[u].y : c == 2 ? w[u].z : w[u].w);
        acc_lds[k * slot_stride] = s;
      }
    }
  }
}

// Class sums in registers for K <= VK (vector kernels with VK = 2, 4 or 8, one or two 16-byte
// groups per leaf row): every class of the padded row is added, so the padding's zeros land
// in accumulators past K, which are never stored.  Per class the trees are added in order.
// (Deferring each group's adds until after the next group's walk, to hide the L2 round trip,
// was measured slower for K <= 4 and cost occupancy for K <= 8.)
template <int VK>
__device__ __forceinline__ void vec_init_reg(const LaunchArgs &a, double (&acc)[VK],
                                             bool first_group) {
#pragma unroll
  for (int k = 0; k < VK; ++k) acc[k] = k < a.K ? class_init(a, k, first_group) : 0.0;
}

template <int N, int VK>
__device__ __forceinline__ void vec_add_reg(const LaunchArgs &a, double (&acc)[VK],
                                            const int64_t (&leaf)[N]) {
#pragma unroll
  for (int u = 0; u < N; ++u) {
    const float4 *v = reinterpret_cast<const float4 *>(a.leaf_vec) + leaf[u] * (VK / 4);
#pragma unroll
    for (int g = 0; g < VK / 4; ++g) {
      const float4 w = v[g];
      acc[4 * g + 0] += (double)w.x;
      acc[4 * g + 1] += (double)w.y;
      acc[4 * g + 2] += (double)w.z;
      acc[4 * g + 3] += (double)w.w;
    }
  }
}

// The same with the leaf rows in LDS (the chunked PERFECT kernel stages them with the tree
// blocks): addr[u] is the byte address of tree u's leaf row, VK floats, 16-byte aligned.
template <int N, int VK>
__device__ __forceinline__ void vec_add_lds(double (&acc)[VK], const uint32_t (&addr)[N]) {
  typedef float f4 __attribute__((ext_vector_type(4)));
  typedef float f2 __attribute__((ext_vector_type(2)));
#pragma unroll
  for (int u = 0; u < N; ++u) {
    if constexpr (VK == 2) {  // two classes: the first half of the 16-byte row
      const f2 w = *(const __attribute__((address_space(3))) f2 *)(uintptr_t)addr[u];
      acc[0] += (double)w.x;
      acc[1] += (double)w.y;
      continue;
    }
#pragma unroll
    for (int g = 0; g < VK / 4; ++g) {
      const f4 w = *(const __attribute__((address_space(3))) f4 *)(uintptr_t)(addr[u] + 16u * g);
      acc[4 * g + 0] += (double)w.x;
      acc[4 * g + 1] += (double)w.y;
      acc[4 * g + 2] += (double)w.z;
      acc[4 * g + 3] += (double)w.w;
    }
  }
}

template <int VK>
__device__ __forceinline__ void vec_store_reg(const LaunchArgs &a, const double (&acc)[VK],
                                              double *acc_lds, int slot_stride) {
#pragma unroll
  for (int k = 0; k < VK; ++k)
    if (k < a.K) acc_lds[k * slot_stride] = acc[k];
}

}  // namespace bridger
