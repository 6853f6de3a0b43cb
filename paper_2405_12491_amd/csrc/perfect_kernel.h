// perfect_kernel.h -- the generic chunked PERFECT kernel (any depth 1..10, classes, lane
// groups, scores or leaf ids), templated on the feature element: fp32 (XB = 4, with the
// sign-of-difference step when every threshold is finite) or bins of XB = 2 or 1 bytes.
#pragma once
#include "perfect_walk.h"
#include "vector_leaves.h"

namespace bridger {

// VK: 0 scalar leaves; 2, 4 or 8 vector leaves (K <= VK) with the class sums in registers (for
// VK = 2 and 4 the leaf rows come with the staged tree blocks, for VK = 8 from global memory);
// 64 vector leaves with the class sums in LDS and the rows from global memory.
// KS: scalar leaves of at most KS classes with the lane group's finished class sums kept in
// registers and written to LDS (into the row tile, whose LDS the plan then shares with them)
// only after the walk.
template <int D, int U, bool LEAVES, bool SIMPLE, bool FIN, int XB, int VK = 0, int KS = 0>
__global__ __launch_bounds__(1024) void perfect_kernel(LaunchArgs a) {
  extern __shared__ __attribute__((aligned(16))) uint8_t smem[];
  constexpr bool VK_REG = VK == 2 || VK == 4 || VK == 8;  // vector leaves, sums in registers
  constexpr int VR = VK_REG ? VK : 4;
  const int tid = threadIdx.x;
  const int R = a.rows_per_wg, G = a.groups;
  const uint32_t tb = (uint32_t)a.tree_bytes;
  const int T = a.n_trees, CT = a.trees_per_chunk;
  if (tid >= G * R) {
    staging_wave(smem, a.n_chunks, (uint32_t)a.chunk_bytes, tid & 63, (LEAVES || SIMPLE) ? 0 : 1,
                 [&](int c) {
                   const int n0 = c * CT, n1 = (n0 + CT < T) ? n0 + CT : T;
                   return std::make_pair(a.nodes + (size_t)n0 * tb, (n1 - n0) * (int)tb);
                 }, a.csr ? 1 : 0);
    return;
  }
  const int r = tid & (R - 1);
  // with R >= 64 a wave lies inside one lane group, so the group index (and every tree
  // address derived from it) is wave-uniform and lives in scalar registers
  const int g = SIMPLE ? 0 : (R >= 64 ? __builtin_amdgcn_readfirstlane(tid / R) : tid / R);
  const int64_t row = (int64_t)blockIdx.x * R + r;
  const bool row_ok = row < a.n_rows;
  const uint32_t lane_off = (uint32_t)a.lds_x_off + tile_row_off<XB>(r);
  // leaf j of a tree is at base + 8 * 2^D + 4j, i.e. base + 4m + 4 * 2^D for final slot m
  constexpr uint32_t kLeafOff = 4u << D;
  constexpr uint32_t kFirstLeaf = 1u << D;

  load_tile_any<XB, FIN>(smem, a, r, row, row_ok, g, G);
  __syncthreads();

  double *acc_lds = reinterpret_cast<double *>(smem + a.lds_acc_off) + g * R + r;
  const int slot_stride = G * R;
  ClassAcc ca;
  ca.k = 0;
  ca.acc = SIMPLE ? (a.aggregate == 0 ? (double)a.base[0] : 0.0) : class_init(a, 0, g == 0);
  ca.next_b = SIMPLE ? 0x7fffffff : a.class_begin[1];
  double vacc[VR];
  if (VK_REG) vec_init_reg(a, vacc, g == 0);
  if (VK == 64) vec_init(a, acc_lds, slot_stride, g == 0);
  // KS: a group walks its trees in ascending (class-sorted) order, so each class is summed in
  // one stretch: the running sum moves to cs[k] when the class changes (rarely)
  double cs[KS > 0 ? KS : 1];
  if (KS) {
#pragma unroll
    for (int c = 0; c < KS; ++c) cs[c] = c < a.K ? class_init(a, c, g == 0) : 0.0;
  }
  auto advance_reg = [&](int t) {
    if (t < ca.next_b) return;
#pragma unroll
    for (int c = 0; c < KS; ++c)
      if (c == ca.k) cs[c] = ca.acc;
    while (t >= ca.next_b) {
      ca.k += 1;
      ca.next_b = a.class_begin[ca.k + 1];
    }
    double v = 0.0;
#pragma unroll
    for (int c = 0; c < KS; ++c)
      if (c == ca.k) v = cs[c];
    ca.acc = v;
  };

  // leaf ids or leaf values of N walked trees, kernel trees q .. q + N - 1
  auto finish = [&](auto &m, int q, uint32_t b0) {
    constexpr int N = sizeof(m) / sizeof(m[0]);
    if (LEAVES) {
#pragma unroll
      for (int u = 0; u < N; ++u) {
        if (row_ok) {
          const int t = q + u;
          a.out_leaf[row * (int64_t)T + a.tree_order[t]] =
              a.leaf_map[(int64_t)t * (1 << D) + (m[u] - kFirstLeaf)];
        }
      }
    } else if (VK == 2 || VK == 4) {
      // the leaf rows (16 bytes) follow the records in the staged tree blocks
      uint32_t addr[N];
#pragma unroll
      for (int u = 0; u < N; ++u)
        addr[u] = b0 + (uint32_t)u * tb + (8u << D) + (m[u] - kFirstLeaf) * 16u;
      vec_add_lds(vacc, addr);
    } else if (VK) {
      int64_t leaf[N];
#pragma unroll
      for (int u = 0; u < N; ++u) leaf[u] = (int64_t)(q + u) * (1 << D) + (m[u] - kFirstLeaf);
      if (VK_REG) vec_add_reg(a, vacc, leaf);
      else vec_add(a, acc_lds, slot_stride, leaf);
    } else {
      float lv[N];
#pragma unroll
      for (int u = 0; u < N; ++u) lv[u] = lds_f32(smem, (m[u] << 2) + b0 + (uint32_t)u * tb + kLeafOff);
#pragma unroll
      for (int u = 0; u < N; ++u) {
        if (KS) advance_reg(q + u);
        else if (!SIMPLE) class_advance(a, ca, q + u, acc_lds, slot_stride, g == 0);
        ca.acc += (double)lv[u];
      }
    }
  };

  for (int c = 0; c < a.n_chunks; ++c) {
    const int t0 = c * CT;
    const int t1 = (t0 + CT < T) ? t0 + CT : T;
    const uint32_t buf = (c & 1) ? (uint32_t)a.chunk_bytes : 0u;
    // whole groups of U trees, then (only when the chunk's tree count leaves one) a partial
    // group walked one tree at a time
    int q = t0 + U * g;
    for (; q + U <= t1; q += U * G) {
      const uint32_t b0 = buf + (uint32_t)(q - t0) * tb;
      uint32_t m[U];
      walk_trees<D, U, FIN, XB>(smem, b0, tb, lane_off, m);
      finish(m, q, b0);
    }
    for (; q < t1; ++q) {
      const uint32_t b0 = buf + (uint32_t)(q - t0) * tb;
      uint32_t m[1];
      walk_trees<D, 1, FIN, XB>(smem, b0, tb, lane_off, m);
      finish(m, q, b0);
    }
    __syncthreads();
  }
  if (LEAVES) return;
  if (SIMPLE) {
    if (row_ok) {
      double z = ca.acc;
      if (a.aggregate == 1) z = (double)a.base[0] + z / (double)a.class_count[0];
      store_one(a, row, z);
    }
    return;
  }
  // With acc_alias the sums below go into the row tile: the last chunk's barrier above has
  // already seen every group finish its walk, so the tile is free.
  if (KS) {
#pragma unroll
    for (int c = 0; c < KS; ++c)
      if (c == ca.k) cs[c] = ca.acc;
#pragma unroll
    for (int c = 0; c < KS; ++c)
      if (c < a.K) acc_lds[c * slot_stride] = cs[c];
  } else if (VK_REG) {
    vec_store_reg(a, vacc, acc_lds, slot_stride);
  } else if (!VK) {
    class_flush_all(a, ca, acc_lds, slot_stride, g == 0);
  }
  __syncthreads();
  groups_finalize_store(a, reinterpret_cast<double *>(smem + a.lds_acc_off), R, G, slot_stride,
                        tid, row, row_ok);
}

// Launch for one depth and element size; U is chosen from the plan (lane-group plans pick it
// to fit the LDS; any plan works with any U since a chunk's last partial group is walked one
// tree at a time).
template <int D, bool FIN, int XB>
static int launch_perfect_dfx(const LaunchArgs &a, int waves, int64_t n_wg, int lds_bytes,
                              void *stream) {
  const bool simple = a.K == 1 && a.groups == 1;
  const int threads = 64 * (waves + 1);  // + the staging wave
  if (a.out_leaf)
    return launch_common(perfect_kernel<D, 4, true, false, FIN, XB>, threads, n_wg, lds_bytes, stream, a);
  if (a.vec && a.K == 2)  // vector leaves: K >= 2, so never the simple variant
    return launch_common(perfect_kernel<D, 4, false, false, FIN, XB, 2>, threads, n_wg, lds_bytes, stream, a);
  if (a.vec && a.K <= 4)
    return launch_common(perfect_kernel<D, 4, false, false, FIN, XB, 4>, threads, n_wg, lds_bytes, stream, a);
  if (a.vec && a.K <= 8)  // two trees per lane: the rows of four would cost occupancy
    return launch_common(perfect_kernel<D, 2, false, false, FIN, XB, 8>, threads, n_wg, lds_bytes, stream, a);
  if (a.vec)
    return launch_common(perfect_kernel<D, 4, false, false, FIN, XB, 64>, threads, n_wg, lds_bytes, stream, a);
  if (simple)
    return launch_common(perfect_kernel<D, 4, false, true, FIN, XB>, threads, n_wg, lds_bytes, stream, a);
  if (a.acc_alias && a.K <= 8 && a.ilp == 4)  // class sums in registers, then into the tile
    return launch_common(perfect_kernel<D, 4, false, false, FIN, XB, 0, 8>, threads, n_wg, lds_bytes, stream, a);
  if (a.ilp == 1)
    return launch_common(perfect_kernel<D, 1, false, false, FIN, XB>, threads, n_wg, lds_bytes, stream, a);
  if (a.ilp == 2)
    return launch_common(perfect_kernel<D, 2, false, false, FIN, XB>, threads, n_wg, lds_bytes, stream, a);
  return launch_common(perfect_kernel<D, 4, false, false, FIN, XB>, threads, n_wg, lds_bytes, stream, a);
}

}  // namespace bridger
