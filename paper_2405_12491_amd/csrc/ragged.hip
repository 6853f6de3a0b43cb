// ragged.hip -- gfx950 kernel for forests of trees of any shape, staged through LDS.
#include "perfect_walk.h"
#include "vector_leaves.h"

namespace bridger {

// x (fp32 bits, or a bin) against an internal record's w (threshold bits, or its rank).
template <int XB>
__device__ __forceinline__ bool goes_right(uint32_t x, uint32_t w) {
  if constexpr (XB == 4) return !(__uint_as_float(x) <= __uint_as_float(w));
  else return x > w;
}

// ======================================================================== RAGGED
// Any tree shape.  Each lane runs a state machine over its group's trees of the chunk: at an
// internal record it gathers x[feature], compares and moves to left or left+1; at a leaf it
// adds the value and jumps to the next tree's root.  Lanes never wait for each other inside
// a chunk, so a short path in one tree is not padded to the wave's longest path.
// VK: 0 scalar leaves; 4 or 8 (K <= VK) or 64 vector leaves (class sums in registers / LDS).
template <bool LEAVES, bool SIMPLE, int XB, int VK = 0>
__global__ __launch_bounds__(1024) void ragged_kernel(LaunchArgs a) {
  extern __shared__ __attribute__((aligned(16))) uint8_t smem[];
  constexpr bool VK_REG = VK == 4 || VK == 8;  // vector leaves, class sums in registers
  constexpr int VR = VK_REG ? VK : 4;
  const int tid = threadIdx.x;
  const int R = a.rows_per_wg, G = a.groups;
  if (tid >= G * R) {
    staging_wave(smem, a.n_chunks, (uint32_t)a.chunk_bytes, tid & 63,
                 (LEAVES || (SIMPLE && G == 1)) ? 0 : 1, [&](int c) {
                   return std::make_pair(a.nodes + 8 * (size_t)a.chunk_rec[c],
                                         8 * (a.chunk_rec[c + 1] - a.chunk_rec[c]));
                 }, a.csr ? 1 : 0);
    return;
  }
  const int r = tid & (R - 1);
  const int g = tid / R;
  const int64_t row = (int64_t)blockIdx.x * R + r;
  const bool row_ok = row < a.n_rows;
  const uint32_t lane_off = (uint32_t)a.lds_x_off + tile_row_off<XB>(r);
  const int shift = a.log2_row_bytes;
  const int T = a.n_trees;

  load_tile_any<XB, false>(smem, a, r, row, row_ok, g, G);
  __syncthreads();

  double *acc_lds = reinterpret_cast<double *>(smem + a.lds_acc_off) + g * R + r;
  const int slot_stride = G * R;
  ClassAcc ca;
  ca.k = 0;
  ca.acc = class_init(a, 0, g == 0);
  ca.next_b = SIMPLE ? 0x7fffffff : a.class_begin[1];
  double vacc[VR];
  if (VK_REG) vec_init_reg(a, vacc, g == 0);
  if (VK == 64) vec_init(a, acc_lds, slot_stride, g == 0);

  for (int c = 0; c < a.n_chunks; ++c) {
    const uint32_t buf = (c & 1) ? (uint32_t)a.chunk_bytes : 0u;
    const int ct0 = a.chunk_first[c], ct1 = a.chunk_first[c + 1];
    const int nt = ct1 - ct0;
    const int ga = ct0 + (int)(((int64_t)nt * g) / G);
    const int gb = ct0 + (int)(((int64_t)nt * (g + 1)) / G);
    const int rec0 = a.chunk_rec[c];
    uint32_t addr = buf + 8u * (uint32_t)(a.tree_start[ga] - rec0);
    const uint32_t end = buf + 8u * (uint32_t)(a.tree_start[gb] - rec0);
    int t = ga;
    while (addr < end) {
      const uint2 rec = lds_u64(smem, addr);
      const uint32_t meta = rec.y;
      const uint32_t xv = gather_x<false, XB>(smem, ((meta >> 16) << shift) + lane_off);
      const bool leaf = (meta & (uint32_t)kLeafFlag) != 0;
      const uint32_t rel = meta & (uint32_t)kMaxRel;
      const bool right = goes_right<XB>(xv, rec.x) && !leaf;
      if (leaf) {
        if (LEAVES) {
          if (row_ok)
            a.out_leaf[row * (int64_t)T + a.tree_order[t]] =
                a.leaf_map[rec0 + (int)((addr - buf) >> 3)];
        } else if (VK) {
          const int64_t leaf[1] = {rec0 + (int)((addr - buf) >> 3)};
          if (VK_REG) vec_add_reg(a, vacc, leaf);
          else vec_add(a, acc_lds, slot_stride, leaf);
        } else {
          if (!SIMPLE) class_advance(a, ca, t, acc_lds, slot_stride, g == 0);
          ca.acc += (double)__uint_as_float(rec.x);
        }
        ++t;
      }
      // a valid record always moves forward (left_rel >= 1, next_rel >= 1); the max keeps the
      // loop finite even on a corrupted record
      const uint32_t step = rel + (right ? 1u : 0u);
      addr += 8u * (step > 1u ? step : 1u);
    }
    __syncthreads();
  }
  if (LEAVES) return;
  if (SIMPLE && G == 1) {
    if (row_ok) {
      double z = ca.acc;
      if (a.aggregate == 1) z = (double)a.base[0] + z / (double)a.class_count[0];
      store_one(a, row, z);
    }
    return;
  }
  if (SIMPLE) {
    acc_lds[0] = ca.acc;
  } else if (VK_REG) {
    vec_store_reg(a, vacc, acc_lds, slot_stride);
  } else if (!VK) {
    class_flush_all(a, ca, acc_lds, slot_stride, g == 0);
  }
  __syncthreads();
  if (g == 0) {
    double *z = reinterpret_cast<double *>(smem + a.lds_acc_off) + r;
    for (int k = 0; k < a.K; ++k) {
      double s = z[k * slot_stride];
      for (int gg = 1; gg < G; ++gg) s += z[k * slot_stride + gg * R];
      z[k * slot_stride] = s;
    }
    if (row_ok) finalize_store(a, z, slot_stride, row);
  }
}

// Records read from global memory instead of LDS chunks (big forests on wide rows, where a
// 64-row tile already takes most of the LDS and restaging every tree for every tile is the
// bottleneck).  G lane groups share the row tile; group g walks the contiguous tree range
// [T g / G, T (g + 1) / G), U trees at a time, in lockstep: the lanes of a wave descend the same
// trees together (a lane that reached its leaf idles until the wave's deepest path ends), so
// one wave-wide gather touches only the few cache lines of those trees' current levels
// rather than records of many trees at once.  Leaves are added in tree order.
template <bool LEAVES, bool SIMPLE, int U, int XB, int VK = 0>
__global__ __launch_bounds__(1024) void ragged_global_kernel(LaunchArgs a) {
  extern __shared__ __attribute__((aligned(16))) uint8_t smem[];
  constexpr bool VK_REG = VK == 4 || VK == 8;  // vector leaves, class sums in registers
  constexpr int VR = VK_REG ? VK : 4;
  const int tid = threadIdx.x;
  const int R = a.rows_per_wg, G = a.groups;
  const int r = tid & (R - 1);
  const int g = tid / R;
  const int64_t row = (int64_t)blockIdx.x * R + r;
  const bool row_ok = row < a.n_rows;
  const uint32_t lane_off = (uint32_t)a.lds_x_off + tile_row_off<XB>(r);
  const int shift = a.log2_row_bytes;
  const int T = a.n_trees;

  load_tile_any<XB, false>(smem, a, r, row, row_ok, g, G);
  __syncthreads();

  double *acc_lds = reinterpret_cast<double *>(smem + a.lds_acc_off) + g * R + r;
  const int slot_stride = G * R;
  ClassAcc ca;
  ca.k = 0;
  ca.acc = class_init(a, 0, g == 0);
  ca.next_b = SIMPLE ? 0x7fffffff : a.class_begin[1];
  double vacc[VR];
  if (VK_REG) vec_init_reg(a, vacc, g == 0);
  if (VK == 64) vec_init(a, acc_lds, slot_stride, g == 0);

  const int ga = (int)(((int64_t)T * g) / G), gb = (int)(((int64_t)T * (g + 1)) / G);
  const uint2 *recs = reinterpret_cast<const uint2 *>(a.nodes);
  // trees q .. q + N - 1 from their roots to their leaves
  auto walk = [&](auto n_tag, int q) {
    constexpr int N = decltype(n_tag)::value;
    int64_t idx[N];
    uint2 rec[N];
#pragma unroll
    for (int u = 0; u < N; ++u) {
      idx[u] = a.tree_start[q + u];
      rec[u] = recs[idx[u]];
    }
    // validated trees are at most 64 deep; the bound keeps the loop finite regardless
    for (int level = 0; level <= 64; ++level) {
      bool inner[N];
      bool any = false;
#pragma unroll
      for (int u = 0; u < N; ++u) {
        inner[u] = (rec[u].y & (uint32_t)kLeafFlag) == 0;
        any = any || inner[u];
      }
      if (!any) break;
      uint32_t xv[N];
#pragma unroll
      for (int u = 0; u < N; ++u)
        xv[u] = gather_x<false, XB>(smem, ((rec[u].y >> 16) << shift) + lane_off);
#pragma unroll
      for (int u = 0; u < N; ++u) {
        if (inner[u]) {
          // left child at rel (>= 1), right child next to it
          const uint32_t rel = rec[u].y & (uint32_t)kMaxRel;
          idx[u] += (int64_t)rel + (goes_right<XB>(xv[u], rec[u].x) ? 1 : 0);
          rec[u] = recs[idx[u]];
        }
      }
    }
    if (VK_REG) {
      vec_add_reg(a, vacc, idx);
      return;
    }
    if (VK == 64) {
      vec_add(a, acc_lds, slot_stride, idx);
      return;
    }
#pragma unroll
    for (int u = 0; u < N; ++u) {
      if (LEAVES) {
        if (row_ok) a.out_leaf[row * (int64_t)T + a.tree_order[q + u]] = a.leaf_map[idx[u]];
      } else {
        if (!SIMPLE) class_advance(a, ca, q + u, acc_lds, slot_stride, g == 0);
        ca.acc += (double)__uint_as_float(rec[u].x);
      }
    }
  };
  int q = ga;
  for (; q + U <= gb; q += U) walk(std::integral_constant<int, U>{}, q);
  for (; q < gb; ++q) walk(std::integral_constant<int, 1>{}, q);
  if (LEAVES) return;
  if (SIMPLE) {
    acc_lds[0] = ca.acc;
  } else if (VK_REG) {
    vec_store_reg(a, vacc, acc_lds, slot_stride);
  } else if (!VK) {
    class_flush_all(a, ca, acc_lds, slot_stride, g == 0);
  }
  __syncthreads();
  if (g == 0) {
    double *z = reinterpret_cast<double *>(smem + a.lds_acc_off) + r;
    for (int k = 0; k < a.K; ++k) {
      double s = z[k * slot_stride];
      for (int gg = 1; gg < G; ++gg) s += z[k * slot_stride + gg * R];
      z[k * slot_stride] = s;
    }
    if (row_ok) finalize_store(a, z, slot_stride, row);
  }
}

// ---------------------------------------------------------------------- launchers
template <int XB, int U>
static int launch_ragged_global_xu(const LaunchArgs &a, int waves, int64_t n_wg, int lds_bytes,
                                   void *stream) {
  const int threads = 64 * waves;
  if (a.out_leaf)
    return launch_common(ragged_global_kernel<true, false, U, XB>, threads, n_wg, lds_bytes, stream, a);
  if (a.vec && a.K <= 4)
    return launch_common(ragged_global_kernel<false, false, 4, XB, 4>, threads, n_wg, lds_bytes, stream, a);
  if (a.vec && a.K <= 8)
    return launch_common(ragged_global_kernel<false, false, 4, XB, 8>, threads, n_wg, lds_bytes, stream, a);
  if (a.vec)
    return launch_common(ragged_global_kernel<false, false, 4, XB, 64>, threads, n_wg, lds_bytes, stream, a);
  if (a.K != 1)
    return launch_common(ragged_global_kernel<false, false, U, XB>, threads, n_wg, lds_bytes, stream, a);
  return launch_common(ragged_global_kernel<false, true, U, XB>, threads, n_wg, lds_bytes, stream, a);
}

template <int XB>
static int launch_ragged_global_x(const LaunchArgs &a, int waves, int64_t n_wg, int lds_bytes,
                                  void *stream) {
  if (a.ilp == 1) return launch_ragged_global_xu<XB, 1>(a, waves, n_wg, lds_bytes, stream);
  if (a.ilp == 2) return launch_ragged_global_xu<XB, 2>(a, waves, n_wg, lds_bytes, stream);
  if (a.ilp == 4) return launch_ragged_global_xu<XB, 4>(a, waves, n_wg, lds_bytes, stream);
  return launch_ragged_global_xu<XB, 8>(a, waves, n_wg, lds_bytes, stream);
}

int launch_ragged_global(const LaunchArgs &a, int waves, int64_t n_wg, int lds_bytes,
                         void *stream) {
  if (a.x_bytes == 2) return launch_ragged_global_x<2>(a, waves, n_wg, lds_bytes, stream);
  if (a.x_bytes == 1) return launch_ragged_global_x<1>(a, waves, n_wg, lds_bytes, stream);
  return launch_ragged_global_x<4>(a, waves, n_wg, lds_bytes, stream);
}

template <int XB>
static int launch_ragged_x(const LaunchArgs &a, int waves, int64_t n_wg, int lds_bytes,
                           void *stream) {
  const bool simple = a.K == 1;
  const int threads = 64 * (waves + 1);  // + the staging wave
  if (a.out_leaf)
    return launch_common(ragged_kernel<true, false, XB>, threads, n_wg, lds_bytes, stream, a);
  if (a.vec && a.K <= 4)
    return launch_common(ragged_kernel<false, false, XB, 4>, threads, n_wg, lds_bytes, stream, a);
  if (a.vec && a.K <= 8)
    return launch_common(ragged_kernel<false, false, XB, 8>, threads, n_wg, lds_bytes, stream, a);
  if (a.vec)
    return launch_common(ragged_kernel<false, false, XB, 64>, threads, n_wg, lds_bytes, stream, a);
  if (simple)
    return launch_common(ragged_kernel<false, true, XB>, threads, n_wg, lds_bytes, stream, a);
  return launch_common(ragged_kernel<false, false, XB>, threads, n_wg, lds_bytes, stream, a);
}

int launch_ragged(const LaunchArgs &a, int waves, int64_t n_wg, int lds_bytes, void *stream) {
  if (a.x_bytes == 2) return launch_ragged_x<2>(a, waves, n_wg, lds_bytes, stream);
  if (a.x_bytes == 1) return launch_ragged_x<1>(a, waves, n_wg, lds_bytes, stream);
  return launch_ragged_x<4>(a, waves, n_wg, lds_bytes, stream);
}

}  // namespace bridger
