// perfect_fixed.hip -- compile-time chunk variants of the PERFECT kernel for the common case.
#include "perfect_walk.h"

namespace bridger {

// Compile-time chunk geometry for the common case (one class, one lane group, finite
// thresholds or bins): CT trees per chunk and the tree block size are constants and the chunk
// loop is unrolled over the two buffers, so every tree's LDS base folds into the gathers'
// offset field and a level's node address is a single shift.  A last chunk with fewer than CT
// trees is walked with run-time bases.  XB: fp32 rows (4) or rows of 16- / 8-bit bins.
template <int D, int CT, int XB = 4>
__global__ __launch_bounds__(1024) void perfect_fixed_kernel(LaunchArgs a) {
  extern __shared__ __attribute__((aligned(16))) uint8_t smem[];
  constexpr int U = 4;
  constexpr uint32_t TB = (uint32_t)perfect_tree_bytes(D);
  constexpr uint32_t CB = (uint32_t)CT * TB;
  constexpr uint32_t kLeafOff = 4u << D;
  static_assert(perfect_fixed_ok(D, CT), "chunk geometry outside the offset field");
  const int tid = threadIdx.x;
  const int R = a.rows_per_wg;  // 64 lanes per compute wave, one row each
  const int T = a.n_trees, n_chunks = a.n_chunks;

  if (tid >= R) {
    staging_wave(smem, n_chunks, CB, tid & 63, 0, [&](int c) {
      const int n0 = c * CT, n1 = (n0 + CT < T) ? n0 + CT : T;
      return std::make_pair(a.nodes + (size_t)n0 * TB, (n1 - n0) * (int)TB);
    }, a.csr ? 1 : 0);
    return;
  }

  const int64_t row = (int64_t)blockIdx.x * R + tid;
  const bool row_ok = row < a.n_rows;
  const uint32_t lane_off = (uint32_t)a.lds_x_off + tile_row_off<XB>(tid);
  load_tile_any<XB, true>(smem, a, tid, row, row_ok, 0, 1);
  __syncthreads();

  double acc = a.aggregate == 0 ? (double)a.base[0] : 0.0;
  auto chunk = [&](auto buf_tag, int c) {
    constexpr uint32_t BUF = decltype(buf_tag)::value ? CB : 0u;
    const int t0 = c * CT;
    if (t0 + CT <= T) {
      // the chunk's root records, wave-uniform: scalar loads through the constant address space
      uint2 root[CT];
      typedef __attribute__((address_space(4))) const uint64_t const_u64;
      const_u64 *rt = (const_u64 *)(uintptr_t)a.roots + t0;
#pragma unroll
      for (int j = 0; j < CT; ++j) {
        const uint64_t v = rt[j];
        root[j] = make_uint2((uint32_t)v, (uint32_t)(v >> 32));
      }
#pragma unroll
      for (int j = 0; j < CT / U; ++j) {
        uint32_t m[U];
        walk_trees_root<D, U, XB>(smem, BUF + (uint32_t)(j * U) * TB, TB, lane_off, root + j * U, m);
        float lv[U];
#pragma unroll
        for (int u = 0; u < U; ++u)
          lv[u] = lds_f32(smem, (m[u] << 2) + BUF + (uint32_t)(j * U + u) * TB + kLeafOff);
#pragma unroll
        for (int u = 0; u < U; ++u) acc += (double)lv[u];
      }
    } else {
      int q = t0;
      for (; q + U <= T; q += U) {
        const uint32_t b0 = BUF + (uint32_t)(q - t0) * TB;
        uint32_t m[U];
        walk_trees<D, U, true, XB>(smem, b0, TB, lane_off, m);
        float lv[U];
#pragma unroll
        for (int u = 0; u < U; ++u) lv[u] = lds_f32(smem, (m[u] << 2) + b0 + (uint32_t)u * TB + kLeafOff);
#pragma unroll
        for (int u = 0; u < U; ++u) acc += (double)lv[u];
      }
      for (; q < T; ++q) {
        const uint32_t b0 = BUF + (uint32_t)(q - t0) * TB;
        uint32_t m[1];
        walk_trees<D, 1, true, XB>(smem, b0, TB, lane_off, m);
        acc += (double)lds_f32(smem, (m[0] << 2) + b0 + kLeafOff);
      }
    }
    __syncthreads();
  };
  int c = 0;
  for (; c + 2 <= n_chunks; c += 2) {
    chunk(std::integral_constant<int, 0>{}, c);
    chunk(std::integral_constant<int, 1>{}, c + 1);
  }
  if (c < n_chunks) chunk(std::integral_constant<int, 0>{}, c);
  if (row_ok) {
    double z = acc;
    if (a.aggregate == 1) z = (double)a.base[0] + z / (double)a.class_count[0];
    store_one(a, row, z);
  }
}

// ---------------------------------------------------------------------- launchers
template <int D, int CT>
static int launch_fixed_dc(const LaunchArgs &a, int waves, int64_t n_wg, int lds_bytes,
                           void *stream) {
  if constexpr (perfect_fixed_ok(D, CT)) {
    const int threads = 64 * (waves + 1);
    if (a.x_bytes == 2)
      return launch_common(perfect_fixed_kernel<D, CT, 2>, threads, n_wg, lds_bytes, stream, a);
    if (a.x_bytes == 1)
      return launch_common(perfect_fixed_kernel<D, CT, 1>, threads, n_wg, lds_bytes, stream, a);
    return launch_common(perfect_fixed_kernel<D, CT, 4>, threads, n_wg, lds_bytes, stream, a);
  } else {
    return (int)hipErrorInvalidValue;
  }
}

template <int D>
static int launch_fixed_d(const LaunchArgs &a, int waves, int64_t n_wg, int lds_bytes,
                          void *stream) {
  switch (a.trees_per_chunk) {
    case 4: return launch_fixed_dc<D, 4>(a, waves, n_wg, lds_bytes, stream);
    case 8: return launch_fixed_dc<D, 8>(a, waves, n_wg, lds_bytes, stream);
    case 16: return launch_fixed_dc<D, 16>(a, waves, n_wg, lds_bytes, stream);
    case 32: return launch_fixed_dc<D, 32>(a, waves, n_wg, lds_bytes, stream);
    default: return (int)hipErrorInvalidValue;
  }
}

int launch_perfect_fixed(int depth, const LaunchArgs &a, int waves, int64_t n_wg, int lds_bytes,
                         void *stream) {
  switch (depth) {
    case 2: return launch_fixed_d<2>(a, waves, n_wg, lds_bytes, stream);
    case 3: return launch_fixed_d<3>(a, waves, n_wg, lds_bytes, stream);
    case 4: return launch_fixed_d<4>(a, waves, n_wg, lds_bytes, stream);
    case 5: return launch_fixed_d<5>(a, waves, n_wg, lds_bytes, stream);
    case 6: return launch_fixed_d<6>(a, waves, n_wg, lds_bytes, stream);
    case 7: return launch_fixed_d<7>(a, waves, n_wg, lds_bytes, stream);
    case 8: return launch_fixed_d<8>(a, waves, n_wg, lds_bytes, stream);
    case 9: return launch_fixed_d<9>(a, waves, n_wg, lds_bytes, stream);
    default: return (int)hipErrorInvalidValue;
  }
}

}  // namespace bridger
