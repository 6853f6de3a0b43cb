// kernels.hip -- gfx950 kernels for batched tree-ensemble prediction.
//
// One fused kernel per launch runs the whole lowered pipeline of a tree model (Sec. 4.2 and
// Table 4): gather the split feature of the current node (take/gather), compare it with the
// threshold (less_equal), pick the child (where), descend (loop/while), fetch the leaf and
// aggregate over trees (sum/mean), then apply the link function (exp/add/divide/max).  No
// intermediate tensor leaves the chip (the cross-domain fusion idea of Sec. 4.3 applied to
// one model).
//
// Work decomposition (the "tile", "split" and "parallel" schedules of Table 5, sized by the
// Eq. 1 planner on the host):
//   * a workgroup owns R consecutive rows; their features are copied once from HBM into an
//     LDS tile stored feature-major (x of feature f, row r at byte 4*(f*R + r)).  Lane r of
//     every 32-lane half-wave then reads a different LDS bank whatever feature it needs, so
//     the per-lane feature gather is conflict-free;
//   * the trees stream through two LDS chunk buffers: while the waves traverse chunk c, the
//     direct global->LDS loads for chunk c+1 are in flight (one barrier per chunk);
//   * with 64*waves == R every lane owns one row and adds its leaves in ascending tree order
//     (bit-identical to a sequential sum); with 64*waves > R the G = 64*waves/R lane groups
//     split the trees and their per-class partial sums are added in group order at the end.
// Sums are kept in double precision; the output is rounded once to float.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <map>
#include <utility>
#include <type_traits>
#include <mutex>

#include "internal.h"

namespace bridger {

typedef __attribute__((address_space(3))) uint8_t lds_byte;

// The kernels declare no static LDS, so dynamic LDS starts at LDS address 0 and a byte
// offset into it is directly an LDS address (no base add on every access).
__device__ __forceinline__ float lds_f32(const uint8_t *, uint32_t addr) {
  return *(const __attribute__((address_space(3))) float *)(uintptr_t)addr;
}
__device__ __forceinline__ uint2 lds_u64(const uint8_t *, uint32_t addr) {
  const uint64_t v = *(const __attribute__((address_space(3))) uint64_t *)(uintptr_t)addr;
  return make_uint2((uint32_t)v, (uint32_t)(v >> 32));
}
// Stage `bytes` (multiple of 16) from global memory into LDS at byte offset `dst` with
// direct global->LDS loads: each wave instruction moves 1 KB (64 lanes x 16 bytes).
__device__ __forceinline__ void stage_async(uint8_t *smem, uint32_t dst, const uint8_t *src,
                                            int bytes, int wave, int lane, int waves) {
  for (int off = wave * 1024; off < bytes; off += waves * 1024) {
    if (off + lane * 16 < bytes) {
      __builtin_amdgcn_global_load_lds(
          (const void *)(src + off + lane * 16),
          (__attribute__((address_space(3))) void *)((lds_byte *)smem + dst + off), 16, 0, 0);
    }
  }
}

__device__ __forceinline__ void wait_stage() { __builtin_amdgcn_s_waitcnt(0); }

// Body of the staging wave that the chunked kernels add after their compute waves: it stages
// chunk 0, then during chunk c the chunk c + 1 into the other buffer, and meets the compute
// waves at each of their barriers (1 after the tile load, 1 per chunk, `tail` after the
// loop).  The compute waves never issue direct global->LDS loads, so they never wait for
// staging traffic; the barrier alone orders a chunk's arrival before its use.
// chunk_src(c) -> {global source, bytes} of chunk c.
template <class ChunkSrc>
__device__ __forceinline__ void staging_wave(uint8_t *smem, int n_chunks, uint32_t chunk_bytes,
                                             int lane, int tail, ChunkSrc chunk_src) {
  {
    const auto src = chunk_src(0);
    stage_async(smem, 0, src.first, src.second, 0, lane, 1);
    wait_stage();
  }
  __syncthreads();
  for (int c = 0; c < n_chunks; ++c) {
    if (c + 1 < n_chunks) {
      const auto src = chunk_src(c + 1);
      stage_async(smem, ((c + 1) & 1) ? chunk_bytes : 0u, src.first, src.second, 0, lane, 1);
      wait_stage();
    }
    __syncthreads();
  }
  for (int i = 0; i < tail; ++i) __syncthreads();
}

// Load this lane's row into the feature-major LDS tile (zeros past the last row).  With
// NAN_TO_INF a NaN feature is stored as +inf: against finite thresholds both compare false
// (x <= t), so every split sends them the same way.
template <bool NAN_TO_INF = false>
__device__ __forceinline__ void load_row_tile(uint8_t *smem, const LaunchArgs &a, int r,
                                              int64_t row, bool row_ok) {
  float *xt = reinterpret_cast<float *>(smem + a.lds_x_off);
  const int R = a.rows_per_wg;
  auto put = [&](int f, float v) {
    if (NAN_TO_INF) v = (v != v) ? __builtin_inff() : v;
    xt[f * R + r] = v;
  };
  if (!row_ok) {
    for (int f = 0; f < a.F; ++f) xt[f * R + r] = 0.0f;
    return;
  }
  const float *xr = a.X + row * (int64_t)a.F;
  if (a.x_vec4) {
    const float4 *x4 = reinterpret_cast<const float4 *>(xr);
    const int n4 = a.F >> 2;
    int i = 0;
    for (; i + 2 <= n4; i += 2) {
      float4 v0 = x4[i], v1 = x4[i + 1];
      put(4 * i + 0, v0.x);
      put(4 * i + 1, v0.y);
      put(4 * i + 2, v0.z);
      put(4 * i + 3, v0.w);
      put(4 * i + 4, v1.x);
      put(4 * i + 5, v1.y);
      put(4 * i + 6, v1.z);
      put(4 * i + 7, v1.w);
    }
    for (; i < n4; ++i) {
      float4 v = x4[i];
      put(4 * i + 0, v.x);
      put(4 * i + 1, v.y);
      put(4 * i + 2, v.z);
      put(4 * i + 3, v.w);
    }
  } else {
    for (int f = 0; f < a.F; ++f) put(f, xr[f]);
  }
}

__device__ __forceinline__ double sigmoid_d(double z) {
  if (z >= 0.0) return 1.0 / (1.0 + exp(-z));
  const double e = exp(z);
  return e / (1.0 + e);
}

// Finish class values z[0..K) held in LDS (stride `stride` doubles) and store the row.
__device__ void finalize_store(const LaunchArgs &a, double *z, int stride, int64_t row) {
  const int K = a.K;
  for (int k = 0; k < K; ++k) {
    double v = z[k * stride];
    if (a.aggregate == 1) v = (double)a.base[k] + v / (double)a.class_count[k];
    z[k * stride] = v;
  }
  float *o = a.out + row * (int64_t)K;
  if (a.transform == 1) {
    o[0] = (float)sigmoid_d(z[0]);
  } else if (a.transform == 2) {
    double m = z[0];
    for (int k = 1; k < K; ++k) m = z[k * stride] > m ? z[k * stride] : m;
    double s = 0.0;
    for (int k = 0; k < K; ++k) {
      const double e = exp(z[k * stride] - m);
      z[k * stride] = e;
      s += e;
    }
    for (int k = 0; k < K; ++k) o[k] = (float)(z[k * stride] / s);
  } else {
    for (int k = 0; k < K; ++k) o[k] = (float)z[k * stride];
  }
}

// Per-lane class bookkeeping for forests with several classes or several tree groups.
struct ClassAcc {
  double acc;
  int k;       // class being accumulated
  int next_b;  // first kernel tree of class k+1
};

__device__ __forceinline__ double class_init(const LaunchArgs &a, int k, bool first_group) {
  return (a.aggregate == 0 && first_group) ? (double)a.base[k] : 0.0;
}

__device__ __forceinline__ void class_advance(const LaunchArgs &a, ClassAcc &c, int t,
                                              double *acc_lds, int slot_stride, bool first_group) {
  while (t >= c.next_b) {
    acc_lds[c.k * slot_stride] = c.acc;
    c.k += 1;
    c.acc = class_init(a, c.k, first_group);
    c.next_b = a.class_begin[c.k + 1];
  }
}

__device__ __forceinline__ void class_flush_all(const LaunchArgs &a, ClassAcc &c,
                                                double *acc_lds, int slot_stride,
                                                bool first_group) {
  while (c.k < a.K) {
    acc_lds[c.k * slot_stride] = c.acc;
    c.k += 1;
    if (c.k < a.K) c.acc = class_init(a, c.k, first_group);
  }
}

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
template <int D, int U, bool FIN>
__device__ __forceinline__ void walk_trees(const uint8_t *smem, uint32_t b0, uint32_t tb,
                                           uint32_t lane_off, uint32_t (&m)[U]) {
#pragma unroll
  for (int u = 0; u < U; ++u) m[u] = 1u;
#pragma unroll
  for (int d = 0; d < D; ++d) {
    uint2 rec[U];
    float xv[U];
#pragma unroll
    for (int u = 0; u < U; ++u) rec[u] = lds_u64(smem, (m[u] << 3) + b0 + (uint32_t)u * tb);
#pragma unroll
    for (int u = 0; u < U; ++u) xv[u] = lds_f32(smem, rec[u].y + lane_off);
#pragma unroll
    for (int u = 0; u < U; ++u) {
      if (FIN) {
        const float diff = __uint_as_float(rec[u].x) - xv[u];
        m[u] = __builtin_amdgcn_alignbit(m[u], __float_as_uint(diff), 31);
      } else {
        m[u] = 2u * m[u] + ((xv[u] <= __uint_as_float(rec[u].x)) ? 0u : 1u);
      }
    }
  }
}

// Same walk with the root records given as wave-uniform values (scalar registers): level 0
// then needs only the feature gather.
template <int D, int U>
__device__ __forceinline__ void walk_trees_root(const uint8_t *smem, uint32_t b0, uint32_t tb,
                                                uint32_t lane_off, const uint2 *root,
                                                uint32_t (&m)[U]) {
  {
    float xv[U];
#pragma unroll
    for (int u = 0; u < U; ++u) xv[u] = lds_f32(smem, root[u].y + lane_off);
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const float diff = __uint_as_float(root[u].x) - xv[u];
      m[u] = __builtin_amdgcn_alignbit(1u, __float_as_uint(diff), 31);
    }
  }
#pragma unroll
  for (int d = 1; d < D; ++d) {
    uint2 rec[U];
    float xv[U];
#pragma unroll
    for (int u = 0; u < U; ++u) rec[u] = lds_u64(smem, (m[u] << 3) + b0 + (uint32_t)u * tb);
#pragma unroll
    for (int u = 0; u < U; ++u) xv[u] = lds_f32(smem, rec[u].y + lane_off);
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const float diff = __uint_as_float(rec[u].x) - xv[u];
      m[u] = __builtin_amdgcn_alignbit(m[u], __float_as_uint(diff), 31);
    }
  }
}

template <int D, int U, bool LEAVES, bool SIMPLE, bool FIN>
__global__ __launch_bounds__(1024) void perfect_kernel(LaunchArgs a) {
  extern __shared__ __attribute__((aligned(16))) uint8_t smem[];
  const int tid = threadIdx.x;
  const int R = a.rows_per_wg, G = a.groups;
  const uint32_t tb = (uint32_t)a.tree_bytes;
  const int T = a.n_trees, CT = a.trees_per_chunk;
  if (tid >= G * R) {
    staging_wave(smem, a.n_chunks, (uint32_t)a.chunk_bytes, tid & 63, (LEAVES || SIMPLE) ? 0 : 1,
                 [&](int c) {
                   const int n0 = c * CT, n1 = (n0 + CT < T) ? n0 + CT : T;
                   return std::make_pair(a.nodes + (size_t)n0 * tb, (n1 - n0) * (int)tb);
                 });
    return;
  }
  const int r = tid & (R - 1);
  // with R >= 64 a wave lies inside one lane group, so the group index (and every tree
  // address derived from it) is wave-uniform and lives in scalar registers
  const int g = SIMPLE ? 0 : (R >= 64 ? __builtin_amdgcn_readfirstlane(tid / R) : tid / R);
  const int64_t row = (int64_t)blockIdx.x * R + r;
  const bool row_ok = row < a.n_rows;
  const uint32_t lane_off = (uint32_t)a.lds_x_off + 4u * (uint32_t)r;
  // leaf j of a tree is at base + 8 * 2^D + 4j, i.e. base + 4m + 4 * 2^D for final slot m
  constexpr uint32_t kLeafOff = 4u << D;
  constexpr uint32_t kFirstLeaf = 1u << D;

  if (g == 0) load_row_tile<FIN>(smem, a, r, row, row_ok);
  __syncthreads();

  double *acc_lds = reinterpret_cast<double *>(smem + a.lds_acc_off) + g * R + r;
  const int slot_stride = G * R;
  ClassAcc ca;
  ca.k = 0;
  ca.acc = SIMPLE ? (a.aggregate == 0 ? (double)a.base[0] : 0.0) : class_init(a, 0, g == 0);
  ca.next_b = SIMPLE ? 0x7fffffff : a.class_begin[1];

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
    } else {
      float lv[N];
#pragma unroll
      for (int u = 0; u < N; ++u) lv[u] = lds_f32(smem, (m[u] << 2) + b0 + (uint32_t)u * tb + kLeafOff);
#pragma unroll
      for (int u = 0; u < N; ++u) {
        if (!SIMPLE) class_advance(a, ca, q + u, acc_lds, slot_stride, g == 0);
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
      walk_trees<D, U, FIN>(smem, b0, tb, lane_off, m);
      finish(m, q, b0);
    }
    for (; q < t1; ++q) {
      const uint32_t b0 = buf + (uint32_t)(q - t0) * tb;
      uint32_t m[1];
      walk_trees<D, 1, FIN>(smem, b0, tb, lane_off, m);
      finish(m, q, b0);
    }
    __syncthreads();
  }
  if (LEAVES) return;
  if (SIMPLE) {
    if (row_ok) {
      double z = ca.acc;
      if (a.aggregate == 1) z = (double)a.base[0] + z / (double)a.class_count[0];
      a.out[row] = (float)(a.transform == 1 ? sigmoid_d(z) : z);
    }
    return;
  }
  class_flush_all(a, ca, acc_lds, slot_stride, g == 0);
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

// Compile-time chunk geometry for the common case (one class, one lane group, finite
// thresholds): CT trees per chunk and the tree block size are constants and the chunk loop is
// unrolled over the two buffers, so every tree's LDS base folds into the gathers' offset field
// and a level's node address is a single shift.  A last chunk with fewer than CT trees is
// walked with run-time bases.
template <int D, int CT>
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
    });
    return;
  }

  const int64_t row = (int64_t)blockIdx.x * R + tid;
  const bool row_ok = row < a.n_rows;
  const uint32_t lane_off = (uint32_t)a.lds_x_off + 4u * (uint32_t)tid;
  load_row_tile<true>(smem, a, tid, row, row_ok);
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
        walk_trees_root<D, U>(smem, BUF + (uint32_t)(j * U) * TB, TB, lane_off, root + j * U, m);
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
        walk_trees<D, U, true>(smem, b0, TB, lane_off, m);
        float lv[U];
#pragma unroll
        for (int u = 0; u < U; ++u) lv[u] = lds_f32(smem, (m[u] << 2) + b0 + (uint32_t)u * TB + kLeafOff);
#pragma unroll
        for (int u = 0; u < U; ++u) acc += (double)lv[u];
      }
      for (; q < T; ++q) {
        const uint32_t b0 = BUF + (uint32_t)(q - t0) * TB;
        uint32_t m[1];
        walk_trees<D, 1, true>(smem, b0, TB, lane_off, m);
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
    a.out[row] = (float)(a.transform == 1 ? sigmoid_d(z) : z);
  }
}

// ======================================================================== RAGGED
// Any tree shape.  Each lane runs a state machine over its group's trees of the chunk: at an
// internal record it gathers x[feature], compares and moves to left or left+1; at a leaf it
// adds the value and jumps to the next tree's root.  Lanes never wait for each other inside
// a chunk, so a short path in one tree is not padded to the wave's longest path.
template <bool LEAVES, bool SIMPLE>
__global__ __launch_bounds__(1024) void ragged_kernel(LaunchArgs a) {
  extern __shared__ __attribute__((aligned(16))) uint8_t smem[];
  const int tid = threadIdx.x;
  const int R = a.rows_per_wg, G = a.groups;
  if (tid >= G * R) {
    staging_wave(smem, a.n_chunks, (uint32_t)a.chunk_bytes, tid & 63,
                 (LEAVES || (SIMPLE && G == 1)) ? 0 : 1, [&](int c) {
                   return std::make_pair(a.nodes + 8 * (size_t)a.chunk_rec[c],
                                         8 * (a.chunk_rec[c + 1] - a.chunk_rec[c]));
                 });
    return;
  }
  const int r = tid & (R - 1);
  const int g = tid / R;
  const int64_t row = (int64_t)blockIdx.x * R + r;
  const bool row_ok = row < a.n_rows;
  const uint32_t lane_off = (uint32_t)a.lds_x_off + 4u * (uint32_t)r;
  const int shift = a.log2_row_bytes;
  const int T = a.n_trees;

  if (g == 0) load_row_tile(smem, a, r, row, row_ok);
  __syncthreads();

  double *acc_lds = reinterpret_cast<double *>(smem + a.lds_acc_off) + g * R + r;
  const int slot_stride = G * R;
  ClassAcc ca;
  ca.k = 0;
  ca.acc = class_init(a, 0, g == 0);
  ca.next_b = SIMPLE ? 0x7fffffff : a.class_begin[1];

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
      const float xv = lds_f32(smem, ((meta >> 16) << shift) + lane_off);
      const bool leaf = (meta & (uint32_t)kLeafFlag) != 0;
      const uint32_t rel = meta & (uint32_t)kMaxRel;
      const bool right = !(xv <= __uint_as_float(rec.x)) && !leaf;
      if (leaf) {
        if (LEAVES) {
          if (row_ok)
            a.out_leaf[row * (int64_t)T + a.tree_order[t]] =
                a.leaf_map[rec0 + (int)((addr - buf) >> 3)];
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
      a.out[row] = (float)(a.transform == 1 ? sigmoid_d(z) : z);
    }
    return;
  }
  if (SIMPLE) {
    acc_lds[0] = ca.acc;
  } else {
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

// ======================================================================== DIRECT
// Fallback for any forest: one row per lane, nodes and features read from global memory.
template <bool LEAVES>
__global__ __launch_bounds__(256) void direct_kernel(LaunchArgs a) {
  extern __shared__ __attribute__((aligned(16))) uint8_t smem[];
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
  for (int t = 0; t < T; ++t) {
    int n = a.tree_start[t];
    int4 rc = recs[n];
    while (rc.y >= 0) {
      const float xv = xr[rc.y];
      n = (xv <= __int_as_float(rc.x)) ? rc.z : rc.w;
      rc = recs[n];
    }
    if (LEAVES) {
      if (row_ok) a.out_leaf[row * (int64_t)T + a.tree_order[t]] = a.leaf_map[n];
    } else {
      class_advance(a, ca, t, acc_lds, slot_stride, true);
      ca.acc += (double)__int_as_float(rc.x);
    }
  }
  if (LEAVES) return;
  class_flush_all(a, ca, acc_lds, slot_stride, true);
  if (row_ok) finalize_store(a, reinterpret_cast<double *>(smem) + threadIdx.x, slot_stride, row);
}

// ========================================================================== GEMM
// The matrix-multiply lowering of a tree ensemble (Table 4's matmul and one_hot, in the
// style of the GEMM strategy for shallow trees), kept as a measured alternative to the
// traversal kernels for perfect trees of depth D <= 4, one output class and at most 64
// features.  Per wave: a tile of 16 rows; per block of 16 node columns (16 / 2^D trees,
// column j = tree u = j >> D, 1-based heap slot m = j & (2^D - 1), m = 0 unused):
//   1. S = X_tile (16 x F) . A (F x 16) on v_mfma_f32_16x16x4f32, A one-hot (A[f][j] = 1 iff
//      feature(j) = f): S[i][j] = x[i][feature(j)], exact for finite x;
//   2. bits[i][j] = S[i][j] <= threshold(j) (the direction at every internal node);
//   3. P = bits (16 x 32, upper 16 columns zero) . Cm (32 x 16) on v_mfma_i32_16x16x32_i8, where
//      Cm[j][L] = +1 if node j lies on leaf L's path and the path turns left there, -1 if it
//      turns right, 0 otherwise; the leaf reached is the unique L with P[i][L] equal to the
//      number of left turns on L's path (D - popcount of L's slot);
//   4. that leaf's value is added into per-lane double accumulators, reduced across the 16
//      leaf columns at the end.
// A row holding a non-finite feature breaks step 1 (0 * inf = NaN), so such rows are
// detected while loading and recomputed by a plain root-to-leaf walk.
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef int i32x4 __attribute__((ext_vector_type(4)));

template <int D, bool LEAVES>
__global__ __launch_bounds__(256) void gemm_kernel(LaunchArgs a) {
  constexpr int kSlots = 1 << D;          // heap slots per tree incl. the unused slot 0
  constexpr int kTpb = 16 / kSlots;       // trees per 16-column block
  __shared__ __attribute__((aligned(16))) uint8_t bits_lds[4][16 * 16];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int64_t row0 = ((int64_t)blockIdx.x * 4 + wave) * 16;
  const int F = a.F, T = a.n_trees;
  const int n_steps = (F + 3) >> 2;       // K = 4 features per f32 MFMA
  const uint32_t tb = (uint32_t)a.tree_bytes;
  const uint8_t *blob = a.nodes;
  const int col = lane & 15, grp = lane >> 4;

  // A operand of step 1: lane (i = col, k = grp) holds x[row0 + i][4s + k] for every step s
  float xa[16];
  bool nonfinite = false;
  {
    const int64_t row = row0 + col;
#pragma unroll
    for (int s = 0; s < 16; ++s) {
      const int f = 4 * s + grp;
      float v = 0.0f;
      if (s < n_steps && f < F && row < a.n_rows) v = a.X[row * (int64_t)F + f];
      nonfinite |= !__builtin_isfinite(v);
      xa[s] = v;
    }
  }
  // rows with a non-finite feature: bit i of the mask (lanes i, i+16, i+32, i+48 hold row i)
  uint64_t nf = __ballot(nonfinite);
  const uint32_t nf_rows = (uint32_t)((nf | (nf >> 16) | (nf >> 32) | (nf >> 48)) & 0xFFFFu);

  // B operand of step 3 (constant for depth D): lane (L = col, k-block = grp) holds
  // Cm[8*grp + t][L] for t = 0..7 as signed bytes; node columns >= 16 are zero
  long cm = 0;
  if (grp < 2) {
    const int uL = col >> D, s_leaf = col & (kSlots - 1);
    const int h = kSlots + s_leaf;  // the leaf's 1-based heap slot
    for (int t = 0; t < 8; ++t) {
      const int j = 8 * grp + t;
      const int uj = j >> D, m = j & (kSlots - 1);
      int c = 0;
      if (uj == uL && m >= 1) {
        int dm = 0;
        while ((2 << dm) <= m) ++dm;  // depth of slot m
        const int below = D - dm;     // levels from m down to the leaf
        if ((h >> below) == m) c = ((h >> (below - 1)) & 1) ? -1 : 1;
      }
      cm |= (long)(uint8_t)(int8_t)c << (8 * t);
    }
  }
  const int nleft = D - __builtin_popcount(col & (kSlots - 1));

  double acc[4] = {0.0, 0.0, 0.0, 0.0};
  for (int t0 = 0; t0 < T; t0 += kTpb) {
    // this lane's node column (for steps 1-2) and leaf column (step 4) share index col
    const int u = col >> D, m = col & (kSlots - 1);
    const int t = t0 + u;
    const bool tree_ok = t < T;
    float thr = 0.0f;
    int feat = -1;
    float leaf = 0.0f;
    if (tree_ok) {
      const uint8_t *tp = blob + (size_t)t * tb;
      if (m >= 1) {
        thr = *reinterpret_cast<const float *>(tp + 8 * m);
        feat = *reinterpret_cast<const int32_t *>(tp + 8 * m + 4);
      }
      leaf = *reinterpret_cast<const float *>(tp + 8 * kSlots + 4 * m);
    }
    // step 1: S = X . one_hot
    f32x4 sacc = {0.0f, 0.0f, 0.0f, 0.0f};
    const int fk = feat - grp;  // lane (j, k) contributes 1 at step s iff 4s + k == feat(j)
#pragma unroll
    for (int s = 0; s < 16; ++s) {
      if (s < n_steps) {
        const float b = (fk == 4 * s) ? 1.0f : 0.0f;
        sacc = __builtin_amdgcn_mfma_f32_16x16x4f32(xa[s], b, sacc, 0, 0, 0);
      }
    }
    // step 2: directions; rows 4*grp + r of column col
    uint8_t *bl = bits_lds[wave];
#pragma unroll
    for (int r = 0; r < 4; ++r) bl[(4 * grp + r) * 16 + col] = (sacc[r] <= thr) ? 1 : 0;
    __builtin_amdgcn_s_waitcnt(0xc07f);  // lgkmcnt(0): the wave's own LDS writes are done
    __builtin_amdgcn_wave_barrier();
    long bits = 0;
    if (grp < 2) bits = *reinterpret_cast<const long *>(bl + col * 16 + 8 * grp);
    __builtin_amdgcn_wave_barrier();
    // step 3: path match
    i32x4 z = {0, 0, 0, 0};
    const i32x4 pm = __builtin_amdgcn_mfma_i32_16x16x32_i8(bits, cm, z, 0, 0, 0);
    // step 4: the matching leaf column contributes its value
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const bool hit = tree_ok && pm[r] == nleft;
      if (LEAVES) {
        const int64_t row = row0 + 4 * grp + r;
        if (hit && row < a.n_rows && !((nf_rows >> (4 * grp + r)) & 1))
          a.out_leaf[row * (int64_t)T + a.tree_order[t]] = a.leaf_map[(int64_t)t * kSlots + m];
      } else {
        acc[r] += hit ? (double)leaf : 0.0;
      }
    }
  }
  if (!LEAVES) {
    // sum the 16 leaf columns of each row (lanes 16*grp .. 16*grp + 15), fixed order
#pragma unroll
    for (int r = 0; r < 4; ++r) {
#pragma unroll
      for (int off = 1; off < 16; off <<= 1) acc[r] += __shfl_xor(acc[r], off, 16);
    }
    if (col == 0) {
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int64_t row = row0 + 4 * grp + r;
        if (row < a.n_rows && !((nf_rows >> (4 * grp + r)) & 1)) {
          double zv = acc[r];
          if (a.aggregate == 1) zv = (double)a.base[0] + zv / (double)a.class_count[0];
          else zv += (double)a.base[0];
          a.out[row] = (float)(a.transform == 1 ? sigmoid_d(zv) : zv);
        }
      }
    }
  }
  // rows with a non-finite feature: root-to-leaf walk, one lane per row
  if (nf_rows && lane < 16 && ((nf_rows >> lane) & 1)) {
    const int64_t row = row0 + lane;
    if (row < a.n_rows) {
      const float *xr = a.X + row * (int64_t)F;
      double zv = a.aggregate == 0 ? (double)a.base[0] : 0.0;
      for (int t = 0; t < T; ++t) {
        const uint8_t *tp = blob + (size_t)t * tb;
        int mm = 1;
        for (int d = 0; d < D; ++d) {
          const float th = *reinterpret_cast<const float *>(tp + 8 * mm);
          const int f = *reinterpret_cast<const int32_t *>(tp + 8 * mm + 4);
          mm = 2 * mm + ((xr[f] <= th) ? 0 : 1);
        }
        if (LEAVES)
          a.out_leaf[row * (int64_t)T + a.tree_order[t]] =
              a.leaf_map[(int64_t)t * kSlots + (mm - kSlots)];
        else
          zv += (double)*reinterpret_cast<const float *>(tp + 8 * kSlots + 4 * (mm - kSlots));
      }
      if (!LEAVES) {
        if (a.aggregate == 1) zv = (double)a.base[0] + zv / (double)a.class_count[0];
        a.out[row] = (float)(a.transform == 1 ? sigmoid_d(zv) : zv);
      }
    }
  }
}

// ====================================================================== launchers
// Raise a kernel's dynamic-LDS limit once per (kernel, device) to the largest size used.
static int ensure_lds_limit(const void *kernel, int lds_bytes) {
  static std::mutex mu;
  static std::map<std::pair<const void *, int>, int> limits;
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return (int)hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(mu);
  int &cur = limits[{kernel, dev}];
  if (lds_bytes <= cur) return 0;
  hipError_t e = hipFuncSetAttribute(kernel, hipFuncAttributeMaxDynamicSharedMemorySize, lds_bytes);
  if (e != hipSuccess) return (int)e;
  cur = lds_bytes;
  return 0;
}

template <class K>
static int launch_common(K kernel, int threads, int64_t n_wg, int lds_bytes, void *stream,
                         const LaunchArgs &a) {
  const int e = ensure_lds_limit((const void *)kernel, lds_bytes);
  if (e != 0) return e;
  hipLaunchKernelGGL(kernel, dim3((unsigned)n_wg), dim3(threads), lds_bytes,
                     (hipStream_t)stream, a);
  return (int)hipGetLastError();
}

template <int D, bool FIN>
static int launch_perfect_df(const LaunchArgs &a, int waves, int64_t n_wg, int lds_bytes,
                             void *stream) {
  const bool simple = a.K == 1 && a.groups == 1;
  const int threads = 64 * (waves + 1);  // + the staging wave
  if (a.out_leaf)
    return launch_common(perfect_kernel<D, 4, true, false, FIN>, threads, n_wg, lds_bytes, stream, a);
  if (a.ilp == 8) {
    if (simple)
      return launch_common(perfect_kernel<D, 8, false, true, FIN>, threads, n_wg, lds_bytes, stream, a);
    return launch_common(perfect_kernel<D, 8, false, false, FIN>, threads, n_wg, lds_bytes, stream, a);
  }
  if (simple)
    return launch_common(perfect_kernel<D, 4, false, true, FIN>, threads, n_wg, lds_bytes, stream, a);
  return launch_common(perfect_kernel<D, 4, false, false, FIN>, threads, n_wg, lds_bytes, stream, a);
}

template <int D>
static int launch_perfect_d(const LaunchArgs &a, int waves, int64_t n_wg, int lds_bytes,
                            void *stream) {
  return a.finite_thresholds ? launch_perfect_df<D, true>(a, waves, n_wg, lds_bytes, stream)
                             : launch_perfect_df<D, false>(a, waves, n_wg, lds_bytes, stream);
}

int launch_perfect(int depth, const LaunchArgs &a, int waves, int64_t n_wg, int lds_bytes,
                   void *stream) {
  switch (depth) {
    case 1: return launch_perfect_d<1>(a, waves, n_wg, lds_bytes, stream);
    case 2: return launch_perfect_d<2>(a, waves, n_wg, lds_bytes, stream);
    case 3: return launch_perfect_d<3>(a, waves, n_wg, lds_bytes, stream);
    case 4: return launch_perfect_d<4>(a, waves, n_wg, lds_bytes, stream);
    case 5: return launch_perfect_d<5>(a, waves, n_wg, lds_bytes, stream);
    case 6: return launch_perfect_d<6>(a, waves, n_wg, lds_bytes, stream);
    case 7: return launch_perfect_d<7>(a, waves, n_wg, lds_bytes, stream);
    case 8: return launch_perfect_d<8>(a, waves, n_wg, lds_bytes, stream);
    case 9: return launch_perfect_d<9>(a, waves, n_wg, lds_bytes, stream);
    case 10: return launch_perfect_d<10>(a, waves, n_wg, lds_bytes, stream);
    default: return (int)hipErrorInvalidValue;
  }
}

template <int D, int CT>
static int launch_fixed_dc(const LaunchArgs &a, int waves, int64_t n_wg, int lds_bytes,
                           void *stream) {
  if constexpr (perfect_fixed_ok(D, CT))
    return launch_common(perfect_fixed_kernel<D, CT>, 64 * (waves + 1), n_wg, lds_bytes, stream, a);
  else
    return (int)hipErrorInvalidValue;
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

int launch_ragged(const LaunchArgs &a, int waves, int64_t n_wg, int lds_bytes, void *stream) {
  const bool simple = a.K == 1;
  const int threads = 64 * (waves + 1);  // + the staging wave
  if (a.out_leaf) return launch_common(ragged_kernel<true, false>, threads, n_wg, lds_bytes, stream, a);
  if (simple) return launch_common(ragged_kernel<false, true>, threads, n_wg, lds_bytes, stream, a);
  return launch_common(ragged_kernel<false, false>, threads, n_wg, lds_bytes, stream, a);
}

int launch_direct(const LaunchArgs &a, int64_t n_wg, void *stream) {
  const int lds = a.out_leaf ? 0 : 256 * 8 * a.K;
  if (a.out_leaf) return launch_common(direct_kernel<true>, 256, n_wg, lds, stream, a);
  return launch_common(direct_kernel<false>, 256, n_wg, lds, stream, a);
}

int launch_gemm(int depth, const LaunchArgs &a, int64_t n_wg, void *stream) {
#define BRIDGER_GEMM_CASE(DD)                                                                 \
  case DD:                                                                                   \
    return a.out_leaf ? launch_common(gemm_kernel<DD, true>, 256, n_wg, 0, stream, a)        \
                      : launch_common(gemm_kernel<DD, false>, 256, n_wg, 0, stream, a);
  switch (depth) {
    BRIDGER_GEMM_CASE(1)
    BRIDGER_GEMM_CASE(2)
    BRIDGER_GEMM_CASE(3)
    BRIDGER_GEMM_CASE(4)
    default: return (int)hipErrorInvalidValue;
  }
#undef BRIDGER_GEMM_CASE
}

}  // namespace bridger
