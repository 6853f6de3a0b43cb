// perfect_global.hip -- PERFECT forests on wide rows: the LDS holds only the row tile and the
// node records are read from global memory, where a forest of a few MB stays in L2.
//
// With wide rows (hundreds of features) a row tile of 32 rows already fills most of the LDS,
// so streaming the forest through LDS chunks leaves one or two compute waves per CU and the
// chunk staging latency-bound; restaging the whole forest for every 32 rows also multiplies
// the L2->LDS traffic.  Here G lane groups share each row tile and split the trees into
// contiguous ranges (no chunks, no staging, no barriers inside the walk), so a CU runs as
// many waves as the tile and the per-group class sums allow.
#include "perfect_walk.h"
#include "vector_leaves.h"

namespace bridger {

// Whether a row goes right at a node: the step bit of step_slot.
template <bool FIN, int XB>
__device__ __forceinline__ uint32_t go_right(uint32_t w, uint32_t x) {
  if constexpr (XB != 4) return (w - x) >> 31;
  else if constexpr (FIN) return __float_as_uint(__uint_as_float(w) - __uint_as_float(x)) >> 31;
  else return (__uint_as_float(x) <= __uint_as_float(w)) ? 0u : 1u;
}

// VK: 0 scalar leaves; 4 or 8 (K <= VK) or 64 vector leaves (class sums in registers / LDS).
// TL: 0, or the number of top levels read from per-wave LDS copies (scalar leaves only).
// DEEP: below the top levels the walk reads the deep blocks (layout in internal.h): one
// 16-byte load per pair of levels; the last level's block carries its two leaf values, or
// (an even number of deep levels) the last pair's load goes out together with that of the
// four leaves under its node, so no load waits for the last pair.  DEEP with 16 trees per
// lane holds 16 blocks of 16 bytes per lane: workgroups of at most 8 waves, so that a lane
// may use 256 registers; with 8 trees per lane, 16-wave workgroups.  GB: bytes of a lane
// group's top-level copy (one batch of U trees).  KS: scalar leaves, and the class sums of
// the (at most KS) classes of a group's trees in registers, written only after the walk into
// the row tile's LDS (acc_alias), which leaves the LDS to the tile and the top-level copies
// during the walk.
template <int D, int U, bool LEAVES, bool FIN, int XB, int VK = 0, int TL = 0, bool DEEP = false,
          int GB = 1024, int KS = 0>
__global__ __launch_bounds__(DEEP && U > 8 ? 512 : 1024) void perfect_global_kernel(LaunchArgs a) {
  static_assert(TL == 0 || (VK == 0 && U * (8 << TL) == GB && TL < D && GB % 1024 == 0),
                "top levels: scalar leaves, one lane group's batch in GB bytes");
  static_assert(!DEEP || TL > 0, "deep blocks follow LDS top levels");
  static_assert(KS == 0 || (TL > 0 && !LEAVES), "register class sums: the top-level walk");
  extern __shared__ __attribute__((aligned(16))) uint8_t smem[];
  constexpr bool VK_REG = VK == 4 || VK == 8;  // vector leaves, class sums in registers
  constexpr int VR = VK_REG ? VK : 4;
  const int tid = threadIdx.x;
  const int R = a.rows_per_wg, G = a.groups;
  const uint32_t tb = (uint32_t)a.tree_bytes;
  const int T = a.n_trees;
  const int r = tid & (R - 1);
  const int g = R >= 64 ? __builtin_amdgcn_readfirstlane(tid / R) : tid / R;
  const int64_t row = (int64_t)blockIdx.x * R + r;
  const bool row_ok = row < a.n_rows;
  const uint32_t lane_off = (uint32_t)a.lds_x_off + tile_row_off<XB>(r);
  constexpr uint32_t kLeafOff = 4u << D;
  constexpr uint32_t kFirstLeaf = 1u << D;

  // Top levels from LDS (TL > 0): the wave's copies of its lane groups' first batch are issued
  // before the row tile, so their latency overlaps the tile's.
  constexpr uint32_t TBT = 8u << TL;  // bytes of one tree's top levels
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int gpw = R < 64 ? 64 / R : 1;              // lane groups per wave
  const int gi = R < 64 ? lane / R : 0;             // this lane's group within the wave
  const int gw0 = __builtin_amdgcn_readfirstlane((wave * 64) / R);  // the wave's first group
  const uint32_t wave_bytes = (uint32_t)gpw * GB;
  const uint32_t buf = (uint32_t)a.lds_top_off + (uint32_t)wave * wave_bytes;
  static_assert(TL == 0 || U * TBT == GB,
                "one lane group's batch is GB / 1024 16-byte-per-lane loads");
  const int NB = ((T + G - 1) / G + U - 1) / U;     // batches of the largest group
  // the tree ranges of the wave's (at most two) lane groups
  int cb0[2], cb1[2];
#pragma unroll
  for (int i = 0; i < 2; ++i) {
    const int gc = gw0 + (i < gpw ? i : 0);
    cb0[i] = (int)(((int64_t)T * gc) / G);
    cb1[i] = (int)(((int64_t)T * (gc + 1)) / G);
  }
  constexpr int LPT = (int)TBT / 16;                 // 16-byte pieces per tree of the copy
  auto copy_batch = [&](int j) {
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      if (i < gpw) {
#pragma unroll
        for (int k = 0; k < GB / 1024; ++k) {
          const int piece = k * 64 + lane;           // this lane's piece of the batch
          const int t = min(cb0[i] + j * U + piece / LPT, cb1[i] - 1);
          __builtin_amdgcn_global_load_lds(
              (const void *)(a.nodes + (size_t)t * tb + (uint32_t)(piece % LPT) * 16),
              (__attribute__((address_space(3))) void *)((lds_byte *)smem + buf +
                                                         (uint32_t)i * GB + k * 1024u),
              16, 0, 0);
        }
      }
    }
  };
  if constexpr (TL > 0) copy_batch(0);
  load_tile_any<XB, FIN>(smem, a, r, row, row_ok, g, G);
  __syncthreads();

  double *acc_lds = reinterpret_cast<double *>(smem + a.lds_acc_off) + g * R + r;
  const int slot_stride = G * R;
  const int t_begin = (int)(((int64_t)T * g) / G), t_end = (int)(((int64_t)T * (g + 1)) / G);
  // KS: the class of the group's first tree (register class slot 0)
  int k0 = 0;
  if (KS)
    while (k0 + 1 < a.K && t_begin >= a.class_begin[k0 + 1]) ++k0;
  ClassAcc ca;
  ca.k = k0;
  ca.acc = class_init(a, k0, g == 0);
  ca.next_b = a.class_begin[k0 + 1];
  double vacc[VR];
  if (VK_REG) vec_init_reg(a, vacc, g == 0);
  if (VK == 64) vec_init(a, acc_lds, slot_stride, g == 0);
  // KS: a group's trees are contiguous and class-sorted, so each class is summed in one
  // stretch; when the class changes its finished sum is shifted into cs (cs[j] then holds class
  // ca.k - 1 - j), so that no register is indexed at run time (the host takes this kernel only
  // when every group's trees span at most KS classes)
  double cs[KS > 0 ? KS : 1];
#pragma unroll
  for (int j = 0; j < (KS > 0 ? KS : 1); ++j) cs[j] = 0.0;
  auto advance_reg = [&](int t) {
    while (t >= ca.next_b) {
#pragma unroll
      for (int j = KS - 1; j > 0; --j) cs[j] = cs[j - 1];
      cs[0] = ca.acc;
      ca.k += 1;
      ca.acc = class_init(a, ca.k, g == 0);
      ca.next_b = a.class_begin[ca.k + 1];
    }
  };

  auto finish = [&](auto &m, int q) {
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
    } else if (VK) {
      int64_t leaf[N];
#pragma unroll
      for (int u = 0; u < N; ++u) leaf[u] = (int64_t)(q + u) * (1 << D) + (m[u] - kFirstLeaf);
      if (VK_REG) vec_add_reg(a, vacc, leaf);
      else vec_add(a, acc_lds, slot_stride, leaf);
    } else {
      float lv[N];
#pragma unroll
      for (int u = 0; u < N; ++u)
        lv[u] = *reinterpret_cast<const float *>(a.nodes + (size_t)(q + u) * tb + kLeafOff +
                                                 (m[u] << 2));
#pragma unroll
      for (int u = 0; u < N; ++u) {
        class_advance(a, ca, q + u, acc_lds, slot_stride, g == 0);
        ca.acc += (double)lv[u];
      }
    }
  };

  if constexpr (TL > 0) {
    // Top levels from LDS: every wave copies the first TL levels (records of heap slots 1 ..
    // 2^TL - 1, 8 << TL bytes from the start of each tree block) of the next U trees of each of
    // its lane groups into its own LDS buffer with 16-byte global->LDS loads (1 KB per
    // instruction), issued as soon as the current batch has left its top levels.  The batch
    // loop is wave-uniform: batch j covers trees t_begin + jU .. + U - 1 of every group, slots
    // past a group's last tree walk that tree again and are not added.
    // deep blocks through a buffer resource: 32-bit byte offsets, and a read outside the blocks
    // returns zeros instead of faulting
    typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
    const __amdgpu_buffer_rsrc_t drs = __builtin_amdgcn_make_buffer_rsrc(
        (void *)a.deep, (short)0, T * a.deep_tree_bytes, kBufferRsrcWord3);
    for (int j = 0; j < NB; ++j) {
      const int q = t_begin + j * U;
      wait_stage();  // this batch's top levels have landed
      uint32_t m[U];
      size_t base[U];
#pragma unroll
      for (int u = 0; u < U; ++u) {
        m[u] = 1u;
        base[u] = (size_t)min(q + u, t_end - 1) * tb;
      }
      const uint32_t lbuf = buf + (uint32_t)gi * GB;
#pragma unroll
      for (int d = 0; d < (DEEP ? TL : D); ++d) {
        uint2 rec[U];
        uint32_t xv[U];
#pragma unroll
        for (int u = 0; u < U; ++u)
          rec[u] = d < TL ? lds_u64(smem, lbuf + (uint32_t)u * TBT + (m[u] << 3))
                          : *reinterpret_cast<const uint2 *>(a.nodes + base[u] + (m[u] << 3));
#pragma unroll
        for (int u = 0; u < U; ++u) xv[u] = gather_x<FIN, XB>(smem, rec[u].y + lane_off);
#pragma unroll
        for (int u = 0; u < U; ++u) m[u] = step_slot<FIN, XB>(m[u], rec[u].x, xv[u]);
        if (d == TL - 1 && j + 1 < NB) copy_batch(j + 1);
      }
      float lv[U];
      if constexpr (DEEP) {
        constexpr int ND = D - TL, NP = ND / 2;
        // D - TL even: the last pair's node m has the four leaves of its grandchildren, 16
        // contiguous bytes of the leaf array, loaded with its block (not with 16 register class
        // sums in a 1024-thread workgroup: no registers left for them)
        constexpr bool QUAD = !(ND & 1) && !LEAVES && !(KS > 4 && U <= 8);
        const uint32_t l2rb = (uint32_t)a.log2_row_bytes;
        uint32_t doff[U];  // byte offsets of the trees' blocks (below 2^31, checked on the host)
#pragma unroll
        for (int u = 0; u < U; ++u)
          doff[u] = (uint32_t)min(q + u, t_end - 1) * (uint32_t)a.deep_tree_bytes;
#pragma unroll
        for (int i = 0; i < NP; ++i) {
          // levels d and d + 1: node m's block holds both children's thresholds and features
          const int d = TL + 2 * i;
          const uint32_t off = (uint32_t)(deep_pair_off(TL, i) - (16 << d));
          uint4 blk[U];
          uint4 quad[QUAD ? U : 1];
          uint32_t xv[U], b[U];
#pragma unroll
          for (int u = 0; u < U; ++u) {
            const u32x4 v = __builtin_amdgcn_raw_buffer_load_b128(drs, doff[u] + off + (m[u] << 4), 0, 0);
            blk[u] = make_uint4(v.x, v.y, v.z, v.w);
          }
          if (QUAD && i == NP - 1) {
            constexpr uint32_t qoff = (uint32_t)(deep_pair_off(TL, NP) - (16 << (D - 2)));
#pragma unroll
            for (int u = 0; u < U; ++u) {
              const u32x4 v = __builtin_amdgcn_raw_buffer_load_b128(drs, doff[u] + qoff + (m[u] << 4), 0, 0);
              quad[QUAD ? u : 0] = make_uint4(v.x, v.y, v.z, v.w);
            }
          }
#pragma unroll
          for (int u = 0; u < U; ++u)
            xv[u] = gather_x<FIN, XB>(smem, ((blk[u].w & 1023u) << l2rb) + lane_off);
#pragma unroll
          for (int u = 0; u < U; ++u) {
            b[u] = go_right<FIN, XB>(blk[u].x, xv[u]);
            const uint32_t f2 = (blk[u].w >> (b[u] ? 20 : 10)) & 1023u;
            blk[u].x = b[u] ? blk[u].z : blk[u].y;  // the child's threshold
            xv[u] = gather_x<FIN, XB>(smem, (f2 << l2rb) + lane_off);
          }
#pragma unroll
          for (int u = 0; u < U; ++u) {
            const uint32_t b2 = go_right<FIN, XB>(blk[u].x, xv[u]);
            if (QUAD && i == NP - 1) {
              const uint4 qv = quad[QUAD ? u : 0];
              const uint32_t lo = b2 ? qv.y : qv.x, hi = b2 ? qv.w : qv.z;
              lv[u] = __uint_as_float(b[u] ? hi : lo);
            }
            m[u] = 4u * m[u] + 2u * b[u] + b2;
          }
        }
        if constexpr (ND & 1) {
          // level D - 1 with its two leaf values
          constexpr uint32_t off = (uint32_t)(deep_pair_off(TL, NP) - (16 << (D - 1)));
          uint4 blk[U];
          uint32_t xv[U];
#pragma unroll
          for (int u = 0; u < U; ++u)
          {
            const u32x4 v = __builtin_amdgcn_raw_buffer_load_b128(drs, doff[u] + off + (m[u] << 4), 0, 0);
            blk[u] = make_uint4(v.x, v.y, v.z, v.w);
          }
#pragma unroll
          for (int u = 0; u < U; ++u) xv[u] = gather_x<FIN, XB>(smem, (blk[u].y << l2rb) + lane_off);
#pragma unroll
          for (int u = 0; u < U; ++u) {
            const uint32_t bb = go_right<FIN, XB>(blk[u].x, xv[u]);
            lv[u] = __uint_as_float(bb ? blk[u].w : blk[u].z);
            m[u] = 2u * m[u] + bb;
          }
        }
      } else if (!LEAVES) {
#pragma unroll
        for (int u = 0; u < U; ++u)
          lv[u] = *reinterpret_cast<const float *>(a.nodes + base[u] + kLeafOff + (m[u] << 2));
      }
      if (LEAVES) {
#pragma unroll
        for (int u = 0; u < U; ++u) {
          if (row_ok && q + u < t_end)
            a.out_leaf[row * (int64_t)T + a.tree_order[q + u]] =
                a.leaf_map[(int64_t)(q + u) * (1 << D) + (m[u] - kFirstLeaf)];
        }
      } else {
#pragma unroll
        for (int u = 0; u < U; ++u) {
          if (q + u < t_end) {
            if (KS) advance_reg(q + u);
            else class_advance(a, ca, q + u, acc_lds, slot_stride, g == 0);
            ca.acc += (double)lv[u];
          }
        }
      }
    }
  } else {
    int q = t_begin;
    for (; q + U <= t_end; q += U) {
      uint32_t m[U];
      walk_trees_global<D, U, FIN, XB>(smem, a.nodes, (size_t)q * tb, tb, lane_off, m);
      finish(m, q);
    }
    for (; q < t_end; ++q) {
      uint32_t m[1];
      walk_trees_global<D, 1, FIN, XB>(smem, a.nodes, (size_t)q * tb, tb, lane_off, m);
      finish(m, q);
    }
  }
  if (LEAVES) return;
  if (KS) {
    // the sums go into the row tile's LDS: every group must be done with the tile (no copy of
    // top levels is in flight after the last batch); classes outside the group's span get
    // their initial value (the base score in the first group)
    __syncthreads();
    for (int c = 0; c < a.K; ++c) {
      const int d = ca.k - c;  // class c's sum: ca.acc (d = 0) or cs[d - 1] (k0 <= c < ca.k)
      double v = d == 0 ? ca.acc : class_init(a, c, g == 0);
#pragma unroll
      for (int j = 0; j < KS; ++j)
        if (c >= k0 && d == j + 1) v = cs[j];
      acc_lds[c * slot_stride] = v;
    }
  } else if (VK_REG) {
    vec_store_reg(a, vacc, acc_lds, slot_stride);
  } else if (!VK) {
    class_flush_all(a, ca, acc_lds, slot_stride, g == 0);
  }
  __syncthreads();
  groups_finalize_store(a, reinterpret_cast<double *>(smem + a.lds_acc_off), R, G, slot_stride,
                        tid, row, row_ok);
}

// ---------------------------------------------------------------------- launchers
// The deep-block walk: top levels TL and group copies of GB bytes (3 levels of 16 trees in
// 1 KB; 4 levels of 16 trees or 5 of 8 in 2 KB), class sums in registers (acc_alias) or LDS.
template <int D, bool FIN, int XB, int TL, int GB>
static int launch_global_deep_tg(const LaunchArgs &a, int threads, int64_t n_wg, int lds_bytes,
                                 void *stream) {
  constexpr int U = GB / (8 << TL);
  if constexpr (TL < D && (U == 8 || U == 16)) {
    if (a.out_leaf)
      return launch_common(perfect_global_kernel<D, U, true, FIN, XB, 0, TL, true, GB>, threads,
                           n_wg, lds_bytes, stream, a);
    if (a.acc_alias && a.class_span <= 4)
      return launch_common(perfect_global_kernel<D, U, false, FIN, XB, 0, TL, true, GB, 4>,
                           threads, n_wg, lds_bytes, stream, a);
    if (a.acc_alias)
      return launch_common(perfect_global_kernel<D, U, false, FIN, XB, 0, TL, true, GB, 16>,
                           threads, n_wg, lds_bytes, stream, a);
    return launch_common(perfect_global_kernel<D, U, false, FIN, XB, 0, TL, true, GB>, threads,
                         n_wg, lds_bytes, stream, a);
  } else {
    return (int)hipErrorInvalidValue;
  }
}

template <int D, bool FIN, int XB>
static int launch_global_deep(const LaunchArgs &a, int waves, int64_t n_wg, int lds_bytes,
                              void *stream) {
  const int threads = 64 * waves;
  const int gb = a.top_group_bytes ? a.top_group_bytes : 1024;
  if (a.top_levels == 3 && gb == 1024)
    return launch_global_deep_tg<D, FIN, XB, 3, 1024>(a, threads, n_wg, lds_bytes, stream);
  if (a.top_levels == 4 && gb == 1024)
    return launch_global_deep_tg<D, FIN, XB, 4, 1024>(a, threads, n_wg, lds_bytes, stream);
  if (a.top_levels == 4 && gb == 2048)
    return launch_global_deep_tg<D, FIN, XB, 4, 2048>(a, threads, n_wg, lds_bytes, stream);
  if (a.top_levels == 5 && gb == 2048)
    return launch_global_deep_tg<D, FIN, XB, 5, 2048>(a, threads, n_wg, lds_bytes, stream);
  return (int)hipErrorInvalidValue;
}

template <int D, bool FIN, int XB>
static int launch_global_dfx(const LaunchArgs &a, int waves, int64_t n_wg, int lds_bytes,
                             void *stream) {
  const int threads = 64 * waves;
  // 16 trees per lane: at most 8 waves (256 registers a lane); 8 trees: up to 16 waves
  if (a.top_levels && !a.vec && a.deep &&
      waves <= (a.top_group_bytes / (8 << a.top_levels) > 8 ? 8 : 16))
    return launch_global_deep<D, FIN, XB>(a, waves, n_wg, lds_bytes, stream);
  if constexpr (D > 4) {
    if (a.top_levels == 4 && !a.vec) {  // 8 trees per lane
      if (a.out_leaf)
        return launch_common(perfect_global_kernel<D, 8, true, FIN, XB, 0, 4>, threads, n_wg,
                             lds_bytes, stream, a);
      return launch_common(perfect_global_kernel<D, 8, false, FIN, XB, 0, 4>, threads, n_wg,
                           lds_bytes, stream, a);
    }
  }
  if constexpr (D > 3) {
    if (a.top_levels == 3 && !a.vec) {  // 16 trees per lane
      if (a.out_leaf)
        return launch_common(perfect_global_kernel<D, 16, true, FIN, XB, 0, 3>, threads, n_wg,
                             lds_bytes, stream, a);
      return launch_common(perfect_global_kernel<D, 16, false, FIN, XB, 0, 3>, threads, n_wg,
                           lds_bytes, stream, a);
    }
  }
  if (a.out_leaf)
    return launch_common(perfect_global_kernel<D, 4, true, FIN, XB>, threads, n_wg, lds_bytes, stream, a);
  if (a.vec && a.K <= 4)
    return launch_common(perfect_global_kernel<D, 4, false, FIN, XB, 4>, threads, n_wg, lds_bytes, stream, a);
  if (a.vec && a.K <= 8)  // two trees per lane: the rows of four would cost occupancy
    return launch_common(perfect_global_kernel<D, 2, false, FIN, XB, 8>, threads, n_wg, lds_bytes, stream, a);
  if (a.vec)
    return launch_common(perfect_global_kernel<D, 4, false, FIN, XB, 64>, threads, n_wg, lds_bytes, stream, a);
  if (a.ilp == 4)
    return launch_common(perfect_global_kernel<D, 4, false, FIN, XB>, threads, n_wg, lds_bytes, stream, a);
  return launch_common(perfect_global_kernel<D, 8, false, FIN, XB>, threads, n_wg, lds_bytes, stream, a);
}

template <int D>
static int launch_global_d(const LaunchArgs &a, int waves, int64_t n_wg, int lds_bytes,
                           void *stream) {
  if (a.x_bytes == 2) return launch_global_dfx<D, true, 2>(a, waves, n_wg, lds_bytes, stream);
  if (a.x_bytes == 1) return launch_global_dfx<D, true, 1>(a, waves, n_wg, lds_bytes, stream);
  return a.finite_thresholds ? launch_global_dfx<D, true, 4>(a, waves, n_wg, lds_bytes, stream)
                             : launch_global_dfx<D, false, 4>(a, waves, n_wg, lds_bytes, stream);
}

int launch_perfect_global(int depth, const LaunchArgs &a, int waves, int64_t n_wg, int lds_bytes,
                          void *stream) {
  switch (depth) {
    case 1: return launch_global_d<1>(a, waves, n_wg, lds_bytes, stream);
    case 2: return launch_global_d<2>(a, waves, n_wg, lds_bytes, stream);
    case 3: return launch_global_d<3>(a, waves, n_wg, lds_bytes, stream);
    case 4: return launch_global_d<4>(a, waves, n_wg, lds_bytes, stream);
    case 5: return launch_global_d<5>(a, waves, n_wg, lds_bytes, stream);
    case 6: return launch_global_d<6>(a, waves, n_wg, lds_bytes, stream);
    case 7: return launch_global_d<7>(a, waves, n_wg, lds_bytes, stream);
    case 8: return launch_global_d<8>(a, waves, n_wg, lds_bytes, stream);
    case 9: return launch_global_d<9>(a, waves, n_wg, lds_bytes, stream);
    case 10: return launch_global_d<10>(a, waves, n_wg, lds_bytes, stream);
    default: return (int)hipErrorInvalidValue;
  }
}

}  // namespace bridger
