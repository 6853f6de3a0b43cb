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
  groups_finalize_store(a, reinterpret_cast<double *>(smem + a.lds_acc_off), R, G, slot_stride,
                        tid, row, row_ok);
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

  load_tile_all<XB, false>(smem, a, r, row, row_ok, g, G);
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
  groups_finalize_store(a, reinterpret_cast<double *>(smem + a.lds_acc_off), R, G, slot_stride,
                        tid, row, row_ok);
}

// The same lockstep walk for one output class with scalar leaves (or leaf ids), when every
// lane group is a whole number of waves (R >= 64): all lanes of a wave then walk the same
// batch of U = top_batch(L) trees, so each tree's first L levels come from a per-wave LDS copy
// of the trees' top-level heaps (layout in internal.h) instead of one wave-wide global load per
// level.  One 16-byte-per-lane global->LDS load copies a whole batch's heaps (1 KB); the next
// batch's copy is issued as soon as the current batch has left its top levels, so it lands
// while the deeper levels are walked.  The texture addresser, which resolves every wave-wide
// global load and bounds the walk, sees L fewer loads per tree.  A batch is always U slots;
// slots past the group's last tree start at a leaf and are never added.  Leaves are added in
// tree order; the G groups' partial sums meet in the waves' copy buffers at the end.
template <bool LEAVES, int XB, int L>
__global__ __launch_bounds__(1024) void ragged_top_kernel(LaunchArgs a) {
  extern __shared__ __attribute__((aligned(16))) uint8_t smem[];
  constexpr int U = top_batch(L);
  constexpr int kTopLevels = L;
  constexpr uint32_t kTopBytes = (uint32_t)top_bytes(L);
  const int tid = threadIdx.x;
  const int R = a.rows_per_wg, G = a.groups;
  const int r = tid & (R - 1);
  const int g = __builtin_amdgcn_readfirstlane(tid / R);
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int lane = tid & 63;
  const int64_t row = (int64_t)blockIdx.x * R + r;
  const bool row_ok = row < a.n_rows;
  const uint32_t lane_off = (uint32_t)a.lds_x_off + tile_row_off<XB>(r);
  const int shift = a.log2_row_bytes;
  const int T = a.n_trees;
  const uint32_t buf = (uint32_t)a.lds_top_off + (uint32_t)wave * kTopWaveBytes;

  load_tile_all<XB, false>(smem, a, r, row, row_ok, g, G);
  __syncthreads();

  const int ga = (int)(((int64_t)T * g) / G), gb = (int)(((int64_t)T * (g + 1)) / G);
  const uint8_t *tops = reinterpret_cast<const uint8_t *>(a.tops);
  const uint8_t *recs = a.nodes;
  // the heaps of trees q .. q + U - 1 (one 16-byte load per lane) into this wave's buffer
  auto copy_tops = [&](int q) {
    __builtin_amdgcn_global_load_lds(
        (const void *)(tops + (size_t)q * kTopBytes + (size_t)lane * 16),
        (__attribute__((address_space(3))) void *)((lds_byte *)smem + buf), 16, 0, 0);
  };
  // record i through a buffer resource: a 32-bit byte offset (one shift per load), and a read
  // outside the records returns zeros instead of faulting
  const __amdgpu_buffer_rsrc_t rsrc = __builtin_amdgcn_make_buffer_rsrc(
      (void *)recs, (short)0, (int)a.nodes_bytes, kBufferRsrcWord3);
  auto load_rec = [&](uint32_t i) {
    typedef unsigned int u32x2 __attribute__((ext_vector_type(2)));
    const u32x2 v = __builtin_amdgcn_raw_buffer_load_b64(rsrc, i * 8u, 0, 0);
    return make_uint2(v.x, v.y);
  };
  double acc = (!LEAVES && a.aggregate == 0 && g == 0) ? (double)a.base[0] : 0.0;
  if (ga < gb) copy_tops(ga);
  for (int q = ga; q < gb; q += U) {
    const int nvalid = gb - q < U ? gb - q : U;
    wait_stage();  // this batch's heaps have landed
    uint32_t idx[U], m[U];
    uint2 rec[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const uint32_t tb = buf + (uint32_t)u * kTopBytes;
      idx[u] = lds_u64(smem, tb).x;
      rec[u] = u < nvalid ? lds_u64(smem, tb + 8) : make_uint2(0u, (uint32_t)kLeafFlag);
      m[u] = 1u;
    }
    // levels 0 .. kTopLevels - 1: every record from the copy, the last level's children from
    // global memory
    // One level of all U slots: gather every slot's feature value (a slot at a leaf reads
    // feature 0 harmlessly), then step the slots that sit on an internal node.  Returns
    // whether any slot of this lane was internal.
    bool inner[U];
    auto step = [&]() {
      bool any = false;
      uint32_t xv[U];
#pragma unroll
      for (int u = 0; u < U; ++u)
        xv[u] = gather_x<false, XB>(smem, ((rec[u].y >> 16) << shift) + lane_off);
#pragma unroll
      for (int u = 0; u < U; ++u) {
        // branch-free: keep = all ones on an internal node, zero at a leaf
        const uint32_t meta = rec[u].y;
        const uint32_t keep = ((meta >> 15) & 1u) - 1u;
        inner[u] = keep != 0u;
        any = any || inner[u];
        const uint32_t right = (goes_right<XB>(xv[u], rec[u].x) ? 1u : 0u) & keep;
        idx[u] += ((meta & (uint32_t)kMaxRel) + right) & keep;
        m[u] += (m[u] + right) & keep;
      }
      return any;
    };
    // levels 0 .. kTopLevels - 2 read the next record from the copy (slots at a leaf re-read
    // their own); the last top level reads the children from global memory
    bool live = true;
#pragma unroll
    for (int level = 0; level + 1 < kTopLevels; ++level) {
      if (live) {
        live = step();
#pragma unroll
        for (int u = 0; u < U; ++u)
          rec[u] = lds_u64(smem, buf + (uint32_t)u * kTopBytes + 8u * m[u]);
      }
    }
    if (live) {
      live = step();
#pragma unroll
      for (int u = 0; u < U; ++u)
        if (inner[u]) rec[u] = load_rec(idx[u]);
    }
    // the top levels are read: the next batch's heaps can land while the deeper levels run
    if (q + U < gb) copy_tops(q + U);
    // deeper levels: a slot whose lanes all sit at leaves skips its work (the branch is taken
    // on the slot's own lane mask), so a finished tree costs neither loads nor arithmetic
    // validated trees are at most 64 deep; the bound keeps the loop finite regardless
    for (int level = kTopLevels; live && level <= 64; ++level) {
      bool any = false;
#pragma unroll
      for (int u = 0; u < U; ++u) {
        inner[u] = (rec[u].y & (uint32_t)kLeafFlag) == 0;
        any = any || inner[u];
      }
      if (!any) break;
      uint32_t xv[U];
#pragma unroll
      for (int u = 0; u < U; ++u)
        xv[u] = gather_x<false, XB>(smem, ((rec[u].y >> 16) << shift) + lane_off);
#pragma unroll
      for (int u = 0; u < U; ++u) {
        if (inner[u]) {
          idx[u] += (rec[u].y & (uint32_t)kMaxRel) + (goes_right<XB>(xv[u], rec[u].x) ? 1u : 0u);
          rec[u] = load_rec(idx[u]);
        }
      }
    }
#pragma unroll
    for (int u = 0; u < U; ++u) {
      if (u < nvalid) {
        if (LEAVES) {
          if (row_ok) a.out_leaf[row * (int64_t)T + a.tree_order[q + u]] = a.leaf_map[idx[u]];
        } else {
          acc += (double)__uint_as_float(rec[u].x);
        }
      }
    }
  }
  if (LEAVES) return;
  // group sums: each thread's partial in its own wave's copy buffer (free once no copy is in
  // flight), then group 0 adds the groups' partials of its row in group order
  wait_stage();
  auto slot = [&](int t) {
    return reinterpret_cast<double *>(smem + a.lds_top_off + (t >> 6) * kTopWaveBytes +
                                      (t & 63) * 8);
  };
  *slot(tid) = acc;
  __syncthreads();
  if (g == 0 && row_ok) {
    double z = *slot(r);
    for (int gg = 1; gg < G; ++gg) z += *slot(gg * R + r);
    if (a.aggregate == 1) z = (double)a.base[0] + z / (double)a.class_count[0];
    store_one(a, row, z);
  }
}

// The lockstep global-node walk over two-level treelets (layout in internal.h): one 16-byte
// load brings a node's threshold and feature and both children's (or their leaf values), so a
// load covers two levels and a leaf child ends the walk without a load of its own.  Each wave
// copies the first slots of its next U trees to its LDS buffer with one 16-byte load per lane
// (slots 0-20, tree levels 0-5, of three trees; or slots 0-4 of four); deeper slots come from
// global memory through a buffer resource (32-bit offsets; a read past the blocks returns
// zeros).  One class, scalar leaves; lane groups of whole waves.
// LT: treelet levels read from the copy, 2 (slots 0-4, kTreeletCopyBytes per tree) or 3
// (slots 0-20, 336 bytes per tree: three trees per buffer).
template <bool LEAVES, int XB, int U, int LT = 2>
__global__ __launch_bounds__(1024) void ragged_treelet_kernel(LaunchArgs a) {
  extern __shared__ __attribute__((aligned(16))) uint8_t smem[];
  static_assert(LT == 2 || LT == 3, "two or three treelet levels from the copy");
  constexpr uint32_t kSlots = LT == 2 ? (uint32_t)kTreeletTopSlots : 21u;
  constexpr uint32_t kCopy = LT == 2 ? (uint32_t)kTreeletCopyBytes : 16u * kSlots;
  static_assert(U * kCopy <= (uint32_t)kTopWaveBytes, "a batch's copies fit the wave's buffer");
  const int tid = threadIdx.x;
  const int R = a.rows_per_wg, G = a.groups;
  const int r = tid & (R - 1);
  const int g = __builtin_amdgcn_readfirstlane(tid / R);
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int lane = tid & 63;
  const int64_t row = (int64_t)blockIdx.x * R + r;
  const bool row_ok = row < a.n_rows;
  const uint32_t lane_off = (uint32_t)a.lds_x_off + tile_row_off<XB>(r);
  const int shift = a.log2_row_bytes;
  const int T = a.n_trees;
  const uint32_t buf = (uint32_t)a.lds_top_off + (uint32_t)wave * kTopWaveBytes;

  load_tile_all<XB, false>(smem, a, r, row, row_ok, g, G);
  __syncthreads();

  const int ga = (int)(((int64_t)T * g) / G), gb = (int)(((int64_t)T * (g + 1)) / G);
  const uint8_t *blocks = a.nodes;
  // slots 0 .. kCopy / 16 - 1 of trees q .. q + U - 1 (the last tree of the group repeated past
  // the group's end) into this wave's buffer, tree u at buf + u * kCopy; returns this lane's
  // tree's first slot, which lane 8u holds for tree u of the batch
  auto copy_tops = [&](int q) {
    const int t = min(q + lane / (int)(kCopy / 16), gb - 1);
    const uint32_t piece = (uint32_t)(lane % (int)(kCopy / 16));
    const int32_t first = a.tree_start[t];
    __builtin_amdgcn_global_load_lds(
        (const void *)(blocks + ((size_t)first + piece) * 16),
        (__attribute__((address_space(3))) void *)((lds_byte *)smem + buf), 16, 0, 0);
    return first;
  };
  const __amdgpu_buffer_rsrc_t rsrc = __builtin_amdgcn_make_buffer_rsrc(
      (void *)blocks, (short)0, (int)a.nodes_bytes, kBufferRsrcWord3);
  auto load_block = [&](uint32_t slot) {
    typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
    const u32x4 v = __builtin_amdgcn_raw_buffer_load_b128(rsrc, slot * 16u, 0, 0);
    return make_uint4(v.x, v.y, v.z, v.w);
  };
  double acc = (!LEAVES && a.aggregate == 0 && g == 0) ? (double)a.base[0] : 0.0;
  int32_t firsts = ga < gb ? copy_tops(ga) : 0;
  for (int q = ga; q < gb; q += U) {
    const int nvalid = gb - q < U ? gb - q : U;
    wait_stage();  // this batch's slots have landed
    uint32_t s[U], out[U];  // slot within the tree; on finishing: leaf value or leaf-id index
    bool live[U];
    uint4 blk[U];
    int32_t base[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      base[u] = __builtin_amdgcn_readlane(firsts, u * (int)(kCopy / 16));
      s[u] = 0u;
      out[u] = 0u;
      live[u] = true;
    }
    // one step of every live slot from its block: the node, then the child it chooses; a leaf
    // child finishes the slot, an internal one moves it to the grandchild's slot
    auto step = [&]() {
      uint32_t x1[U], wc[U], fc[U], b1[U], x2[U];
#pragma unroll
      for (int u = 0; u < U; ++u)
        x1[u] = gather_x<false, XB>(smem, ((blk[u].w & 1023u) << shift) + lane_off);
#pragma unroll
      for (int u = 0; u < U; ++u) {
        b1[u] = goes_right<XB>(x1[u], blk[u].x) ? 1u : 0u;
        wc[u] = b1[u] ? blk[u].z : blk[u].y;
        fc[u] = (blk[u].w >> (b1[u] ? 20 : 10)) & 1023u;
        x2[u] = gather_x<false, XB>(smem, (fc[u] << shift) + lane_off);
      }
#pragma unroll
      for (int u = 0; u < U; ++u) {
        if (live[u]) {
          if ((blk[u].w >> (30 + b1[u])) & 1u) {
            live[u] = false;
            out[u] = LEAVES ? ((uint32_t)base[u] + s[u]) * 2u + b1[u] : wc[u];
          } else {
            s[u] = 4u * s[u] + 1u + 2u * b1[u] + (goes_right<XB>(x2[u], wc[u]) ? 1u : 0u);
          }
        }
      }
    };
    // treelet levels 0 .. LT - 1 (slots 0 .. kSlots - 1) from the copy
#pragma unroll
    for (int lv = 0; lv < LT; ++lv) {
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const uint32_t addr = buf + (uint32_t)u * kCopy + 16u * (s[u] < kSlots ? s[u] : 0u);
        const uint2 lo = lds_u64(smem, addr), hi = lds_u64(smem, addr + 8u);
        blk[u] = make_uint4(lo.x, lo.y, hi.x, hi.y);
      }
      step();
    }
    // the copy is read: the next batch's slots can land while the deeper levels run
    if (q + U < gb) firsts = copy_tops(q + U);
    // deeper treelets from global memory; a slot whose lanes have all finished skips its load
    // (trees are at most 64 levels deep: 32 treelet levels; the bound keeps the loop finite)
    for (int lv = LT; lv < 34; ++lv) {
      bool any = false;
#pragma unroll
      for (int u = 0; u < U; ++u) any = any || live[u];
      if (!any) break;
#pragma unroll
      for (int u = 0; u < U; ++u)
        if (live[u]) blk[u] = load_block((uint32_t)base[u] + s[u]);
      step();
    }
#pragma unroll
    for (int u = 0; u < U; ++u) {
      if (u < nvalid) {
        if (LEAVES) {
          if (row_ok) a.out_leaf[row * (int64_t)T + a.tree_order[q + u]] = a.leaf_map[out[u]];
        } else {
          acc += (double)__uint_as_float(out[u]);
        }
      }
    }
  }
  if (LEAVES) return;
  // group sums: each thread's partial in its own wave's copy buffer (free once no copy is in
  // flight), then group 0 adds the groups' partials of its row in group order
  wait_stage();
  auto slot = [&](int t) {
    return reinterpret_cast<double *>(smem + a.lds_top_off + (t >> 6) * kTopWaveBytes +
                                      (t & 63) * 8);
  };
  *slot(tid) = acc;
  __syncthreads();
  if (g == 0 && row_ok) {
    double z = *slot(r);
    for (int gg = 1; gg < G; ++gg) z += *slot(gg * R + r);
    if (a.aggregate == 1) z = (double)a.base[0] + z / (double)a.class_count[0];
    store_one(a, row, z);
  }
}

// ---------------------------------------------------------------------- launchers
template <int XB, int L>
static int launch_ragged_top_xl(const LaunchArgs &a, int waves, int64_t n_wg, int lds_bytes,
                                void *stream) {
  const int threads = 64 * waves;
  if (a.out_leaf)
    return launch_common(ragged_top_kernel<true, XB, L>, threads, n_wg, lds_bytes, stream, a);
  return launch_common(ragged_top_kernel<false, XB, L>, threads, n_wg, lds_bytes, stream, a);
}

template <int XB>
static int launch_ragged_top_x(const LaunchArgs &a, int waves, int64_t n_wg, int lds_bytes,
                               void *stream) {
  if (a.top_levels == 5) return launch_ragged_top_xl<XB, 5>(a, waves, n_wg, lds_bytes, stream);
  if (a.top_levels == 4) return launch_ragged_top_xl<XB, 4>(a, waves, n_wg, lds_bytes, stream);
  return (int)hipErrorInvalidValue;
}

// Two treelet levels from the copy: four trees per batch; with eight (72 registers) one
// 16-wave workgroup fits a CU instead of two (4M x 256 rows: 19.8 against 14.2 ms); six
// measured 21.3 ms.  Three levels from the copy: three trees per batch.
template <int XB>
static int launch_ragged_treelet_x(const LaunchArgs &a, int waves, int64_t n_wg, int lds_bytes,
                                   void *stream) {
  const int threads = 64 * waves;
  if (a.top_levels == 3) {  // three treelet levels from the copy, three trees per batch
    if (a.out_leaf)
      return launch_common(ragged_treelet_kernel<true, XB, 3, 3>, threads, n_wg, lds_bytes, stream, a);
    return launch_common(ragged_treelet_kernel<false, XB, 3, 3>, threads, n_wg, lds_bytes, stream, a);
  }
  if (a.out_leaf)
    return launch_common(ragged_treelet_kernel<true, XB, 4>, threads, n_wg, lds_bytes, stream, a);
  return launch_common(ragged_treelet_kernel<false, XB, 4>, threads, n_wg, lds_bytes, stream, a);
}

int launch_ragged_treelet(const LaunchArgs &a, int waves, int64_t n_wg, int lds_bytes,
                          void *stream) {
  if (a.x_bytes == 2) return launch_ragged_treelet_x<2>(a, waves, n_wg, lds_bytes, stream);
  if (a.x_bytes == 1) return launch_ragged_treelet_x<1>(a, waves, n_wg, lds_bytes, stream);
  return launch_ragged_treelet_x<4>(a, waves, n_wg, lds_bytes, stream);
}

int launch_ragged_top(const LaunchArgs &a, int waves, int64_t n_wg, int lds_bytes, void *stream) {
  if (a.x_bytes == 2) return launch_ragged_top_x<2>(a, waves, n_wg, lds_bytes, stream);
  if (a.x_bytes == 1) return launch_ragged_top_x<1>(a, waves, n_wg, lds_bytes, stream);
  return launch_ragged_top_x<4>(a, waves, n_wg, lds_bytes, stream);
}

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
