// internal.h -- layouts and launch descriptors shared by the host code and the HIP kernels.
//
// Packed layouts (all little-endian, built once by bridger_forest_create):
//
// PERFECT (every tree perfect with one depth D, 1 <= D <= kMaxPerfectDepth):
//   one block of tree_bytes = 12 * 2^D per tree, in kernel tree order (trees stably sorted
//   by class):
//     [0, 8)                  unused
//     [8, 8*2^D)              internal records {float threshold; uint32 feature} in a 1-based
//                             breadth-first heap: slot m at byte 8m, children 2m and 2m+1
//     [8*2^D, 12*2^D)         leaf values: leaf j is heap slot 2^D + j; the two leaves of
//                             last-level slot m form an 8-byte pair 4*2^D bytes past that
//                             slot's record
//   Every level's records and the leaf block start 16-byte aligned.
//   Vector leaves with K <= 4 classes: the leaf block holds the leaves' class rows instead,
//   4 floats each (leaf j at 8 * 2^D + 16 j), so the tree chunks bring them to LDS with the
//   records; tree_bytes = 24 * 2^D.
//   The PERFECT kernel reads a traversal copy of this layout in which each record holds
//   {threshold with -0 stored as +0; byte offset feature * 4R of the feature's row in the
//   LDS tile of R rows}; the copy is rebuilt whenever the launch plan (and so R) is chosen.
//
// RAGGED (any tree whose records fit one LDS chunk):
//   8-byte records {uint32 w; uint32 meta}, trees contiguous in kernel order, each tree
//   breadth-first with the two children of a node adjacent (right = left + 1):
//     internal: w = threshold bits, meta = feature << 16 | left_rel   (1 <= left_rel <= 0x7FFF,
//               left child = this record + left_rel)
//     leaf    : w = value bits,     meta = 0x8000 | next_rel           (next_rel = records to the
//               next tree's root, i.e. to the end of this tree)
//   Trees are grouped into chunks of at most chunk_bytes; a chunk is staged to LDS whole.
//   Top levels (for the lockstep kernel with one tree per wave in every slot), L = 4 or 5: per
//   kernel tree 2^L records of 8 bytes, a 1-based heap of the tree's first L levels (slot 1 the
//   root, the children of slot m at 2m and 2m + 1, each a copy of the node's packed record;
//   slots under a leaf hold a leaf record) with slot 0 holding the root's record index in its
//   low word; then top_batch(L) empty trees, so that a batch copy never reads past the end.
//
// DIRECT (any forest): 16-byte records {float w; int32 feature (-1 at a leaf); int32 left;
//   int32 right} with absolute record indices; kernel tree t starts at record root[t].
#pragma once
#include <stdint.h>

namespace bridger {

constexpr int kMaxPerfectDepth = 10;
constexpr int kLdsBytesPerCU = 163840;
constexpr int kLeafFlag = 0x8000;
constexpr int kMaxRel = 0x7FFF;
constexpr int kMaxRaggedFeatures = 0xFFFF;
// RAGGED top-level heaps: a wave's LDS copy holds one batch of top_batch(L) trees' heaps, 1 KB
// (one 16-byte load per lane); L top levels per tree.
constexpr int kTopWaveBytes = 1024;
// PERFECT trees on the global-node kernel: the first L levels (default kPerfectTopLevels) of
// each of the 1024 / 2^(L+3) trees a lane group walks at once are copied to the wave's LDS
// (1 KB per lane group).
constexpr int kPerfectTopLevels = 4;
constexpr int kTopLevelsDefault = 5;
constexpr int top_bytes(int L) { return 8 << L; }
constexpr int top_batch(int L) { return kTopWaveBytes / top_bytes(L); }
// Rows per dispatch: every launch shape then stays far below the 32-bit work-item count of a
// dispatch; predictions over more rows are issued as several launches.
constexpr int64_t kMaxRowsPerLaunch = int64_t(1) << 24;
constexpr int kMaxClasses = 64;  // class sums of one 256-row block fit LDS in every kernel
// Rows per call of the allocation-free predict (its row-norm scratch: one double per row, a
// file-scope device array of 16 MiB per GPU).
constexpr int64_t kNoAllocMaxRows = int64_t(1) << 21;

enum Kernel { kAuto = 0, kPerfect = 1, kRagged = 2, kDirect = 3, kGemm = 4 };

// Bytes of one PERFECT tree block of depth D (records, then leaves; 16-byte multiple).
constexpr int perfect_tree_bytes(int D) { return ((12 << D) + 15) & ~15; }

// The PERFECT kernel has compile-time chunk variants (trees per chunk CT in 4..32, a power of
// two; both chunk buffers addressable by the 16-bit offset field of an LDS instruction) for
// one class, one lane group and finite thresholds.
constexpr bool perfect_fixed_ok(int D, int CT) {
  return D >= 2 && D <= 9 && (CT == 4 || CT == 8 || CT == 16 || CT == 32) &&
         2 * CT * perfect_tree_bytes(D) <= 65536;
}
// PERFECT deep blocks, read from global memory by the wide-row kernel below its first TL levels
// (which come from per-wave LDS copies): per kernel tree, for the deep levels TL, TL + 2, ...
// taken in pairs, one 16-byte block per node m of the pair's upper level, {w(m), w(2m),
// w(2m + 1), f(m) | f(2m) << 10 | f(2m + 1) << 20} (w: the threshold's bits, or its rank for
// bins; f: the feature index, below kDeepMaxFeatures); then, when D - TL is odd, one block per
// node m of level D - 1, {w(m), f(m), leaf value of 2m, leaf value of 2m + 1}, else the 2^D
// leaf values.  Every block of a level is indexed by m - 2^level.
constexpr int kDeepMaxFeatures = 1024;
// RAGGED treelets (the global-node ragged kernel): per kernel tree a 4-ary heap of 16-byte
// blocks, slot s holding the node n at tree level 2l of treelet level l and its two children:
// {w(n), v(c0), v(c1), f(n) | f(c0) << 10 | f(c1) << 20 | leaf(c0) << 30 | leaf(c1) << 31},
// v(c) = w(c) for an internal child, its leaf value for a leaf; the grandchild reached by
// steps b1 (at n) and b2 (at c_b1) sits in slot 4s + 1 + 2 b1 + b2.  A leaf n takes {0, v(n),
// v(n), 3 << 30}; unreachable slots are zero.  Feature indices below kDeepMaxFeatures.  The
// first kTreeletTopSlots slots (levels 0-3) of each tree of a batch are copied to the wave's
// LDS, kTreeletCopyBytes per tree (or the first 21 slots, levels 0-5, 336 bytes per tree);
// the last tree is followed by 21 zero slots.
constexpr int kTreeletTopSlots = 5;
constexpr int kTreeletCopyBytes = 128;
constexpr int kTreeletBatch = kTopWaveBytes / kTreeletCopyBytes;
constexpr int deep_pair_off(int TL, int i) {
  int o = 0;
  for (int j = 0; j < i; ++j) o += 16 << (TL + 2 * j);
  return o;
}
constexpr int deep_tree_bytes(int D, int TL) {
  return deep_pair_off(TL, (D - TL) / 2) + (((D - TL) & 1) ? (16 << (D - 1)) : (4 << D));
}
constexpr int kMaxGemmDepth = 4;
constexpr int kMaxGemmFeatures = 64;

// Launch plan (host side), chosen by the data-movement model of Eq. 1.
struct Plan {
  int32_t waves;           // waves per workgroup
  int32_t rows_per_wg;     // R: rows held in the LDS feature tile (power of two, >= 32)
  int32_t groups;          // G = 64*waves / R: tree groups sharing the row tile
  int32_t chunk_bytes;     // bytes of one LDS chunk buffer (two are used, double-buffered)
  int32_t trees_per_chunk; // PERFECT: fixed trees per chunk; RAGGED: 0 (variable)
  int32_t n_chunks;
  int32_t lds_bytes;       // dynamic LDS per workgroup
  int32_t acc_in_lds;      // class/group partial sums kept in LDS
  int32_t ilp;             // trees walked at once per lane: chunked PERFECT 1, 2 or 4; global
                           // PERFECT 4 or 8; global RAGGED 1, 2, 4 or 8
  int32_t global_nodes;    // records read from global memory, LDS holds only the tile
  int32_t waves_per_cu;    // resident compute waves per CU
  int32_t acc_alias;       // class sums written after the walk into the row tile's LDS
  int32_t tops;            // RAGGED global: 0, or L, the top levels read from a per-wave LDS
                           // copy (after the row tile, kTopWaveBytes per wave, which then
                           // holds the group sums); PERFECT global: the top levels read from
                           // per-lane-group LDS copies
  int32_t top_group_bytes; // PERFECT global with tops: bytes of one lane group's copy (1 or 2 KB)
  double hbm_bytes, stage_bytes, lds_read_bytes, est_seconds;
};

// Everything a kernel needs; passed by value (lands in SGPRs / the kernarg segment).
struct LaunchArgs {
  const float *X;
  int64_t n_rows;
  int32_t F;
  int32_t x_vec4;          // rows are 16-byte aligned and F % 4 == 0
  float *out;              // [n_rows, K] (scores) or nullptr
  int32_t *out_leaf;       // [n_rows, n_trees] (leaf ids) or nullptr
  int32_t *out_label;      // [n_rows] (class labels) or nullptr
  const uint8_t *nodes;    // packed records of the kernel family
  const int32_t *tree_start;   // RAGGED: record index of each kernel tree's root; DIRECT: same
  const int32_t *chunk_first;  // RAGGED: first kernel tree of each chunk [n_chunks + 1]
  const int32_t *chunk_rec;    // RAGGED: first record of each chunk [n_chunks + 1]
  const int32_t *class_begin;  // [K + 1] first kernel tree of each class
  const int32_t *class_count;  // [K] trees per class
  const float *base;           // [K]
  const int32_t *tree_order;   // kernel tree -> caller tree
  const int32_t *leaf_map;     // PERFECT: kernel tree * 2^D + slot -> caller node id;
                               // RAGGED/DIRECT: record -> caller node id
  int32_t n_trees;
  int32_t K;
  int32_t aggregate;
  int32_t transform;
  int32_t tree_bytes;          // PERFECT
  int32_t trees_per_chunk;     // PERFECT
  int32_t n_chunks;
  int32_t rows_per_wg;         // R
  int32_t log2_row_bytes;      // log2(4 * R): feature f's row of the LDS tile starts at f << this
  int32_t groups;              // G
  int32_t chunk_bytes;
  int32_t lds_x_off;           // byte offset of the feature tile in dynamic LDS
  int32_t lds_acc_off;         // byte offset of the partial-sum area (acc_in_lds)
  int32_t acc_alias;           // that area is the row tile's, written only after the walk
  int32_t class_span;          // acc_alias: the most classes one lane group's trees span
  int32_t acc_in_lds;
  int32_t ilp;                 // trees walked at once per lane (the plan's ilp)
  int32_t finite_thresholds;   // PERFECT: every threshold is finite (sign-of-difference step)
  const uint32_t *roots;       // PERFECT: per kernel tree the root's traversal record (2 words)
  int32_t x_bytes;             // element of X and of the LDS tile: 4 (fp32) or 2 / 1 (bins)
  const float *q_values;       // binning: sorted distinct thresholds of every feature
  const int32_t *q_off;        // binning: [F + 1] offsets into q_values
  void *xq;                    // binning: output bins [n_rows, F] of x_bytes each
  int32_t csr;                 // rows in CSR form: X = values, plus the two arrays below
  const int64_t *csr_indptr;   // [n_rows + 1]
  const int32_t *csr_indices;  // [nnz] feature of each stored value
  int32_t pre_kind;            // fused preprocessing (BRIDGER_PRE_*), 0 = none
  const double *pre_a, *pre_b; // its per-feature parameters
  const double *row_norm;      // NORMALIZE: each row's L2 norm in double (1 for a zero row)
  int32_t vec;                 // vector leaves: K class values per leaf in leaf_vec
  const float *leaf_vec;       // [leaf index][vec_stride(K)], as the family numbers leaves
  const uint64_t *tops;        // RAGGED top-level heaps ([n_trees + top_batch(L)][2^L])
  int32_t top_levels;          // L
  uint32_t nodes_bytes;        // bytes of `nodes` (RAGGED top-level kernel: < 2^31)
  int32_t lds_top_off;         // byte offset of the per-wave top-level copies in dynamic LDS
  const uint8_t *deep;         // PERFECT deep blocks of the top_levels plan, or nullptr
  int32_t deep_tree_bytes;     // their bytes per kernel tree (deep_tree_bytes(D, top_levels))
  int32_t top_group_bytes;     // PERFECT global: bytes of a lane group's top-level copy
  int32_t tile_coalesced;      // global-node RAGGED kernels: the row tile read 8 rows x 128 B a load
};

// Vector leaves: floats per leaf in leaf_vec, K rounded up to whole 16-byte groups.
constexpr int32_t vec_stride(int32_t K) { return (K + 3) & ~3; }

// Kernel launchers (defined in the .hip files).  Return a hipError_t as int.
int launch_perfect(int depth, const LaunchArgs &a, int waves, int64_t n_wg, int lds_bytes,
                   void *stream);
int launch_perfect_binned(int depth, const LaunchArgs &a, int waves, int64_t n_wg, int lds_bytes,
                          void *stream);
int launch_bin(const LaunchArgs &a, void *stream);
int launch_row_norm(const LaunchArgs &a, double *norm, void *stream);
// Device address of the allocation-free predict's row-norm scratch on the current device
// (kNoAllocMaxRows doubles); looked up once per device.  Returns a hipError_t as int.
int noalloc_norm_scratch(double **ptr);
int launch_perfect_global(int depth, const LaunchArgs &a, int waves, int64_t n_wg, int lds_bytes,
                          void *stream);
int launch_perfect_fixed(int depth, const LaunchArgs &a, int waves, int64_t n_wg, int lds_bytes,
                         void *stream);
int launch_ragged(const LaunchArgs &a, int waves, int64_t n_wg, int lds_bytes, void *stream);
int launch_ragged_global(const LaunchArgs &a, int waves, int64_t n_wg, int lds_bytes,
                         void *stream);
int launch_ragged_top(const LaunchArgs &a, int waves, int64_t n_wg, int lds_bytes, void *stream);
int launch_ragged_treelet(const LaunchArgs &a, int waves, int64_t n_wg, int lds_bytes,
                          void *stream);
int launch_direct(const LaunchArgs &a, int64_t n_wg, void *stream);
int launch_gemm(int depth, const LaunchArgs &a, int64_t n_wg, void *stream);

}  // namespace bridger
