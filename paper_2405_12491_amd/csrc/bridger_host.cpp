// bridger_host.cpp -- C ABI, forest validation, packing and launch planning.
//
// create: validate the caller's node arrays, order trees by class (stable, so the per-class
// sum keeps ascending tree order), detect perfect trees, pack the layouts of internal.h
// ("data type rewriting" and "redundant operator elimination" of Table 2: narrow node
// records, no stored child indices for perfect trees, no values at internal nodes), plan the
// launch with the data-movement model of Eq. 1, and upload.  predict: check arguments and
// launch on the caller's stream.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdint>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <deque>
#include <new>
#include <string>
#include <tuple>
#include <vector>

#include "bridger.h"
#include "internal.h"

using namespace bridger;

namespace {

thread_local std::string g_last_error;

bridger_status fail(bridger_status s, const std::string &msg) {
  g_last_error = msg;
  return s;
}

// ---------------------------------------------------------------- machine model
// Constants of the Eq. 1 model (bytes/s per level).  HBM and LDS figures are measured on
// MI355X by the calibration microbenchmarks; L2 is the per-XCD L2 request bandwidth summed
// over the 8 XCDs.  The LDS level is counted in wave-wide instructions: a conflict-free
// 32- or 64-bit per-lane gather costs one slot either way.
constexpr double kHbmBytesPerSec = 5.0e12;
constexpr double kL2BytesPerSec = 30.0e12;
constexpr double kLdsInstrPerSec = 0.44 * 256 * 2.4e9;
constexpr int kMaxWavesPerCU = 32;
constexpr double kL2BytesPerXcd = 4.0 * 1024 * 1024;
constexpr int kMinWavesPerCU = 8;
constexpr int kNumCUs = 256;
constexpr int64_t kLastLevelCacheBytes = int64_t(256) << 20;  // MI355X Infinity Cache
// Latency terms for small batches, where a workgroup's walk over its share of the trees, not
// the throughput of the LDS, sets the time: one dependent LDS gather (two per level, and the
// leaf), and the barrier and L2 round trip of a chunk.  Fitted by least squares to batches
// that take one round of workgroups (the 500-tree depth-6 and 100-tree depth-8 forests, one to
// sixteen lane groups, 7 to 32 chunks; 15 to 81 us): 35 ns and 0.63 us.
constexpr double kLdsLatencySec = 35e-9;
constexpr double kChunkLatencySec = 0.63e-6;
// Batch-size classes: besides the plan for large batches, each forest keeps plans made for
// batches of at most these many rows (a predict takes the smallest class that holds it).
constexpr int64_t kSizeClasses[] = {int64_t(1) << 13, int64_t(1) << 15, int64_t(1) << 17,
                                    int64_t(1) << 19};

int env_int(const char *name, int dflt) {
  const char *v = std::getenv(name);
  if (!v || !*v) return dflt;
  return std::atoi(v);
}

int ilog2(int64_t v) {
  int r = 0;
  while ((int64_t(1) << (r + 1)) <= v) ++r;
  return r;
}

struct DevArrays {
  void *nodes = nullptr;
  void *tree_start = nullptr;
  void *chunk_first = nullptr;
  void *chunk_rec = nullptr;
  void *leaf_map = nullptr;
};

}  // namespace

struct bridger_forest {
  int32_t n_trees = 0, F = 0, K = 1, aggregate = 0, transform = 0;
  int64_t n_nodes = 0;
  int32_t max_depth = 0, all_perfect = 0, perfect_depth = -1;
  bool host_only = false;
  int device = -1;
  int32_t kernel_active = kDirect;

  std::vector<int32_t> tree_order;   // kernel position -> caller tree
  std::vector<int32_t> class_begin;  // [K+1]
  std::vector<int32_t> class_count;  // [K]
  std::vector<float> base;           // [K]

  // PERFECT
  bool perfect_ok = false;
  int32_t perfect_tree_bytes = 0;
  std::vector<uint8_t> perfect_blob;
  std::vector<uint8_t> perfect_trav;  // traversal copy: {threshold, feature * 4R}
  std::vector<uint32_t> perfect_roots;  // per tree: the traversal copy's root record
  std::vector<int32_t> perfect_leaf_map;
  bool finite_thresholds = false;
  bool fixed_chunks = true;           // allow the compile-time chunk kernel variants
  Plan perfect_plan{};

  // RAGGED
  bool ragged_ok = false;
  std::vector<uint64_t> ragged_rec;
  std::vector<int32_t> ragged_tree_start;  // [T+1]
  std::vector<int32_t> ragged_rec_node;
  std::vector<int32_t> ragged_chunk_first, ragged_chunk_rec;
  int64_t ragged_max_tree_bytes = 0;
  Plan ragged_plan{};

  // exact feature quantization (Table 2 "data type rewriting"): per feature the distinct
  // thresholds ascending (-0 stored as +0); a binned forest keeps each threshold's rank
  int32_t bin_bytes = 0;                // 2 or 1; 0: some feature has 2^16 or more thresholds
  std::vector<float> q_values;
  std::vector<int32_t> q_off;           // [F + 1]
  Plan perfect_bplan{}, ragged_bplan{};
  bool perfect_bok = false, ragged_bok = false;
  std::vector<uint8_t> perfect_btrav;   // PERFECT traversal copy for bins: {rank, f * R * bytes}
  std::vector<uint32_t> perfect_broots;  // per tree: the binned copy's root record
  // PERFECT plans for small batches (kSizeClasses; the plans above serve larger batches), with
  // the traversal copies for their row tiles (copy -1: the one above serves)
  struct TravCopy {
    int32_t R;
    std::vector<uint8_t> trav;
    std::vector<uint32_t> roots;
    void *d_trav = nullptr, *d_roots = nullptr;
  };
  struct SizedPlan {
    int64_t max_rows;
    Plan plan;
    int copy;
  };
  std::vector<SizedPlan> perfect_sized, perfect_bsized;
  std::deque<TravCopy> perfect_copies, perfect_bcopies;
  // PERFECT deep blocks (layout in internal.h) below deep_tl top levels: thresholds' bits,
  // and ranks for bins; empty when the forest has more than kDeepMaxFeatures features
  std::vector<uint8_t> perfect_deep, perfect_bdeep;
  int32_t deep_tl = 0;
  void *d_perfect_deep = nullptr, *d_perfect_bdeep = nullptr;
  // RAGGED treelets (layout in internal.h): blocks (fp32 thresholds / ranks), per kernel tree
  // the first slot, per slot the leaf ids of its two children (4 words, 4 words, 1, 2 per slot)
  std::vector<uint32_t> treelets, btreelets;
  std::vector<int32_t> treelet_start, treelet_leaf;
  void *d_treelets = nullptr, *d_btreelets = nullptr, *d_treelet_start = nullptr,
       *d_treelet_leaf = nullptr;
  std::vector<uint64_t> ragged_brec;    // RAGGED records with ranks in place of thresholds
  std::vector<uint64_t> ragged_tops, ragged_btops;  // top-level heaps (fp32 / binned records)
  std::vector<int32_t> ragged_bchunk_first, ragged_bchunk_rec;

  // fused preprocessing (BRIDGER_PRE_*)
  int32_t pre_kind = 0;
  std::vector<double> pre_a, pre_b;
  void *d_pre_a = nullptr, *d_pre_b = nullptr;

  // vector leaves (BRIDGER_CREATE_VECTOR_LEAVES): K class values per leaf, numbered as each
  // kernel family finds its leaves (PERFECT: kernel tree x 2^D + leaf slot; RAGGED: record
  // index; DIRECT: record index)
  bool vec = false;
  std::vector<float> vec_perfect, vec_ragged, vec_direct;
  void *d_vec_perfect = nullptr, *d_vec_ragged = nullptr, *d_vec_direct = nullptr;

  // DIRECT
  std::vector<int32_t> direct_rec;  // 4 ints per record
  std::vector<int32_t> direct_root;
  std::vector<int32_t> direct_rec_node;

  // device copies
  void *d_class_begin = nullptr, *d_class_count = nullptr, *d_base = nullptr,
       *d_tree_order = nullptr;
  DevArrays d_perfect, d_ragged, d_direct;
  void *d_perfect_trav = nullptr, *d_perfect_roots = nullptr, *d_perfect_broots = nullptr;
  void *d_q_values = nullptr, *d_q_off = nullptr, *d_perfect_btrav = nullptr,
       *d_ragged_brec = nullptr, *d_ragged_bchunk_first = nullptr, *d_ragged_tops = nullptr,
       *d_ragged_btops = nullptr,
       *d_ragged_bchunk_rec = nullptr;
  double visits_per_row_est = 0;  // for the model: mean internal visits per row (all trees)
};

namespace {

// ------------------------------------------------------------------ validation
struct TreeShape {
  int32_t depth;    // max leaf depth
  bool perfect;     // all leaves at depth `depth` and 2^(depth+1)-1 nodes
  double mean_path; // mean leaf depth weighted uniformly (for the cost model only)
};

bridger_status validate_tree(int32_t t, int64_t n, const int32_t *feat, const float *thr,
                             const int32_t *left, const int32_t *right, int32_t F,
                             std::vector<int32_t> &depth_scratch, TreeShape &shape) {
  if (n < 1)
    return fail(BRIDGER_ERR_INVALID_FOREST, "tree " + std::to_string(t) + " has no nodes");
  std::vector<int32_t> parents(n, 0);
  for (int64_t i = 0; i < n; ++i) {
    const bool l_leaf = left[i] == -1, r_leaf = right[i] == -1;
    if (l_leaf != r_leaf)
      return fail(BRIDGER_ERR_INVALID_FOREST, "tree " + std::to_string(t) + " node " +
                                                  std::to_string(i) + " has exactly one child");
    if (l_leaf) continue;
    if (left[i] < 0 || left[i] >= n || right[i] < 0 || right[i] >= n)
      return fail(BRIDGER_ERR_INVALID_FOREST, "tree " + std::to_string(t) + " node " +
                                                  std::to_string(i) + " child out of range");
    if (left[i] == right[i])
      return fail(BRIDGER_ERR_INVALID_FOREST, "tree " + std::to_string(t) + " node " +
                                                  std::to_string(i) + " has identical children");
    if (feat[i] < 0 || feat[i] >= F)
      return fail(BRIDGER_ERR_INVALID_FOREST, "tree " + std::to_string(t) + " node " +
                                                  std::to_string(i) + " feature out of range");
    if (std::isnan(thr[i]))
      return fail(BRIDGER_ERR_INVALID_FOREST, "tree " + std::to_string(t) + " node " +
                                                  std::to_string(i) + " has a NaN threshold");
    parents[left[i]]++;
    parents[right[i]]++;
  }
  if (parents[0] != 0)
    return fail(BRIDGER_ERR_INVALID_FOREST, "tree " + std::to_string(t) + ": root is a child");
  for (int64_t i = 1; i < n; ++i)
    if (parents[i] != 1)
      return fail(BRIDGER_ERR_INVALID_FOREST,
                  "tree " + std::to_string(t) + " node " + std::to_string(i) +
                      (parents[i] ? " has several parents" : " is unreachable"));
  // breadth-first from the root: depths, reachability (parents==1 everywhere + reached all)
  depth_scratch.assign(n, -1);
  std::vector<int64_t> q;
  q.reserve(n);
  q.push_back(0);
  depth_scratch[0] = 0;
  int32_t maxd = 0;
  int64_t leaves = 0;
  double path_sum = 0;
  for (size_t qi = 0; qi < q.size(); ++qi) {
    int64_t i = q[qi];
    int32_t d = depth_scratch[i];
    if (left[i] == -1) {
      maxd = std::max(maxd, d);
      ++leaves;
      path_sum += d;
      continue;
    }
    if (d + 1 > 64)
      return fail(BRIDGER_ERR_INVALID_FOREST, "tree " + std::to_string(t) + " deeper than 64");
    for (int32_t c : {left[i], right[i]}) {
      if (depth_scratch[c] != -1)
        return fail(BRIDGER_ERR_INVALID_FOREST, "tree " + std::to_string(t) + " has a cycle");
      depth_scratch[c] = d + 1;
      q.push_back(c);
    }
  }
  if ((int64_t)q.size() != n)
    return fail(BRIDGER_ERR_INVALID_FOREST, "tree " + std::to_string(t) + " has unreachable nodes");
  shape.depth = maxd;
  shape.perfect = (maxd <= 30) && (n == (int64_t(2) << maxd) - 1);
  if (shape.perfect)
    for (int64_t i = 0; i < n; ++i)
      if (left[i] == -1 && depth_scratch[i] != maxd) shape.perfect = false;
  shape.mean_path = leaves ? path_sum / leaves : 0;
  return BRIDGER_OK;
}

// -------------------------------------------------------------------- packing
// Vector leaves of at most 4 classes are read by the chunked PERFECT kernel from LDS: their
// class rows sit in the tree blocks in place of the scalar leaves (measured 4-8% faster for
// K = 2..4; with 8-float rows the larger blocks pushed the plan to one workgroup per CU and
// the 8-class GBDT forest ran 6% slower, so 5..8 classes keep their rows in global memory).
bool perfect_vec_rows(const bridger_forest *h) { return h->vec && h->K <= 4; }

void pack_perfect(bridger_forest *h, int D, const int64_t *offs, const int32_t *feat,
                  const float *thr, const int32_t *left, const int32_t *right,
                  const float *value) {
  const int n_int = (1 << D) - 1, n_leaf = 1 << D;
  const int leaf_off = 8 * (n_int + 1);   // 1-based heap: slots 1 .. 2^D - 1, slot 0 unused
  // vector leaves (K <= 4): the leaf block holds class rows, filled by build_vector_leaves
  const bool rows = perfect_vec_rows(h);
  const int tb = rows ? (8 + 4 * vec_stride(h->K)) << D : perfect_tree_bytes(D);
  h->perfect_tree_bytes = tb;
  h->perfect_blob.assign((size_t)tb * h->n_trees, 0);
  h->perfect_leaf_map.assign((size_t)n_leaf * h->n_trees, -1);
  std::vector<int32_t> heap_to_node((size_t)2 * n_leaf);
  for (int32_t k = 0; k < h->n_trees; ++k) {
    const int32_t t = h->tree_order[k];
    const int64_t a = offs[t];
    // 1-based heap slot -> caller node
    heap_to_node[1] = 0;
    for (int m = 1; m <= n_int; ++m) {
      const int32_t nd = heap_to_node[m];
      heap_to_node[2 * m] = left[a + nd];
      heap_to_node[2 * m + 1] = right[a + nd];
    }
    uint8_t *blk = h->perfect_blob.data() + (size_t)k * tb;
    for (int m = 1; m <= n_int; ++m) {
      const int32_t nd = heap_to_node[m];
      const float th = thr[a + nd];
      const uint32_t f = (uint32_t)feat[a + nd];
      std::memcpy(blk + 8 * m, &th, 4);
      std::memcpy(blk + 8 * m + 4, &f, 4);
    }
    for (int j = 0; j < n_leaf; ++j) {
      const int32_t nd = heap_to_node[n_leaf + j];
      const float v = value[a + nd];
      if (!rows) std::memcpy(blk + leaf_off + 4 * j, &v, 4);
      h->perfect_leaf_map[(size_t)k * n_leaf + j] = nd;
    }
  }
}

// Records of the PERFECT kernel: the feature index becomes the byte offset of the feature's
// row in the LDS tile of the chosen plan (row stride 4R bytes), and a threshold of -0 is
// stored as +0 (equal under <=; the sign-of-difference step needs the +0).
void make_perfect_trav(const bridger_forest *h, int32_t R, std::vector<uint8_t> &trav,
                       std::vector<uint32_t> &roots) {
  const int D = h->perfect_depth;
  const int tb = h->perfect_tree_bytes;
  const uint32_t row_bytes = 4u * (uint32_t)R;
  trav = h->perfect_blob;
  for (int32_t k = 0; k < h->n_trees; ++k) {
    uint8_t *blk = trav.data() + (size_t)k * tb;
    for (int m = 1; m < (1 << D); ++m) {
      float th;
      uint32_t f;
      std::memcpy(&th, blk + 8 * m, 4);
      std::memcpy(&f, blk + 8 * m + 4, 4);
      if (th == 0.0f) th = 0.0f;
      f *= row_bytes;
      std::memcpy(blk + 8 * m, &th, 4);
      std::memcpy(blk + 8 * m + 4, &f, 4);
    }
  }
  roots.assign((size_t)2 * h->n_trees, 0);
  for (int32_t k = 0; k < h->n_trees; ++k)
    std::memcpy(&roots[2 * (size_t)k], trav.data() + (size_t)k * tb + 8, 8);
}

void build_perfect_trav(bridger_forest *h) {
  make_perfect_trav(h, h->perfect_plan.rows_per_wg, h->perfect_trav, h->perfect_roots);
}

// Breadth-first record order with adjacent children; returns false if a tree cannot be
// encoded (child offset or feature index too large).
bool pack_ragged(bridger_forest *h, const int64_t *offs, const int32_t *feat, const float *thr,
                 const int32_t *left, const int32_t *right, const float *value) {
  if (h->F > kMaxRaggedFeatures) return false;
  h->ragged_rec.clear();
  h->ragged_rec.reserve(h->n_nodes);
  h->ragged_rec_node.clear();
  h->ragged_rec_node.reserve(h->n_nodes);
  h->ragged_tree_start.assign(h->n_trees + 1, 0);
  h->ragged_max_tree_bytes = 0;
  std::vector<int32_t> order;
  std::vector<int32_t> slot;
  for (int32_t k = 0; k < h->n_trees; ++k) {
    const int32_t t = h->tree_order[k];
    const int64_t a = offs[t], n = offs[t + 1] - offs[t];
    const int64_t base = (int64_t)h->ragged_rec.size();
    if (base + n + 1 > INT32_MAX) return false;
    h->ragged_tree_start[k] = (int32_t)base;
    order.assign(1, 0);
    slot.assign(n, -1);
    slot[0] = 0;
    for (size_t qi = 0; qi < order.size(); ++qi) {
      const int32_t nd = order[qi];
      if (left[a + nd] == -1) continue;
      slot[left[a + nd]] = (int32_t)order.size();
      order.push_back(left[a + nd]);
      slot[right[a + nd]] = (int32_t)order.size();
      order.push_back(right[a + nd]);
    }
    const int64_t n_padded = n + (n & 1);  // even record count: trees start 16-byte aligned
    for (int64_t s = 0; s < n; ++s) {
      const int32_t nd = order[s];
      uint32_t w, meta;
      if (left[a + nd] == -1) {
        const int64_t next_rel = n_padded - s;
        if (next_rel > kMaxRel) return false;
        std::memcpy(&w, &value[a + nd], 4);
        meta = (uint32_t)kLeafFlag | (uint32_t)next_rel;
      } else {
        const int64_t rel = slot[left[a + nd]] - s;
        if (rel < 1 || rel > kMaxRel) return false;
        std::memcpy(&w, &thr[a + nd], 4);
        meta = ((uint32_t)feat[a + nd] << 16) | (uint32_t)rel;
      }
      h->ragged_rec.push_back((uint64_t)w | ((uint64_t)meta << 32));
      h->ragged_rec_node.push_back(nd);
    }
    if (n_padded != n) {  // filler record, never visited
      h->ragged_rec.push_back((uint64_t)kLeafFlag << 32);
      h->ragged_rec_node.push_back(-1);
    }
    h->ragged_max_tree_bytes = std::max<int64_t>(h->ragged_max_tree_bytes, 8 * n_padded);
  }
  h->ragged_tree_start[h->n_trees] = (int32_t)h->ragged_rec.size();
  return true;
}

void pack_direct(bridger_forest *h, const int64_t *offs, const int32_t *feat, const float *thr,
                 const int32_t *left, const int32_t *right, const float *value) {
  h->direct_rec.assign((size_t)4 * h->n_nodes, 0);
  h->direct_rec_node.assign(h->n_nodes, 0);
  h->direct_root.assign(h->n_trees, 0);
  int64_t r = 0;
  for (int32_t k = 0; k < h->n_trees; ++k) {
    const int32_t t = h->tree_order[k];
    const int64_t a = offs[t], n = offs[t + 1] - offs[t];
    h->direct_root[k] = (int32_t)r;
    for (int64_t i = 0; i < n; ++i) {
      int32_t *rec = &h->direct_rec[(size_t)4 * (r + i)];
      float w = left[a + i] == -1 ? value[a + i] : thr[a + i];
      std::memcpy(&rec[0], &w, 4);
      rec[1] = left[a + i] == -1 ? -1 : feat[a + i];
      rec[2] = left[a + i] == -1 ? -1 : (int32_t)(r + left[a + i]);
      rec[3] = left[a + i] == -1 ? -1 : (int32_t)(r + right[a + i]);
      h->direct_rec_node[r + i] = (int32_t)i;
    }
    r += n;
  }
}

// Vector leaves: the K class values of every leaf (rows of vec_stride(K) floats), numbered as
// each kernel family finds its leaves (PERFECT: kernel tree x 2^D + leaf slot; RAGGED and
// DIRECT: record index); zeros for internal and filler records and for the padding.
void build_vector_leaves(bridger_forest *h, const int64_t *offs, const int32_t *left,
                         const float *value) {
  const int K = h->K, KS = vec_stride(K);  // rows padded with zeros to whole 16-byte groups
  auto put = [&](std::vector<float> &dst, size_t slot, int32_t t, int32_t nd) {
    if (nd < 0) return;  // filler record
    const int64_t i = offs[t] + nd;
    if (left[i] != -1) return;
    std::memcpy(&dst[slot * KS], &value[i * K], sizeof(float) * K);
  };
  if (!h->perfect_leaf_map.empty()) {
    const size_t n_leaf = (size_t)1 << h->perfect_depth;
    h->vec_perfect.assign(n_leaf * h->n_trees * KS, 0.0f);
    for (int32_t k = 0; k < h->n_trees; ++k)
      for (size_t j = 0; j < n_leaf; ++j)
        put(h->vec_perfect, k * n_leaf + j, h->tree_order[k], h->perfect_leaf_map[k * n_leaf + j]);
    if (perfect_vec_rows(h)) {  // the rows also go into every copy of the tree blocks
      const size_t tb = (size_t)h->perfect_tree_bytes, row = 4 * (size_t)KS;
      std::vector<std::vector<uint8_t> *> blobs{&h->perfect_blob, &h->perfect_trav,
                                                &h->perfect_btrav};
      for (auto *cs : {&h->perfect_copies, &h->perfect_bcopies})
        for (auto &c : *cs) blobs.push_back(&c.trav);
      for (std::vector<uint8_t> *blob : blobs) {
        if (blob->empty()) continue;
        for (int32_t k = 0; k < h->n_trees; ++k)
          std::memcpy(blob->data() + k * tb + 8 * n_leaf, &h->vec_perfect[k * n_leaf * KS],
                      n_leaf * row);
      }
    }
  }
  if (!h->ragged_rec.empty()) {
    h->vec_ragged.assign(h->ragged_rec.size() * KS, 0.0f);
    for (int32_t k = 0; k < h->n_trees; ++k)
      for (int32_t r = h->ragged_tree_start[k]; r < h->ragged_tree_start[k + 1]; ++r)
        put(h->vec_ragged, r, h->tree_order[k], h->ragged_rec_node[r]);
  }
  h->vec_direct.assign(h->direct_rec_node.size() * KS, 0.0f);
  for (int32_t k = 0; k < h->n_trees; ++k) {
    const int32_t t = h->tree_order[k];
    const int64_t n = offs[t + 1] - offs[t];
    for (int64_t i = 0; i < n; ++i)
      put(h->vec_direct, h->direct_root[k] + i, t, h->direct_rec_node[h->direct_root[k] + i]);
  }
}

// -------------------------------------------------------------- Eq. 1 planner
// Choose (waves per workgroup, rows per tile, chunk size) minimising the slowest level's
// data-movement time max_l DataMove_l / BandWidth_l, subject to the LDS capacity of a CU
// (DataOccupy_LDS < Capacity_LDS) and to keeping at least kMinWavesPerCU waves resident
// (relaxed if nothing satisfies it).  Levels: HBM (X once, output once, forest once), L2->LDS
// (the forest is staged once per workgroup), LDS reads (per-visit node and feature gathers,
// plus one leaf read per tree).  Ties (the usual case: the LDS level binds) go to higher
// occupancy, then to fewer chunks.
struct PlanInput {
  int64_t n_rows;
  int32_t F, K, n_trees;
  double forest_bytes;
  int32_t tree_bytes;      // PERFECT: fixed block; RAGGED: largest tree
  bool perfect;
  double visits_per_row;
  int32_t x_bytes = 4;     // element of the LDS tile: 4 (fp32) or 2 / 1 (bins)
  bool vec = false;        // vector leaves
  int32_t depth = 0;       // PERFECT: the trees' depth
  bool deep = false;       // PERFECT: deep blocks exist (wide-row plans may use them)
};

// Smallest tile: bins pack 4 / x_bytes rows per 32-bit word and a half-wave's 32 rows must
// fill 32 words of each feature's row, so R >= 32 * 4 / x_bytes.
int min_rows(const PlanInput &in) { return 32 * (4 / in.x_bytes); }

Plan choose_plan(const PlanInput &in) {
  // trees walked at once per lane (PERFECT): 4 unless the LDS only fits fewer trees per lane
  // group; forced with BRIDGER_ILP
  const int force_ilp = env_int("BRIDGER_ILP", 0);
  std::vector<int> ilps;
  if (force_ilp == 1 || force_ilp == 2 || force_ilp == 4) ilps = {force_ilp};
  else if (in.perfect) ilps = {4, 2, 1};
  else ilps = {4};
  const int force_waves = env_int("BRIDGER_WAVES", 0);
  const int force_rows = env_int("BRIDGER_ROWS", 0);
  const int force_ct = env_int("BRIDGER_CHUNK_TREES", 0);
  const int force_wg_per_cu = env_int("BRIDGER_WG_PER_CU", 0);
  const int64_t n = std::max<int64_t>(in.n_rows, 1);
  struct Cand {
    Plan p;
    int waves_cu, single, overlap;
  };
  std::vector<Cand> cands;
  for (int pass = 0; pass < 2 && cands.empty(); ++pass) {
   for (const int ilp : ilps) {
    const int kTreesMultiple = ilp;
    for (int W : {1, 2, 4, 8}) {  // compute waves; each workgroup also has a staging wave
      if (force_waves && W != force_waves) continue;
      for (int R = min_rows(in); R <= 64 * W; R *= 2) {
        if (force_rows && R != force_rows) continue;
        const int G = 64 * W / R;
        if (G > 1 && !in.perfect && R < 64) continue;
        const bool acc_lds = in.K > 1 || G > 1;
        const int64_t x_tile = (int64_t)in.F * R * in.x_bytes;
        // PERFECT with at most 8 classes (vector leaves, or scalar leaves walked 4 trees at a
        // time) keeps the class sums in registers and writes them only after the walk, into
        // the row tile's LDS
        const bool alias = in.perfect && acc_lds && in.K <= 8 && (in.vec || ilp == 4) &&
                           (int64_t)in.K * G * R * 8 <= x_tile;
        const int64_t acc_bytes = acc_lds && !alias ? (int64_t)in.K * G * R * 8 : 0;
        for (int m = 1; m <= kMaxWavesPerCU / (W + 1); ++m) {  // workgroups per CU
          if (force_wg_per_cu && m != force_wg_per_cu) continue;
          if (pass == 0 && m * W < kMinWavesPerCU) continue;
          const int64_t budget = kLdsBytesPerCU / m - x_tile - acc_bytes;
          if (budget < 2 * (int64_t)in.tree_bytes) continue;
          int64_t chunk = std::min<int64_t>(budget / 2, 65536);
          int ct = 0;
          int n_chunks;
          if (in.perfect) {
            ct = (int)(chunk / in.tree_bytes);
            ct -= ct % kTreesMultiple;
            if (ct < kTreesMultiple) {
              if (in.n_trees < kTreesMultiple && ct >= in.n_trees) ct = in.n_trees;
              else continue;
            }
            ct = std::min(ct, ((in.n_trees + kTreesMultiple - 1) / kTreesMultiple) * kTreesMultiple);
            // a power of two, so that the compile-time chunk variants of the kernel apply
            if (ct >= kTreesMultiple)
              while (ct & (ct - 1)) ct &= ct - 1;
            if (force_ct) {
              if (force_ct * (int64_t)in.tree_bytes > chunk) continue;
              ct = force_ct;
            }
            // every lane group needs at least one group of trees per chunk
            if (ct < kTreesMultiple * G && in.n_trees >= kTreesMultiple * G) continue;
            chunk = (int64_t)ct * in.tree_bytes;
            n_chunks = (in.n_trees + ct - 1) / ct;
          } else {
            if (chunk < in.tree_bytes) continue;
            chunk &= ~int64_t(1023);
            if (chunk < in.tree_bytes) continue;
            // lane groups split a chunk's trees by count: want about one tree per group at
            // least (a walk costs its path length, not the tree's size, so equal counts
            // balance the groups)
            if (G > 1 && chunk < 0.8 * G * in.forest_bytes / in.n_trees) continue;
            n_chunks = (int)std::ceil(in.forest_bytes / (0.9 * chunk));
          }
          const int64_t lds = 2 * chunk + x_tile + acc_bytes;
          if (lds > kLdsBytesPerCU) continue;
          const double n_wg = std::ceil((double)n / R);
          const double hbm = (double)n * in.F * 4 + (double)n * in.K * 4 + in.forest_bytes;
          const double stage = n_wg * in.forest_bytes + (double)n * in.F * 4;
          const double lds_instr =
              (double)n / 64.0 * (2.0 * in.visits_per_row + in.n_trees) +
              n_wg * (in.forest_bytes / 1024.0);
          // fewer workgroups than resident slots leave CUs idle; and a workgroup cannot finish
          // before its lanes' dependent gathers over their share of the trees, once per round
          // of resident workgroups
          const double slots = (double)kNumCUs * m;
          const double fill = std::min(1.0, n_wg / slots);
          const double rounds = std::ceil(n_wg / slots);
          const double per_tree_visits = in.visits_per_row / std::max(in.n_trees, 1);
          const double chain = rounds * (std::ceil((double)in.n_trees / ((double)G * ilp)) *
                                             (2.0 * per_tree_visits + 1.0) * kLdsLatencySec +
                                         n_chunks * kChunkLatencySec);
          Cand c{};
          c.p.waves = W;
          c.p.rows_per_wg = R;
          c.p.groups = G;
          c.p.chunk_bytes = (int32_t)chunk;
          c.p.trees_per_chunk = ct;
          c.p.n_chunks = n_chunks;
          c.p.lds_bytes = (int32_t)lds;
          c.p.acc_in_lds = acc_lds;
          c.p.acc_alias = alias ? 1 : 0;
          c.p.ilp = ilp;
          c.p.hbm_bytes = hbm;
          c.p.stage_bytes = stage;
          c.p.lds_read_bytes = lds_instr * 256.0;
          c.p.est_seconds = std::max({hbm / kHbmBytesPerSec, stage / kL2BytesPerSec,
                                      lds_instr / kLdsInstrPerSec}) / fill;
          c.p.est_seconds = std::max(c.p.est_seconds, chain);
          c.waves_cu = m * W;
          c.p.waves_per_cu = m * W;
          c.single = G == 1;
          c.overlap = m >= 2;
          cands.push_back(c);
        }
      }
    }
   }
  }
  Plan best{};
  if (cands.empty()) return best;  // infeasible: waves == 0
  double t_min = 1e300;
  for (const Cand &c : cands) t_min = std::min(t_min, c.p.est_seconds);
  // The model resolves a few percent; among plans within 2% of the fastest prefer enough
  // resident waves to keep every SIMD issuing, then one lane group (each lane walks every
  // tree of its row: no split of a chunk's trees and no partial sums), then more trees per
  // lane, then more resident waves (latency hiding), then two or more workgroups per CU (one
  // workgroup's barrier and tail overlap another's work), then fewer chunks.
  const Cand *pick = nullptr;
  const bool log = env_int("BRIDGER_LOG", 0) != 0;
  for (const Cand &c : cands) {
    if (log)
      std::fprintf(stderr, "[bridger plan] W=%d R=%d G=%d U=%d waves/CU=%d chunk=%d ct=%d chunks=%d lds=%d est=%.1fus%s\n",
                   c.p.waves, c.p.rows_per_wg, c.p.groups, c.p.ilp, c.waves_cu, c.p.chunk_bytes,
                   c.p.trees_per_chunk, c.p.n_chunks, c.p.lds_bytes, c.p.est_seconds * 1e6,
                   c.p.est_seconds > 1.02 * t_min ? "" : "  (tie)");
    if (c.p.est_seconds > 1.02 * t_min) continue;
    if (!pick) { pick = &c; continue; }
    // a CU issues from its four SIMDs: below two compute waves per SIMD, more waves come
    // before a single lane group.  Bins: at equal resident waves, 4-wave workgroups before
    // 8-wave ones (measured on the depth-6, 500-tree, 28-feature forest with 16-bit bins: 8
    // waves x 3 workgroups 0.46 ms, 4 waves x 6 workgroups 0.42 ms; fp32 tiles show no
    // difference, 0.423 against 0.424 ms, and keep the fewer chunks)
    const bool bins = in.x_bytes < 4;
    auto key = [bins](const Cand &x) {
      return std::make_tuple(std::min(x.waves_cu, kMinWavesPerCU), x.single, x.p.ilp,
                             x.waves_cu, bins ? -std::max(x.p.waves, 4) : 0, x.overlap,
                             -x.p.n_chunks);
    };
    if (key(c) > key(*pick)) pick = &c;
  }
  return pick->p;
}

// Wide rows: a plan for the global-node kernels (PERFECT and RAGGED).  The LDS holds the row
// tile and the per-group class sums only; G lane groups split the trees; up to 16 waves per
// workgroup (no staging wave).  Picks the most resident waves (every wave hides L2 round
// trips), then fewer lane groups, then more rows per tile.
// Top levels of the RAGGED lockstep kernel read from LDS: 5 (4 trees per batch) measured at
// least as fast as 4 (8 trees per batch) on the ragged forests, fp32 and binned, and 6 (2 trees
// per batch) slower; BRIDGER_TOP_LEVELS=4 overrides.
int top_levels_default() {
  const int l = env_int("BRIDGER_TOP_LEVELS", kTopLevelsDefault);
  return (l == 4 || l == 5) ? l : kTopLevelsDefault;
}

// Top levels of the PERFECT global-node kernel read from LDS (BRIDGER_PERFECT_TOP_LEVELS
// overrides).  With the deep blocks, on the 10-class 784-feature forest: 4 levels of 8 trees per
// lane in workgroups of 16 waves 0.489 ms (16-bit bins 0.370); 3 levels of 16 trees, whose
// registers allow 8 waves, 0.536 (0.443); 4 levels of 16 trees in 2 KB copies 0.535; 5 of 8,
// 0.551.  Without deep blocks: 3 levels 0.629, 4 levels 0.685; 2 levels with 32 trees per lane
// spill registers.
int perfect_top_levels(int depth) {
  const int dflt = depth > kPerfectTopLevels ? kPerfectTopLevels : 3;
  const int l = env_int("BRIDGER_PERFECT_TOP_LEVELS", dflt);
  return (l >= 3 && l <= 5) ? l : dflt;
}

// Bytes of a lane group's copy of top levels: 1 KB (3 levels of 16 trees, 4 of 8), 2 KB (4
// levels of 16 trees, 5 of 8; with deep blocks only).
int perfect_top_group_bytes(int L, bool deep) {
  if (!deep) return 1024;
  if (L == 5) return 2048;
  return env_int("BRIDGER_TOP_GROUP_KB", 1) == 2 ? 2048 : 1024;
}

// Deep blocks: scalar leaves, feature indices in 10 bits, trees deeper than the top levels,
// all of them addressed by 32-bit byte offsets.
bool deep_possible(bool vec, int F, int depth, int64_t n_trees) {
  const int tl = perfect_top_levels(depth);
  return env_int("BRIDGER_DEEP", 1) != 0 && !vec && F <= kDeepMaxFeatures && depth > tl &&
         n_trees * deep_tree_bytes(depth, tl) < (int64_t(1) << 31);
}

// tops: the RAGGED variant whose top levels come from per-wave LDS copies (one class, scalar
// leaves, lane groups of whole waves): the LDS holds the row tile and kTopWaveBytes per wave,
// which also take the group sums at the end.
Plan choose_global_plan(const PlanInput &in, bool tops = false) {
  Plan best{};
  const int force_waves = env_int("BRIDGER_WAVES", 0);
  const int force_rows = env_int("BRIDGER_ROWS", 0);
  const int wave_cap = env_int("BRIDGER_GLOBAL_WAVES_CU", 32);
  auto key = [wave_cap](const Plan &p) {
    return std::make_tuple(std::min(p.waves_per_cu, wave_cap), -p.groups, p.rows_per_wg);
  };
  for (int W : {1, 2, 4, 8, 16}) {
    if (force_waves && W != force_waves) continue;
    for (int R = min_rows(in); R <= 64 * W; R *= 2) {
      if (force_rows && R != force_rows) continue;
      const int G = 64 * W / R;
      if (G > 1 && (int64_t)G * 4 > in.n_trees) continue;  // a few trees per lane group
      if (tops && !in.perfect && R < 64) continue;         // a group is whole waves
      // PERFECT top levels: 1 or 2 KB per lane group of each wave (a wave holds 64 / R groups
      // when R < 64), besides the class sums, which the deep-block kernel keeps in registers
      // (at most 16 classes) and writes into the row tile after the walk
      const int tl = perfect_top_levels(in.depth);
      const int gb_deep = perfect_top_group_bytes(tl, true);
      const int u_deep = gb_deep / (8 << tl);  // trees per lane
      const bool deep = tops && in.perfect && in.deep && W <= (u_deep > 8 ? 8 : 16);
      const int gb = perfect_top_group_bytes(tl, deep);
      const int64_t tile = (int64_t)in.F * R * in.x_bytes;
      const int64_t acc = (int64_t)in.K * G * R * 8;
      const bool alias = deep && in.K <= 16 && acc <= tile && env_int("BRIDGER_REG_SUMS", 1) != 0;
      const int64_t top_bytes_wg =
          !tops ? 0 : in.perfect ? (int64_t)W * std::max(1, 64 / R) * gb
                                 : (int64_t)W * kTopWaveBytes;
      const int64_t lds = tile + top_bytes_wg + ((tops && !in.perfect) || alias ? 0 : acc);
      if (lds > kLdsBytesPerCU) continue;
      const int m = (int)std::min<int64_t>(kLdsBytesPerCU / lds, kMaxWavesPerCU / W);
      if (m < 1) continue;
      Plan p{};
      p.waves = W;
      p.rows_per_wg = R;
      p.groups = G;
      p.lds_bytes = (int32_t)lds;
      p.acc_in_lds = 1;
      p.ilp = env_int("BRIDGER_ILP", 8) == 4 ? 4 : 8;  // L2 round trips: keep 8 in flight
      p.global_nodes = 1;
      p.tops = !tops ? 0 : in.perfect ? tl : top_levels_default();
      p.acc_alias = alias ? 1 : 0;
      p.top_group_bytes = tops && in.perfect ? gb : 0;
      p.waves_per_cu = m * W;
      const double n = (double)std::max<int64_t>(in.n_rows, 1);
      p.hbm_bytes = n * in.F * 4 + n * in.K * 4 + in.forest_bytes;
      p.lds_read_bytes = 256.0 * n / 64.0 * in.visits_per_row;
      if (best.waves == 0 || key(p) > key(best)) best = p;
    }
  }
  return best;
}

// Cut the RAGGED trees into chunks of at most chunk_bytes (whole trees, in kernel order).
int32_t ragged_chunks(const bridger_forest *h, int64_t chunk_bytes, std::vector<int32_t> &first,
                      std::vector<int32_t> &rec) {
  first.assign(1, 0);
  rec.assign(1, 0);
  int64_t cur = 0;
  for (int32_t k = 0; k < h->n_trees; ++k) {
    const int64_t tbytes = 8 * (int64_t)(h->ragged_tree_start[k + 1] - h->ragged_tree_start[k]);
    if (cur > 0 && cur + tbytes > chunk_bytes) {
      first.push_back(k);
      rec.push_back(h->ragged_tree_start[k]);
      cur = 0;
    }
    cur += tbytes;
  }
  first.push_back(h->n_trees);
  rec.push_back(h->ragged_tree_start[h->n_trees]);
  return (int32_t)first.size() - 1;
}

// The chunked plan, or the global-node plan when the chunked one leaves fewer than eight
// compute waves per CU (wide rows) and, for PERFECT, the forest fits in L2, or when a RAGGED
// forest does not fit in L2.
Plan pick_plan(const PlanInput &pin) {
  Plan p = choose_plan(pin);
  const int gmode = env_int("BRIDGER_GLOBAL", -1);  // tuning override: 0 off, 1 on
  if (gmode == 0) return p;
  Plan g = choose_global_plan(pin);
  if (g.waves == 0) return p;
  if (!pin.perfect) {  // trees walked at once per lane (8: 3% faster than 4 on ragged forests)
    const int u = env_int("BRIDGER_ILP", 8);
    g.ilp = (u == 1 || u == 2 || u == 4) ? u : 8;
    // one class with scalar leaves: the top levels from per-wave LDS copies when that keeps as
    // many resident waves (BRIDGER_TOPS=0 turns it off)
    if (pin.K == 1 && !pin.vec && pin.forest_bytes < 2147483648.0 &&
        env_int("BRIDGER_TOPS", 1) != 0 && !env_int("BRIDGER_ILP", 0)) {
      Plan t = choose_global_plan(pin, true);
      if (t.waves && t.waves_per_cu >= g.waves_per_cu) {
        t.ilp = top_batch(t.tops);
        g = t;
      }
    }
  }
  // Ragged trees: the global-node kernel, whose lanes walk their trees in lockstep with no
  // barrier inside the walk, measured as fast or faster than the LDS-chunked state machine on
  // every ragged forest tried (up to 1.9x on depth 10-12 trees, where a chunk holds few trees
  // and every chunk's barrier waits for its deepest path); a forest larger than L2 would
  // moreover be restaged from memory for every row tile.
  if (!pin.perfect) return g;
  // PERFECT trees deeper than the copied levels, scalar leaves, eight trees per lane: the top
  // levels from per-wave LDS copies when that keeps as many resident waves
  if (!pin.vec && pin.depth > perfect_top_levels(pin.depth) && g.ilp == 8 &&
      env_int("BRIDGER_TOPS", 1) != 0) {
    Plan t = choose_global_plan(pin, true);
    if (t.waves && t.waves_per_cu >= g.waves_per_cu) {
      t.ilp = 1024 / (8 << t.tops);
      g = t;
    }
  }
  const bool few = p.waves == 0 || p.waves_per_cu < kMinWavesPerCU;
  const bool fits = pin.forest_bytes <= kL2BytesPerXcd;
  if (gmode == 1 || (few && fits && g.waves_per_cu > p.waves_per_cu)) return g;
  return p;
}

// Per feature, the distinct thresholds ascending; false if a feature has 2^16 or more.
bool build_quantization(bridger_forest *h, const int32_t *feat, const float *thr,
                        const int32_t *left) {
  std::vector<std::vector<float>> per(h->F);
  for (int64_t i = 0; i < h->n_nodes; ++i)
    if (left[i] != -1) per[feat[i]].push_back(thr[i] == 0.0f ? 0.0f : thr[i]);
  size_t max_n = 0;
  h->q_off.assign(h->F + 1, 0);
  h->q_values.clear();
  for (int32_t f = 0; f < h->F; ++f) {
    std::vector<float> &u = per[f];
    std::sort(u.begin(), u.end());
    u.erase(std::unique(u.begin(), u.end()), u.end());
    max_n = std::max(max_n, u.size());
    h->q_off[f] = (int32_t)h->q_values.size();
    h->q_values.insert(h->q_values.end(), u.begin(), u.end());
  }
  h->q_off[h->F] = (int32_t)h->q_values.size();
  // a bin ranges over 0 .. n (n = the feature's threshold count, for values above all of them)
  h->bin_bytes = max_n <= 255 ? 1 : (max_n <= 65535 ? 2 : 0);
  return h->bin_bytes != 0;
}

uint32_t rank_of(const bridger_forest *h, int32_t f, float t) {
  const float *b = h->q_values.data() + h->q_off[f];
  const float *e = h->q_values.data() + h->q_off[f + 1];
  return (uint32_t)(std::lower_bound(b, e, t == 0.0f ? 0.0f : t) - b);
}

// PERFECT traversal copy for bins: {rank, byte offset f * R * bin_bytes of the feature's row}.
void make_perfect_btrav(const bridger_forest *h, int32_t R, std::vector<uint8_t> &trav,
                        std::vector<uint32_t> &roots) {
  const int D = h->perfect_depth;
  const int tb = h->perfect_tree_bytes;
  const uint32_t row_bytes = (uint32_t)R * (uint32_t)h->bin_bytes;
  trav = h->perfect_blob;
  for (int32_t k = 0; k < h->n_trees; ++k) {
    uint8_t *blk = trav.data() + (size_t)k * tb;
    for (int m = 1; m < (1 << D); ++m) {
      float th;
      uint32_t f;
      std::memcpy(&th, blk + 8 * m, 4);
      std::memcpy(&f, blk + 8 * m + 4, 4);
      const uint32_t r = rank_of(h, (int32_t)f, th), off = f * row_bytes;
      std::memcpy(blk + 8 * m, &r, 4);
      std::memcpy(blk + 8 * m + 4, &off, 4);
    }
  }
  roots.assign((size_t)2 * h->n_trees, 0);
  for (int32_t k = 0; k < h->n_trees; ++k)
    std::memcpy(&roots[2 * (size_t)k], trav.data() + (size_t)k * tb + 8, 8);
}

void build_perfect_btrav(bridger_forest *h) {
  make_perfect_btrav(h, h->perfect_bplan.rows_per_wg, h->perfect_btrav, h->perfect_broots);
}

// Deep blocks of the PERFECT trees below TL top levels (layout in internal.h) from the packed
// blocks: thresholds as stored (-0 as +0, as in the traversal copy), or their ranks (binned).
void make_perfect_deep(const bridger_forest *h, int TL, bool binned, std::vector<uint8_t> &deep) {
  const int D = h->perfect_depth, tb = h->perfect_tree_bytes;
  const int dtb = deep_tree_bytes(D, TL), ND = D - TL, NP = ND / 2;
  deep.assign((size_t)dtb * h->n_trees, 0);
  for (int32_t k = 0; k < h->n_trees; ++k) {
    const uint8_t *blk = h->perfect_blob.data() + (size_t)k * tb;
    uint8_t *out = deep.data() + (size_t)k * dtb;
    auto rec = [&](int m, uint32_t &w, uint32_t &f) {
      float th;
      std::memcpy(&th, blk + 8 * m, 4);
      std::memcpy(&f, blk + 8 * m + 4, 4);
      if (th == 0.0f) th = 0.0f;
      if (binned) w = rank_of(h, (int32_t)f, th);
      else std::memcpy(&w, &th, 4);
    };
    auto leaf = [&](int j) {
      uint32_t v;
      std::memcpy(&v, blk + (8 << D) + 4 * j, 4);
      return v;
    };
    for (int i = 0; i < NP; ++i) {
      const int d = TL + 2 * i;
      for (int m = 1 << d; m < (2 << d); ++m) {
        uint32_t w[3], f[3];
        rec(m, w[0], f[0]);
        rec(2 * m, w[1], f[1]);
        rec(2 * m + 1, w[2], f[2]);
        const uint32_t q[4] = {w[0], w[1], w[2], f[0] | f[1] << 10 | f[2] << 20};
        std::memcpy(out + deep_pair_off(TL, i) + 16 * (m - (1 << d)), q, 16);
      }
    }
    uint8_t *tail = out + deep_pair_off(TL, NP);
    if (ND & 1) {
      for (int m = 1 << (D - 1); m < (1 << D); ++m) {
        uint32_t q[4];
        rec(m, q[0], q[1]);
        q[2] = leaf(2 * m - (1 << D));
        q[3] = leaf(2 * m + 1 - (1 << D));
        std::memcpy(tail + 16 * (m - (1 << (D - 1))), q, 16);
      }
    } else {
      for (int j = 0; j < (1 << D); ++j) {
        const uint32_t v = leaf(j);
        std::memcpy(tail + 4 * j, &v, 4);
      }
    }
  }
}

// The deep blocks serve the wide-row plans whose top levels come from LDS copies.
bool deep_wanted(const bridger_forest *h) {
  return deep_possible(h->vec, h->F, h->perfect_depth, h->n_trees);
}

// The most classes the trees of one lane group span when G groups split the kernel trees
// (class-sorted) into contiguous ranges.
int class_span(const bridger_forest *h, int G) {
  auto class_of = [&](int t) {
    return (int)(std::upper_bound(h->class_begin.begin(), h->class_begin.end(), t) -
                 h->class_begin.begin()) - 1;
  };
  int span = 1;
  for (int g = 0; g < G; ++g) {
    const int t0 = (int)((int64_t)h->n_trees * g / G), t1 = (int)((int64_t)h->n_trees * (g + 1) / G);
    if (t0 < t1) span = std::max(span, class_of(t1 - 1) - class_of(t0) + 1);
  }
  return span;
}

bool same_plan(const Plan &a, const Plan &b) {
  return a.waves == b.waves && a.rows_per_wg == b.rows_per_wg && a.groups == b.groups &&
         a.chunk_bytes == b.chunk_bytes && a.trees_per_chunk == b.trees_per_chunk &&
         a.n_chunks == b.n_chunks && a.lds_bytes == b.lds_bytes && a.ilp == b.ilp &&
         a.global_nodes == b.global_nodes && a.acc_alias == b.acc_alias && a.tops == b.tops &&
         a.top_group_bytes == b.top_group_bytes;
}

// PERFECT plans for the batch-size classes that differ from the large-batch plan `big`, each
// with a traversal copy for its row tile unless `big`'s serves (binned: bin copies).
void build_sized_plans(bridger_forest *h, PlanInput pin, const Plan &big, bool binned) {
  auto &sized = binned ? h->perfect_bsized : h->perfect_sized;
  auto &copies = binned ? h->perfect_bcopies : h->perfect_copies;
  sized.clear();
  copies.clear();
  if (env_int("BRIDGER_SIZED_PLANS", 1) == 0) return;
  for (const int64_t n : kSizeClasses) {
    pin.n_rows = n;
    const Plan p = pick_plan(pin);
    if (p.waves == 0 || same_plan(p, big)) continue;
    int copy = -1;
    if (p.rows_per_wg != big.rows_per_wg) {
      for (size_t i = 0; i < copies.size(); ++i)
        if (copies[i].R == p.rows_per_wg) copy = (int)i;
      if (copy < 0) {
        copies.emplace_back();
        copies.back().R = p.rows_per_wg;
        if (binned) make_perfect_btrav(h, p.rows_per_wg, copies.back().trav, copies.back().roots);
        else make_perfect_trav(h, p.rows_per_wg, copies.back().trav, copies.back().roots);
        copy = (int)copies.size() - 1;
      }
    }
    sized.push_back({n, p, copy});
  }
}

// RAGGED treelets (layout in internal.h) of every kernel tree, thresholds as bits or (binned)
// their ranks; false when a tree needs more than 2^27 slots in all (32-bit byte offsets).
bool make_treelets(const bridger_forest *h, const int64_t *offs, const int32_t *feat,
                   const float *thr, const int32_t *left, const int32_t *right,
                   const float *value, bool binned, std::vector<uint32_t> &blk,
                   std::vector<int32_t> &start, std::vector<int32_t> *leaf_ids) {
  start.assign((size_t)h->n_trees + 1, 0);
  int64_t total = 0;
  std::vector<std::pair<int32_t, int32_t>> stack;
  for (int32_t k = 0; k < h->n_trees; ++k) {
    const int32_t t = h->tree_order[k];
    const int64_t a = offs[t];
    int32_t depth = 0;  // the tree's largest leaf depth
    stack.assign(1, {0, 0});
    while (!stack.empty()) {
      const auto [nd, d] = stack.back();
      stack.pop_back();
      depth = std::max(depth, d);
      if (left[a + nd] != -1) {
        stack.push_back({left[a + nd], d + 1});
        stack.push_back({right[a + nd], d + 1});
      }
    }
    const int levels = depth / 2 + 1;  // treelet levels: nodes at tree levels 0, 2, ..., 2(levels-1)
    if (2 * levels > 26) return false;
    start[k] = (int32_t)total;
    total += ((int64_t(1) << (2 * levels)) - 1) / 3;
    if (total > (int64_t(1) << 27)) return false;
  }
  // the heaps are sparse (a ragged tree fills few of its deep slots): at most 8x the packed
  // records' bytes and 512 MB, else the record walk serves (1000 trees up to depth 12: 74 MB
  // against 11.3 MB)
  if (total * 16 > std::min<int64_t>(8 * 8 * (int64_t)h->ragged_rec.size() + (1 << 20),
                                     int64_t(512) << 20))
    return false;
  start[h->n_trees] = (int32_t)total;
  // an LDS copy reads up to 21 slots (treelet levels 0-2) from every tree's first slot, so the
  // last tree is followed by that many zero slots
  const int64_t pad = 21;
  blk.assign((size_t)(total + pad) * 4, 0u);
  if (leaf_ids) leaf_ids->assign((size_t)(total + pad) * 2, -1);
  auto w_of = [&](int64_t i) {
    float th = thr[i];
    if (th == 0.0f) th = 0.0f;
    uint32_t w;
    if (binned) w = rank_of(h, feat[i], th);
    else std::memcpy(&w, &th, 4);
    return w;
  };
  auto bits = [](float v) {
    uint32_t w;
    std::memcpy(&w, &v, 4);
    return w;
  };
  std::vector<std::pair<int64_t, int32_t>> todo;  // (slot, node)
  for (int32_t k = 0; k < h->n_trees; ++k) {
    const int32_t t = h->tree_order[k];
    const int64_t a = offs[t];
    todo.assign(1, {0, 0});
    while (!todo.empty()) {
      const auto [sl, nd] = todo.back();
      todo.pop_back();
      uint32_t *b = &blk[(size_t)(start[k] + sl) * 4];
      int32_t *lid = leaf_ids ? &(*leaf_ids)[(size_t)(start[k] + sl) * 2] : nullptr;
      if (left[a + nd] == -1) {
        b[0] = 0u;
        b[1] = b[2] = bits(value[a + nd]);
        b[3] = 3u << 30;
        if (lid) lid[0] = lid[1] = nd;
        continue;
      }
      const int32_t c[2] = {left[a + nd], right[a + nd]};
      b[0] = w_of(a + nd);
      b[3] = (uint32_t)feat[a + nd];
      for (int j = 0; j < 2; ++j) {
        const int64_t ci = a + c[j];
        if (left[ci] == -1) {
          b[1 + j] = bits(value[ci]);
          b[3] |= 1u << (30 + j);
          if (lid) lid[j] = c[j];
        } else {
          b[1 + j] = w_of(ci);
          b[3] |= (uint32_t)feat[ci] << (10 + 10 * j);
          todo.push_back({4 * sl + 1 + 2 * j, left[ci]});
          todo.push_back({4 * sl + 2 + 2 * j, right[ci]});
        }
      }
    }
  }
  return true;
}

bool treelets_wanted(const bridger_forest *h) {
  return env_int("BRIDGER_TREELETS", 1) != 0 && !h->vec && h->F <= kDeepMaxFeatures;
}

// RAGGED records for bins: an internal record's threshold becomes its rank.
void build_ragged_brec(bridger_forest *h) {
  h->ragged_brec = h->ragged_rec;
  for (uint64_t &rec : h->ragged_brec) {
    const uint32_t meta = (uint32_t)(rec >> 32);
    if (meta & (uint32_t)kLeafFlag) continue;
    float th;
    const uint32_t w = (uint32_t)rec;
    std::memcpy(&th, &w, 4);
    rec = (uint64_t)rank_of(h, (int32_t)(meta >> 16), th) | ((uint64_t)meta << 32);
  }
}

// Top-level heaps of the RAGGED trees (layout in internal.h): per kernel tree the records of its
// first L levels at heap slots 1 .. 2^L - 1 (copies of the packed records `rec`, found by
// following each internal record's left_rel), slot 0 the root's record index; slots under a
// leaf, and top_batch(L) trailing trees, hold a leaf record.
void build_ragged_tops(const std::vector<uint64_t> &rec, const std::vector<int32_t> &start,
                       int32_t n_trees, int L, std::vector<uint64_t> &tops) {
  const uint64_t leaf = (uint64_t)kLeafFlag << 32;
  const int slots = 1 << L;
  tops.assign((size_t)(n_trees + top_batch(L)) * slots, leaf);
  std::vector<int64_t> idx(slots);
  for (int32_t k = 0; k < n_trees; ++k) {
    uint64_t *t = &tops[(size_t)k * slots];
    t[0] = (uint64_t)(uint32_t)start[k];
    idx[1] = start[k];
    for (int m = 2; m < slots; ++m) idx[m] = -1;
    for (int m = 1; m < slots; ++m) {
      if (idx[m] < 0) continue;
      t[m] = rec[idx[m]];
      const uint32_t meta = (uint32_t)(rec[idx[m]] >> 32);
      if (2 * m + 1 < slots && !(meta & (uint32_t)kLeafFlag)) {
        idx[2 * m] = idx[m] + (meta & (uint32_t)kMaxRel);
        idx[2 * m + 1] = idx[2 * m] + 1;
      }
    }
  }
}

// ------------------------------------------------------------------- device io
// Test hook: with BRIDGER_TEST_ALLOC_LIMIT=<bytes> in the environment, every device allocation
// of the library larger than <bytes> fails as an exhausted device would (read at each
// allocation), so that the out-of-memory paths of create, set_preprocess and the Normalizer's
// scratch can be exercised.
bool alloc_refused(size_t bytes) {
  const char *v = std::getenv("BRIDGER_TEST_ALLOC_LIMIT");
  if (!v || !*v) return false;
  return bytes > (size_t)std::strtoull(v, nullptr, 10);
}

template <class T>
bridger_status upload(void **dst, const std::vector<T> &src, size_t pad = 0) {
  const size_t bytes = src.size() * sizeof(T);
  if (alloc_refused(bytes + pad + 16) || hipMalloc(dst, bytes + pad + 16) != hipSuccess) {
    *dst = nullptr;
    (void)hipGetLastError();
    return fail(BRIDGER_ERR_OUT_OF_MEMORY, "device allocation failed");
  }
  if (pad && hipMemset(*dst, 0, bytes + pad + 16) != hipSuccess)
    return fail(BRIDGER_ERR_DEVICE, "hipMemset failed");
  if (bytes && hipMemcpy(*dst, src.data(), bytes, hipMemcpyHostToDevice) != hipSuccess)
    return fail(BRIDGER_ERR_DEVICE, "hipMemcpy to device failed");
  return BRIDGER_OK;
}

void free_dev(void *&p) {
  if (p) (void)hipFree(p);
  p = nullptr;
}

void free_all(bridger_forest *h) {
  free_dev(h->d_class_begin);
  free_dev(h->d_class_count);
  free_dev(h->d_base);
  free_dev(h->d_tree_order);
  free_dev(h->d_perfect_trav);
  free_dev(h->d_perfect_roots);
  free_dev(h->d_perfect_broots);
  for (auto *cs : {&h->perfect_copies, &h->perfect_bcopies})
    for (auto &c : *cs) {
      free_dev(c.d_trav);
      free_dev(c.d_roots);
    }
  for (void **q : {&h->d_treelets, &h->d_btreelets, &h->d_treelet_start, &h->d_treelet_leaf,
                   &h->d_perfect_deep, &h->d_perfect_bdeep, &h->d_ragged_tops,
                   &h->d_ragged_btops, &h->d_q_values, &h->d_q_off,
                   &h->d_perfect_btrav, &h->d_ragged_brec,
                   &h->d_ragged_bchunk_first, &h->d_ragged_bchunk_rec, &h->d_pre_a, &h->d_pre_b,
                   &h->d_vec_perfect, &h->d_vec_ragged, &h->d_vec_direct})
    free_dev(*q);
  for (DevArrays *d : {&h->d_perfect, &h->d_ragged, &h->d_direct}) {
    free_dev(d->nodes);
    free_dev(d->tree_start);
    free_dev(d->chunk_first);
    free_dev(d->chunk_rec);
    free_dev(d->leaf_map);
  }
}

bridger_status upload_all(bridger_forest *h) {
  bridger_status s;
  if ((s = upload(&h->d_class_begin, h->class_begin)) != BRIDGER_OK) return s;
  if ((s = upload(&h->d_class_count, h->class_count)) != BRIDGER_OK) return s;
  if ((s = upload(&h->d_base, h->base)) != BRIDGER_OK) return s;
  if ((s = upload(&h->d_tree_order, h->tree_order)) != BRIDGER_OK) return s;
  if (h->perfect_ok) {
    if ((s = upload(&h->d_perfect.nodes, h->perfect_blob, 1024)) != BRIDGER_OK) return s;
    if ((s = upload(&h->d_perfect_trav, h->perfect_trav, 1024)) != BRIDGER_OK) return s;
    if ((s = upload(&h->d_perfect_roots, h->perfect_roots)) != BRIDGER_OK) return s;
    for (auto &c : h->perfect_copies) {
      if ((s = upload(&c.d_trav, c.trav, 1024)) != BRIDGER_OK) return s;
      if ((s = upload(&c.d_roots, c.roots)) != BRIDGER_OK) return s;
    }
    if ((s = upload(&h->d_perfect.leaf_map, h->perfect_leaf_map)) != BRIDGER_OK) return s;
    if (!h->perfect_deep.empty() &&
        (s = upload(&h->d_perfect_deep, h->perfect_deep, 1024)) != BRIDGER_OK)
      return s;
  }
  if (h->ragged_ok) {
    if ((s = upload(&h->d_ragged.nodes, h->ragged_rec, 1024)) != BRIDGER_OK) return s;
    if ((s = upload(&h->d_ragged.tree_start, h->ragged_tree_start)) != BRIDGER_OK) return s;
    if ((s = upload(&h->d_ragged.chunk_first, h->ragged_chunk_first)) != BRIDGER_OK) return s;
    if ((s = upload(&h->d_ragged.chunk_rec, h->ragged_chunk_rec)) != BRIDGER_OK) return s;
    if ((s = upload(&h->d_ragged.leaf_map, h->ragged_rec_node)) != BRIDGER_OK) return s;
    if (!h->ragged_tops.empty() && (s = upload(&h->d_ragged_tops, h->ragged_tops)) != BRIDGER_OK)
      return s;
    if (!h->treelets.empty()) {
      if ((s = upload(&h->d_treelets, h->treelets, 1024)) != BRIDGER_OK) return s;
      if ((s = upload(&h->d_treelet_start, h->treelet_start)) != BRIDGER_OK) return s;
      if ((s = upload(&h->d_treelet_leaf, h->treelet_leaf)) != BRIDGER_OK) return s;
    }
  }
  if (h->bin_bytes) {
    if ((s = upload(&h->d_q_values, h->q_values)) != BRIDGER_OK) return s;
    if ((s = upload(&h->d_q_off, h->q_off)) != BRIDGER_OK) return s;
  }
  if (h->perfect_bok) {
    if ((s = upload(&h->d_perfect_btrav, h->perfect_btrav, 1024)) != BRIDGER_OK) return s;
    if ((s = upload(&h->d_perfect_broots, h->perfect_broots)) != BRIDGER_OK) return s;
    for (auto &c : h->perfect_bcopies) {
      if ((s = upload(&c.d_trav, c.trav, 1024)) != BRIDGER_OK) return s;
      if ((s = upload(&c.d_roots, c.roots)) != BRIDGER_OK) return s;
    }
    if (!h->perfect_bdeep.empty() &&
        (s = upload(&h->d_perfect_bdeep, h->perfect_bdeep, 1024)) != BRIDGER_OK)
      return s;
  }
  if (h->ragged_bok) {
    if ((s = upload(&h->d_ragged_brec, h->ragged_brec, 1024)) != BRIDGER_OK) return s;
    if ((s = upload(&h->d_ragged_bchunk_first, h->ragged_bchunk_first)) != BRIDGER_OK) return s;
    if ((s = upload(&h->d_ragged_bchunk_rec, h->ragged_bchunk_rec)) != BRIDGER_OK) return s;
    if (!h->ragged_btops.empty() &&
        (s = upload(&h->d_ragged_btops, h->ragged_btops)) != BRIDGER_OK)
      return s;
    if (!h->btreelets.empty() && (s = upload(&h->d_btreelets, h->btreelets, 1024)) != BRIDGER_OK)
      return s;
  }
  if ((s = upload(&h->d_direct.nodes, h->direct_rec)) != BRIDGER_OK) return s;
  if ((s = upload(&h->d_direct.tree_start, h->direct_root)) != BRIDGER_OK) return s;
  if ((s = upload(&h->d_direct.leaf_map, h->direct_rec_node)) != BRIDGER_OK) return s;
  if (h->vec) {
    if (!h->vec_perfect.empty() && (s = upload(&h->d_vec_perfect, h->vec_perfect)) != BRIDGER_OK)
      return s;
    if (!h->vec_ragged.empty() && (s = upload(&h->d_vec_ragged, h->vec_ragged)) != BRIDGER_OK)
      return s;
    if ((s = upload(&h->d_vec_direct, h->vec_direct)) != BRIDGER_OK) return s;
  }
  return BRIDGER_OK;
}

// The Normalizer's row norms: n_rows doubles of stream-ordered scratch from the device's default
// memory pool, filled by the row-norm pass ahead of the fused kernel and handed back to the pool
// on the same stream when this object goes out of scope (after the kernel is enqueued).
struct RowNorms {
  double *p = nullptr;
  hipStream_t stream = nullptr;
  ~RowNorms() {
    if (p) (void)hipFreeAsync(p, stream);
  }
};

// `scratch` (the allocation-free entry point) replaces the pool allocation when given.
bridger_status prepare_row_norms(const bridger_forest *h, LaunchArgs &a, void *stream,
                                 RowNorms &rn, double *scratch = nullptr) {
  if (h->pre_kind != BRIDGER_PRE_NORMALIZE) return BRIDGER_OK;
  if (scratch) {
    const int err = launch_row_norm(a, scratch, stream);
    if (err != 0)
      return fail(BRIDGER_ERR_DEVICE, std::string("row-norm launch failed: ") +
                                          hipGetErrorString((hipError_t)err));
    a.row_norm = scratch;
    return BRIDGER_OK;
  }
  if (alloc_refused((size_t)a.n_rows * sizeof(double)) ||
      hipMallocAsync((void **)&rn.p, (size_t)a.n_rows * sizeof(double), (hipStream_t)stream) !=
          hipSuccess) {
    (void)hipGetLastError();
    rn.p = nullptr;
    return fail(BRIDGER_ERR_OUT_OF_MEMORY, "no stream-ordered scratch for the row norms");
  }
  rn.stream = (hipStream_t)stream;
  const int err = launch_row_norm(a, rn.p, stream);
  if (err != 0)
    return fail(BRIDGER_ERR_DEVICE, std::string("row-norm launch failed: ") +
                                        hipGetErrorString((hipError_t)err));
  a.row_norm = rn.p;
  return BRIDGER_OK;
}

void set_preprocess_args(const bridger_forest *h, LaunchArgs &a) {
  a.pre_kind = h->pre_kind;
  a.pre_a = (const double *)h->d_pre_a;
  a.pre_b = (const double *)h->d_pre_b;
}

bool gemm_ok(const bridger_forest *h) {
  return h->perfect_ok && h->perfect_depth >= 1 && h->perfect_depth <= kMaxGemmDepth &&
         h->K == 1 && h->F <= kMaxGemmFeatures;
}

int32_t resolve_auto(const bridger_forest *h) {
  if (h->perfect_ok) return kPerfect;
  if (h->ragged_ok) return kRagged;
  return kDirect;
}

bridger_status check_predict(const bridger_forest *h, const void *X, int64_t n_rows,
                             int32_t n_features, const void *out, int x_align = 4,
                             bool x_may_be_null = false) {
  if (!h) return fail(BRIDGER_ERR_INVALID_ARGUMENT, "null handle");
  if (h->host_only) return fail(BRIDGER_ERR_INVALID_ARGUMENT, "handle was created host-only");
  if (n_rows < 0) return fail(BRIDGER_ERR_INVALID_ARGUMENT, "n_rows < 0");
  if (n_features != h->F)
    return fail(BRIDGER_ERR_INVALID_ARGUMENT,
                "n_features " + std::to_string(n_features) + " != forest's " + std::to_string(h->F));
  if (n_rows == 0) return BRIDGER_OK;
  if ((!X && !x_may_be_null) || !out)
    return fail(BRIDGER_ERR_INVALID_ARGUMENT, "null X or output pointer");
  if (((uintptr_t)X % (uintptr_t)x_align) || ((uintptr_t)out & 3))
    return fail(BRIDGER_ERR_INVALID_ARGUMENT,
                "X must be aligned to its element size and the output to 4 bytes");
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev != h->device)
    return fail(BRIDGER_ERR_INVALID_ARGUMENT, "the handle's device is not current");
  if (n_rows > (int64_t)INT32_MAX * 64)
    return fail(BRIDGER_ERR_INVALID_ARGUMENT, "n_rows too large");
  return BRIDGER_OK;
}

// The PERFECT plan made for the smallest batch-size class holding n_rows, or null (the plan
// for large batches serves).
const bridger_forest::SizedPlan *sized_plan(const bridger_forest *h, int64_t n_rows,
                                            bool binned) {
  for (const auto &sp : binned ? h->perfect_bsized : h->perfect_sized)
    if (n_rows <= sp.max_rows) return &sp;
  return nullptr;
}

// X is fp32 rows, or (binned) rows of bin_bytes-wide bins from bridger_forest_bin.
struct CsrRows {
  const int64_t *indptr = nullptr;
  const int32_t *indices = nullptr;
};

// One launch (plus the Normalizer's row-norm pass) over n_rows rows; do_predict splits larger
// batches.
bridger_status launch_rows(bridger_forest *h, const void *X, int64_t n_rows, float *out,
                           int32_t *out_leaf, int32_t *out_label, const CsrRows *csr,
                           void *stream, bool binned, int xsz, double *norm_scratch) {
  bridger_status s = BRIDGER_OK;
  LaunchArgs a{};
  a.X = (const float *)X;
  a.n_rows = n_rows;
  a.F = h->F;
  a.x_bytes = xsz;
  a.x_vec4 = !csr && ((uintptr_t)X % 16 == 0) && (((int64_t)h->F * xsz) % 16 == 0);
  if (csr) {
    a.csr = 1;
    a.csr_indptr = csr->indptr;
    a.csr_indices = csr->indices;
  }
  a.out = out;
  a.out_leaf = out_leaf;
  a.out_label = out_label;
  a.class_begin = (const int32_t *)h->d_class_begin;
  a.class_count = (const int32_t *)h->d_class_count;
  a.base = (const float *)h->d_base;
  a.tree_order = (const int32_t *)h->d_tree_order;
  a.n_trees = h->n_trees;
  a.K = h->K;
  a.aggregate = h->aggregate;
  a.transform = h->transform;
  a.tile_coalesced = env_int("BRIDGER_COALESCED_TILE", 1) != 0 ? 1 : 0;
  RowNorms norms;
  if (!binned) {
    set_preprocess_args(h, a);
    if ((s = prepare_row_norms(h, a, stream, norms, norm_scratch)) != BRIDGER_OK) return s;
  }
  int err = 0;
  if (h->kernel_active == kPerfect || h->kernel_active == kRagged) {
    const bool perfect = h->kernel_active == kPerfect;
    const bridger_forest::SizedPlan *sp = perfect ? sized_plan(h, n_rows, binned) : nullptr;
    const Plan &p = sp ? sp->plan
                       : perfect ? (binned ? h->perfect_bplan : h->perfect_plan)
                                 : (binned ? h->ragged_bplan : h->ragged_plan);
    const DevArrays &d = perfect ? h->d_perfect : h->d_ragged;
    if (perfect)
      a.nodes = (const uint8_t *)(binned ? h->d_perfect_btrav : h->d_perfect_trav);
    else
      a.nodes = (const uint8_t *)(binned ? h->d_ragged_brec : d.nodes);
    a.finite_thresholds = h->finite_thresholds ? 1 : 0;
    a.roots = (const uint32_t *)(binned ? h->d_perfect_broots : h->d_perfect_roots);
    if (sp && sp->copy >= 0) {  // the small-batch plan's own row tile
      const auto &c = (binned ? h->perfect_bcopies : h->perfect_copies)[sp->copy];
      a.nodes = (const uint8_t *)c.d_trav;
      a.roots = (const uint32_t *)c.d_roots;
    }
    a.tree_start = (const int32_t *)d.tree_start;
    a.chunk_first = (const int32_t *)(binned && !perfect ? h->d_ragged_bchunk_first : d.chunk_first);
    a.chunk_rec = (const int32_t *)(binned && !perfect ? h->d_ragged_bchunk_rec : d.chunk_rec);
    a.leaf_map = (const int32_t *)d.leaf_map;
    a.vec = h->vec ? 1 : 0;
    a.leaf_vec = (const float *)(perfect ? h->d_vec_perfect : h->d_vec_ragged);
    a.tree_bytes = h->perfect_tree_bytes;
    a.trees_per_chunk = p.trees_per_chunk;
    a.n_chunks = p.n_chunks;
    a.rows_per_wg = p.rows_per_wg;
    a.log2_row_bytes = ilog2((int64_t)xsz * p.rows_per_wg);
    a.groups = p.groups;
    a.chunk_bytes = p.chunk_bytes;
    a.lds_x_off = p.global_nodes ? 0 : 2 * p.chunk_bytes;
    a.lds_acc_off = a.lds_x_off + h->F * p.rows_per_wg * xsz;
    a.acc_in_lds = p.acc_in_lds;
    if (p.acc_alias && !p.global_nodes) {  // class sums written into the tile after the walk
      a.acc_alias = 1;
      a.lds_acc_off = a.lds_x_off;
    }
    a.ilp = p.ilp;
    const int64_t n_wg = (n_rows + p.rows_per_wg - 1) / p.rows_per_wg;
    // (bins compare exactly whatever the thresholds; fp32 needs them finite)
    const bool fixed = h->kernel_active == kPerfect && !out_leaf && h->K == 1 && !h->vec &&
                       p.groups == 1 && p.waves <= 8 && (binned || h->finite_thresholds) &&
                       p.ilp == 4 &&
                       perfect_fixed_ok(h->perfect_depth, p.trees_per_chunk) &&
                       p.chunk_bytes == p.trees_per_chunk * h->perfect_tree_bytes &&
                       h->fixed_chunks;
    if (h->kernel_active == kPerfect && p.global_nodes) {
      if (p.tops) {  // after the row tile and the class sums
        a.top_levels = p.tops;
        a.top_group_bytes = p.top_group_bytes;
        a.lds_top_off = a.lds_acc_off + h->K * p.groups * p.rows_per_wg * 8;
        void *deep = binned ? h->d_perfect_bdeep : h->d_perfect_deep;
        if (deep && p.tops == h->deep_tl) {
          a.deep = (const uint8_t *)deep;
          a.deep_tree_bytes = deep_tree_bytes(h->perfect_depth, p.tops);
        }
        if (p.acc_alias) {  // class sums in registers, then into the row tile: no sum area
          if (!a.deep)
            return fail(BRIDGER_ERR_DEVICE, "plan without the deep blocks it was made for");
          a.acc_alias = 1;
          a.lds_acc_off = a.lds_x_off;
          a.lds_top_off = a.lds_x_off + h->F * p.rows_per_wg * xsz;
          a.class_span = class_span(h, p.groups);
        }
      }
      err = launch_perfect_global(h->perfect_depth, a, p.waves, n_wg, p.lds_bytes, stream);
    }
    else if (fixed)
      err = launch_perfect_fixed(h->perfect_depth, a, p.waves, n_wg, p.lds_bytes, stream);
    else if (h->kernel_active == kPerfect)
      err = launch_perfect(h->perfect_depth, a, p.waves, n_wg, p.lds_bytes, stream);
    else if (p.global_nodes && p.tops && (binned ? h->d_btreelets : h->d_treelets)) {
      a.nodes = (const uint8_t *)(binned ? h->d_btreelets : h->d_treelets);
      a.nodes_bytes = (uint32_t)(4 * (binned ? h->btreelets.size() : h->treelets.size()));
      a.tree_start = (const int32_t *)h->d_treelet_start;
      a.leaf_map = (const int32_t *)h->d_treelet_leaf;
      a.lds_top_off = h->F * p.rows_per_wg * xsz;
      // treelet levels from the LDS copy: 3 (three trees a batch; 4M x 256 rows 14.15 ms,
      // 1M x 28 rows 0.362 ms) or 2 (four trees: 14.22 and 0.374 ms)
      a.top_levels = env_int("BRIDGER_TREELET_LDS_LEVELS", 3) == 2 ? 2 : 3;
      err = launch_ragged_treelet(a, p.waves, n_wg, p.lds_bytes, stream);
    } else if (p.global_nodes && p.tops) {
      a.tops = (const uint64_t *)(binned ? h->d_ragged_btops : h->d_ragged_tops);
      a.nodes_bytes = (uint32_t)(8 * h->ragged_rec.size());
      a.top_levels = p.tops;
      a.lds_top_off = h->F * p.rows_per_wg * xsz;
      err = launch_ragged_top(a, p.waves, n_wg, p.lds_bytes, stream);
    } else if (p.global_nodes)
      err = launch_ragged_global(a, p.waves, n_wg, p.lds_bytes, stream);
    else
      err = launch_ragged(a, p.waves, n_wg, p.lds_bytes, stream);
  } else if (h->kernel_active == kGemm) {
    a.nodes = (const uint8_t *)h->d_perfect.nodes;
    a.leaf_map = (const int32_t *)h->d_perfect.leaf_map;
    a.tree_bytes = h->perfect_tree_bytes;
    const int64_t n_wg = (n_rows + 63) / 64;  // 4 waves x 16 rows
    err = launch_gemm(h->perfect_depth, a, n_wg, stream);
  } else {
    a.nodes = (const uint8_t *)h->d_direct.nodes;
    a.tree_start = (const int32_t *)h->d_direct.tree_start;
    a.leaf_map = (const int32_t *)h->d_direct.leaf_map;
    a.vec = h->vec ? 1 : 0;
    a.leaf_vec = (const float *)h->d_vec_direct;
    const int64_t n_wg = (n_rows + 255) / 256;
    err = launch_direct(a, n_wg, stream);
  }
  if (err != 0)
    return fail(BRIDGER_ERR_DEVICE, std::string("kernel launch failed: ") +
                                        hipGetErrorString((hipError_t)err));
  return BRIDGER_OK;
}

bridger_status do_predict(bridger_forest *h, const void *X, int64_t n_rows, int32_t n_features,
                          float *out, int32_t *out_leaf, void *stream, bool binned,
                          int32_t *out_label = nullptr, const CsrRows *csr = nullptr,
                          bool no_alloc = false) {
  g_last_error.clear();
  if (csr && h && !(h->kernel_active == kPerfect || h->kernel_active == kRagged))
    return fail(BRIDGER_ERR_UNSUPPORTED, "CSR rows run on the perfect and ragged kernels only");
  // CSR: indptr is always read; indices and values only inside the rows' ranges, so they may
  // be null when no entry is stored
  if (csr && n_rows > 0 && !csr->indptr)
    return fail(BRIDGER_ERR_INVALID_ARGUMENT, "null CSR indptr");
  if (out_label && h && h->K == 1 && h->transform != BRIDGER_XFORM_SIGMOID)
    return fail(BRIDGER_ERR_UNSUPPORTED,
                "labels need several classes or a sigmoid output (a classifier)");
  if (binned && h && !h->bin_bytes)
    return fail(BRIDGER_ERR_UNSUPPORTED, "a feature has 65536 or more distinct thresholds");
  const int xsz = binned && h ? h->bin_bytes : 4;
  void *dst = out ? (void *)out : (out_leaf ? (void *)out_leaf : (void *)out_label);
  bridger_status s = check_predict(h, X, n_rows, n_features, dst, xsz, csr != nullptr);
  if (s != BRIDGER_OK || n_rows == 0) return s;
  if (binned && !((h->kernel_active == kPerfect && h->perfect_bok) ||
                  (h->kernel_active == kRagged && h->ragged_bok)))
    return fail(BRIDGER_ERR_UNSUPPORTED,
                "binned prediction runs on the perfect and ragged kernels only");
  const uint8_t *xb = (const uint8_t *)X;
  const uint8_t *ob = (const uint8_t *)dst;
  const size_t xbytes = (size_t)n_rows * h->F * xsz;
  const size_t obytes = (size_t)n_rows * (out ? h->K : (out_leaf ? h->n_trees : 1)) * 4;
  if (!csr && xb < ob + obytes && ob < xb + xbytes)
    return fail(BRIDGER_ERR_INVALID_ARGUMENT, "output overlaps X");

  // The allocation-free entry point: the row norms go to the library's static scratch.
  double *norm_scratch = nullptr;
  if (no_alloc) {
    if (n_rows > kNoAllocMaxRows)
      return fail(BRIDGER_ERR_INVALID_ARGUMENT,
                  "n_rows " + std::to_string(n_rows) + " exceeds the allocation-free limit of " +
                      std::to_string(kNoAllocMaxRows) + " rows per call");
    if (h->pre_kind == BRIDGER_PRE_NORMALIZE) {
      const int err = noalloc_norm_scratch(&norm_scratch);
      if (err != 0)
        return fail(BRIDGER_ERR_DEVICE, std::string("scratch lookup failed: ") +
                                            hipGetErrorString((hipError_t)err));
    }
  }
  // A dispatch counts its work-items in 32 bits: larger batches go out as several launches of
  // at most kMaxRowsPerLaunch rows each (tile boundaries are unaffected: every tile size divides
  // it).  CSR rows keep absolute entry offsets, so only indptr moves.
  for (int64_t r0 = 0; r0 < n_rows; r0 += kMaxRowsPerLaunch) {
    const int64_t nr = std::min<int64_t>(kMaxRowsPerLaunch, n_rows - r0);
    CsrRows part;
    if (csr) part = {csr->indptr + r0, csr->indices};
    const void *xr = csr ? X : (const void *)((const uint8_t *)X + r0 * (int64_t)h->F * xsz);
    s = launch_rows(h, xr, nr, out ? out + r0 * h->K : nullptr,
                    out_leaf ? out_leaf + r0 * h->n_trees : nullptr,
                    out_label ? out_label + r0 : nullptr, csr ? &part : nullptr, stream, binned,
                    xsz, norm_scratch);
    if (s != BRIDGER_OK) return s;
  }
  return BRIDGER_OK;
}

}  // namespace

// ========================================================================== ABI
extern "C" {

const char *bridger_last_error(void) { return g_last_error.c_str(); }

bridger_status bridger_forest_create_ex(int32_t n_trees, const int64_t *tree_offsets,
                                        const int32_t *feature, const float *threshold,
                                        const int32_t *left, const int32_t *right,
                                        const float *value, int32_t n_features,
                                        int32_t n_classes, const int32_t *tree_class,
                                        int32_t aggregate, int32_t transform,
                                        const float *base_score, uint32_t flags,
                                        bridger_forest_t *out) {
  g_last_error.clear();
  if (!out) return fail(BRIDGER_ERR_INVALID_ARGUMENT, "null output handle pointer");
  *out = nullptr;
  if (n_trees < 1) return fail(BRIDGER_ERR_INVALID_ARGUMENT, "n_trees must be >= 1");
  if (!tree_offsets || !feature || !threshold || !left || !right || !value)
    return fail(BRIDGER_ERR_INVALID_ARGUMENT, "null forest array");
  if (n_features < 1) return fail(BRIDGER_ERR_INVALID_ARGUMENT, "n_features must be >= 1");
  if (n_classes < 1) return fail(BRIDGER_ERR_INVALID_ARGUMENT, "n_classes must be >= 1");
  if (n_classes > kMaxClasses)
    return fail(BRIDGER_ERR_UNSUPPORTED, "n_classes above " + std::to_string(kMaxClasses));
  if (aggregate != BRIDGER_AGG_SUM && aggregate != BRIDGER_AGG_MEAN)
    return fail(BRIDGER_ERR_INVALID_ARGUMENT, "unknown aggregate");
  if (transform < BRIDGER_XFORM_IDENTITY || transform > BRIDGER_XFORM_SOFTMAX)
    return fail(BRIDGER_ERR_INVALID_ARGUMENT, "unknown transform");
  if (transform == BRIDGER_XFORM_SIGMOID && n_classes != 1)
    return fail(BRIDGER_ERR_INVALID_ARGUMENT, "sigmoid needs n_classes == 1");
  if (transform == BRIDGER_XFORM_SOFTMAX && n_classes < 2)
    return fail(BRIDGER_ERR_INVALID_ARGUMENT, "softmax needs n_classes >= 2");
  if (flags & ~(uint32_t)(BRIDGER_CREATE_HOST_ONLY | BRIDGER_CREATE_VECTOR_LEAVES))
    return fail(BRIDGER_ERR_INVALID_ARGUMENT, "unknown flags");
  // one class: a vector leaf is a scalar leaf
  const bool vec = (flags & BRIDGER_CREATE_VECTOR_LEAVES) && n_classes > 1;
  if (vec && tree_class)
    return fail(BRIDGER_ERR_INVALID_ARGUMENT, "vector leaves take no tree_class");
  if (tree_offsets[0] != 0) return fail(BRIDGER_ERR_INVALID_FOREST, "tree_offsets[0] != 0");
  for (int32_t t = 0; t < n_trees; ++t)
    if (tree_offsets[t + 1] <= tree_offsets[t])
      return fail(BRIDGER_ERR_INVALID_FOREST, "tree " + std::to_string(t) + " has no nodes");
  if (tree_offsets[n_trees] > (int64_t)INT32_MAX / 4)
    return fail(BRIDGER_ERR_UNSUPPORTED, "too many nodes");
  std::vector<int32_t> klass(n_trees);
  for (int32_t t = 0; t < n_trees; ++t) {
    klass[t] = vec ? 0 : (tree_class ? tree_class[t] : t % n_classes);
    if (klass[t] < 0 || klass[t] >= n_classes)
      return fail(BRIDGER_ERR_INVALID_ARGUMENT, "tree_class out of range");
  }

  bridger_forest *h = new (std::nothrow) bridger_forest();
  if (!h) return fail(BRIDGER_ERR_OUT_OF_MEMORY, "host allocation failed");
  try {
    h->n_trees = n_trees;
    h->F = n_features;
    h->K = n_classes;
    h->aggregate = aggregate;
    h->transform = transform;
    h->n_nodes = tree_offsets[n_trees];
    h->host_only = (flags & BRIDGER_CREATE_HOST_ONLY) != 0;

    // validation and shape
    std::vector<int32_t> scratch;
    int32_t common_depth = -2;
    bool all_perfect = true;
    double visits = 0;
    for (int32_t t = 0; t < n_trees; ++t) {
      const int64_t a = tree_offsets[t], n = tree_offsets[t + 1] - a;
      TreeShape sh;
      bridger_status s = validate_tree(t, n, feature + a, threshold + a, left + a, right + a,
                                       n_features, scratch, sh);
      if (s != BRIDGER_OK) {
        delete h;
        return s;
      }
      h->max_depth = std::max(h->max_depth, sh.depth);
      if (!sh.perfect) all_perfect = false;
      if (common_depth == -2) common_depth = sh.depth;
      else if (common_depth != sh.depth) all_perfect = false;
      visits += sh.perfect ? sh.depth : sh.mean_path;
    }
    h->visits_per_row_est = visits;
    h->finite_thresholds = env_int("BRIDGER_NO_SIGN_STEP", 0) == 0;
    h->fixed_chunks = env_int("BRIDGER_NO_FIXED", 0) == 0;
    for (int64_t i = 0; i < h->n_nodes && h->finite_thresholds; ++i)
      if (left[i] != -1 && !std::isfinite(threshold[i])) h->finite_thresholds = false;
    h->all_perfect = all_perfect ? 1 : 0;
    h->perfect_depth = all_perfect ? common_depth : -1;

    // class-major stable tree order (vector leaves: caller order, every tree in every class)
    h->vec = vec;
    h->class_count.assign(n_classes, 0);
    for (int32_t t = 0; t < n_trees; ++t) h->class_count[klass[t]]++;
    if (vec) h->class_count.assign(n_classes, n_trees);
    if (aggregate == BRIDGER_AGG_MEAN)
      for (int32_t k = 0; k < n_classes; ++k)
        if (h->class_count[k] == 0) {
          delete h;
          return fail(BRIDGER_ERR_INVALID_ARGUMENT,
                      "mean needs at least one tree in class " + std::to_string(k));
        }
    h->class_begin.assign(n_classes + 1, 0);
    for (int32_t k = 0; k < n_classes; ++k)
      h->class_begin[k + 1] = h->class_begin[k] + (vec ? (k == 0 ? n_trees : 0) : h->class_count[k]);
    h->tree_order.resize(n_trees);
    {
      std::vector<int32_t> fill(h->class_begin.begin(), h->class_begin.end() - 1);
      for (int32_t t = 0; t < n_trees; ++t) h->tree_order[fill[klass[t]]++] = t;
    }
    h->base.assign(n_classes, 0.0f);
    if (base_score)
      for (int32_t k = 0; k < n_classes; ++k) h->base[k] = base_score[k];

    // packing (vector leaves: the packers lay out class 0's values; the class vectors follow)
    std::vector<float> value0;
    const float *value_vec = value;
    if (vec) {
      value0.resize(h->n_nodes);
      for (int64_t i = 0; i < h->n_nodes; ++i) value0[i] = value[i * n_classes];
      value = value0.data();
    }
    pack_direct(h, tree_offsets, feature, threshold, left, right, value);
    const int D = h->perfect_depth;
    if (all_perfect && D >= 1 && D <= kMaxPerfectDepth) {
      pack_perfect(h, D, tree_offsets, feature, threshold, left, right, value);
      PlanInput pin{1 << 20, n_features, n_classes, n_trees,
                    (double)h->perfect_blob.size(), h->perfect_tree_bytes, true, visits};
      pin.vec = vec;
      pin.depth = D;
      pin.deep = deep_possible(vec, n_features, D, n_trees);
      h->perfect_plan = pick_plan(pin);
      h->perfect_ok = h->perfect_plan.waves > 0;
      if (h->perfect_ok) {
        build_perfect_trav(h);
        build_sized_plans(h, pin, h->perfect_plan, false);
        if (deep_wanted(h)) {
          h->deep_tl = perfect_top_levels(h->perfect_depth);
          make_perfect_deep(h, h->deep_tl, false, h->perfect_deep);
        }
      }
    }
    const bool ragged_packed = pack_ragged(h, tree_offsets, feature, threshold, left, right, value);
    if (ragged_packed) {
      PlanInput pin{1 << 20, n_features, n_classes, n_trees, 8.0 * h->ragged_rec.size(),
                    (int32_t)std::min<int64_t>(h->ragged_max_tree_bytes, INT32_MAX), false, visits};
      pin.vec = vec;
      h->ragged_plan = pick_plan(pin);
      h->ragged_ok = h->ragged_plan.waves > 0;
      if (h->ragged_ok && !h->ragged_plan.global_nodes)
        h->ragged_plan.n_chunks = ragged_chunks(h, h->ragged_plan.chunk_bytes,
                                                h->ragged_chunk_first, h->ragged_chunk_rec);
      if (h->ragged_ok && h->ragged_plan.tops) {
        build_ragged_tops(h->ragged_rec, h->ragged_tree_start, h->n_trees, h->ragged_plan.tops,
                          h->ragged_tops);
        if (treelets_wanted(h) &&
            !make_treelets(h, tree_offsets, feature, threshold, left, right, value, false,
                           h->treelets, h->treelet_start, &h->treelet_leaf))
          h->treelets.clear();
      }
    }
    // binned variants of the same layouts (used by bridger_forest_predict_binned)
    if (build_quantization(h, feature, threshold, left)) {
      if (h->perfect_ok) {
        PlanInput pin{1 << 20, n_features, n_classes, n_trees, (double)h->perfect_blob.size(),
                      h->perfect_tree_bytes, true, visits, h->bin_bytes};
        pin.vec = vec;
        pin.depth = D;
        pin.deep = deep_possible(vec, n_features, D, n_trees);
        h->perfect_bplan = pick_plan(pin);
        h->perfect_bok = h->perfect_bplan.waves > 0;
        if (h->perfect_bok) {
          build_perfect_btrav(h);
          build_sized_plans(h, pin, h->perfect_bplan, true);
          if (!h->perfect_deep.empty()) make_perfect_deep(h, h->deep_tl, true, h->perfect_bdeep);
        }
      }
      if (ragged_packed) {
        PlanInput pin{1 << 20, n_features, n_classes, n_trees, 8.0 * h->ragged_rec.size(),
                      (int32_t)std::min<int64_t>(h->ragged_max_tree_bytes, INT32_MAX), false,
                      visits, h->bin_bytes};
        pin.vec = vec;
        h->ragged_bplan = pick_plan(pin);
        h->ragged_bok = h->ragged_bplan.waves > 0;
        if (h->ragged_bok) {
          build_ragged_brec(h);
          if (h->ragged_bplan.tops) {
            build_ragged_tops(h->ragged_brec, h->ragged_tree_start, h->n_trees,
                              h->ragged_bplan.tops, h->ragged_btops);
            if (!h->treelets.empty() &&
                !make_treelets(h, tree_offsets, feature, threshold, left, right, value, true,
                               h->btreelets, h->treelet_start, nullptr))
              h->btreelets.clear();
          }
          if (!h->ragged_bplan.global_nodes)
            h->ragged_bplan.n_chunks = ragged_chunks(h, h->ragged_bplan.chunk_bytes,
                                                     h->ragged_bchunk_first, h->ragged_bchunk_rec);
        }
      }
    }
    if (vec) build_vector_leaves(h, tree_offsets, left, value_vec);
    if (env_int("BRIDGER_LOG", 0)) {
      auto show = [](const char *what, const Plan &p) {
        if (p.waves)
          std::fprintf(stderr,
                       "[bridger] %s plan: W=%d R=%d G=%d U=%d global=%d waves/CU=%d chunk=%d "
                       "ct=%d chunks=%d lds=%d\n",
                       what, p.waves, p.rows_per_wg, p.groups, p.ilp, p.global_nodes,
                       p.waves_per_cu, p.chunk_bytes, p.trees_per_chunk, p.n_chunks, p.lds_bytes);
      };
      show("perfect", h->perfect_plan);
      show("perfect binned", h->perfect_bplan);
      show("ragged", h->ragged_plan);
      show("ragged binned", h->ragged_bplan);
      for (const auto &sp : h->perfect_sized) {
        const std::string what = "perfect <= " + std::to_string(sp.max_rows) + " rows";
        show(what.c_str(), sp.plan);
      }
      for (const auto &sp : h->perfect_bsized) {
        const std::string what = "perfect binned <= " + std::to_string(sp.max_rows) + " rows";
        show(what.c_str(), sp.plan);
      }
    }
    h->kernel_active = resolve_auto(h);
    const int forced = env_int("BRIDGER_KERNEL", 0);
    if (forced == kPerfect && h->perfect_ok) h->kernel_active = kPerfect;
    if (forced == kRagged && h->ragged_ok) h->kernel_active = kRagged;
    if (forced == kDirect) h->kernel_active = kDirect;
    if (forced == kGemm && gemm_ok(h)) h->kernel_active = kGemm;

    if (!h->host_only) {
      int ndev = 0;
      if (hipGetDeviceCount(&ndev) != hipSuccess || ndev < 1) {
        (void)hipGetLastError();
        delete h;
        return fail(BRIDGER_ERR_DEVICE, "no HIP device available");
      }
      if (hipGetDevice(&h->device) != hipSuccess) {
        delete h;
        return fail(BRIDGER_ERR_DEVICE, "hipGetDevice failed");
      }
      bridger_status s = upload_all(h);
      if (s != BRIDGER_OK) {
        std::string msg = g_last_error;
        free_all(h);
        delete h;
        return fail(s, msg);
      }
    }
  } catch (const std::bad_alloc &) {
    free_all(h);
    delete h;
    return fail(BRIDGER_ERR_OUT_OF_MEMORY, "host allocation failed");
  }
  *out = h;
  return BRIDGER_OK;
}

bridger_status bridger_forest_create(int32_t n_trees, const int64_t *tree_offsets,
                                     const int32_t *feature, const float *threshold,
                                     const int32_t *left, const int32_t *right,
                                     const float *value, int32_t n_features, int32_t n_classes,
                                     const int32_t *tree_class, int32_t aggregate,
                                     int32_t transform, const float *base_score,
                                     bridger_forest_t *out) {
  return bridger_forest_create_ex(n_trees, tree_offsets, feature, threshold, left, right, value,
                                  n_features, n_classes, tree_class, aggregate, transform,
                                  base_score, 0u, out);
}

bridger_status bridger_forest_predict(bridger_forest_t h, const float *X, int64_t n_rows,
                                      int32_t n_features, float *out, void *stream) {
  return do_predict(h, X, n_rows, n_features, out, nullptr, stream, false);
}

bridger_status bridger_forest_predict_noalloc(bridger_forest_t h, const float *X, int64_t n_rows,
                                              int32_t n_features, float *out, void *stream) {
  if (n_rows > kNoAllocMaxRows) {  // before any other check: a size error is the first answer
    g_last_error.clear();
    return fail(BRIDGER_ERR_INVALID_ARGUMENT,
                "n_rows " + std::to_string(n_rows) + " exceeds the allocation-free limit of " +
                    std::to_string(kNoAllocMaxRows) + " rows per call");
  }
  return do_predict(h, X, n_rows, n_features, out, nullptr, stream, false, nullptr, nullptr,
                    true);
}

bridger_status bridger_forest_predict_leaves(bridger_forest_t h, const float *X, int64_t n_rows,
                                             int32_t n_features, int32_t *out_leaf,
                                             void *stream) {
  return do_predict(h, X, n_rows, n_features, nullptr, out_leaf, stream, false);
}

bridger_status bridger_forest_predict_csr(bridger_forest_t h, const int64_t *indptr,
                                          const int32_t *indices, const float *values,
                                          int64_t n_rows, int32_t n_features, float *out,
                                          void *stream) {
  CsrRows c{indptr, indices};
  return do_predict(h, values, n_rows, n_features, out, nullptr, stream, false, nullptr, &c);
}

bridger_status bridger_forest_predict_csr_leaves(bridger_forest_t h, const int64_t *indptr,
                                                 const int32_t *indices, const float *values,
                                                 int64_t n_rows, int32_t n_features,
                                                 int32_t *out_leaf, void *stream) {
  CsrRows c{indptr, indices};
  return do_predict(h, values, n_rows, n_features, nullptr, out_leaf, stream, false, nullptr, &c);
}

bridger_status bridger_forest_predict_labels(bridger_forest_t h, const float *X, int64_t n_rows,
                                             int32_t n_features, int32_t *labels, void *stream) {
  return do_predict(h, X, n_rows, n_features, nullptr, nullptr, stream, false, labels);
}

bridger_status bridger_forest_bin_info(bridger_forest_t h, int32_t *bin_bytes,
                                       int64_t *n_thresholds) {
  g_last_error.clear();
  if (!h) return fail(BRIDGER_ERR_INVALID_ARGUMENT, "null handle");
  if (bin_bytes) *bin_bytes = h->bin_bytes;
  if (n_thresholds) *n_thresholds = (int64_t)h->q_values.size();
  return BRIDGER_OK;
}

bridger_status bridger_forest_bin(bridger_forest_t h, const float *X, int64_t n_rows,
                                  int32_t n_features, void *Xq, void *stream) {
  g_last_error.clear();
  if (h && !h->bin_bytes)
    return fail(BRIDGER_ERR_UNSUPPORTED, "a feature has 65536 or more distinct thresholds");
  bridger_status s = check_predict(h, X, n_rows, n_features, Xq, 4);
  if (s != BRIDGER_OK || n_rows == 0) return s;
  if ((uintptr_t)Xq % (uintptr_t)h->bin_bytes)
    return fail(BRIDGER_ERR_INVALID_ARGUMENT, "Xq must be aligned to the bin size");
  const uint8_t *xb = (const uint8_t *)X, *qb = (const uint8_t *)Xq;
  const size_t xbytes = (size_t)n_rows * h->F * 4, qbytes = (size_t)n_rows * h->F * h->bin_bytes;
  if (xb < qb + qbytes && qb < xb + xbytes)
    return fail(BRIDGER_ERR_INVALID_ARGUMENT, "Xq overlaps X");
  for (int64_t r0 = 0; r0 < n_rows; r0 += kMaxRowsPerLaunch) {  // bounded dispatches
    const int64_t nr = std::min<int64_t>(kMaxRowsPerLaunch, n_rows - r0);
    LaunchArgs a{};
    a.X = X + r0 * (int64_t)h->F;
    a.n_rows = nr;
    a.F = h->F;
    a.x_bytes = h->bin_bytes;
    a.q_values = (const float *)h->d_q_values;
    a.q_off = (const int32_t *)h->d_q_off;
    a.xq = (uint8_t *)Xq + r0 * (int64_t)h->F * h->bin_bytes;
    a.x_vec4 = ((uintptr_t)a.X % 16 == 0) && (h->F % 4 == 0);
    a.rows_per_wg = env_int("BRIDGER_BIN_ROWS", 0);  // tuning overrides: stream kernel's rows
    a.trees_per_chunk = env_int("BRIDGER_BIN_CHUNKS", 0);  // and row kernel's 512-row chunks
    {  // tuning override of the LDS table buffer
      const int kb = env_int("BRIDGER_BIN_LDS_KB", 0);
      if (kb > 0) a.chunk_bytes = (int32_t)std::min<int64_t>((int64_t)kb * 1024, kLdsBytesPerCU);
    }
    // the largest number of LDS loads of tables (runs of whole tables within 64 KB, or the
    // override) any group of 32 features needs; it picks the binning kernel
    {
      const int cap = (a.chunk_bytes > 0 ? a.chunk_bytes : 65536) / 4;
      int max_runs = 0;
      for (int f0 = 0; f0 < h->F; f0 += 32) {
        const int f1 = std::min(h->F, f0 + 32);
        int runs = 0;
        for (int f = f0; f < f1;) {
          int fe = f;
          while (fe < f1 && h->q_off[fe + 1] - h->q_off[f] <= cap) ++fe;
          f = fe > f ? fe : f + 1;
          ++runs;
        }
        max_runs = std::max(max_runs, runs);
      }
      // the row kernel when the stream kernel's re-reads of the rows (one per run) would miss
      // the last-level cache: more than two runs and more row bytes than the cache holds
      const bool rows_kernel = max_runs > 2 && nr * (int64_t)h->F * 4 > kLastLevelCacheBytes;
      const int force = env_int("BRIDGER_BIN_KERNEL", 0);
      a.n_chunks = force == 1 ? std::max(max_runs, 3)
                   : force == 2 ? 1 : rows_kernel ? max_runs : 1;
    }
    set_preprocess_args(h, a);
    RowNorms norms;
    if ((s = prepare_row_norms(h, a, stream, norms)) != BRIDGER_OK) return s;
    const int err = launch_bin(a, stream);
    if (err != 0)
      return fail(BRIDGER_ERR_DEVICE, std::string("kernel launch failed: ") +
                                          hipGetErrorString((hipError_t)err));
  }
  return BRIDGER_OK;
}

bridger_status bridger_forest_predict_binned(bridger_forest_t h, const void *Xq, int64_t n_rows,
                                             int32_t n_features, float *out, void *stream) {
  return do_predict(h, Xq, n_rows, n_features, out, nullptr, stream, true);
}

bridger_status bridger_forest_predict_binned_leaves(bridger_forest_t h, const void *Xq,
                                                    int64_t n_rows, int32_t n_features,
                                                    int32_t *out_leaf, void *stream) {
  return do_predict(h, Xq, n_rows, n_features, nullptr, out_leaf, stream, true);
}

bridger_status bridger_forest_set_preprocess(bridger_forest_t h, int32_t kind, const double *pa,
                                             const double *pb) {
  g_last_error.clear();
  if (!h) return fail(BRIDGER_ERR_INVALID_ARGUMENT, "null handle");
  if (kind < BRIDGER_PRE_NONE || kind > BRIDGER_PRE_NORMALIZE)
    return fail(BRIDGER_ERR_INVALID_ARGUMENT, "unknown preprocessing kind");
  const bool params = kind != BRIDGER_PRE_NONE && kind != BRIDGER_PRE_NORMALIZE;
  if (params && !pa) return fail(BRIDGER_ERR_INVALID_ARGUMENT, "null parameter array a");
  if ((kind == BRIDGER_PRE_MINMAX || kind == BRIDGER_PRE_CENTER_SCALE) && !pb)
    return fail(BRIDGER_ERR_INVALID_ARGUMENT, "null parameter array b");
  std::vector<double> va, vb;
  if (params) {
    va.assign(pa, pa + h->F);
    vb = pb ? std::vector<double>(pb, pb + h->F) : std::vector<double>(h->F, 0.0);
  }
  if (!h->host_only && params) {
    if (!h->d_pre_a) {
      bridger_status s = upload(&h->d_pre_a, va);
      if (s != BRIDGER_OK) return s;
      if ((s = upload(&h->d_pre_b, vb)) != BRIDGER_OK) {
        free_dev(h->d_pre_a);  // both or neither: a later call uploads both again
        return s;
      }
    } else if (hipMemcpy(h->d_pre_a, va.data(), 8 * va.size(), hipMemcpyHostToDevice) !=
                   hipSuccess ||
               hipMemcpy(h->d_pre_b, vb.data(), 8 * vb.size(), hipMemcpyHostToDevice) !=
                   hipSuccess) {
      return fail(BRIDGER_ERR_DEVICE, "hipMemcpy to device failed");
    }
  }
  h->pre_kind = kind;
  h->pre_a = std::move(va);
  h->pre_b = std::move(vb);
  return BRIDGER_OK;
}

bridger_status bridger_forest_info(bridger_forest_t h, int32_t *n_trees, int32_t *n_features,
                                   int32_t *n_outputs, int32_t *max_depth, int32_t *all_perfect) {
  g_last_error.clear();
  if (!h) return fail(BRIDGER_ERR_INVALID_ARGUMENT, "null handle");
  if (n_trees) *n_trees = h->n_trees;
  if (n_features) *n_features = h->F;
  if (n_outputs) *n_outputs = h->K;
  if (max_depth) *max_depth = h->max_depth;
  if (all_perfect) *all_perfect = h->all_perfect;
  return BRIDGER_OK;
}

bridger_status bridger_forest_set_kernel(bridger_forest_t h, int32_t kernel) {
  g_last_error.clear();
  if (!h) return fail(BRIDGER_ERR_INVALID_ARGUMENT, "null handle");
  switch (kernel) {
    case BRIDGER_KERNEL_AUTO: h->kernel_active = resolve_auto(h); return BRIDGER_OK;
    case BRIDGER_KERNEL_PERFECT:
      if (!h->perfect_ok)
        return fail(BRIDGER_ERR_UNSUPPORTED, "forest is not all perfect trees of one depth 1..10");
      h->kernel_active = kPerfect;
      return BRIDGER_OK;
    case BRIDGER_KERNEL_RAGGED:
      if (!h->ragged_ok)
        return fail(BRIDGER_ERR_UNSUPPORTED, "a tree does not fit the LDS-chunked layout");
      h->kernel_active = kRagged;
      return BRIDGER_OK;
    case BRIDGER_KERNEL_DIRECT: h->kernel_active = kDirect; return BRIDGER_OK;
    case BRIDGER_KERNEL_GEMM:
      if (!gemm_ok(h))
        return fail(BRIDGER_ERR_UNSUPPORTED,
                    "the matrix lowering needs perfect trees of depth 1..4, one class and at "
                    "most 64 features");
      h->kernel_active = kGemm;
      return BRIDGER_OK;
    default: return fail(BRIDGER_ERR_INVALID_ARGUMENT, "unknown kernel");
  }
}

bridger_status bridger_forest_get_kernel(bridger_forest_t h, int32_t *kernel) {
  g_last_error.clear();
  if (!h || !kernel) return fail(BRIDGER_ERR_INVALID_ARGUMENT, "null argument");
  *kernel = h->kernel_active;
  return BRIDGER_OK;
}

bridger_status bridger_forest_plan(bridger_forest_t h, int64_t n_rows, int32_t *rows_per_wg,
                                   int32_t *chunk_bytes, int32_t *trees_per_chunk,
                                   int32_t *n_chunks, int32_t *lds_bytes, double *hbm_bytes,
                                   double *stage_bytes, double *lds_read_bytes) {
  g_last_error.clear();
  if (!h) return fail(BRIDGER_ERR_INVALID_ARGUMENT, "null handle");
  if (n_rows < 0) return fail(BRIDGER_ERR_INVALID_ARGUMENT, "n_rows < 0");
  Plan p{};
  double forest_bytes = 0;
  if (h->kernel_active == kPerfect) {
    const bridger_forest::SizedPlan *sp = sized_plan(h, n_rows, false);
    p = sp ? sp->plan : h->perfect_plan;
    forest_bytes = (double)h->perfect_blob.size();
  } else if (h->kernel_active == kRagged) {
    p = h->ragged_plan;
    forest_bytes = 8.0 * h->ragged_rec.size();
  } else if (h->kernel_active == kGemm) {
    p.rows_per_wg = 64;
    p.waves = 4;
    forest_bytes = (double)h->perfect_blob.size();
  } else {
    p.rows_per_wg = 256;
    p.waves = 4;
    forest_bytes = 16.0 * h->n_nodes;
  }
  const double n = (double)n_rows;
  const double n_wg = std::ceil(n / std::max(p.rows_per_wg, 1));
  if (rows_per_wg) *rows_per_wg = p.rows_per_wg;
  if (chunk_bytes) *chunk_bytes = p.chunk_bytes;
  if (trees_per_chunk) *trees_per_chunk = p.trees_per_chunk;
  if (n_chunks) *n_chunks = p.n_chunks;
  if (lds_bytes) *lds_bytes = p.lds_bytes;
  if (hbm_bytes) *hbm_bytes = n * h->F * 4 + n * h->K * 4 + forest_bytes;
  const bool no_lds = h->kernel_active == kDirect || h->kernel_active == kGemm;
  const bool no_chunks = no_lds || p.global_nodes;
  if (stage_bytes) *stage_bytes = no_lds ? 0.0 : (no_chunks ? 0.0 : n_wg * forest_bytes) + n * h->F * 4;
  if (lds_read_bytes)
    *lds_read_bytes = no_lds
                          ? 0.0
                          : 256.0 * (n / 64.0 * (2.0 * h->visits_per_row_est + h->n_trees) +
                                     n_wg * forest_bytes / 1024.0);
  return BRIDGER_OK;
}

bridger_status bridger_forest_packed(bridger_forest_t h, int32_t which, const void **ptr,
                                     int64_t *bytes) {
  g_last_error.clear();
  if (!h || !ptr || !bytes) return fail(BRIDGER_ERR_INVALID_ARGUMENT, "null argument");
  *ptr = nullptr;
  *bytes = 0;
  auto give = [&](const void *p, size_t b) {
    *ptr = p;
    *bytes = (int64_t)b;
    return BRIDGER_OK;
  };
  if (which == 3) return give(h->tree_order.data(), h->tree_order.size() * 4);
  if (which == 5) return give(h->q_values.data(), h->q_values.size() * 4);
  if (which == 6) return give(h->q_off.data(), h->q_off.size() * 4);
  switch (h->kernel_active) {
    case kPerfect:
    case kGemm:
      if (which == 0) return give(h->perfect_blob.data(), h->perfect_blob.size());
      if (which == 2) return give(h->perfect_leaf_map.data(), h->perfect_leaf_map.size() * 4);
      if (which == 8 && !h->perfect_deep.empty())
        return give(h->perfect_deep.data(), h->perfect_deep.size());
      if (which == 9 && !h->perfect_bdeep.empty())
        return give(h->perfect_bdeep.data(), h->perfect_bdeep.size());
      break;
    case kRagged:
      if (which == 0) return give(h->ragged_rec.data(), h->ragged_rec.size() * 8);
      if (which == 1) return give(h->ragged_tree_start.data(), h->ragged_tree_start.size() * 4);
      if (which == 2) return give(h->ragged_rec_node.data(), h->ragged_rec_node.size() * 4);
      if (which == 4) return give(h->ragged_chunk_first.data(), h->ragged_chunk_first.size() * 4);
      if (which == 10 && !h->treelets.empty())
        return give(h->treelets.data(), h->treelets.size() * 4);
      if (which == 11 && !h->treelet_start.empty())
        return give(h->treelet_start.data(), h->treelet_start.size() * 4);
      if (which == 12 && !h->treelet_leaf.empty())
        return give(h->treelet_leaf.data(), h->treelet_leaf.size() * 4);
      if (which == 13 && !h->btreelets.empty())
        return give(h->btreelets.data(), h->btreelets.size() * 4);
      if (which == 7 && !h->ragged_tops.empty())
        return give(h->ragged_tops.data(), h->ragged_tops.size() * 8);
      break;
    default:
      if (which == 0) return give(h->direct_rec.data(), h->direct_rec.size() * 4);
      if (which == 1) return give(h->direct_root.data(), h->direct_root.size() * 4);
      if (which == 2) return give(h->direct_rec_node.data(), h->direct_rec_node.size() * 4);
      break;
  }
  return fail(BRIDGER_ERR_INVALID_ARGUMENT, "no such packed array for the active kernel");
}

void bridger_forest_destroy(bridger_forest_t h) {
  if (!h) return;
  if (!h->host_only) free_all(h);
  delete h;
}

}  // extern "C"
