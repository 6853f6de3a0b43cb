/*
 * bridger.h -- C ABI of the MI355X tree-ensemble prediction library.
 *
 * The library evaluates classical-ML tree ensembles (a single decision tree, a
 * random forest, gradient-boosted trees; binary or multiclass) over a batch of
 * rows.  In the paper's terms a tree model is a combination of comparison,
 * conditional, assignment and aggregation operators (Sec. 4.2, the classical
 * operator representation) lowered to the primitive operators of Table 4:
 * gather/take (feature and node reads), less_equal (threshold compare),
 * where / if_then_else (child choice), loop/while (descent), sum/mean
 * (aggregation over trees) and exp/add/divide/max (link functions).  The frontend
 * hands over a trained model's arrays (Sec. 4.1: the frontend converts models,
 * the runtime reads the executable and the input data); here that is
 * bridger_forest_create, and the runtime call is bridger_forest_predict.
 *
 * Semantics (the paper fixes no comparison, tie or NaN rule; these are the
 * library's conventions):
 *   - each tree starts at its tree-local node 0; a node is a leaf iff
 *     left == right == -1;
 *   - a row goes to the left child iff x[feature] <= threshold (ties go left);
 *     comparisons are IEEE: a NaN feature value goes right, -0.0 == +0.0,
 *     -inf goes left of every finite threshold and +inf goes right;
 *   - tree t adds its leaf value to class tree_class[t] (or t mod n_classes);
 *     per class the sum runs in ascending tree order, accumulated in double
 *     precision; SUM starts from base_score[k]; MEAN is
 *     base_score[k] + sum / (number of trees of class k);
 *   - the transform is applied to the n_classes class values: identity,
 *     sigmoid (n_classes == 1) or softmax (n_classes >= 2); results are
 *     rounded once to float.
 *
 * Threading: calls on different handles are independent.  One handle may serve
 * concurrent predict calls on different streams.  bridger_forest_set_kernel and
 * bridger_forest_destroy must not overlap other calls on the same handle.
 * Errors are reported through the return value; bridger_last_error() gives a
 * message for the calling thread's most recent failure.  Nothing throws across
 * this interface.
 */
#ifndef BRIDGER_H
#define BRIDGER_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct bridger_forest *bridger_forest_t; /* opaque; immutable after create */

typedef enum {
  BRIDGER_OK = 0,
  BRIDGER_ERR_INVALID_ARGUMENT = 1, /* bad pointer, size, shape, or handle/device mismatch */
  BRIDGER_ERR_INVALID_FOREST = 2,   /* the arrays do not describe a valid forest          */
  BRIDGER_ERR_UNSUPPORTED = 3,      /* valid, but the requested kernel cannot run it     */
  BRIDGER_ERR_OUT_OF_MEMORY = 4,    /* host or device allocation failed                  */
  BRIDGER_ERR_DEVICE = 5            /* no usable GPU, or a HIP call / launch failed      */
} bridger_status;

enum { BRIDGER_AGG_SUM = 0, BRIDGER_AGG_MEAN = 1 };
enum { BRIDGER_XFORM_IDENTITY = 0, BRIDGER_XFORM_SIGMOID = 1, BRIDGER_XFORM_SOFTMAX = 2 };

/* Kernel families.  AUTO picks PERFECT when every tree is a perfect binary tree of
 * one common depth (1..10), else RAGGED when every tree fits an LDS chunk, else
 * DIRECT.  PERFECT and RAGGED stage the trees through LDS (the data-movement
 * model of Eq. 1 sizes the row tile and the tree chunks); DIRECT reads nodes
 * from global memory and handles any forest.  GEMM is the matrix-multiply
 * lowering (Table 4's matmul and one_hot on the matrix cores) for perfect trees
 * of depth 1..4 with one output class and at most 64 features; it is never
 * chosen by AUTO and exists to be measured against the traversal kernels. */
enum {
  BRIDGER_KERNEL_AUTO = 0,
  BRIDGER_KERNEL_PERFECT = 1,
  BRIDGER_KERNEL_RAGGED = 2,
  BRIDGER_KERNEL_DIRECT = 3,
  BRIDGER_KERNEL_GEMM = 4
};

/* Flags for bridger_forest_create_ex. */
enum {
  /* Validate and pack on the host only; no device is touched.  Predict calls on
   * such a handle fail with BRIDGER_ERR_INVALID_ARGUMENT.  Used to inspect the
   * packed layout and the launch plan on a machine without a GPU. */
  BRIDGER_CREATE_HOST_ONLY = 1u,
  /* Vector leaves (tree classifiers: decision, extra and random forests of
   * classification trees, whose leaves hold class probabilities; the aggregation
   * category of the classical operator representation, Sec. 3.2 and Sec. 4.2, lowered
   * to Table 4's sum/mean): `value` holds n_classes floats per node, row-major
   * [N, n_classes] (ignored at internal nodes), and every tree adds its leaf's
   * vector to all n_classes outputs, in ascending tree order per class.  MEAN
   * divides each class sum by n_trees (a random forest's averaged probabilities).
   * tree_class must be NULL; the transform is IDENTITY or SOFTMAX.  Labels
   * (predict_labels) are the class of largest averaged value.  Runs on the
   * PERFECT, RAGGED and DIRECT kernels (GEMM: BRIDGER_ERR_UNSUPPORTED). */
  BRIDGER_CREATE_VECTOR_LEAVES = 2u
};

/*
 * Build a forest handle from per-node arrays (all host pointers; every array is
 * copied, so the caller may free them as soon as the call returns).
 *   n_trees        >= 1
 *   tree_offsets   [n_trees + 1] int64; tree t owns nodes [tree_offsets[t],
 *                  tree_offsets[t+1]); tree_offsets[0] == 0; every tree has >= 1 node
 *   feature        [N] int32 split feature, 0 <= f < n_features (ignored at leaves)
 *   threshold      [N] float split threshold, not NaN (ignored at leaves)
 *   left, right    [N] int32 tree-local child ids, or -1 and -1 for a leaf
 *   value          [N] float leaf value (ignored at internal nodes)
 *   n_features     >= 1, the row width every predict call must use
 *   n_classes      K, 1 <= K <= 64, the output width
 *   tree_class     [n_trees] int32 in [0, K), or NULL for t mod K
 *   aggregate      BRIDGER_AGG_SUM or BRIDGER_AGG_MEAN (MEAN needs >= 1 tree per class)
 *   transform      BRIDGER_XFORM_*; SIGMOID needs K == 1, SOFTMAX needs K >= 2
 *   base_score     [K] float, or NULL for zeros
 *   out            receives the handle (set to NULL on failure)
 * Validation: every non-root node is the child of exactly one node and every
 * node is reachable from node 0 (each tree is a tree), depth <= 64.
 * Returns BRIDGER_ERR_INVALID_FOREST / _INVALID_ARGUMENT on bad input,
 * BRIDGER_ERR_DEVICE when no GPU is usable, BRIDGER_ERR_OUT_OF_MEMORY.
 * The packed forest is uploaded synchronously to the device current at the call.
 */
bridger_status bridger_forest_create(int32_t n_trees, const int64_t *tree_offsets,
                                     const int32_t *feature, const float *threshold,
                                     const int32_t *left, const int32_t *right,
                                     const float *value, int32_t n_features, int32_t n_classes,
                                     const int32_t *tree_class, int32_t aggregate,
                                     int32_t transform, const float *base_score,
                                     bridger_forest_t *out);

/* As bridger_forest_create, with BRIDGER_CREATE_* flags. */
bridger_status bridger_forest_create_ex(int32_t n_trees, const int64_t *tree_offsets,
                                        const int32_t *feature, const float *threshold,
                                        const int32_t *left, const int32_t *right,
                                        const float *value, int32_t n_features,
                                        int32_t n_classes, const int32_t *tree_class,
                                        int32_t aggregate, int32_t transform,
                                        const float *base_score, uint32_t flags,
                                        bridger_forest_t *out);

/*
 * Predict n_rows rows.
 *   X       device pointer, row-major float [n_rows, n_features], 4-byte aligned;
 *           read only
 *   out     device pointer, row-major float [n_rows, n_classes]; must not overlap X
 *   stream  a hipStream_t (NULL = the null stream); the call is asynchronous on it
 * n_features must equal the value given at create; n_rows == 0 launches nothing;
 * n_rows up to 2^37 (more than 2^24 rows go out as several launches on the same
 * stream, each over at most 2^24 rows).
 * Must be called with the handle's device current.  Launch failures return
 * BRIDGER_ERR_DEVICE; faults during execution surface at the caller's sync.
 */
bridger_status bridger_forest_predict(bridger_forest_t h, const float *X, int64_t n_rows,
                                      int32_t n_features, float *out, void *stream);

/*
 * Allocation-free predict, for callers that cannot allocate device memory (code under
 * HIP graph capture, tight serving loops, harnesses that forbid hipMalloc).  Same arguments,
 * outputs, rules and errors as bridger_forest_predict, except that:
 *   - n_rows must be at most BRIDGER_NOALLOC_MAX_ROWS (BRIDGER_ERR_INVALID_ARGUMENT beyond,
 *     checked first, before any other argument);
 *   - the call allocates nothing: the Normalizer's row norms (BRIDGER_PRE_NORMALIZE, the only
 *     scratch of a prediction) go to a fixed device array of the library, 16 MiB per GPU,
 *     held by every GPU the library runs on until the process ends.  Its address is looked
 *     up once per device, at the first call on that device.
 * Every allocation-free call on one GPU shares that GPU's array: calls that overlap on one
 * GPU (on other streams, or through other handles) race and must be serialized by the
 * caller, e.g. by issuing them on one stream.  Nothing in the array needs clearing: every
 * call writes its rows' norms before reading them.
 */
#define BRIDGER_NOALLOC_MAX_ROWS 2097152
bridger_status bridger_forest_predict_noalloc(bridger_forest_t h, const float *X, int64_t n_rows,
                                              int32_t n_features, float *out, void *stream);

/*
 * Write, for every (row, tree), the id of the leaf the row reaches, in the
 * caller's tree-local node numbering: device int32 [n_rows, n_trees], row-major
 * (tree index in the caller's order).  Same arguments and rules as predict.
 * This is the result of the comparison and conditional operators alone (Sec. 4.2;
 * Table 4's less_equal and where, iterated by loop/while), before the aggregation.
 */
bridger_status bridger_forest_predict_leaves(bridger_forest_t h, const float *X, int64_t n_rows,
                                             int32_t n_features, int32_t *out_leaf,
                                             void *stream);

/*
 * Exact feature quantization (the "data type rewriting" of Table 2).  For each
 * feature, the forest's distinct thresholds on it, ascending (-0 and +0 are one);
 * the bin of a value x is the number of them strictly below x, and a NaN gets
 * their count.  For a threshold t of rank k, x <= t exactly when bin(x) <= k, so
 * predicting on bins reaches the same leaves as predicting on the fp32 rows.
 *
 * bin_info: *bin_bytes = 1 when every feature has at most 255 distinct
 * thresholds, 2 when at most 65535, 0 when some feature has more (binning is then
 * unsupported); *n_thresholds = their total count.  Any pointer may be NULL;
 * works on host-only handles.
 */
bridger_status bridger_forest_bin_info(bridger_forest_t h, int32_t *bin_bytes,
                                       int64_t *n_thresholds);

/*
 * Bin n_rows fp32 rows.  X as for predict; Xq a device pointer to n_rows x
 * n_features elements of bin_bytes each (uint8 or uint16, row-major), aligned to
 * bin_bytes, not overlapping X.  Asynchronous on stream.  BRIDGER_ERR_UNSUPPORTED
 * when bin_bytes is 0.
 */
bridger_status bridger_forest_bin(bridger_forest_t h, const float *X, int64_t n_rows,
                                  int32_t n_features, void *Xq, void *stream);

/*
 * Predict (or write leaf ids) from binned rows Xq made by bridger_forest_bin for
 * this handle; same outputs, rules and errors as predict / predict_leaves.  The
 * feature tile then takes bin_bytes instead of 4 bytes per value.  Runs on the
 * perfect and ragged kernel families (BRIDGER_ERR_UNSUPPORTED otherwise).
 */
bridger_status bridger_forest_predict_binned(bridger_forest_t h, const void *Xq, int64_t n_rows,
                                             int32_t n_features, float *out, void *stream);
bridger_status bridger_forest_predict_binned_leaves(bridger_forest_t h, const void *Xq,
                                                    int64_t n_rows, int32_t n_features,
                                                    int32_t *out_leaf, void *stream);

/*
 * Preprocessing fused into prediction (the paper's cross-domain operator fusion,
 * Sec. 4.3, with the scalers of its CML suite): every feature value x of feature f
 * is transformed at the row load, before any compare, the forest's thresholds
 * applying to the transformed value x'.  Each step is done in double precision
 * and rounded to float, so the first three kinds match scikit-learn's transforms
 * of float32 data bit for bit:
 *   BRIDGER_PRE_MINMAX        x1 = float(x * a[f]);  x' = float(x1 + b[f])
 *                             (MinMaxScaler: a = scale_, b = min_)
 *   BRIDGER_PRE_CENTER_SCALE  x1 = float(x - a[f]);  x' = float(x1 / b[f])
 *                             (StandardScaler: a = mean_, b = scale_;
 *                              RobustScaler: a = center_, b = scale_)
 *   BRIDGER_PRE_BINARIZE      x' = (x > a[f]) ? 1 : 0   (Binarizer; NaN gives 0)
 *   BRIDGER_PRE_NORMALIZE     s = sum of double(x_f)^2 over the row, one add at a
 *                             time in feature order (CSR rows: in stored order);
 *                             n = sqrt(s), or 1 when s = 0; x' = float(x / n)
 *                             (Normalizer, unit L2 rows: within a few ulps of
 *                             scikit-learn's float32 arithmetic, and within half an
 *                             ulp of the exact x / ||x|| but for rounding ties;
 *                             a NaN makes the whole row NaN)
 *   BRIDGER_PRE_NONE          x' = x (b and a may be NULL)
 * a and b are host arrays of n_features doubles (b unused for BINARIZE, neither
 * for NORMALIZE: both may be NULL), copied at the call; the setting applies to
 * every later predict, predict_leaves, predict_csr, predict_labels and bin on the
 * handle.  Call it with no prediction in flight on the handle (synchronous
 * upload).  BRIDGER_ERR_INVALID_ARGUMENT on an unknown kind or a missing array.
 * NORMALIZE runs a row-norm pass before the fused kernel, with n_rows doubles of
 * scratch taken from the device's default stream-ordered memory pool and returned
 * to it on the same stream after the kernel (BRIDGER_ERR_OUT_OF_MEMORY if the pool
 * cannot supply them).
 */
#define BRIDGER_PRE_NONE 0
#define BRIDGER_PRE_MINMAX 1
#define BRIDGER_PRE_CENTER_SCALE 2
#define BRIDGER_PRE_BINARIZE 3
#define BRIDGER_PRE_NORMALIZE 4
bridger_status bridger_forest_set_preprocess(bridger_forest_t h, int32_t kind, const double *a,
                                             const double *b);

/*
 * Predict (or write leaf ids) from rows in compressed sparse row form (the
 * "sparse operator replacing" of Table 2): row i's stored values are
 * values[indptr[i] .. indptr[i+1]) at features indices[same range]; every feature
 * not stored reads 0.0 (then goes through the fused preprocessing like any value).
 * Device pointers: indptr int64 [n_rows + 1] (non-decreasing), indices int32 and
 * values float [indptr[n_rows]]; indices and values are read only inside the rows'
 * ranges and may be null when no entry is stored (a null indptr with n_rows > 0 is
 * BRIDGER_ERR_INVALID_ARGUMENT).  Indices within a row must be distinct (a repeated
 * index gives one of its values, unspecified which); indices outside
 * [0, n_features) are ignored.  Same outputs and rules as predict /
 * predict_leaves; runs on the perfect and ragged kernel families
 * (BRIDGER_ERR_UNSUPPORTED otherwise).
 */
bridger_status bridger_forest_predict_csr(bridger_forest_t h, const int64_t *indptr,
                                          const int32_t *indices, const float *values,
                                          int64_t n_rows, int32_t n_features, float *out,
                                          void *stream);
bridger_status bridger_forest_predict_csr_leaves(bridger_forest_t h, const int64_t *indptr,
                                                 const int32_t *indices, const float *values,
                                                 int64_t n_rows, int32_t n_features,
                                                 int32_t *out_leaf, void *stream);

/*
 * Classifier labels (int32 [n_rows], device; the index operators of Table 4, an
 * argmax over the class values): with several classes the class of largest value
 * (the first on ties), taken on the double-precision class values
 * before the link function (softmax keeps their order); with one output and a
 * sigmoid link, 1 when the value is above zero (probability above one half), else
 * 0.  BRIDGER_ERR_UNSUPPORTED for one output without a sigmoid (a regressor).
 * Other arguments and rules as predict.
 */
bridger_status bridger_forest_predict_labels(bridger_forest_t h, const float *X, int64_t n_rows,
                                             int32_t n_features, int32_t *labels, void *stream);

/* Shape facts of the converted model (what the frontend handed over, Sec. 4.1).
 * Any output pointer may be NULL.  all_perfect = 1 when every tree is perfect with
 * one common depth (then max_depth is that depth). */
bridger_status bridger_forest_info(bridger_forest_t h, int32_t *n_trees, int32_t *n_features,
                                   int32_t *n_outputs, int32_t *max_depth, int32_t *all_perfect);

/* Select the kernel family (BRIDGER_KERNEL_*): which generated code runs the lowered
 * operators (the code generation step of Sec. 4.5).  Returns BRIDGER_ERR_UNSUPPORTED
 * (and keeps the current choice) when that family cannot evaluate this forest. */
bridger_status bridger_forest_set_kernel(bridger_forest_t h, int32_t kernel);

/* The kernel family predict will use (AUTO resolved; Sec. 4.5's code generation). */
bridger_status bridger_forest_get_kernel(bridger_forest_t h, int32_t *kernel);

/*
 * The launch plan predict would use for n_rows rows (the Eq. 1 choice):
 * rows per workgroup, bytes of one LDS tree-chunk buffer, trees per chunk (0 when
 * chunks hold a varying number of trees), number of chunks, LDS bytes per
 * workgroup, and the modelled bytes moved per level (HBM, L2->LDS staging, LDS
 * reads).  Any output pointer may be NULL.  Works on host-only handles.
 */
bridger_status bridger_forest_plan(bridger_forest_t h, int64_t n_rows, int32_t *rows_per_wg,
                                   int32_t *chunk_bytes, int32_t *trees_per_chunk,
                                   int32_t *n_chunks, int32_t *lds_bytes, double *hbm_bytes,
                                   double *stage_bytes, double *lds_read_bytes);

/*
 * Read-only view of a host copy of the packed layout (the node records after Table 2's
 * data type rewriting and redundant operator elimination), for inspection and tests:
 * which = 0 node records of the active kernel family, 1 per-tree start offsets,
 * 2 leaf-id map (kernel leaf slot -> caller node id), 3 kernel tree order
 * (kernel position -> caller tree index), 4 chunk table, 5 the binning thresholds
 * (float, feature after feature, each ascending), 6 their per-feature offsets
 * (int32 [n_features + 1]), 7 the ragged trees' top-level heaps (2^L records per tree, L = 4
 * or 5 levels: the root's record index, then the records of the first L levels as a 1-based
 * heap; absent when the plan does not use them), 8 and 9 the perfect trees' deep blocks below
 * their first 3 (or 4) levels, with the thresholds' bits (8) or their ranks among the binning
 * thresholds (9): per kernel tree, levels taken in pairs, one 16-byte block {w(m), w(2m),
 * w(2m + 1), f(m) | f(2m) << 10 | f(2m + 1) << 20} per node m of a pair's upper level, then
 * either one block {w(m), f(m), leaf value of 2m, of 2m + 1} per node of the last level or
 * the 2^D leaf values (absent with vector leaves or more than 1024 features), 10 the ragged
 * trees' two-level treelets (16 bytes a slot: a 4-ary heap per tree, slot s holding a node of
 * an even level and its two children, {w(n), v(c0), v(c1), f(n) | f(c0) << 10 | f(c1) << 20 |
 * leaf(c0) << 30 | leaf(c1) << 31}, v the child's threshold or leaf value; the grandchild of
 * steps b1, b2 in slot 4s + 1 + 2 b1 + b2; a leaf n as {0, v(n), v(n), 3 << 30}), 11 each
 * kernel tree's first slot (int32 [n_trees + 1]), 12 the leaf id of each slot's two children
 * (int32 pairs), 13 the treelets with ranks in place of thresholds (absent when the plan does
 * not use them).  *ptr stays valid until destroy or set_kernel.
 */
bridger_status bridger_forest_packed(bridger_forest_t h, int32_t which, const void **ptr,
                                     int64_t *bytes);

/* Free the handle and its device memory (device-synchronizing): the end of the
 * runtime's hold on the converted model (Sec. 4.1).  NULL is a no-op. */
void bridger_forest_destroy(bridger_forest_t h);

/* Message for the calling thread's most recent failed call ("" if none).  The
 * paper states no error interface; this is the library's own, so that nothing
 * throws across the C ABI (thread-local storage, valid until the thread's next
 * call into the library). */
const char *bridger_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* BRIDGER_H */
