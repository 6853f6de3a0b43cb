/*
 * forest_oracle.c -- TEST INFRASTRUCTURE, not part of the library.
 *
 * A plain, slow, scalar CPU evaluation of a tree ensemble.  Only the test suite,
 * the smoke check and the benchmark's CPU-baseline leg use it.  It shares no code,
 * header, table or constant with the HIP library.
 *
 * What it computes (the method's own definition, written out):
 *   A classical-ML model is a combination of assignment, basic arithmetic,
 *   aggregation, comparison and conditional operators (Sec. 4.2, the classical
 *   operator representation), lowered to the primitive operators of Table 4:
 *   take/gather (read a node, read x[f]), less_equal (compare), where /
 *   if_then_else (pick a child), loop/while (descend), sum/mean (aggregate over
 *   trees) and exp/add/divide/max (link functions).  For every row r:
 *
 *     acc[k] = base[k]                      (SUM)   or 0 (MEAN)
 *     for t = 0 .. T-1 in ascending order:
 *         n = 0                              root = tree-local node 0
 *         while n is internal:               a node is a leaf iff left == right == -1
 *             n = (x[r, feature[n]] <= threshold[n]) ? left[n] : right[n]
 *         leaf[r, t] = n
 *         acc[class(t)] += value[n]
 *     z[k] = acc[k]                          (SUM)
 *     z[k] = base[k] + acc[k] / count[k]     (MEAN; count[k] = trees of class k)
 *     out  = z | sigmoid(z) | softmax(z)
 *
 * Readings where the paper is silent (each is a stated convention):
 *   - a row goes left iff x <= t; ties go left;
 *   - comparisons are IEEE: NaN compares false (goes right), -0.0 == +0.0,
 *     -inf goes left of every finite threshold, +inf goes right;
 *   - the tree-to-class map is tree_class[t], or t mod K when none is given;
 *   - accumulation is in double precision, strictly in ascending tree order;
 *   - sigmoid(z) = 1/(1+exp(-z)) for z >= 0 and exp(z)/(1+exp(z)) otherwise;
 *     softmax subtracts the max logit and sums exponentials in class order.
 * Inputs (x, thresholds, leaf values) are fp32 data; widening them to double is
 * exact, so the comparison decides exactly as an fp32 comparison would.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>

#define ORACLE_OK 0
#define ORACLE_BAD_TREE (-1)
#define ORACLE_BAD_ARG (-2)

/* Descend one tree for one row; returns the tree-local leaf id or ORACLE_BAD_TREE. */
static int64_t walk_tree(int64_t n_nodes, const int32_t *feature, const float *threshold,
                         const int32_t *left, const int32_t *right, const float *x,
                         int32_t n_features, int64_t *visits) {
  int64_t n = 0;
  int64_t steps = 0;
  if (n_nodes <= 0) return ORACLE_BAD_TREE;
  while (left[n] != -1 || right[n] != -1) {
    int32_t f = feature[n];
    if (f < 0 || f >= n_features) return ORACLE_BAD_TREE;
    double xv = (double)x[f];
    double tv = (double)threshold[n];
    int64_t next = (xv <= tv) ? (int64_t)left[n] : (int64_t)right[n];
    if (next < 0 || next >= n_nodes) return ORACLE_BAD_TREE;
    n = next;
    *visits += 1;
    if (++steps > n_nodes) return ORACLE_BAD_TREE; /* a cycle */
  }
  return n;
}

static double sigmoid(double z) {
  if (z >= 0.0) return 1.0 / (1.0 + exp(-z));
  double e = exp(z);
  return e / (1.0 + e);
}

/*
 * Evaluate rows [0, n_rows) of X (row-major, n_rows x n_features, fp32).
 *   out    : n_rows x n_classes doubles (required)
 *   leaves : n_rows x n_trees tree-local leaf ids (nullable)
 *   visits : total internal nodes visited (nullable)
 * Returns ORACLE_OK or a negative error code.
 */
int oracle_predict(int32_t n_trees, const int64_t *tree_offsets, const int32_t *feature,
                   const float *threshold, const int32_t *left, const int32_t *right,
                   const float *value, int32_t n_features, int32_t n_classes,
                   const int32_t *tree_class, int32_t aggregate, int32_t transform,
                   const float *base_score, const float *X, int64_t n_rows, double *out,
                   int32_t *leaves, int64_t *visits) {
  if (n_trees < 1 || n_classes < 1 || n_features < 1 || n_rows < 0 || !out) return ORACLE_BAD_ARG;
  if (aggregate != 0 && aggregate != 1) return ORACLE_BAD_ARG;
  if (transform < 0 || transform > 2) return ORACLE_BAD_ARG;
  double *acc = (double *)malloc(sizeof(double) * (size_t)n_classes);
  int64_t *count = (int64_t *)calloc((size_t)n_classes, sizeof(int64_t));
  if (!acc || !count) { free(acc); free(count); return ORACLE_BAD_ARG; }
  for (int32_t t = 0; t < n_trees; ++t) {
    int32_t k = tree_class ? tree_class[t] : t % n_classes;
    if (k < 0 || k >= n_classes) { free(acc); free(count); return ORACLE_BAD_ARG; }
    count[k] += 1;
  }
  int64_t nvis = 0;
  int rc = ORACLE_OK;
  for (int64_t r = 0; r < n_rows && rc == ORACLE_OK; ++r) {
    const float *x = X + r * (int64_t)n_features;
    for (int32_t k = 0; k < n_classes; ++k)
      acc[k] = (aggregate == 0 && base_score) ? (double)base_score[k] : 0.0;
    for (int32_t t = 0; t < n_trees; ++t) {
      int64_t a = tree_offsets[t];
      int64_t b = tree_offsets[t + 1];
      int64_t leaf = walk_tree(b - a, feature + a, threshold + a, left + a, right + a, x,
                               n_features, &nvis);
      if (leaf < 0) { rc = ORACLE_BAD_TREE; break; }
      if (leaves) leaves[r * (int64_t)n_trees + t] = (int32_t)leaf;
      int32_t k = tree_class ? tree_class[t] : t % n_classes;
      acc[k] = acc[k] + (double)value[a + leaf];
    }
    if (rc != ORACLE_OK) break;
    double *z = out + r * (int64_t)n_classes;
    for (int32_t k = 0; k < n_classes; ++k) {
      if (aggregate == 0) {
        z[k] = acc[k];
      } else {
        double base = base_score ? (double)base_score[k] : 0.0;
        z[k] = count[k] > 0 ? base + acc[k] / (double)count[k] : NAN;
      }
    }
    if (transform == 1) {
      for (int32_t k = 0; k < n_classes; ++k) z[k] = sigmoid(z[k]);
    } else if (transform == 2) {
      double m = z[0];
      for (int32_t k = 1; k < n_classes; ++k) if (z[k] > m) m = z[k];
      double s = 0.0;
      for (int32_t k = 0; k < n_classes; ++k) { z[k] = exp(z[k] - m); s += z[k]; }
      for (int32_t k = 0; k < n_classes; ++k) z[k] = z[k] / s;
    }
  }
  if (visits) *visits = nvis;
  free(acc);
  free(count);
  return rc;
}
