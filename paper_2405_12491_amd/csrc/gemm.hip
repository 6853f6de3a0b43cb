// gemm.hip -- gfx950 matrix-multiply lowering of shallow perfect forests (MFMA).
#include "kernel_common.h"

namespace bridger {

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
      if (s < n_steps && f < F && row < a.n_rows) {
        v = a.X[row * (int64_t)F + f];
        if (a.pre_kind) v = preprocess(a, f, row, v);
      }
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
          store_one(a, row, zv);
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
          const float xv = a.pre_kind ? preprocess(a, f, row, xr[f]) : xr[f];
          mm = 2 * mm + ((xv <= th) ? 0 : 1);
        }
        if (LEAVES)
          a.out_leaf[row * (int64_t)T + a.tree_order[t]] =
              a.leaf_map[(int64_t)t * kSlots + (mm - kSlots)];
        else
          zv += (double)*reinterpret_cast<const float *>(tp + 8 * kSlots + 4 * (mm - kSlots));
      }
      if (!LEAVES) {
        if (a.aggregate == 1) zv = (double)a.base[0] + zv / (double)a.class_count[0];
        store_one(a, row, zv);
      }
    }
  }
}

// ---------------------------------------------------------------------- launchers
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
