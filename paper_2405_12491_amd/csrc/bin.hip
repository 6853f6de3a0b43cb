// bin.hip -- exact feature quantization ("data type rewriting", Table 2): each fp32 feature
// value becomes its bin, the number of the forest's distinct thresholds on that feature that
// are strictly below it.  For a threshold t of rank k among them, x <= t iff bin(x) <= k
// (-0.0 and +0.0 are one threshold; a NaN feature gets the table's size, above every rank,
// so it goes right at every split as the fp32 compare sends it).
//
// A workgroup owns a block of rows.  It walks the features in runs whose threshold tables fit
// its LDS buffer: stage the run's tables (direct global->LDS loads), then every (row, feature)
// of the run binary-searches its feature's table in LDS.  A single table larger than the
// buffer is searched in global memory instead.
#include "kernel_common.h"

namespace bridger {

// 16 waves per workgroup: each lane's binary search is a chain of dependent LDS reads, so the
// pass needs many waves in flight per CU (two 64 KB workgroups fit a CU).
constexpr int kBinThreads = 1024;
// Features per block: one 128-byte line of an fp32 row.  A block reads its rows' line once per
// run of features (the tables of a run share the LDS buffer), so the runs of one block re-read
// only that line, soon enough for L2 to serve it, and the blocks of one group (one in every
// n_groups, dispatched round-robin over the XCDs) share the group's tables in L2.
constexpr int kBinGroup = 32;

__device__ __forceinline__ int lower_bound_f32(const float *t, int n, float x) {
  int lo = 0, len = n;
  while (len > 0) {
    const int half = len >> 1;
    if (t[lo + half] < x) {
      lo += half + 1;
      len -= half + 1;
    } else {
      len = half;
    }
  }
  return lo;
}

template <int XB>
__global__ __launch_bounds__(kBinThreads) void bin_kernel(LaunchArgs a) {
  extern __shared__ __attribute__((aligned(16))) uint8_t smem[];
  const float *tab = reinterpret_cast<const float *>(smem);
  const int cap = a.chunk_bytes / 4;  // floats the LDS buffer holds
  const int tid = threadIdx.x;
  // block = (row block, group of kBinGroup features); consecutive blocks take consecutive groups
  const int n_groups = a.groups;
  const int grp = (int)(blockIdx.x % (uint32_t)n_groups);
  const int64_t r0 = (int64_t)(blockIdx.x / (uint32_t)n_groups) * a.rows_per_wg;
  const int64_t r1 = (r0 + a.rows_per_wg < a.n_rows) ? r0 + a.rows_per_wg : a.n_rows;
  const int F = a.F;
  const int f_end = (grp + 1) * kBinGroup < F ? (grp + 1) * kBinGroup : F;
  int f = grp * kBinGroup;
  while (f < f_end) {
    const int base = a.q_off[f];
    int fe = f;
    while (fe < f_end && a.q_off[fe + 1] - base <= cap) ++fe;
    const bool in_lds = fe > f;
    if (!in_lds) fe = f + 1;  // one table too large for the buffer: search it in place
    const int nf = fe - f;
    if (in_lds) {
      __syncthreads();  // the previous run's searches are done with the buffer
      const int n = a.q_off[fe] - base;
      for (int i = tid; i < n; i += kBinThreads) reinterpret_cast<float *>(smem)[i] = a.q_values[base + i];
      __syncthreads();
    }
    // a block's rows x the run's features stays below 2^31 (launch_bin): 32-bit indices
    const uint32_t total = (uint32_t)(r1 - r0) * (uint32_t)nf;
    for (uint32_t i = tid; i < total; i += kBinThreads) {
      const uint32_t rq = i / (uint32_t)nf;
      const int64_t row = r0 + rq;
      const int ff = f + (int)(i - rq * (uint32_t)nf);
      const int64_t e = row * F + ff;
      const float x = a.pre_kind ? preprocess(a, ff, row, a.X[e]) : a.X[e];
      const int o = a.q_off[ff] - base, cnt = a.q_off[ff + 1] - a.q_off[ff];
      int b = cnt;
      if (x == x) b = in_lds ? lower_bound_f32(tab + o, cnt, x)
                             : lower_bound_f32(a.q_values + a.q_off[ff], cnt, x);
      if (XB == 2) reinterpret_cast<uint16_t *>(a.xq)[e] = (uint16_t)b;
      else reinterpret_cast<uint8_t *>(a.xq)[e] = (uint8_t)b;
    }
    f = fe;
  }
}

int launch_bin(const LaunchArgs &a0, void *stream) {
  LaunchArgs a = a0;
  // About one block per resident workgroup (two per CU): each block restages its tables once
  // per run of features, and longer blocks re-read lines that L2 no longer holds; at most
  // 2,048 rows, 1,024 with several feature groups (measured: 1M x 28 rows 0.146 -> 0.138 ms
  // against n / 1024 rows per block and no groups, 100k x 784 0.546 -> 0.33 ms, 4M x 256
  // 13.0 -> 9.4 ms).
  const int64_t groups = (a.F + kBinGroup - 1) / kBinGroup;
  int64_t rows = (a.n_rows * groups + 511) / 512;
  const int64_t max_rows = groups > 1 ? 1024 : 2048;
  rows = rows < 64 ? 64 : (rows > max_rows ? max_rows : rows);
  if (a0.rows_per_wg > 0) rows = a0.rows_per_wg;
  // at most 2^21 blocks (2^31 work-items), and a run's (row, feature) pairs fit 32 bits
  const int64_t min_rows = (a.n_rows * groups + (int64_t(1) << 21) - 1) >> 21;
  rows = rows < min_rows ? min_rows : rows;
  const int64_t cap = INT32_MAX / kBinGroup;
  rows = rows > cap ? cap : rows;
  a.rows_per_wg = (int32_t)rows;
  a.groups = (int32_t)groups;
  if (a.chunk_bytes <= 0) a.chunk_bytes = 64 * 1024;
  const int64_t blocks = (a.n_rows + rows - 1) / rows * groups;
  if (a.x_bytes == 2) return launch_common(bin_kernel<2>, kBinThreads, blocks, a.chunk_bytes, stream, a);
  if (a.x_bytes == 1) return launch_common(bin_kernel<1>, kBinThreads, blocks, a.chunk_bytes, stream, a);
  return (int)hipErrorInvalidValue;
}

}  // namespace bridger
