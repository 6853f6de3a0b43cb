// bin.hip -- exact feature quantization ("data type rewriting", Table 2): each fp32 feature
// value becomes its bin, the number of the forest's distinct thresholds on that feature that
// are strictly below it.  For a threshold t of rank k among them, x <= t iff bin(x) <= k
// (-0.0 and +0.0 are one threshold; a NaN feature gets the table's size, above every rank,
// so it goes right at every split as the fp32 compare sends it).
//
// Two kernels; launch_bin (at the end) picks one by how many LDS loads of tables a group of 32
// features needs.
//
// Row kernel: a workgroup owns 512 rows and one group of 32 features (one 128-byte line of an
// fp32 row): every thread holds its row's 32 values of the group in registers, read once.  The
// group's features are then taken in runs whose threshold tables fit the workgroup's LDS
// buffer: stage the run's tables, then each thread binary-searches its values of the run's
// features, four features at a time (four independent chains of LDS reads).  The bins stay in
// registers until every run is done and are written once, whole (16-byte stores where the
// layout allows).  X is read once and the bins written once whatever the tables' size; what
// grows with the tables is the L2->LDS staging (the tables, a few MB at most, stay in L2).  A
// single table larger than the buffer is searched in global memory instead.
#include "kernel_common.h"

namespace bridger {

constexpr int kBinThreads = 512;  // rows per workgroup, one per thread; two workgroups a CU
constexpr int kBinGroup = 32;     // features per workgroup
constexpr int kBinIlp = 4;        // searches in flight per thread

// Number of the n[j] ascending values at t[j] strictly below x[j] (x not NaN), for N tables at
// once, by a binary search over power-of-two steps: lo only grows, by `step` when the step's
// last element is below x.  The same trip count (floor(log2 max_n) + 1 steps) for every lane
// searching the same tables.  LDS: t holds element offsets into the staged (padded) run; else
// global element offsets into g.
// In LDS the staged tables keep one unused float after every 32 (element e at e + e / 32): a
// search's lanes sit at positions that differ by multiples of its step, and without the pad
// every step of 32 or more would send all of them to one bank.
__device__ __forceinline__ uint32_t padded(uint32_t e) { return e + (e >> 5); }

template <int N, bool LDS>
__device__ __forceinline__ void count_below(const float *g, const uint32_t (&t)[N],
                                            const int (&n)[N], const float (&x)[N], int max_n,
                                            int (&lo)[N]) {
#pragma unroll
  for (int j = 0; j < N; ++j) lo[j] = 0;
  if (max_n <= 0) return;
  for (int step = 1 << (31 - __builtin_clz((unsigned)max_n)); step > 0; step >>= 1) {
    float v[N];
#pragma unroll
    for (int j = 0; j < N; ++j) {
      const int i = lo[j] + step - 1;
      const uint32_t k = (uint32_t)(i < n[j] ? i : (n[j] > 0 ? n[j] - 1 : 0));
      v[j] = LDS ? lds_f32(nullptr, 4u * padded(t[j] + k)) : g[t[j] + k];
    }
#pragma unroll
    for (int j = 0; j < N; ++j)
      if (lo[j] + step <= n[j] && v[j] < x[j]) lo[j] += step;
  }
}

template <int XB>
__global__ __launch_bounds__(kBinThreads, 4) void bin_rows_kernel(LaunchArgs a) {  // 2 per CU
  extern __shared__ __attribute__((aligned(16))) uint8_t smem[];
  // floats of tables the LDS buffer holds: padded, with up to 3 leading and 3 trailing slack
  const int cap = (a.chunk_bytes / 4) * 32 / 33 - 8;
  const int tid = threadIdx.x;
  const int n_groups = a.groups;
  const int grp = (int)(blockIdx.x % (uint32_t)n_groups);
  // this block's rows: trees_per_chunk chunks of kBinThreads rows (the host's choice)
  const int chunks = a.trees_per_chunk;
  const int64_t rb = (int64_t)(blockIdx.x / (uint32_t)n_groups) * chunks * kBinThreads;
  const int F = a.F;
  const int f0 = grp * kBinGroup;
  const int nf = F - f0 < kBinGroup ? F - f0 : kBinGroup;
  const int f_end = f0 + nf;
  int staged = -1, staged_end = -1;  // the run whose tables the buffer holds

  for (int c = 0; c < chunks; ++c) {
    const int64_t row = rb + (int64_t)c * kBinThreads + tid;
    if (__builtin_amdgcn_readfirstlane((int)(rb + (int64_t)c * kBinThreads < a.n_rows)) == 0)
      break;  // uniform: no row of this chunk exists
    const bool row_ok = row < a.n_rows;

    // the row's values of the group (zeros past the row's end or the last feature)
    float x[kBinGroup];
    const float *xr = a.X + (row_ok ? row : 0) * (int64_t)F + f0;
    if (a.x_vec4 && nf == kBinGroup) {
      const float4 *x4 = reinterpret_cast<const float4 *>(xr);
#pragma unroll
      for (int k = 0; k < kBinGroup / 4; ++k) {
        const float4 v = row_ok ? x4[k] : make_float4(0.f, 0.f, 0.f, 0.f);
        x[4 * k] = v.x;
        x[4 * k + 1] = v.y;
        x[4 * k + 2] = v.z;
        x[4 * k + 3] = v.w;
      }
    } else {
#pragma unroll
      for (int j = 0; j < kBinGroup; ++j) x[j] = (row_ok && j < nf) ? xr[j] : 0.0f;
    }
    if (a.pre_kind && row_ok) {
#pragma unroll
      for (int j = 0; j < kBinGroup; ++j)
        if (j < nf) x[j] = preprocess(a, f0 + j, row, x[j]);
    }

    uint32_t bin[kBinGroup];
#pragma unroll
    for (int j = 0; j < kBinGroup; ++j) bin[j] = 0;
    int f = f0;
    while (f < f_end) {  // runs of features whose tables fit the buffer (uniform control flow)
      const int base = a.q_off[f];
      int fe = f;
      while (fe < f_end && a.q_off[fe + 1] - base <= cap) ++fe;
      const bool in_lds = fe > f;
      if (!in_lds) fe = f + 1;  // one table too large for the buffer: search it in place
      // the run's tables, copied in 16-byte pieces from the aligned global offset abase <= base
      // into the padded layout; a group with one run stages it once for all its chunks
      const int abase = base & ~3;
      if (in_lds && !(staged == base && staged_end == fe)) {
        __syncthreads();  // the previous run's searches are done with the buffer
        const int n4 = (a.q_off[fe] - abase + 3) >> 2;  // 16-byte pieces
        const float4 *src4 = reinterpret_cast<const float4 *>(a.q_values + abase);
        for (int i = tid; i < n4; i += kBinThreads) {
          const float4 v = src4[i];
          const uint32_t p = 4u * padded(4u * (uint32_t)i);  // four elements of one 32-row
          *(__attribute__((address_space(3))) float *)(uintptr_t)(p) = v.x;
          *(__attribute__((address_space(3))) float *)(uintptr_t)(p + 4) = v.y;
          *(__attribute__((address_space(3))) float *)(uintptr_t)(p + 8) = v.z;
          *(__attribute__((address_space(3))) float *)(uintptr_t)(p + 12) = v.w;
        }
        __syncthreads();
        staged = base;
        staged_end = fe;
      }
#pragma unroll
      for (int j0 = 0; j0 < kBinGroup; j0 += kBinIlp) {
        if (f0 + j0 + kBinIlp <= f || f0 + j0 >= fe) continue;  // no feature of the run here
        uint32_t t[kBinIlp];
        int n[kBinIlp], lo[kBinIlp];
        float xv[kBinIlp];
        int max_n = 0;
#pragma unroll
        for (int j = 0; j < kBinIlp; ++j) {
          const int ff = f0 + j0 + j;
          const bool in_run = ff >= f && ff < fe;
          const int o = in_run ? a.q_off[ff] : base;
          n[j] = in_run ? a.q_off[ff + 1] - o : 0;
          // the table's element offset in the staged run (the buffer starts at LDS 0), or in
          // the global array
          t[j] = in_lds ? (uint32_t)(o - abase) : (uint32_t)o;
          xv[j] = x[j0 + j];
          max_n = n[j] > max_n ? n[j] : max_n;
        }
        if (in_lds) count_below<kBinIlp, true>(a.q_values, t, n, xv, max_n, lo);
        else count_below<kBinIlp, false>(a.q_values, t, n, xv, max_n, lo);
#pragma unroll
        for (int j = 0; j < kBinIlp; ++j) {
          const int ff = f0 + j0 + j;
          if (ff >= f && ff < fe)
            bin[j0 + j] = (xv[j] == xv[j]) ? (uint32_t)lo[j] : (uint32_t)n[j];
        }
      }
      f = fe;
    }

    if (row_ok) {
      uint8_t *q = reinterpret_cast<uint8_t *>(a.xq) + (row * (int64_t)F + f0) * XB;
      constexpr int kBytes = kBinGroup * XB;  // one row's bins of the group
      if (nf == kBinGroup && ((uintptr_t)q & 15) == 0) {
        uint32_t w[kBytes / 4];
#pragma unroll
        for (int i = 0; i < kBytes / 4; ++i) {
          if (XB == 2)
            w[i] = bin[2 * i] | (bin[2 * i + 1] << 16);
          else
            w[i] = bin[4 * i] | (bin[4 * i + 1] << 8) | (bin[4 * i + 2] << 16) |
                   (bin[4 * i + 3] << 24);
        }
        uint4 *q4 = reinterpret_cast<uint4 *>(q);
#pragma unroll
        for (int i = 0; i < kBytes / 16; ++i)
          q4[i] = make_uint4(w[4 * i], w[4 * i + 1], w[4 * i + 2], w[4 * i + 3]);
      } else {
#pragma unroll
        for (int j = 0; j < kBinGroup; ++j) {
          if (j < nf) {
            if (XB == 2) reinterpret_cast<uint16_t *>(q)[j] = (uint16_t)bin[j];
            else q[j] = (uint8_t)bin[j];
          }
        }
      }
    }
  }
}

static int launch_bin_rows(const LaunchArgs &a0, void *stream) {
  LaunchArgs a = a0;
  const int64_t groups = (a.F + kBinGroup - 1) / kBinGroup;
  a.groups = (int32_t)groups;
  if (a.chunk_bytes <= 0) a.chunk_bytes = 64 * 1024;  // two workgroups per CU
  // chunks of kBinThreads rows per block: about two blocks per CU slot while that keeps a
  // feature group's tables staged once for several chunks, at most 8
  const int64_t n_chunks = (a.n_rows + kBinThreads - 1) / kBinThreads;
  int64_t per = (n_chunks * groups) / 2048;
  per = per < 1 ? 1 : (per > 8 ? 8 : per);
  if (a0.trees_per_chunk > 0) per = a0.trees_per_chunk;  // tuning override
  a.trees_per_chunk = (int32_t)per;
  const int64_t blocks = (n_chunks + per - 1) / per * groups;
  if (a.x_bytes == 2) return launch_common(bin_rows_kernel<2>, kBinThreads, blocks, a.chunk_bytes, stream, a);
  if (a.x_bytes == 1) return launch_common(bin_rows_kernel<1>, kBinThreads, blocks, a.chunk_bytes, stream, a);
  return (int)hipErrorInvalidValue;
}

// ====================================================== stream kernel
// A workgroup owns a block of rows and one group of 32 features and walks the group's runs of
// features whose tables fit its LDS buffer: stage the run's tables, then every (row, feature)
// of the run binary-searches its feature's table, one element per lane at a time, writing its
// bin at once.  The block re-reads its rows' 128-byte line once per run (from L2 while it
// holds them), and the blocks of one group (one in every n_groups, dispatched round-robin
// over the XCDs) share the group's tables in L2.  16 waves per workgroup: each lane's binary
// search is a chain of dependent LDS reads, so the pass needs many waves in flight per CU (two
// 64 KB workgroups fit a CU).
constexpr int kBinStreamThreads = 1024;

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
__global__ __launch_bounds__(kBinStreamThreads) void bin_stream_kernel(LaunchArgs a) {
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
      for (int i = tid; i < n; i += kBinStreamThreads) reinterpret_cast<float *>(smem)[i] = a.q_values[base + i];
      __syncthreads();
    }
    // a block's rows x the run's features stays below 2^31 (launch_bin): 32-bit indices
    const uint32_t total = (uint32_t)(r1 - r0) * (uint32_t)nf;
    for (uint32_t i = tid; i < total; i += kBinStreamThreads) {
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

static int launch_bin_stream(const LaunchArgs &a0, void *stream) {
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
  if (a.x_bytes == 2) return launch_common(bin_stream_kernel<2>, kBinStreamThreads, blocks, a.chunk_bytes, stream, a);
  if (a.x_bytes == 1) return launch_common(bin_stream_kernel<1>, kBinStreamThreads, blocks, a.chunk_bytes, stream, a);
  return (int)hipErrorInvalidValue;
}

// Runs of table staging per feature group decide the kernel: with one or two runs the stream
// kernel (1,024 lanes, many searches in flight, a second read of the rows from L2) is the
// faster (16-bit bins of 1M x 28 rows: 0.138 against 0.276 ms), and so it is with more runs
// while the rows fit the last-level cache that serves its re-reads (1M x 28 rows, five runs:
// 0.167 against 0.323 ms); with more runs over larger rows its re-reads of X go to memory (7.3x
// the rows' bytes read and 4.0x the bins written for 4M x 256 rows with seven runs a group),
// and the row kernel, which reads X and writes the bins once, is the faster (8.7 against
// 9.5 ms).  The host passes a.n_chunks = the largest number of runs of any group when it
// wants the row kernel, else 1.
int launch_bin(const LaunchArgs &a, void *stream) {
  return a.n_chunks > 2 ? launch_bin_rows(a, stream) : launch_bin_stream(a, stream);
}

}  // namespace bridger
