// kernel_common.h -- device helpers shared by the gfx950 kernels (LDS access, chunk staging,
// the feature tile, class bookkeeping, the link functions) and the launch helper.
//
// One fused kernel per launch runs the whole lowered pipeline of a tree model (Sec. 4.2 and
// Table 4): gather the split feature of the current node (take/gather), compare it with the
// threshold (less_equal), pick the child (where), descend (loop/while), fetch the leaf and
// aggregate over trees (sum/mean), then apply the link function (exp/add/divide/max).  No
// intermediate tensor leaves the chip (the cross-domain fusion idea of Sec. 4.3 applied to
// one model).
//
// Work decomposition of the chunked kernels (the "tile", "split" and "parallel" schedules of
// Table 5, sized by the Eq. 1 planner on the host):
//   * a workgroup owns R consecutive rows; their features are copied once from HBM into an
//     LDS tile stored feature-major (x of feature f, row r at byte 4*(f*R + r)).  Lane r of
//     every 32-lane half-wave then reads a different LDS bank whatever feature it needs, so
//     the per-lane feature gather is conflict-free;
//   * the trees stream through two LDS chunk buffers.  One extra wave per workgroup does
//     nothing but stage: while the compute waves traverse chunk c it loads chunk c + 1 into the
//     other buffer with direct global->LDS loads; one barrier per chunk;
//   * with 64*waves == R every lane owns one row and adds its leaves in ascending tree order
//     (bit-identical to a sequential sum); with 64*waves > R the G = 64*waves/R lane groups
//     split the trees and their per-class partial sums are added in group order at the end.
// Sums are kept in double precision; the output is rounded once to float.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <map>
#include <mutex>
#include <type_traits>
#include <utility>

#include "internal.h"

namespace bridger {

typedef __attribute__((address_space(3))) uint8_t lds_byte;

// Fourth word of a raw (untyped, unswizzled) buffer resource on gfx9-family CDNA parts.
constexpr int kBufferRsrcWord3 = 0x00020000;

// The kernels declare no static LDS, so dynamic LDS starts at LDS address 0 and a byte
// offset into it is directly an LDS address (no base add on every access).
__device__ __forceinline__ float lds_f32(const uint8_t *, uint32_t addr) {
  return *(const __attribute__((address_space(3))) float *)(uintptr_t)addr;
}
__device__ __forceinline__ uint32_t lds_u16(const uint8_t *, uint32_t addr) {
  return *(const __attribute__((address_space(3))) uint16_t *)(uintptr_t)addr;
}
__device__ __forceinline__ uint32_t lds_u8(const uint8_t *, uint32_t addr) {
  return *(const __attribute__((address_space(3))) uint8_t *)(uintptr_t)addr;
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
                                             int lane, int tail, ChunkSrc chunk_src,
                                             int lead = 0) {
  {
    const auto src = chunk_src(0);
    stage_async(smem, 0, src.first, src.second, 0, lane, 1);
    wait_stage();
  }
  for (int i = 0; i < lead; ++i) __syncthreads();  // extra barriers of the tile load
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

// The fused preprocessing of feature f (BRIDGER_PRE_* in bridger.h) with the kind fixed at
// compile time: each step in double, rounded to float.  rn is the row's norm (NORMALIZE only).
template <int KIND>
__device__ __forceinline__ float preprocess_k(const LaunchArgs &a, int f, double rn, float x) {
  if (KIND == 1) {
    const float x1 = (float)((double)x * a.pre_a[f]);
    return (float)((double)x1 + a.pre_b[f]);
  }
  if (KIND == 2) {
    const float x1 = (float)((double)x - a.pre_a[f]);
    return (float)((double)x1 / a.pre_b[f]);
  }
  if (KIND == 3) return ((double)x > a.pre_a[f]) ? 1.0f : 0.0f;
  if (KIND == 4) return (float)((double)x / rn);
  return x;
}

// The same with the kind read at run time; rn as above.
__device__ __forceinline__ float preprocess_rt(const LaunchArgs &a, int f, double rn, float x) {
  switch (a.pre_kind) {
    case 1: return preprocess_k<1>(a, f, rn, x);
    case 2: return preprocess_k<2>(a, f, rn, x);
    case 3: return preprocess_k<3>(a, f, rn, x);
    case 4: return preprocess_k<4>(a, f, rn, x);
    default: return x;
  }
}

// The same for feature f of row `row`.
__device__ __forceinline__ float preprocess(const LaunchArgs &a, int f, int64_t row, float x) {
  return preprocess_rt(a, f, a.pre_kind == 4 ? a.row_norm[row] : 1.0, x);
}

// Load part `part` of `parts` of this lane's row into the feature-major LDS tile (zeros past
// the last row): the lane groups sharing a tile split each row's features between them.  With
// NAN_TO_INF a NaN feature is stored as +inf: against finite thresholds both compare false
// (x <= t), so every split sends them the same way.  The row's norm (NORMALIZE) is loaded once
// ahead of the loop.
template <bool NAN_TO_INF = false>
__device__ __forceinline__ void load_row_tile(uint8_t *smem, const LaunchArgs &a, int r,
                                              int64_t row, bool row_ok, int part = 0,
                                              int parts = 1) {
  float *xt = reinterpret_cast<float *>(smem + a.lds_x_off);
  const int R = a.rows_per_wg;
  if (!row_ok) {
    const int f0 = (a.F * part) / parts, f1 = (a.F * (part + 1)) / parts;
    for (int f = f0; f < f1; ++f) xt[f * R + r] = 0.0f;
    return;
  }
  const float *xr = a.X + row * (int64_t)a.F;
  auto body = [&](auto pre_tag) {
    constexpr bool PRE = decltype(pre_tag)::value;
    const double rn = (PRE && a.pre_kind == 4) ? a.row_norm[row] : 1.0;
    auto put = [&](int f, float v) {
      if (PRE) v = preprocess_rt(a, f, rn, v);
      if (NAN_TO_INF) v = (v != v) ? __builtin_inff() : v;
      xt[f * R + r] = v;
    };
    if (a.x_vec4) {
      const float4 *x4 = reinterpret_cast<const float4 *>(xr);
      const int n4 = a.F >> 2;
      const int i0 = (n4 * part) / parts, i1 = (n4 * (part + 1)) / parts;
      int i = i0;
      for (; i + 2 <= i1; i += 2) {
        const float4 v0 = x4[i], v1 = x4[i + 1];
        put(4 * i + 0, v0.x);
        put(4 * i + 1, v0.y);
        put(4 * i + 2, v0.z);
        put(4 * i + 3, v0.w);
        put(4 * i + 4, v1.x);
        put(4 * i + 5, v1.y);
        put(4 * i + 6, v1.z);
        put(4 * i + 7, v1.w);
      }
      for (; i < i1; ++i) {
        const float4 v = x4[i];
        put(4 * i + 0, v.x);
        put(4 * i + 1, v.y);
        put(4 * i + 2, v.z);
        put(4 * i + 3, v.w);
      }
    } else {
      const int f0 = (a.F * part) / parts, f1 = (a.F * (part + 1)) / parts;
      for (int f = f0; f < f1; ++f) put(f, xr[f]);
    }
  };
  if (a.pre_kind) body(std::true_type{});
  else body(std::false_type{});
}

// Byte offset of row r's element inside a feature's row of the LDS tile, for elements of XB
// bytes.  fp32 (XB = 4): 4r.  Bins (XB = 2 or 1) pack P = 4 / XB rows per 32-bit word: row r
// sits in word (r mod 32) + 32 (r div 32P), sub-word (r div 32) mod P, so the 32 rows of a
// half-wave always hit 32 different banks whatever features they read (R is a multiple of 32P).
template <int XB>
__device__ __forceinline__ uint32_t tile_row_off(int r) {
  if (XB == 4) return 4u * (uint32_t)r;
  constexpr int P = 4 / XB;
  return 4u * (uint32_t)((r & 31) + 32 * (r / (32 * P))) + (uint32_t)(XB * ((r >> 5) & (P - 1)));
}

// Load part `part` of `parts` of this lane's row of bins (F elements of XB bytes each,
// row-major in global memory) into the feature-major LDS tile (zeros past the last row).
// x_vec4: rows 16-byte aligned.
template <int XB>
__device__ __forceinline__ void load_row_tile_binned(uint8_t *smem, const LaunchArgs &a, int r,
                                                     int64_t row, bool row_ok, int part,
                                                     int parts) {
  static_assert(XB == 1 || XB == 2, "bins are 8 or 16 bits");
  const uint32_t stride = (uint32_t)a.rows_per_wg * XB;  // one feature's row of the tile
  const uint32_t base = (uint32_t)a.lds_x_off + tile_row_off<XB>(r);
  auto put = [&](int f, uint32_t v) {
    const uint32_t addr = base + (uint32_t)f * stride;
    if (XB == 2) *(__attribute__((address_space(3))) uint16_t *)(uintptr_t)addr = (uint16_t)v;
    else *(__attribute__((address_space(3))) uint8_t *)(uintptr_t)addr = (uint8_t)v;
  };
  const int f0 = (a.F * part) / parts, f1 = (a.F * (part + 1)) / parts;
  if (!row_ok) {
    for (int f = f0; f < f1; ++f) put(f, 0u);
    return;
  }
  const uint8_t *xr = reinterpret_cast<const uint8_t *>(a.X) + row * (int64_t)a.F * XB;
  if (a.x_vec4) {
    constexpr int E = 16 / XB;  // elements per 16-byte load
    const uint4 *x4 = reinterpret_cast<const uint4 *>(xr);
    const int n4 = (a.F * XB) >> 4;
    const int i0 = (n4 * part) / parts, i1 = (n4 * (part + 1)) / parts;
    for (int i = i0; i < i1; ++i) {
      const uint4 v = x4[i];
      const uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
      for (int e = 0; e < E; ++e) {
        const uint32_t word = w[(e * XB) >> 2];
        put(i * E + e, (word >> (8 * ((e * XB) & 3))) & (XB == 2 ? 0xFFFFu : 0xFFu));
      }
    }
  } else {
    for (int f = f0; f < f1; ++f)
      put(f, XB == 2 ? (uint32_t)reinterpret_cast<const uint16_t *>(xr)[f] : (uint32_t)xr[f]);
  }
}

// Rows given in CSR form (a.csr: X = values, a.csr_indptr, a.csr_indices), absent features
// reading 0: fill this lane's part of its row with (preprocessed) zeros, wait for every part,
// then write this lane's share of the row's stored entries.  Entries whose index lies outside
// [0, F) are ignored.  Contains one barrier (every compute wave of the workgroup calls it).
template <bool NAN_TO_INF>
__device__ __forceinline__ void load_row_tile_csr(uint8_t *smem, const LaunchArgs &a, int r,
                                                  int64_t row, bool row_ok, int part, int parts) {
  float *xt = reinterpret_cast<float *>(smem + a.lds_x_off);
  const int R = a.rows_per_wg, F = a.F;
  auto fix = [&](int f, float v) {
    if (a.pre_kind) v = preprocess(a, f, row, v);
    if (NAN_TO_INF) v = (v != v) ? __builtin_inff() : v;
    return v;
  };
  const int f0 = (F * part) / parts, f1 = (F * (part + 1)) / parts;
  for (int f = f0; f < f1; ++f) xt[f * R + r] = row_ok ? fix(f, 0.0f) : 0.0f;
  __syncthreads();
  if (!row_ok) return;
  const int64_t p0 = a.csr_indptr[row], n = a.csr_indptr[row + 1] - p0;
  const int64_t e0 = p0 + (n * part) / parts, e1 = p0 + (n * (part + 1)) / parts;
  for (int64_t e = e0; e < e1; ++e) {
    const int f = a.csr_indices[e];
    if (f >= 0 && f < F) xt[f * R + r] = fix(f, a.X[e]);
  }
}

// The tile load for element size XB (fp32 with NaN stored as +inf when NAN_TO_INF); part
// `part` of `parts` of the row's features.  A CSR load adds one barrier (staging waves match
// it with their `lead` barrier).
template <int XB, bool NAN_TO_INF>
__device__ __forceinline__ void load_tile_any(uint8_t *smem, const LaunchArgs &a, int r,
                                              int64_t row, bool row_ok, int part, int parts) {
  if constexpr (XB == 4) {
    if (a.csr) load_row_tile_csr<NAN_TO_INF>(smem, a, r, row, row_ok, part, parts);
    else load_row_tile<NAN_TO_INF>(smem, a, r, row, row_ok, part, parts);
  } else {
    load_row_tile_binned<XB>(smem, a, r, row, row_ok, part, parts);
  }
}

// The row tile of a workgroup whose threads all load (the global-node RAGGED kernels), for dense
// fp32 rows without preprocessing (16-byte aligned, F % 4 == 0): each wave instruction reads 8
// rows x 128 consecutive bytes (8 lanes per row, one cache line each) instead of 64 rows x 16
// bytes, and writes the values into the same feature-major tile.  In that tile a feature's row
// spans the 32 banks once, so the 8 lanes of a row write to one bank: the L2 reads touch 8
// lines instead of 64 and the LDS writes conflict 8-way.  That pays where two workgroups per
// CU overlap one's tile load with the other's walk (4M x 256 rows: 15.02 -> 14.82 ms); with one
// workgroup per CU waiting on its tile it does not (the 784-feature perfect forest: 0.538 ->
// 0.572 ms), so the PERFECT kernels keep load_tile_any.  Other rows and element types take
// load_tile_any.
template <int XB, bool NAN_TO_INF>
__device__ __forceinline__ void load_tile_all(uint8_t *smem, const LaunchArgs &a, int r,
                                              int64_t row, bool row_ok, int g, int G) {
  if constexpr (XB == 4) {
    if (a.tile_coalesced && a.x_vec4 && !a.csr && a.pre_kind == 0) {
      float *xt = reinterpret_cast<float *>(smem + a.lds_x_off);
      const int R = a.rows_per_wg, F4 = a.F >> 2;
      const int n_rb = R / 8, n_inst = n_rb * ((F4 + 7) / 8);
      const int tid = threadIdx.x, lane = tid & 63, waves = (int)(blockDim.x >> 6);
      const int64_t row0 = (int64_t)blockIdx.x * R;
      const float4 *x4 = reinterpret_cast<const float4 *>(a.X);
      for (int q = tid >> 6; q < n_inst; q += waves) {
        const int rr = (q % n_rb) * 8 + (lane & 7), c = (q / n_rb) * 8 + (lane >> 3);
        if (c < F4) {
          const int64_t gr = row0 + rr;
          float4 v = gr < a.n_rows ? x4[gr * F4 + c] : make_float4(0.f, 0.f, 0.f, 0.f);
          if (NAN_TO_INF) {
            v.x = (v.x != v.x) ? __builtin_inff() : v.x;
            v.y = (v.y != v.y) ? __builtin_inff() : v.y;
            v.z = (v.z != v.z) ? __builtin_inff() : v.z;
            v.w = (v.w != v.w) ? __builtin_inff() : v.w;
          }
          xt[(4 * c + 0) * R + rr] = v.x;
          xt[(4 * c + 1) * R + rr] = v.y;
          xt[(4 * c + 2) * R + rr] = v.z;
          xt[(4 * c + 3) * R + rr] = v.w;
        }
      }
      return;
    }
  }
  load_tile_any<XB, NAN_TO_INF>(smem, a, r, row, row_ok, g, G);
}

__device__ __forceinline__ double sigmoid_d(double z) {
  if (z >= 0.0) return 1.0 / (1.0 + exp(-z));
  const double e = exp(z);
  return e / (1.0 + e);
}

// Store the finished value z of a one-output row: its score, or its label (z > 0, i.e. the
// sigmoid above one half).
__device__ __forceinline__ void store_one(const LaunchArgs &a, int64_t row, double z) {
  if (a.out_label) a.out_label[row] = z > 0.0 ? 1 : 0;
  else a.out[row] = (float)(a.transform == 1 ? sigmoid_d(z) : z);
}

// Finish class values z[0..K) held in LDS (stride `stride` doubles) and store the row: the
// scores, or the label (the first class of largest value; one output: z > 0).
__device__ void finalize_store(const LaunchArgs &a, double *z, int stride, int64_t row) {
  const int K = a.K;
  for (int k = 0; k < K; ++k) {
    double v = z[k * stride];
    if (a.aggregate == 1) v = (double)a.base[k] + v / (double)a.class_count[k];
    z[k * stride] = v;
  }
  if (a.out_label) {
    if (K == 1) {
      a.out_label[row] = z[0] > 0.0 ? 1 : 0;
    } else {
      int best = 0;
      for (int k = 1; k < K; ++k) best = z[k * stride] > z[best * stride] ? k : best;
      a.out_label[row] = best;
    }
    return;
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

// Tile epilogue of the kernels whose G lane groups hold partial class sums: slot (k, g, r) at
// z0[k * stride + g * R + r].  Each (row, class) sum is added in group order by one of the R * G
// compute threads (threads 0 .. R * G - 1 of a tile of rows blockIdx.x * R + r, R a power of
// two; every one of them calls this after a barrier) into slot (k, 0, r); then the first
// group's lanes (tid < R) finish and store their rows.
__device__ void groups_finalize_store(const LaunchArgs &a, double *z0, int R, int G, int stride,
                                      int tid, int64_t row, bool row_ok) {
  if (G > 1) {
    for (int i = tid; i < R * a.K; i += R * G) {
      const int k = i / R;
      double *z = z0 + k * stride + (i - k * R);
      double s = z[0];
      for (int gg = 1; gg < G; ++gg) s += z[gg * R];
      z[0] = s;
    }
    __syncthreads();
    if (a.transform == 2 && !a.out_label && a.K > 1) {
      // softmax, one (row, class) per thread as well: each thread finishes its row's K values
      // as finalize_store does (same operations, same order) and writes its exponential into
      // the second group's slot, free now; then each divides by the row's sum
      const int K = a.K;
      const int64_t row0 = (int64_t)blockIdx.x * R;  // the tile's first row
      for (int i = tid; i < R * K; i += R * G) {
        const int k = i / R, rr = i - k * R;
        const double *z = z0 + rr;
        auto v = [&](int j) {
          const double x = z[j * stride];
          return a.aggregate == 1 ? (double)a.base[j] + x / (double)a.class_count[j] : x;
        };
        double m = v(0);
        for (int j = 1; j < K; ++j) m = v(j) > m ? v(j) : m;
        z0[k * stride + R + rr] = exp(v(k) - m);
      }
      __syncthreads();
      for (int i = tid; i < R * K; i += R * G) {
        const int k = i / R, rr = i - k * R;
        if (row0 + rr >= a.n_rows) continue;
        const double *e = z0 + R + rr;
        double sum = 0.0;
        for (int j = 0; j < K; ++j) sum += e[j * stride];
        a.out[(row0 + rr) * (int64_t)K + k] = (float)(e[k * stride] / sum);
      }
      return;
    }
  }
  if (tid < R && row_ok) finalize_store(a, z0 + tid, stride, row);
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

// ====================================================================== launchers
// Raise a kernel's dynamic-LDS limit once per (kernel, device) to the largest size used.
static inline int ensure_lds_limit(const void *kernel, int lds_bytes) {
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
static inline int launch_common(K kernel, int threads, int64_t n_wg, int lds_bytes, void *stream,
                         const LaunchArgs &a) {
  const int e = ensure_lds_limit((const void *)kernel, lds_bytes);
  if (e != 0) return e;
  hipLaunchKernelGGL(kernel, dim3((unsigned)n_wg), dim3(threads), lds_bytes,
                     (hipStream_t)stream, a);
  return (int)hipGetLastError();
}

}  // namespace bridger
