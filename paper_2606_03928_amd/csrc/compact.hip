// compact.hip -- in-place stable compaction of the K survivors (gfx950).
//
// After selection, the cache keeps K of its N = K + B slots.  The survivor map
// src is strictly increasing with src[j] >= j, so every row moves towards lower
// slots by at most B.  The destination range [0, K) of an instance is cut into
// parts of T rows, one workgroup each:
//
//   * rows that part p reads but part p+1 overwrites (the source range
//     [(p+1)T, src[(p+1)T - 1]], at most B rows) are first copied to a staging
//     workspace by a separate kernel, so parts never race with each other;
//   * inside a part, chunks of rows are processed in ascending order, and each
//     chunk's loads complete (s_waitcnt + barrier) before any of its stores:
//     later chunks only read rows at or above their own destination, which no
//     earlier store touches.
//
// Rows in the unmoved prefix (src[j] == j) are skipped; src[j] - j is
// non-decreasing, so that prefix is found by binary search.
#include "vase_internal.hpp"
#include "vase.h"

namespace vase {
namespace {

constexpr int kCompBlock = 256;

// first j in [lo, hi) with src[j] != j, or hi
__device__ __forceinline__ int first_moved(const int32_t* s, int lo, int hi) {
  while (lo < hi) {
    const int mid = (lo + hi) >> 1;
    if (s[mid] > mid) hi = mid; else lo = mid + 1;
  }
  return lo;
}

__device__ __forceinline__ int clamp_slot(int s, int N) { return s < 0 ? 0 : (s >= N ? N - 1 : s); }

__device__ __forceinline__ void wait_vmem() { __builtin_amdgcn_s_waitcnt(0x0f70); }  // vmcnt(0)

// Stage the rows [(p+1)T, src[(p+1)T-1]] of part p (p < n_part-1) into ws.
// ws layout: [inst][n_part-1][2][B][row_u4] uint4.
template <int ROW_U4>
__global__ __launch_bounds__(kCompBlock) void compact_stage_kernel(
    const uint4* __restrict__ k, const uint4* __restrict__ v, const int32_t* __restrict__ src,
    int K, int B, int T, int n_part, uint4* __restrict__ ws) {
  const int p = blockIdx.x, inst = blockIdx.y;
  const int N = K + B;
  const int32_t* s = src + (size_t)inst * K;
  const int lo = (p + 1) * T;
  const int last = clamp_slot(s[min((p + 1) * T, K) - 1], N);
  const int cnt = min(last - lo + 1, B);
  if (cnt <= 0) return;
  const uint4* kb = k + (size_t)inst * N * ROW_U4;
  const uint4* vb = v + (size_t)inst * N * ROW_U4;
  uint4* wk = ws + (((size_t)inst * (n_part - 1) + p) * 2 + 0) * (size_t)B * ROW_U4;
  uint4* wv = ws + (((size_t)inst * (n_part - 1) + p) * 2 + 1) * (size_t)B * ROW_U4;
  for (int e = threadIdx.x; e < cnt * ROW_U4; e += kCompBlock) {
    const size_t off = (size_t)lo * ROW_U4 + e;
    wk[e] = kb[off];
    wv[e] = vb[off];
  }
}

template <int ROW_U4, int CHUNK>
__global__ __launch_bounds__(kCompBlock) void compact_move_kernel(
    uint4* __restrict__ k, uint4* __restrict__ v, const int32_t* __restrict__ src, int K, int B,
    int T, int n_part, const uint4* __restrict__ ws) {
  constexpr int kRowsPerPass = kCompBlock / ROW_U4;   // rows covered by one block-wide load
  constexpr int kPasses = CHUNK / kRowsPerPass;
  static_assert(CHUNK % kRowsPerPass == 0, "chunk must be a multiple of rows per pass");
  __shared__ int s_start;
  const int p = blockIdx.x, inst = blockIdx.y;
  const int N = K + B;
  const int32_t* s = src + (size_t)inst * K;
  const int j_lo = p * T;
  const int j_hi = min(K, (p + 1) * T);
  const int stage_lo = (p + 1) * T;     // rows >= stage_lo come from the staging area
  if (threadIdx.x == 0) s_start = first_moved(s, j_lo, j_hi);
  __syncthreads();
  const int start = s_start;
  uint4* kb = k + (size_t)inst * N * ROW_U4;
  uint4* vb = v + (size_t)inst * N * ROW_U4;
  const uint4* wk = nullptr;
  const uint4* wv = nullptr;
  if (p + 1 < n_part) {
    wk = ws + (((size_t)inst * (n_part - 1) + p) * 2 + 0) * (size_t)B * ROW_U4;
    wv = ws + (((size_t)inst * (n_part - 1) + p) * 2 + 1) * (size_t)B * ROW_U4;
  }
  const int col = threadIdx.x % ROW_U4;
  const int row0 = threadIdx.x / ROW_U4;
  for (int c0 = start; c0 < j_hi; c0 += CHUNK) {
    uint4 rk[kPasses], rv[kPasses];
#pragma unroll
    for (int u = 0; u < kPasses; ++u) {
      // rows past the part's end load a valid row and are not stored
      const int j = min(c0 + row0 + u * kRowsPerPass, j_hi - 1);
      const int sj = clamp_slot(s[j], N);
      const bool staged = wk != nullptr && sj >= stage_lo;
      const size_t off = staged ? (size_t)min(sj - stage_lo, B - 1) * ROW_U4 + col
                                : (size_t)sj * ROW_U4 + col;
      rk[u] = (staged ? wk : kb)[off];
      rv[u] = (staged ? wv : vb)[off];
    }
    wait_vmem();
    __syncthreads();
#pragma unroll
    for (int u = 0; u < kPasses; ++u) {
      const int j = c0 + row0 + u * kRowsPerPass;
      if (j < j_hi) {
        const size_t off = (size_t)j * ROW_U4 + col;
        kb[off] = rk[u];
        vb[off] = rv[u];
      }
    }
  }
}

// ---------------------------------------------------------------------------
// Compaction fused with one decode-attention step (Eq. 1) over the compacted
// cache.  One workgroup per instance reads every survivor row exactly once (the
// unmoved prefix is read but not written), stores the rows that move, and
// accumulates the G query heads' online softmax over the rows it holds in
// registers, so the decode costs no extra pass over the cache.
//
// Rows go in chunks, in ascending order.  A chunk's stores wait until every
// thread's loads of that chunk have completed (vmcnt, then a barrier): a row
// may be read and overwritten within one chunk.  The loads of the next two
// chunks are in flight meanwhile: they read rows src[j] >= j at or above the
// next chunk's first row, which no store of this or an earlier chunk touches.  The survivor map sits in LDS, so no load waits for an index.
// ---------------------------------------------------------------------------
template <typename T, int D, int G, bool CARRY>
__global__ __launch_bounds__(kCompBlock) void compact_decode_kernel(
    uint4* __restrict__ k, uint4* __restrict__ v, const int32_t* __restrict__ src, int K, int B,
    const T* __restrict__ q, T* __restrict__ out, float scale_log2, int value_kind,
    float* __restrict__ vrange) {
  constexpr int VEC = Vec16<T>::n;            // elements per 16-byte piece
  constexpr int ROW_U4 = D / VEC;             // pieces (lanes) per row
  constexpr int kRowsPerPass = kCompBlock / ROW_U4;
  constexpr int kPasses = 2;
  constexpr int CHUNK = kRowsPerPass * kPasses;
  constexpr int kWaves = kCompBlock / kWave;
  __shared__ int s_start;
  __shared__ float s_o[kWaves][G][D];
  __shared__ float s_ml[kWaves][G][2];
  extern __shared__ int s_src[];              // [K] survivor map of this instance
  const int inst = blockIdx.x;
  const int N = K + B;
  const int32_t* s = src + (size_t)inst * K;
  for (int i = threadIdx.x; i < K; i += kCompBlock) s_src[i] = clamp_slot(s[i], N);
  __syncthreads();
  if (threadIdx.x == 0) s_start = first_moved(s_src, 0, K);
  const int lane = threadIdx.x % kWave, wave = threadIdx.x / kWave;
  const int col = threadIdx.x % ROW_U4;
  const int row0 = threadIdx.x / ROW_U4;
  uint4* kb = k + (size_t)inst * N * ROW_U4;
  uint4* vb = v + (size_t)inst * N * ROW_U4;
  float qf[G][VEC];
#pragma unroll
  for (int g = 0; g < G; ++g) {
    const uint4 w = reinterpret_cast<const uint4*>(q + ((size_t)inst * G + g) * D)[col];
    Vec16<T>::unpack(w, qf[g]);
#pragma unroll
    for (int e = 0; e < VEC; ++e) qf[g][e] *= scale_log2;
  }
  float m[G], l[G], o[G][VEC];
#pragma unroll
  for (int g = 0; g < G; ++g) {
    m[g] = -1.0e30f;
    l[g] = 0.f;
#pragma unroll
    for (int e = 0; e < VEC; ++e) o[g][e] = 0.f;
  }
  __syncthreads();
  const int start = s_start;
  // register stages: chunk c in (ak, av), c+1 in (bk, bv), c+2 in (ck, cv)
  uint4 ak[kPasses], av[kPasses], bk[kPasses], bv[kPasses], ck[kPasses], cv[kPasses];
  auto load = [&](int c0, uint4 (&rk)[kPasses], uint4 (&rv)[kPasses]) {
#pragma unroll
    for (int u = 0; u < kPasses; ++u) {
      const int j = min(c0 + row0 + u * kRowsPerPass, K - 1);
      const size_t off = (size_t)s_src[j] * ROW_U4 + col;
      rk[u] = kb[off];
      rv[u] = vb[off];
    }
  };
  const int last = (K - 1) / CHUNK * CHUNK;             // first row of the last chunk
  load(0, ak, av);
  load(min(CHUNK, last), bk, bv);
  for (int c0 = 0; c0 < K; c0 += CHUNK) {
    load(min(c0 + 2 * CHUNK, last), ck, cv);           // two chunks ahead (the last repeats)
    // this thread's loads of chunk c0 are done (only the next two chunks'
    // 4*kPasses loads may remain), then every thread's are
    __builtin_amdgcn_s_waitcnt(0x0f70 | (4 * kPasses));   // vmcnt(4*kPasses)
    __syncthreads();
    // move the rows of this chunk that are not already in place
    if (c0 + CHUNK > start) {
#pragma unroll
      for (int u = 0; u < kPasses; ++u) {
        const int j = c0 + row0 + u * kRowsPerPass;
        if (j < K && j >= start) {
          const size_t off = (size_t)j * ROW_U4 + col;
          kb[off] = ak[u];
          vb[off] = av[u];
        }
      }
    }
    // decode: scores of the rows, one online-softmax update per chunk
    float sc[kPasses][G];
#pragma unroll
    for (int u = 0; u < kPasses; ++u) {
      float kf[VEC];
      Vec16<T>::unpack(ak[u], kf);
      const bool ok = c0 + row0 + u * kRowsPerPass < K;
#pragma unroll
      for (int g = 0; g < G; ++g) {
        float acc = 0.f;
#pragma unroll
        for (int e = 0; e < VEC; ++e) acc = __builtin_fmaf(qf[g][e], kf[e], acc);
        acc = lanes_sum<ROW_U4>(acc);
        sc[u][g] = ok ? acc : -INFINITY;
      }
    }
#pragma unroll
    for (int g = 0; g < G; ++g) {
      float mn = m[g];
#pragma unroll
      for (int u = 0; u < kPasses; ++u) mn = fmaxf(mn, sc[u][g]);
      const float alpha = __builtin_amdgcn_exp2f(m[g] - mn);
      l[g] *= alpha;
#pragma unroll
      for (int e = 0; e < VEC; ++e) o[g][e] *= alpha;
      m[g] = mn;
    }
#pragma unroll
    for (int u = 0; u < kPasses; ++u) {
      float vf[VEC];
      Vec16<T>::unpack(av[u], vf);
      if (CARRY) {
        // the value score of compacted row j, which the next round's candidates
        // keep unchanged (only the buffer slots are written until then)
        const float val = row_value_score<VEC, ROW_U4>(vf, value_kind);
        const int j = c0 + row0 + u * kRowsPerPass;
        if (col == 0 && j < K) vrange[(size_t)inst * K + j] = val;
      }
#pragma unroll
      for (int g = 0; g < G; ++g) {
        const float p = __builtin_amdgcn_exp2f(sc[u][g] - m[g]);
        l[g] += p;
#pragma unroll
        for (int e = 0; e < VEC; ++e) o[g][e] = __builtin_fmaf(p, vf[e], o[g][e]);
      }
    }
#pragma unroll
    for (int u = 0; u < kPasses; ++u) {
      ak[u] = bk[u];
      av[u] = bv[u];
      bk[u] = ck[u];
      bv[u] = cv[u];
    }
  }
  // merge the row groups of each wave (lane bits above log2(ROW_U4)), fixed order
#pragma unroll
  for (int off = ROW_U4; off < kWave; off <<= 1) {
#pragma unroll
    for (int g = 0; g < G; ++g) {
      const float m2 = __shfl_xor(m[g], off, kWave);
      const float l2 = __shfl_xor(l[g], off, kWave);
      const float mn = fmaxf(m[g], m2);
      const float a1 = __builtin_amdgcn_exp2f(m[g] - mn), a2 = __builtin_amdgcn_exp2f(m2 - mn);
      l[g] = l[g] * a1 + l2 * a2;
#pragma unroll
      for (int e = 0; e < VEC; ++e) {
        const float o2 = __shfl_xor(o[g][e], off, kWave);
        o[g][e] = o[g][e] * a1 + o2 * a2;
      }
      m[g] = mn;
    }
  }
  if (lane < ROW_U4) {
#pragma unroll
    for (int g = 0; g < G; ++g) {
#pragma unroll
      for (int e = 0; e < VEC; ++e) s_o[wave][g][col * VEC + e] = o[g][e];
      if (col == 0) {
        s_ml[wave][g][0] = m[g];
        s_ml[wave][g][1] = l[g];
      }
    }
  }
  __syncthreads();
  for (int t = threadIdx.x; t < G * D; t += kCompBlock) {
    const int g = t / D, dd = t % D;
    float mn = s_ml[0][g][0];
#pragma unroll
    for (int w = 1; w < kWaves; ++w) mn = fmaxf(mn, s_ml[w][g][0]);
    float lt = 0.f, ot = 0.f;
#pragma unroll
    for (int w = 0; w < kWaves; ++w) {
      const float a = __builtin_amdgcn_exp2f(s_ml[w][g][0] - mn);
      lt += s_ml[w][g][1] * a;
      ot += s_o[w][g][dd] * a;
    }
    store_out<T>(out + ((size_t)inst * G + g) * D + dd, ot / lt);
  }
}

template <typename T, int D>
hipError_t launch_cd_d(uint4* k, uint4* v, const int32_t* src, int n_inst, int K, int B, int G,
                       const void* q, void* out, int value_kind, float* vrange,
                       hipStream_t stream) {
  const float sl = 1.4426950408889634f / sqrtf((float)D);
  const T* qq = static_cast<const T*>(q);
  T* oo = static_cast<T*>(out);
#define VASE_CD(GG)                                                                          \
  case GG:                                                                                   \
    if (vrange)                                                                              \
      hipLaunchKernelGGL((compact_decode_kernel<T, D, GG, true>), dim3(n_inst),              \
                         dim3(kCompBlock), sizeof(int) * (size_t)K, stream, k, v, src, K, B, \
                         qq, oo, sl, value_kind, vrange);                                    \
    else                                                                                     \
      hipLaunchKernelGGL((compact_decode_kernel<T, D, GG, false>), dim3(n_inst),             \
                         dim3(kCompBlock), sizeof(int) * (size_t)K, stream, k, v, src, K, B, \
                         qq, oo, sl, value_kind, vrange);                                    \
    break;
  switch (G) {
    VASE_CD(1) VASE_CD(2) VASE_CD(3) VASE_CD(4) VASE_CD(5) VASE_CD(6) VASE_CD(7) VASE_CD(8)
    default: return hipErrorInvalidValue;
  }
#undef VASE_CD
  return hipGetLastError();
}

template <int ROW_U4>
hipError_t launch_rows(uint4* k, uint4* v, int n_inst, int K, int B, const int32_t* src,
                       uint4* ws, const CompactPlan& plan, hipStream_t stream) {
  if (plan.n_part > 1) {
    hipLaunchKernelGGL(compact_stage_kernel<ROW_U4>, dim3(plan.n_part - 1, n_inst),
                       dim3(kCompBlock), 0, stream, k, v, src, K, B, plan.rows_per_part,
                       plan.n_part, ws);
  }
  constexpr int kChunk = (kCompBlock / ROW_U4) * 4;
  hipLaunchKernelGGL((compact_move_kernel<ROW_U4, kChunk>), dim3(plan.n_part, n_inst),
                     dim3(kCompBlock), 0, stream, k, v, src, K, B, plan.rows_per_part,
                     plan.n_part, ws);
  return hipGetLastError();
}

}  // namespace

CompactPlan compact_plan(int dtype, int n_inst, int K, int B, int d) {
  CompactPlan pl;
  const size_t row_bytes = (size_t)d * (dtype == VASE_BF16 ? 2 : 4);
  // enough workgroups to cover the chip; parts of at least 256 rows
  int want = (1024 + n_inst - 1) / n_inst;
  int max_parts = K / 256 > 0 ? K / 256 : 1;
  pl.n_part = want < max_parts ? want : max_parts;
  if (pl.n_part < 1) pl.n_part = 1;
  pl.rows_per_part = (K + pl.n_part - 1) / pl.n_part;
  pl.n_part = (K + pl.rows_per_part - 1) / pl.rows_per_part;
  pl.bytes = pl.n_part > 1 ? (size_t)n_inst * (pl.n_part - 1) * 2 * (size_t)B * row_bytes : 0;
  return pl;
}

hipError_t launch_compact_decode(void* k, void* v, int dtype, int n_inst, int K, int B, int d,
                                 const int32_t* src, const void* q, int G, void* out,
                                 int value_kind, float* vrange, hipStream_t stream) {
  uint4* kk = static_cast<uint4*>(k);
  uint4* vv = static_cast<uint4*>(v);
  const int vk = value_kind;
  if (dtype == VASE_BF16) {
    if (d == 128) return launch_cd_d<bf16_t, 128>(kk, vv, src, n_inst, K, B, G, q, out, vk, vrange, stream);
    if (d == 64) return launch_cd_d<bf16_t, 64>(kk, vv, src, n_inst, K, B, G, q, out, vk, vrange, stream);
  } else {
    if (d == 128) return launch_cd_d<float, 128>(kk, vv, src, n_inst, K, B, G, q, out, vk, vrange, stream);
    if (d == 64) return launch_cd_d<float, 64>(kk, vv, src, n_inst, K, B, G, q, out, vk, vrange, stream);
  }
  return hipErrorInvalidValue;
}

hipError_t launch_compact(void* k, void* v, int dtype, int n_inst, int K, int B, int d,
                          const int32_t* src, void* ws, const CompactPlan& plan,
                          hipStream_t stream) {
  const int row_u4 = d * (dtype == VASE_BF16 ? 2 : 4) / 16;
  uint4* kk = static_cast<uint4*>(k);
  uint4* vv = static_cast<uint4*>(v);
  uint4* w = static_cast<uint4*>(ws);
  switch (row_u4) {
    case 8: return launch_rows<8>(kk, vv, n_inst, K, B, src, w, plan, stream);
    case 16: return launch_rows<16>(kk, vv, n_inst, K, B, src, w, plan, stream);
    case 32: return launch_rows<32>(kk, vv, n_inst, K, B, src, w, plan, stream);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace vase
