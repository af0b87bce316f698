// decode.hip -- decode attention over the compacted cache (Eq. 1 of the paper), gfx950.
//
// For each head instance, the G query heads of its GQA group attend to the same
// n_valid (k, v) rows, so each row is read from HBM once for all G queries.
// A row of d elements is spread over LPR = d*e/16 lanes (16 bytes each); a wave
// covers 64/LPR rows per load.  Each row group keeps an online softmax state in
// log2 units (scores pre-scaled by log2(e)/sqrt(d)); row groups, waves and key
// splits are merged in a fixed order, so the output is bitwise reproducible.
//
// Optionally the kernels also emit, per query head, the log-sum-exp of its
// scores over the first n_persist slots (the persistent part of Eq. (1)'s
// normaliser, which the next eviction round reuses).  Splits [0, s1) start
// below n_persist.  On the VALU path (fp32), and on the MFMA path (bf16) when
// n_persist is not a multiple of 16, none straddles it and the splits
// [s1, n_split) cover [n_persist, n_valid).  Otherwise the MFMA path has no
// such splits: the last split also takes the buffer rows [n_persist,
// n_valid), which would make one more small workgroup per instance (at one
// split per instance, half of the grid), and each of its waves keeps the
// normaliser of the rows below n_persist beside the full one.  A split's
// partial is (m, l, m_p, l_p, o[D]): the full state and the persistent one.
constexpr int kPartHead = 4;   // floats ahead of o[D] in a split's partial
#include "vase_internal.hpp"
#include "vase.h"

#include <mutex>
#include <type_traits>

namespace vase {
namespace {

// Device-resident scratch for the decode split partials of
// vase_decode_step_noalloc (callers that cannot allocate).  Each GPU the library
// runs on holds its own copy from the first use until the process ends.  In
// host code the name below is only a stand-in for the device symbol: kernels
// receive the address that hipGetSymbolAddress returns for the current device.
__device__ __align__(256) char scratch[kDecodeScratchBytes];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_lock;
void* g_scratch_ptr[kMaxDevices] = {};

constexpr int kDecBlock = 256;
constexpr int kDecWaves = kDecBlock / kWave;
constexpr float kNegBig = -1.0e30f;

constexpr float kLn2 = 0.69314718055994531f;

// natural-log LSE from a state (m, l) in scaled log2 units
__device__ __forceinline__ float lse_nat(float m, float l) {
  return (m + __builtin_amdgcn_logf(l)) * kLn2;
}

template <typename T, int D, int G, int UNROLL>
__global__ __launch_bounds__(kDecBlock) void decode_split_kernel(
    const T* __restrict__ k, const T* __restrict__ v, const T* __restrict__ q, int N,
    int n_valid, int n_persist, int s1, int rows_per_split, int n_split, float scale_log2,
    float* __restrict__ part /* [n_inst][n_split][G][kPartHead + D] */, T* __restrict__ out,
    float* __restrict__ lse, int lse_ld) {
  constexpr int VEC = Vec16<T>::n;          // elements per lane
  constexpr int LPR = D / VEC;              // lanes per row
  constexpr int RPW = kWave / LPR;          // rows per wave per load
  constexpr int RPB = RPW * kDecWaves;      // rows per block per step
  __shared__ float s_o[kDecWaves][G][D];
  __shared__ float s_ml[kDecWaves][G][2];

  const int split = blockIdx.x, inst = blockIdx.y;
  const int lane = threadIdx.x % kWave, wave = threadIdx.x / kWave;
  const int seg = lane % LPR, rg = lane / LPR;
  const int r_lo = split < s1 ? split * rows_per_split : n_persist + (split - s1) * rows_per_split;
  const int r_hi = min(split < s1 ? n_persist : n_valid, r_lo + rows_per_split);

  const uint4* kb = reinterpret_cast<const uint4*>(k + (size_t)inst * N * D);
  const uint4* vb = reinterpret_cast<const uint4*>(v + (size_t)inst * N * D);
  float qf[G][VEC];
#pragma unroll
  for (int g = 0; g < G; ++g) {
    const uint4 w = reinterpret_cast<const uint4*>(q + ((size_t)inst * G + g) * D)[seg];
    Vec16<T>::unpack(w, qf[g]);
#pragma unroll
    for (int e = 0; e < VEC; ++e) qf[g][e] *= scale_log2;
  }
  float m[G], l[G], o[G][VEC];
#pragma unroll
  for (int g = 0; g < G; ++g) {
    m[g] = kNegBig;
    l[g] = 0.f;
#pragma unroll
    for (int e = 0; e < VEC; ++e) o[g][e] = 0.f;
  }

  for (int r0 = r_lo + wave * RPW; r0 < r_hi; r0 += RPB * UNROLL) {
    uint4 kw[UNROLL], vw[UNROLL];
    bool ok[UNROLL];
#pragma unroll
    for (int u = 0; u < UNROLL; ++u) {
      const int r = r0 + u * RPB + rg;
      ok[u] = r < r_hi;
      const int rr = ok[u] ? r : r_lo;
      kw[u] = kb[(size_t)rr * LPR + seg];
      vw[u] = vb[(size_t)rr * LPR + seg];
    }
    float s[UNROLL][G];
#pragma unroll
    for (int u = 0; u < UNROLL; ++u) {
      float kf[VEC];
      Vec16<T>::unpack(kw[u], kf);
#pragma unroll
      for (int g = 0; g < G; ++g) {
        float acc = 0.f;
#pragma unroll
        for (int e = 0; e < VEC; ++e) acc = __builtin_fmaf(qf[g][e], kf[e], acc);
        acc = lanes_sum<LPR>(acc);
        s[u][g] = ok[u] ? acc : -INFINITY;
      }
    }
#pragma unroll
    for (int g = 0; g < G; ++g) {
      float mn = m[g];
#pragma unroll
      for (int u = 0; u < UNROLL; ++u) mn = fmaxf(mn, s[u][g]);
      const float alpha = __builtin_amdgcn_exp2f(m[g] - mn);
      l[g] *= alpha;
#pragma unroll
      for (int e = 0; e < VEC; ++e) o[g][e] *= alpha;
      m[g] = mn;
    }
#pragma unroll
    for (int u = 0; u < UNROLL; ++u) {
      float vf[VEC];
      Vec16<T>::unpack(vw[u], vf);
#pragma unroll
      for (int g = 0; g < G; ++g) {
        const float p = __builtin_amdgcn_exp2f(s[u][g] - m[g]);
        l[g] += p;
#pragma unroll
        for (int e = 0; e < VEC; ++e) o[g][e] = __builtin_fmaf(p, vf[e], o[g][e]);
      }
    }
  }

  // merge the RPW row groups of the wave (lane bits above log2(LPR)), fixed order
#pragma unroll
  for (int off = LPR; off < kWave; off <<= 1) {
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
  if (rg == 0) {
#pragma unroll
    for (int g = 0; g < G; ++g) {
#pragma unroll
      for (int e = 0; e < VEC; ++e) s_o[wave][g][seg * VEC + e] = o[g][e];
      if (seg == 0) {
        s_ml[wave][g][0] = m[g];
        s_ml[wave][g][1] = l[g];
      }
    }
  }
  __syncthreads();
  // merge the waves: one thread per (g, dim)
  for (int t = threadIdx.x; t < G * D; t += kDecBlock) {
    const int g = t / D, dd = t % D;
    float mn = s_ml[0][g][0];
#pragma unroll
    for (int w = 1; w < kDecWaves; ++w) mn = fmaxf(mn, s_ml[w][g][0]);
    float lt = 0.f, ot = 0.f;
#pragma unroll
    for (int w = 0; w < kDecWaves; ++w) {
      const float a = __builtin_amdgcn_exp2f(s_ml[w][g][0] - mn);
      lt += s_ml[w][g][1] * a;
      ot += s_o[w][g][dd] * a;
    }
    if (n_split == 1) {
      store_out<T>(out + ((size_t)inst * G + g) * D + dd, ot / lt);
      if (lse && dd == 0) lse[((size_t)inst * G + g) * lse_ld] = lse_nat(mn, lt);
    } else {
      // no split straddles n_persist here: a persistent split's own state is
      // its persistent part
      float* pp = part + (((size_t)inst * n_split + split) * G + g) * (kPartHead + D);
      pp[kPartHead + dd] = ot;
      if (dd == 0) {
        pp[0] = mn;
        pp[1] = lt;
        pp[2] = mn;
        pp[3] = lt;
      }
    }
  }
}

// ---------------------------------------------------------------------------
// bf16 caches: the G query heads' scores come from v_mfma_f32_16x16x32_bf16.
// A wave takes 16-row tiles of its split: the tile's K rows are the A operand
// (lane l holds row l % 16, depth [8 (l / 16), +8) of each 32-deep step, read
// straight from HBM), the queries the B operand (head l % 16, zero beyond
// G), so each lane gets 4 rows of one head.  Each head's running maximum is
// wave-uniform (a max over the 4 lanes that hold the head), and the tile's
// probabilities reach the P.V layout (lane l: 16-byte piece l % PPR of rows
// l / PPR + LG i) through a per-wave LDS tile.  P.V stays on the VALU in fp32.
// ---------------------------------------------------------------------------
typedef __bf16 dbf16x8 __attribute__((ext_vector_type(8)));
typedef float df32x4 __attribute__((ext_vector_type(4)));

template <int D, int G>
__global__ __launch_bounds__(kDecBlock) void decode_mfma_kernel(
    const uint4* __restrict__ k, const uint4* __restrict__ v, const uint4* __restrict__ q, int N,
    int n_valid, int n_persist, int s1, int rows_per_split, int n_split, float scale_log2,
    float* __restrict__ part, bf16_t* __restrict__ out, float* __restrict__ lse, int lse_ld) {
  constexpr int KS = D / 32;           // MFMA depth steps
  constexpr int PPR = D / 8;           // 16-byte pieces per row
  constexpr int LG = kWave / PPR;      // lane groups of the P.V layout
  constexpr int RPL = 16 / LG;         // tile rows per lane in the P.V layout
  static_assert(G >= 1 && G <= 16 && RPL >= 1, "shape");
  __shared__ float s_p[kDecWaves][16][16];     // [row][head]
  __shared__ float s_alpha[kDecWaves][16];
  __shared__ float s_o[kDecWaves][G][D];
  __shared__ float s_ml[kDecWaves][G][2];
  __shared__ float s_mlp[kDecWaves][G][2];   // the persistent rows' state

  const int split = blockIdx.x, inst = blockIdx.y;
  const int lane = threadIdx.x % kWave, wave = threadIdx.x / kWave;
  // when n_split = s1, split s1 - 1 also covers [n_persist, n_valid)
  const int r_lo = split < s1 ? split * rows_per_split : n_persist + (split - s1) * rows_per_split;
  const int r_hi = split == n_split - 1 ? n_valid
                                        : min(split < s1 ? n_persist : n_valid, r_lo + rows_per_split);
  const uint4* kb = k + (size_t)inst * N * PPR;
  const uint4* vb = v + (size_t)inst * N * PPR;
  const int hm = lane % 16, hq = lane / 16;    // MFMA layout
  const int pp = lane % PPR, lg = lane / PPR;  // P.V layout

  dbf16x8 bq[KS];
#pragma unroll
  for (int ks = 0; ks < KS; ++ks) {
    const uint4 w = hm < G ? q[((size_t)inst * G + hm) * PPR + 4 * ks + hq] : make_uint4(0u, 0u, 0u, 0u);
    bq[ks] = __builtin_bit_cast(dbf16x8, w);
  }
  float o[G][8];
#pragma unroll
  for (int g = 0; g < G; ++g)
#pragma unroll
    for (int e = 0; e < 8; ++e) o[g][e] = 0.f;
  float m_run = kNegBig, l_run = 0.f;          // head hm
  // the state over the rows below n_persist: a copy of the running state
  // taken at this wave's first tile at or above n_persist (a split that goes
  // past n_persist starts a multiple of 16 rows below it, so no tile straddles)
  float m_p = kNegBig, l_p = 0.f;
  bool p_open = true;

  const int n_tiles = (r_hi - r_lo + 15) / 16;
  for (int t = wave; t < n_tiles; t += kDecWaves) {
    const int row0 = r_lo + 16 * t;
    if (p_open && row0 >= n_persist) {
      m_p = m_run;
      l_p = l_run;
      p_open = false;
    }
    uint4 ka[KS], vv[RPL];
    const int rk = min(row0 + hm, r_hi - 1);
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) ka[ks] = kb[(size_t)rk * PPR + 4 * ks + hq];
#pragma unroll
    for (int i = 0; i < RPL; ++i) vv[i] = vb[(size_t)min(row0 + lg + LG * i, r_hi - 1) * PPR + pp];
    df32x4 c = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int ks = 0; ks < KS; ++ks)
      c = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(dbf16x8, ka[ks]), bq[ks], c, 0, 0, 0);
    float sc[4], tmax = -INFINITY;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      sc[i] = row0 + 4 * hq + i < r_hi ? c[i] * scale_log2 : -INFINITY;
      tmax = fmaxf(tmax, sc[i]);
    }
    tmax = fmaxf(tmax, __shfl_xor(tmax, 16, kWave));
    tmax = fmaxf(tmax, __shfl_xor(tmax, 32, kWave));
    const float m_new = fmaxf(m_run, tmax);
    const float alpha = __builtin_amdgcn_exp2f(m_run - m_new);
    m_run = m_new;
    float ps = 0.f;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const float p = __builtin_amdgcn_exp2f(sc[i] - m_new);
      ps += p;
      s_p[wave][4 * hq + i][hm] = p;
    }
    l_run = l_run * alpha + ps;
    if (hq == 0) s_alpha[wave][hm] = alpha;
    __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
    float al[G];
#pragma unroll
    for (int g = 0; g < G; ++g) al[g] = s_alpha[wave][g];
#pragma unroll
    for (int g = 0; g < G; ++g)
#pragma unroll
      for (int e = 0; e < 8; ++e) o[g][e] *= al[g];
#pragma unroll
    for (int i = 0; i < RPL; ++i) {
      float vf[8];
      Vec16<bf16_t>::unpack(vv[i], vf);
      const float* prow = s_p[wave][lg + LG * i];
#pragma unroll
      for (int g = 0; g < G; ++g) {
        const float pg = prow[g];
#pragma unroll
        for (int e = 0; e < 8; ++e) o[g][e] = __builtin_fmaf(pg, vf[e], o[g][e]);
      }
    }
    __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");   // reads done before the next tile's writes
  }
  if (p_open) {
    m_p = m_run;
    l_p = l_run;
  }
  // the head's sum over its 4 lanes; the output over the LG lane groups (same maxima)
  l_run += __shfl_xor(l_run, 16, kWave);
  l_run += __shfl_xor(l_run, 32, kWave);
  l_p += __shfl_xor(l_p, 16, kWave);
  l_p += __shfl_xor(l_p, 32, kWave);
#pragma unroll
  for (int off = PPR; off < kWave; off <<= 1)
#pragma unroll
    for (int g = 0; g < G; ++g)
#pragma unroll
      for (int e = 0; e < 8; ++e) o[g][e] += __shfl_xor(o[g][e], off, kWave);
  if (lane < G) {
    s_ml[wave][lane][0] = m_run;
    s_ml[wave][lane][1] = l_run;
    s_mlp[wave][lane][0] = m_p;
    s_mlp[wave][lane][1] = l_p;
  }
  if (lg == 0) {
#pragma unroll
    for (int g = 0; g < G; ++g)
#pragma unroll
      for (int e = 0; e < 8; ++e) s_o[wave][g][8 * pp + e] = o[g][e];
  }
  __syncthreads();
  // merge the waves: one thread per (g, dim), as in decode_split_kernel
  for (int t = threadIdx.x; t < G * D; t += kDecBlock) {
    const int g = t / D, dd = t % D;
    float mn = s_ml[0][g][0];
#pragma unroll
    for (int w = 1; w < kDecWaves; ++w) mn = fmaxf(mn, s_ml[w][g][0]);
    float lt = 0.f, ot = 0.f;
#pragma unroll
    for (int w = 0; w < kDecWaves; ++w) {
      const float a = __builtin_amdgcn_exp2f(s_ml[w][g][0] - mn);
      lt += s_ml[w][g][1] * a;
      ot += s_o[w][g][dd] * a;
    }
    float mp = 0.f, lp = 0.f;
    if (dd == 0) {
      mp = s_mlp[0][g][0];
#pragma unroll
      for (int w = 1; w < kDecWaves; ++w) mp = fmaxf(mp, s_mlp[w][g][0]);
#pragma unroll
      for (int w = 0; w < kDecWaves; ++w) lp += s_mlp[w][g][1] * __builtin_amdgcn_exp2f(s_mlp[w][g][0] - mp);
    }
    if (n_split == 1) {
      store_out<bf16_t>(out + ((size_t)inst * G + g) * D + dd, ot / lt);
      if (lse && dd == 0) lse[((size_t)inst * G + g) * lse_ld] = lse_nat(mp, lp);
    } else {
      float* pq = part + (((size_t)inst * n_split + split) * G + g) * (kPartHead + D);
      pq[kPartHead + dd] = ot;
      if (dd == 0) {
        pq[0] = mn;
        pq[1] = lt;
        pq[2] = mp;
        pq[3] = lp;
      }
    }
  }
}

template <typename T, int D>
__global__ __launch_bounds__(kDecBlock) void decode_combine_kernel(
    const float* __restrict__ part, int n_split, int s1, int G, T* __restrict__ out,
    float* __restrict__ lse, int lse_ld) {
  const int inst = blockIdx.x;
  for (int t = threadIdx.x; t < G * D; t += kDecBlock) {
    const int g = t / D, dd = t % D;
    const float* p0 = part + ((size_t)inst * n_split * G + g) * (kPartHead + D);
    const size_t stride = (size_t)G * (kPartHead + D);
    float mn = p0[0];
    for (int s = 1; s < n_split; ++s) mn = fmaxf(mn, p0[s * stride]);
    float lt = 0.f, ot = 0.f;
    for (int s = 0; s < n_split; ++s) {
      const float a = __builtin_amdgcn_exp2f(p0[s * stride] - mn);
      lt += p0[s * stride + 1] * a;
      ot += p0[s * stride + kPartHead + dd] * a;
    }
    store_out<T>(out + ((size_t)inst * G + g) * D + dd, ot / lt);
    if (lse && dd == 0) {
      // the persistent parts of the splits that start below n_persist, merged
      // in the same order
      float mp = p0[2];
      for (int s = 1; s < s1; ++s) mp = fmaxf(mp, p0[s * stride + 2]);
      float lp = 0.f;
      for (int s = 0; s < s1; ++s) lp += p0[s * stride + 3] * __builtin_amdgcn_exp2f(p0[s * stride + 2] - mp);
      lse[((size_t)inst * G + g) * lse_ld] = lse_nat(mp, lp);
    }
  }
}

struct DecodeArgs {
  const void *k, *v, *q;
  int n_inst, N, n_valid, n_persist;
  void* out;
  float* lse;
  int lse_ld;
};

template <typename T, int D, int G>
hipError_t launch_g(const DecodeArgs& a, float* ws, const DecodePlan& pl, hipStream_t stream) {
  const float scale_log2 = 1.4426950408889634f / sqrtf((float)D);
  if constexpr (std::is_same<T, bf16_t>::value) {
    hipLaunchKernelGGL((decode_mfma_kernel<D, G>), dim3(pl.n_split, a.n_inst), dim3(kDecBlock), 0,
                       stream, static_cast<const uint4*>(a.k), static_cast<const uint4*>(a.v),
                       static_cast<const uint4*>(a.q), a.N, a.n_valid, a.n_persist, pl.s1,
                       pl.rows_per_split, pl.n_split, scale_log2, ws, static_cast<T*>(a.out),
                       a.lse, a.lse_ld);
  } else {
    hipLaunchKernelGGL((decode_split_kernel<T, D, G, 4>), dim3(pl.n_split, a.n_inst),
                       dim3(kDecBlock), 0, stream, static_cast<const T*>(a.k),
                       static_cast<const T*>(a.v), static_cast<const T*>(a.q), a.N, a.n_valid,
                       a.n_persist, pl.s1, pl.rows_per_split, pl.n_split, scale_log2, ws,
                       static_cast<T*>(a.out), a.lse, a.lse_ld);
  }
  if (pl.n_split > 1) {
    hipLaunchKernelGGL((decode_combine_kernel<T, D>), dim3(a.n_inst), dim3(kDecBlock), 0, stream,
                       ws, pl.n_split, pl.s1, G, static_cast<T*>(a.out), a.lse, a.lse_ld);
  }
  return hipGetLastError();
}

template <typename T, int D>
hipError_t launch_d(const DecodeArgs& a, int G, float* ws, const DecodePlan& pl, hipStream_t s) {
  switch (G) {
    case 1: return launch_g<T, D, 1>(a, ws, pl, s);
    case 2: return launch_g<T, D, 2>(a, ws, pl, s);
    case 3: return launch_g<T, D, 3>(a, ws, pl, s);
    case 4: return launch_g<T, D, 4>(a, ws, pl, s);
    case 5: return launch_g<T, D, 5>(a, ws, pl, s);
    case 6: return launch_g<T, D, 6>(a, ws, pl, s);
    case 7: return launch_g<T, D, 7>(a, ws, pl, s);
    case 8: return launch_g<T, D, 8>(a, ws, pl, s);
    default: return hipErrorInvalidValue;
  }
}

// Append one token and cache its query: rows K + pos of k and v take k_new and
// v_new, and q_win[inst][g][pos % w] takes q[inst][g] (byte copies).
__global__ __launch_bounds__(256) void decode_append_kernel(
    uint4* __restrict__ k, uint4* __restrict__ v, const uint4* __restrict__ k_new,
    const uint4* __restrict__ v_new, const uint4* __restrict__ q, uint4* __restrict__ q_win,
    int N, int slot, int G, int w, int ring, int row_u4) {
  const int inst = blockIdx.x;
  for (int t = threadIdx.x; t < (2 + G) * row_u4; t += 256) {
    const int r = t / row_u4, c = t % row_u4;
    if (r == 0) k[((size_t)inst * N + slot) * row_u4 + c] = k_new[(size_t)inst * row_u4 + c];
    else if (r == 1) v[((size_t)inst * N + slot) * row_u4 + c] = v_new[(size_t)inst * row_u4 + c];
    else {
      const int g = r - 2;
      q_win[(((size_t)inst * G + g) * w + ring) * row_u4 + c] = q[((size_t)inst * G + g) * row_u4 + c];
    }
  }
}

}  // namespace

namespace {
// key splits for n_valid rows: at least 4096 workgroups over the chip (one
// workgroup per instance leaves the last of ~2.25 dispatch waves a quarter
// full at 2304 instances; two splits cut a step from 1.10 to 0.87 ms there),
// at least 256 rows per split; non-decreasing in n_valid
int decode_n0(int n_inst, int n_valid) {
  const int want = (4096 + n_inst - 1) / n_inst;
  const int max_split = n_valid / 256 > 0 ? n_valid / 256 : 1;
  const int n0 = want < max_split ? want : max_split;
  return n0 < 1 ? 1 : n0;
}
}  // namespace

DecodePlan decode_plan(int dtype, int n_inst, int K, int B, int d, int G, int n_valid,
                       int n_persist) {
  DecodePlan pl;
  const int n0 = decode_n0(n_inst, n_valid);
  // splits [0, s1) start below n_persist.  The MFMA path puts [n_persist,
  // n_valid) into the last of them when the 16-row tiles of that split meet
  // n_persist at a tile boundary (splits of a multiple of 16 rows, n_persist a
  // multiple of 16); otherwise, and on the VALU path, into splits of its own
  const bool fold = dtype == VASE_BF16 && n_persist % 16 == 0;
  pl.rows_per_split = (n_valid + n0 - 1) / n0;
  if (fold) pl.rows_per_split = (pl.rows_per_split + 15) / 16 * 16;
  pl.s1 = (n_persist + pl.rows_per_split - 1) / pl.rows_per_split;
  pl.n_split =
      fold ? pl.s1 : pl.s1 + (n_valid - n_persist + pl.rows_per_split - 1) / pl.rows_per_split;
  pl.bytes =
      pl.n_split > 1 ? (size_t)n_inst * pl.n_split * G * (kPartHead + d) * sizeof(float) : 0;
  (void)K; (void)B;
  return pl;
}

size_t decode_ws_bytes_max(int dtype, int n_inst, int K, int B, int d, int G) {
  // n_split <= ceil(n_persist / rps) + ceil((n_valid - n_persist) / rps)
  //         <= n0(n_valid) + 1 <= n0(N) + 1 for every n_valid <= N
  (void)dtype;
  const int n0 = decode_n0(n_inst, K + B);
  return (size_t)n_inst * (n0 + 1) * G * (kPartHead + d) * sizeof(float);
}

hipError_t launch_decode(const void* k, const void* v, const void* q, int dtype, int n_inst,
                         int K, int B, int d, int G, int n_valid, int n_persist, void* out,
                         float* lse, int lse_ld, void* ws, const DecodePlan& plan,
                         hipStream_t stream) {
  const DecodeArgs a{k, v, q, n_inst, K + B, n_valid, n_persist, out, lse, lse_ld};
  float* w = static_cast<float*>(ws);
  if (dtype == VASE_BF16) {
    if (d == 128) return launch_d<bf16_t, 128>(a, G, w, plan, stream);
    if (d == 64) return launch_d<bf16_t, 64>(a, G, w, plan, stream);
  } else {
    if (d == 128) return launch_d<float, 128>(a, G, w, plan, stream);
    if (d == 64) return launch_d<float, 64>(a, G, w, plan, stream);
  }
  return hipErrorInvalidValue;
}

hipError_t decode_scratch(void** ptr) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> g(g_scratch_lock);
  if (!g_scratch_ptr[dev]) {
    // once per device, with that device current: the device copy's address
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    if (!p) return hipErrorInvalidSymbol;
    g_scratch_ptr[dev] = p;
  }
  *ptr = g_scratch_ptr[dev];
  return hipSuccess;
}

hipError_t launch_decode_append(void* k, void* v, const void* k_new, const void* v_new,
                                const void* q, void* q_win, int dtype, int n_inst, int K, int B,
                                int d, int G, int w, int pos, hipStream_t stream) {
  const int row_u4 = d * (dtype == VASE_BF16 ? 2 : 4) / 16;
  hipLaunchKernelGGL(decode_append_kernel, dim3(n_inst), dim3(256), 0, stream,
                     static_cast<uint4*>(k), static_cast<uint4*>(v),
                     static_cast<const uint4*>(k_new), static_cast<const uint4*>(v_new),
                     static_cast<const uint4*>(q), static_cast<uint4*>(q_win), K + B, K + pos, G, w,
                     pos % w, row_u4);
  return hipGetLastError();
}

}  // namespace vase
