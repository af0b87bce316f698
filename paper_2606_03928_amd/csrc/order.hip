// order.hip -- the cache under an order map (gfx950).
//
// Under periodic eviction (Sec. 2) the cache returns to K persistent slots after
// every round.  A stable compaction keeps the slots in temporal order, which
// moves every survivor behind the first evicted slot.  With an order map the
// survivors stay where they are:
//
//   ord[inst][t]  physical slot of the persistent token of temporal rank t
//                 (t < K, oldest first); buffer token K + b is in slot K + b
//
// and the round only copies the B buffer rows into the B slots that the evicted
// tokens leave.  Read through the map, the cache is the temporal cache
// T[t] = X[ord[t]], and every step of the round sees exactly that cache:
//   * scores are computed per physical slot (a row's softmax and a slot's
//     column sum do not depend on where the slot sits) and then put into
//     temporal order, where the average pooling of the Sec. 2 footnote runs
//     over temporal neighbours (order_scores_kernel);
//   * selection works on temporal ranks, as it does on a stable cache;
//   * compaction: with e_0 < .. < e_{B-1} the evicted ranks, buffer row K + b
//     goes to slot ord[e_b], and the new map is ord[src[j]] for the K - B
//     surviving ranks followed by ord[e_0 .. e_{B-1}] (compact_map_kernel);
//   * decode attention (Eq. 1) sums over the K slots in any order.
#include "vase_internal.hpp"
#include "vase.h"

#include <type_traits>

namespace vase {
namespace {

constexpr int kOrdBlock = 256;
constexpr int kOrdTile = 256;
constexpr int kOrdMaxHalo = 127;

__device__ __forceinline__ int clampi(int x, int lo, int hi) { return x < lo ? lo : (x > hi ? hi : x); }

// attn_out[t]   = (1/P) sum_{u = t - P/2}^{t + P/2} (0 <= u < K ? attn_phys[ord[u]] : 0)
// vrange_out[t] = vrange_phys[ord[t]]
// With attn_phys the unpooled window mean of each slot, the terms are added in
// the same order as a pooled score over a temporally ordered cache.
__global__ __launch_bounds__(kOrdBlock) void order_scores_kernel(
    const float* __restrict__ attn_phys, const float* __restrict__ vr_phys,
    const int32_t* __restrict__ ord, int K, int pool, float* __restrict__ attn_out,
    float* __restrict__ vr_out) {
  __shared__ float tile[kOrdTile + 2 * kOrdMaxHalo];
  const int inst = blockIdx.y;
  const int i0 = blockIdx.x * kOrdTile;
  const int h = pool / 2;
  const int32_t* o = ord + (size_t)inst * K;
  const float* a = attn_phys + (size_t)inst * K;
  for (int t = threadIdx.x; t < kOrdTile + 2 * h; t += kOrdBlock) {
    const int u = i0 - h + t;
    tile[t] = (u >= 0 && u < K) ? a[clampi(o[u], 0, K - 1)] : 0.f;
  }
  __syncthreads();
  const int i = i0 + threadIdx.x;
  if (i >= K) return;
  float s = 0.f;
  for (int t = 0; t < pool; ++t) s += tile[threadIdx.x + t];
  attn_out[(size_t)inst * K + i] = s / (float)pool;
  if (vr_phys) vr_out[(size_t)inst * K + i] = vr_phys[(size_t)inst * K + clampi(o[i], 0, K - 1)];
}

// ---------------------------------------------------------------------------
// The new order map of one instance, in LDS (16-bit slots and ranks: K <= 8192).
//   on entry  sa = src (clamped to [0, K)), sb = ord (clamped to [0, K))
//   on exit   sa = the new map, also written to ord_g; sb[slot] = its rank
// A rank e between survivors src[j-1] and src[j] (j survivors below it) is the
// (e - j)-th evicted one.  Every index is clamped, so a map that breaks the
// contract gives unspecified results but no access outside the instance.
// ---------------------------------------------------------------------------
template <int NT>
__device__ void build_order_map(uint16_t* sa, uint16_t* sb, int K, int B, int32_t* ord_g) {
  constexpr int kMapPer = VASE_MAX_K / NT;
  const int M = K - B;
  const int tid = threadIdx.x;
  int keep[kMapPer];
#pragma unroll
  for (int u = 0; u < kMapPer; ++u) {
    const int j = tid + u * NT;
    keep[u] = j < M ? sb[sa[j]] : 0;
  }
  // reads of sa stay below M, writes go to [M, K)
  for (int j = tid; j <= M; j += NT) {
    const int lo = j == 0 ? 0 : sa[j - 1] + 1;
    const int hi = j == M ? K : sa[j];
    for (int e = lo; e < hi; ++e) {
      const int b = e - j;
      if (b >= 0 && b < B) sa[M + b] = sb[e];
    }
  }
  __syncthreads();
#pragma unroll
  for (int u = 0; u < kMapPer; ++u) {
    const int j = tid + u * NT;
    if (j < M) sa[j] = (uint16_t)keep[u];
  }
  __syncthreads();
  for (int i = tid; i < K; i += NT) {
    const int sl = sa[i];
    ord_g[i] = sl;
    sb[sl] = (uint16_t)i;
  }
  __syncthreads();
}

template <int NT>
__device__ __forceinline__ void load_maps(uint16_t* sa, uint16_t* sb, const int32_t* src_g,
                                          const int32_t* ord_g, int K) {
  for (int i = threadIdx.x; i < K; i += NT) {
    sa[i] = (uint16_t)clampi(src_g[i], 0, K - 1);
    sb[i] = (uint16_t)clampi(ord_g[i], 0, K - 1);
  }
  __syncthreads();
}

// Compaction alone: the new map, then the B buffer rows into their slots.
// CARRY 1: also the value score of every rank's row (the next round's
// candidates), the survivors' rows read in place; CARRY 2: a survivor keeps the
// score of its old rank from vrange_in (its row has not changed; the output may
// be the input) and only the B buffer rows are scored, from the rows the copy
// holds.
template <typename T, int D, int CARRY>
__global__ __launch_bounds__(kOrdBlock) void compact_map_kernel(
    uint4* __restrict__ k, uint4* __restrict__ v, const int32_t* __restrict__ src,
    int32_t* __restrict__ ord, int K, int B, int value_kind, const float* vrange_in,
    float* vrange) {
  constexpr int VEC = Vec16<T>::n;
  constexpr int ROW_U4 = D / VEC;
  static_assert(kOrdBlock % ROW_U4 == 0 && kWave % ROW_U4 == 0, "a row's lanes share one wave");
  extern __shared__ uint16_t s_map[];
  uint16_t* sa = s_map;
  uint16_t* sb = s_map + K;
  const int inst = blockIdx.x;
  const int N = K + B, M = K - B;
  int32_t* og = ord + (size_t)inst * K;
  float* vr = CARRY != 0 ? vrange + (size_t)inst * K : nullptr;
  load_maps<kOrdBlock>(sa, sb, src + (size_t)inst * K, og, K);
  // survivor j's score, read before the barriers of the map build and written
  // after them
  constexpr int kGather = VASE_MAX_K / kOrdBlock;
  float gv[kGather];
  if (CARRY == 2) {
#pragma unroll
    for (int u = 0; u < kGather; ++u) {
      const int j = threadIdx.x + u * kOrdBlock;
      gv[u] = j < M ? vrange_in[(size_t)inst * K + sa[j]] : 0.f;
    }
  }
  build_order_map<kOrdBlock>(sa, sb, K, B, og);
  if (CARRY == 2) {
#pragma unroll
    for (int u = 0; u < kGather; ++u) {
      const int j = threadIdx.x + u * kOrdBlock;
      if (j < M) vr[j] = gv[u];
    }
  }
  uint4* kb = k + (size_t)inst * N * ROW_U4;
  uint4* vb = v + (size_t)inst * N * ROW_U4;
  // whole rows per pass (kOrdBlock is a multiple of ROW_U4), so the lanes of a
  // row are together for its score
  for (int e = threadIdx.x; e < B * ROW_U4; e += kOrdBlock) {
    const int b = e / ROW_U4, c = e % ROW_U4;
    const size_t from = (size_t)(K + b) * ROW_U4 + c;
    const size_t to = (size_t)sa[M + b] * ROW_U4 + c;
    const uint4 kv = kb[from], vv = vb[from];
    kb[to] = kv;
    vb[to] = vv;
    if (CARRY != 0) {
      float f[VEC];
      Vec16<T>::unpack(vv, f);
      const float val = row_value_score<VEC, ROW_U4>(f, value_kind);
      if (c == 0) vr[M + b] = val;
    }
  }
  if (CARRY == 1) {
    // the survivors' rows, each in its slot sa[j]
    for (int e = threadIdx.x; e < M * ROW_U4; e += kOrdBlock) {
      const int j = e / ROW_U4, c = e % ROW_U4;
      float f[VEC];
      Vec16<T>::unpack(vb[(size_t)sa[j] * ROW_U4 + c], f);
      const float val = row_value_score<VEC, ROW_U4>(f, value_kind);
      if (c == 0) vr[j] = val;
    }
  }
}

// ---------------------------------------------------------------------------
// Compaction under the order map fused with one decode step (Eq. 1) over the K
// persistent slots.  One workgroup per instance builds the new map, then
// streams the K slots in chunks: slot s holds a survivor (read in place) or,
// if it was evicted, receives buffer row K + (rank - (K - B)), which is read
// from the buffer and stored to s.  Stores only reach evicted slots, which no
// load of this kernel reads, so loads run ahead freely (three chunks in
// registers) with no barrier between chunks.  The G heads' online softmax and
// output accumulate from the rows in registers, as in the stable kernel, and
// with CARRY each row's value score is written at its temporal rank.
// ---------------------------------------------------------------------------
template <typename T, int D, int G, bool CARRY>
__global__ __launch_bounds__(kOrdBlock) void compact_map_decode_kernel(
    uint4* __restrict__ k, uint4* __restrict__ v, const int32_t* __restrict__ src,
    int32_t* __restrict__ ord, int K, int B, const T* __restrict__ q, T* __restrict__ out,
    float scale_log2, int value_kind, float* __restrict__ vrange) {
  constexpr int VEC = Vec16<T>::n;
  constexpr int ROW_U4 = D / VEC;
  constexpr int kRowsPerPass = kOrdBlock / ROW_U4;
  constexpr int kPasses = 2;
  constexpr int CHUNK = kRowsPerPass * kPasses;
  constexpr int kWaves = kOrdBlock / kWave;
  __shared__ float s_o[kWaves][G][D];
  __shared__ float s_ml[kWaves][G][2];
  extern __shared__ uint16_t s_map[];
  uint16_t* sa = s_map;
  uint16_t* sb = s_map + K;
  const int inst = blockIdx.x;
  const int N = K + B, M = K - B;
  int32_t* og = ord + (size_t)inst * K;
  load_maps<kOrdBlock>(sa, sb, src + (size_t)inst * K, og, K);
  build_order_map<kOrdBlock>(sa, sb, K, B, og);

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
  // the row that slot s holds after compaction
  auto source = [&](int s) {
    const int t = sb[s];
    return t >= M ? K + (t - M) : s;
  };
  uint4 ak[kPasses], av[kPasses], bk[kPasses], bv[kPasses], ck[kPasses], cv[kPasses];
  auto load = [&](int c0, uint4 (&rk)[kPasses], uint4 (&rv)[kPasses]) {
#pragma unroll
    for (int u = 0; u < kPasses; ++u) {
      const int s = min(c0 + row0 + u * kRowsPerPass, K - 1);
      const size_t off = (size_t)source(s) * ROW_U4 + col;
      rk[u] = kb[off];
      rv[u] = vb[off];
    }
  };
  const int last = (K - 1) / CHUNK * CHUNK;
  load(0, ak, av);
  load(min(CHUNK, last), bk, bv);
  for (int c0 = 0; c0 < K; c0 += CHUNK) {
    load(min(c0 + 2 * CHUNK, last), ck, cv);
#pragma unroll
    for (int u = 0; u < kPasses; ++u) {
      const int s = c0 + row0 + u * kRowsPerPass;
      if (s < K && sb[s] >= M) {
        const size_t off = (size_t)s * ROW_U4 + col;
        kb[off] = ak[u];
        vb[off] = av[u];
      }
    }
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
        // value score of the row at its temporal rank: the next round's
        // candidates, unchanged until then (only buffer slots are written)
        const float val = row_value_score<VEC, ROW_U4>(vf, value_kind);
        const int s = c0 + row0 + u * kRowsPerPass;
        if (col == 0 && s < K) vrange[(size_t)inst * K + sb[s]] = val;
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
  // merge the row groups of each wave, then the waves, in a fixed order
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
  for (int t = threadIdx.x; t < G * D; t += kOrdBlock) {
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

// ---------------------------------------------------------------------------
// bf16: the same compaction and decode step with the scores on MFMA.  One
// workgroup per instance; a wave takes 16-row tiles.  The tile's K rows are the
// A operand of v_mfma_f32_16x16x32_bf16 (lane l: row l % 16, depth
// [8(l/16), +8) of each 32-deep step, 64 contiguous bytes per row per load) and
// the G queries the B operand (zero beyond G), so four MFMAs (d = 128) give
// every head's scores of the tile.  The probabilities go through a per-wave LDS
// tile into the P.V layout (lane l: 16-byte piece l % (d/8) of rows
// l / (d/8) + 64/(d/8) * i), where P.V runs on the VALU in fp32.
// The tiles are the K slots read in place, then the B buffer rows; an evicted
// slot's row is masked out of the softmax, so no load waits for the maps.  The
// buffer rows are copied to the evicted slots after the decode step, as the
// workgroup's last action.  With dlog given (the logits q_g . k_t that the
// score kernel wrote while it streamed the same rows, bit for bit what the
// MFMAs here produce) the tiles read no K rows at all: only V and the logits.
// ---------------------------------------------------------------------------
typedef __bf16 mbf16x8 __attribute__((ext_vector_type(8)));
typedef float mf32x4 __attribute__((ext_vector_type(4)));
constexpr int kMapBlock = 512;
constexpr int kMapWaves = kMapBlock / kWave;
constexpr int kMapMfmaMaxG = 8;

// CARRY: 0 no value scores; 1 every row scored from V; 2 the survivors' scores
// gathered by rank from vrange_in (the scores the selection used: a row that
// survives does not change) and only the buffer rows scored from V
// LOGITS: the scores come from dlog instead of the K rows
template <int D, int G, int CARRY, bool LOGITS>
__global__ __launch_bounds__(kMapBlock) void compact_map_mfma_kernel(
    uint4* __restrict__ k, uint4* __restrict__ v, const int32_t* __restrict__ src,
    int32_t* __restrict__ ord, int K, int B, const uint4* __restrict__ q,
    bf16_t* __restrict__ out, float scale_log2, int value_kind, const float* vrange_in,
    float* vrange, const float* __restrict__ dlog) {
  constexpr int KS = D / 32;           // MFMA depth steps
  constexpr int PPR = D / 8;           // 16-byte pieces per row
  constexpr int LG = kWave / PPR;      // lane groups of the P.V layout
  constexpr int RPL = 16 / LG;         // tile rows per lane in the P.V layout
  static_assert(G >= 1 && G <= 16 && RPL >= 1, "shape");
  __shared__ float s_p[kMapWaves][16][16];     // [row][head]
  __shared__ float s_alpha[kMapWaves][16];
  __shared__ float s_o[kMapWaves][G][D];
  __shared__ float s_ml[kMapWaves][G][2];
  __shared__ uint4 s_q[16][PPR];               // the B operand: G query rows, zero below
  extern __shared__ uint16_t s_map[];
  uint16_t* sa = s_map;
  uint16_t* sb = s_map + K;
  const int inst = blockIdx.x;
  const int N = K + B, M = K - B;
  int32_t* og = ord + (size_t)inst * K;
  for (int i = threadIdx.x; i < 16 * PPR; i += kMapBlock)
    s_q[i / PPR][i % PPR] = i / PPR < G ? q[((size_t)inst * G + i / PPR) * PPR + i % PPR]
                                        : make_uint4(0u, 0u, 0u, 0u);
  load_maps<kMapBlock>(sa, sb, src + (size_t)inst * K, og, K);
  // survivor j keeps the value score of its old rank src[j]; every thread reads
  // its share before the barriers of the map build, and writes after them (the
  // output may be the input)
  constexpr int kGather = VASE_MAX_K / kMapBlock;
  float gv[kGather];
  if (CARRY == 2) {
#pragma unroll
    for (int u = 0; u < kGather; ++u) {
      const int j = threadIdx.x + u * kMapBlock;
      gv[u] = j < M ? vrange_in[(size_t)inst * K + sa[j]] : 0.f;
    }
  }
  build_order_map<kMapBlock>(sa, sb, K, B, og);
  if (CARRY == 2) {
#pragma unroll
    for (int u = 0; u < kGather; ++u) {
      const int j = threadIdx.x + u * kMapBlock;
      if (j < M) vrange[(size_t)inst * K + j] = gv[u];
    }
  }

  const int lane = threadIdx.x % kWave, wave = threadIdx.x / kWave;
  uint4* kb = k + (size_t)inst * N * PPR;
  uint4* vb = v + (size_t)inst * N * PPR;
  const int hm = lane % 16, hq = lane / 16;    // MFMA layout
  // head hm's logits (heads >= G read head G - 1's; their scores are dropped)
  const float* dli = LOGITS ? dlog + ((size_t)inst * G + min(hm, G - 1)) * N : nullptr;
  const int pp = lane % PPR, lg = lane / PPR;  // P.V layout
  float o[G][8];
#pragma unroll
  for (int g = 0; g < G; ++g)
#pragma unroll
    for (int e = 0; e < 8; ++e) o[g][e] = 0.f;
  float m_run = -1.0e30f, l_run = 0.f;         // head hm

  // Tiles [0, n_slot): the K slots, each read in place; a slot whose token was
  // evicted is left out of the softmax.  Tiles [n_slot, n_slot + n_buf): the B
  // buffer rows, which also go to the evicted slots (sa[M + b]).  No load
  // address depends on the maps.
  const int n_slot = (K + 15) / 16, n_buf = (B + 15) / 16;
  for (int t = wave; t < n_slot + n_buf; t += kMapWaves) {
    const bool buf = t >= n_slot;
    const int r0 = buf ? K + 16 * (t - n_slot) : 16 * t;     // first row of the tile
    const int r_end = buf ? N : K;
    uint4 ka[KS], vv[RPL];
    mf32x4 c = {0.f, 0.f, 0.f, 0.f};
    if constexpr (LOGITS) {
#pragma unroll
      for (int i = 0; i < 4; ++i) c[i] = dli[min(r0 + 4 * hq + i, N - 1)];
    } else {
      const int rk = min(r0 + hm, r_end - 1);
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) ka[ks] = kb[(size_t)rk * PPR + 4 * ks + hq];
    }
#pragma unroll
    for (int i = 0; i < RPL; ++i) vv[i] = vb[(size_t)min(r0 + lg + LG * i, r_end - 1) * PPR + pp];
    if constexpr (!LOGITS) {
#pragma unroll
      for (int ks = 0; ks < KS; ++ks)
        c = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(mbf16x8, ka[ks]),
                                                    __builtin_bit_cast(mbf16x8, s_q[hm][4 * ks + hq]),
                                                    c, 0, 0, 0);
    }
    float sc[4], tmax = -INFINITY;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int r = r0 + 4 * hq + i;
      const bool live = buf ? r < N : (r < K && sb[r] < M);
      sc[i] = live ? c[i] * scale_log2 : -INFINITY;
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
      if (CARRY == 1 || (CARRY == 2 && buf)) {
        // value score of the row at its new temporal rank (the next round's
        // candidates): a surviving slot's rank, or M + b for buffer row K + b
        const float val = row_value_score<8, PPR>(vf, value_kind);
        const int r = r0 + lg + LG * i;
        if (pp == 0) {
          if (buf) {
            if (r < N) vrange[(size_t)inst * K + M + (r - K)] = val;
          } else if (r < K && sb[r] < M) {
            vrange[(size_t)inst * K + sb[r]] = val;
          }
        }
      }
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
  // the head's sum over its 4 lanes; the output over the LG lane groups (same maxima)
  l_run += __shfl_xor(l_run, 16, kWave);
  l_run += __shfl_xor(l_run, 32, kWave);
#pragma unroll
  for (int off = PPR; off < kWave; off <<= 1)
#pragma unroll
    for (int g = 0; g < G; ++g)
#pragma unroll
      for (int e = 0; e < 8; ++e) o[g][e] += __shfl_xor(o[g][e], off, kWave);
  if (lane < G) {
    s_ml[wave][lane][0] = m_run;
    s_ml[wave][lane][1] = l_run;
  }
  if (lg == 0) {
#pragma unroll
    for (int g = 0; g < G; ++g)
#pragma unroll
      for (int e = 0; e < 8; ++e) s_o[wave][g][8 * pp + e] = o[g][e];
  }
  __syncthreads();
  // merge the waves in a fixed order: one thread per (head, dimension)
  for (int t = threadIdx.x; t < G * D; t += kMapBlock) {
    const int g = t / D, dd = t % D;
    float mn = s_ml[0][g][0];
#pragma unroll
    for (int w = 1; w < kMapWaves; ++w) mn = fmaxf(mn, s_ml[w][g][0]);
    float lt = 0.f, ot = 0.f;
#pragma unroll
    for (int w = 0; w < kMapWaves; ++w) {
      const float a = __builtin_amdgcn_exp2f(s_ml[w][g][0] - mn);
      lt += s_ml[w][g][1] * a;
      ot += s_o[w][g][dd] * a;
    }
    store_out<bf16_t>(out + ((size_t)inst * G + g) * D + dd, ot / lt);
  }
  // last: the buffer rows into the evicted slots (whole rows, from L2).  Stores
  // are counted by vmcnt, so issued inside the stream they would hold up the
  // loads behind them; here nothing waits for them.
  for (int e = threadIdx.x; e < B * PPR; e += kMapBlock) {
    const int b = e / PPR, c = e % PPR;
    const size_t from = (size_t)(K + b) * PPR + c;
    const size_t to = (size_t)sa[M + b] * PPR + c;
    kb[to] = kb[from];
    vb[to] = vb[from];
  }
}

template <int D>
hipError_t launch_cmm_d(uint4* k, uint4* v, const int32_t* src, int32_t* ord, int n_inst, int K,
                        int B, int G, const void* q, void* out, int value_kind,
                        const float* vrange_in, float* vrange, const float* dlog,
                        hipStream_t stream) {
  const float sl = 1.4426950408889634f / sqrtf((float)D);
  const uint4* qq = static_cast<const uint4*>(q);
  bf16_t* oo = static_cast<bf16_t*>(out);
  const size_t lds = 2 * sizeof(uint16_t) * (size_t)K;
#define VASE_CMM_L(GG, LG)                                                                 \
  if (vrange && vrange_in)                                                                 \
    hipLaunchKernelGGL((compact_map_mfma_kernel<D, GG, 2, LG>), dim3(n_inst), dim3(kMapBlock), \
                       lds, stream, k, v, src, ord, K, B, qq, oo, sl, value_kind, vrange_in, \
                       vrange, dlog);                                                      \
  else if (vrange)                                                                         \
    hipLaunchKernelGGL((compact_map_mfma_kernel<D, GG, 1, LG>), dim3(n_inst), dim3(kMapBlock), \
                       lds, stream, k, v, src, ord, K, B, qq, oo, sl, value_kind, vrange_in, \
                       vrange, dlog);                                                      \
  else                                                                                     \
    hipLaunchKernelGGL((compact_map_mfma_kernel<D, GG, 0, LG>), dim3(n_inst), dim3(kMapBlock), \
                       lds, stream, k, v, src, ord, K, B, qq, oo, sl, value_kind, vrange_in, \
                       vrange, dlog);
#define VASE_CMM(GG)                                                                       \
  case GG:                                                                                 \
    if (dlog) {                                                                            \
      VASE_CMM_L(GG, true)                                                                 \
    } else {                                                                               \
      VASE_CMM_L(GG, false)                                                                \
    }                                                                                      \
    break;
  switch (G) {
    VASE_CMM(1) VASE_CMM(2) VASE_CMM(3) VASE_CMM(4) VASE_CMM(5) VASE_CMM(6) VASE_CMM(7) VASE_CMM(8)
    default: return hipErrorInvalidValue;
  }
#undef VASE_CMM_L
#undef VASE_CMM
  return hipGetLastError();
}

template <typename T, int D>
hipError_t launch_cmd_d(uint4* k, uint4* v, const int32_t* src, int32_t* ord, int n_inst, int K,
                        int B, int G, const void* q, void* out, int value_kind, float* vrange,
                        hipStream_t stream) {
  const float sl = 1.4426950408889634f / sqrtf((float)D);
  const T* qq = static_cast<const T*>(q);
  T* oo = static_cast<T*>(out);
  const size_t lds = 2 * sizeof(uint16_t) * (size_t)K;
#define VASE_CMD(GG)                                                                       \
  case GG:                                                                                 \
    if (vrange)                                                                            \
      hipLaunchKernelGGL((compact_map_decode_kernel<T, D, GG, true>), dim3(n_inst),        \
                         dim3(kOrdBlock), lds, stream, k, v, src, ord, K, B, qq, oo, sl,   \
                         value_kind, vrange);                                              \
    else                                                                                   \
      hipLaunchKernelGGL((compact_map_decode_kernel<T, D, GG, false>), dim3(n_inst),       \
                         dim3(kOrdBlock), lds, stream, k, v, src, ord, K, B, qq, oo, sl,   \
                         value_kind, vrange);                                              \
    break;
  switch (G) {
    VASE_CMD(1) VASE_CMD(2) VASE_CMD(3) VASE_CMD(4) VASE_CMD(5) VASE_CMD(6) VASE_CMD(7) VASE_CMD(8)
    default: return hipErrorInvalidValue;
  }
#undef VASE_CMD
  return hipGetLastError();
}

}  // namespace

hipError_t launch_order_scores(const float* attn_phys, const float* vr_phys, const int32_t* ord,
                               int n_inst, int K, int pool, float* attn_out, float* vr_out,
                               hipStream_t stream) {
  hipLaunchKernelGGL(order_scores_kernel, dim3((K + kOrdTile - 1) / kOrdTile, n_inst),
                     dim3(kOrdBlock), 0, stream, attn_phys, vr_phys, ord, K, pool, attn_out,
                     vr_out);
  return hipGetLastError();
}

hipError_t launch_compact_map(void* k, void* v, int dtype, int n_inst, int K, int B, int d,
                              const int32_t* src, int32_t* ord, const void* q, int G, void* out,
                              int value_kind, const float* vrange_in, float* vrange,
                              const float* dlog, hipStream_t stream) {
  uint4* kk = static_cast<uint4*>(k);
  uint4* vv = static_cast<uint4*>(v);
  if (!q) {
    const size_t lds = 2 * sizeof(uint16_t) * (size_t)K;
    const int carry = vrange ? (vrange_in ? 2 : 1) : 0;
    auto go = [&](auto t_, auto d_) {
      using T = decltype(t_);
      constexpr int D = decltype(d_)::value;
      auto kern = carry == 2 ? compact_map_kernel<T, D, 2>
                  : carry == 1 ? compact_map_kernel<T, D, 1> : compact_map_kernel<T, D, 0>;
      hipLaunchKernelGGL(kern, dim3(n_inst), dim3(kOrdBlock), lds, stream, kk, vv, src, ord, K, B,
                         value_kind, vrange_in, vrange);
      return hipGetLastError();
    };
    using I64 = std::integral_constant<int, 64>;
    using I128 = std::integral_constant<int, 128>;
    if (dtype == VASE_BF16) return d == 128 ? go(bf16_t{}, I128{}) : d == 64 ? go(bf16_t{}, I64{}) : hipErrorInvalidValue;
    return d == 128 ? go(float{}, I128{}) : d == 64 ? go(float{}, I64{}) : hipErrorInvalidValue;
  }
  const int vk = value_kind;
  // supplied logits: the MFMA kernel only
  if (dlog && !(dtype == VASE_BF16 && G <= kMapMfmaMaxG)) return hipErrorInvalidValue;
  if (dtype == VASE_BF16) {
    // scores on MFMA for every group the entry point takes (at G = 8 the heads'
    // outputs hold the kernel at 171 VGPRs, one workgroup per CU)
    if (G <= kMapMfmaMaxG) {
      if (d == 128) return launch_cmm_d<128>(kk, vv, src, ord, n_inst, K, B, G, q, out, vk, vrange_in, vrange, dlog, stream);
      if (d == 64) return launch_cmm_d<64>(kk, vv, src, ord, n_inst, K, B, G, q, out, vk, vrange_in, vrange, dlog, stream);
    }
    if (d == 128) return launch_cmd_d<bf16_t, 128>(kk, vv, src, ord, n_inst, K, B, G, q, out, vk, vrange, stream);
    if (d == 64) return launch_cmd_d<bf16_t, 64>(kk, vv, src, ord, n_inst, K, B, G, q, out, vk, vrange, stream);
  } else {
    if (d == 128) return launch_cmd_d<float, 128>(kk, vv, src, ord, n_inst, K, B, G, q, out, vk, vrange, stream);
    if (d == 64) return launch_cmd_d<float, 64>(kk, vv, src, ord, n_inst, K, B, G, q, out, vk, vrange, stream);
  }
  return hipErrorInvalidValue;
}

}  // namespace vase
