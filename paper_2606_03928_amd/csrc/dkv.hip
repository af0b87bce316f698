// dkv.hip -- VaSE-DKV scoring on gfx950 (Sec. 3.2 of the paper, with CurDKV's
// product score, Eq. 4).
//
// At every eviction step each head instance draws a Gaussian projection
// G_t in R^{d x r} (entries N(0, 1/r)), independent of earlier steps, and
// scores candidate slot i < K by
//     s_i = ||G_t^T k_i||^2 * ||G_t^T v_i||^2.
// Survivors are then the K - B highest scores (vase_select in deterministic
// mode with N_v = 0), and compaction and decode follow as for VaSE-AttnV.
//
// dkv_projection_kernel draws G_t (rng.hpp; this unit is compiled with
// -ffp-contract=off).  The score streams the K candidate key and value rows
// of each instance once, so it is bound by HBM: for bf16 caches the
// projections run on MFMA (v_mfma_f32_32x32x16_bf16) with G^T as the A
// operand, split into a bf16 head and tail (G ~ G_hi + G_lo to 2^-16) so that
// the bf16 rows meet an almost fp32 projection; the accumulator then holds
// 16 projection coordinates x 1 row per lane and the squared norm is a sum
// inside the lane plus one exchange.  fp32 caches use one thread per row.
#include "vase_internal.hpp"
#include "vase.h"

#pragma clang fp contract(off)

#include "rng.hpp"

namespace vase {
namespace {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));

constexpr int kDkvBlock = 256;
constexpr int kDkvTilesPerWave = 8;          // 32-row tiles per wave
constexpr int kDkvRowsPerWave = 32 * kDkvTilesPerWave;
constexpr int kDkvRowsPerBlock = kDkvRowsPerWave * (kDkvBlock / kWave);
constexpr int kDkvMaxR = 32;

__global__ __launch_bounds__(kDkvBlock) void dkv_projection_kernel(int n_inst, uint32_t inst_base,
                                                                 int dr, int r, uint32_t k0,
                                                                 uint32_t k1, uint32_t round,
                                                                 float* __restrict__ g) {
  const size_t i = (size_t)blockIdx.x * kDkvBlock + threadIdx.x;
  if (i >= (size_t)n_inst * dr) return;
  const uint32_t inst = (uint32_t)(i / (size_t)dr);
  const uint32_t e = (uint32_t)(i % (size_t)dr);
  const float scale = 1.0f / __builtin_sqrtf((float)r);
  g[i] = dkv_gaussian_entry(e, inst_base + inst, round, k0, k1, scale);
}

// bf16 head and tail of x: x ~ hi + lo with |x - hi - lo| <= 2^-16 |x|.
__device__ __forceinline__ void split_bf16(float x, __bf16& hi, __bf16& lo) {
  hi = (__bf16)x;
  lo = (__bf16)(x - (float)hi);
}

// One block: kDkvRowsPerBlock consecutive candidate rows of one instance.  With
// dlog given, the rows run to N (the buffer included) and the block also writes
// the decode queries' logits dlog[inst][h][row] = qdec[inst][h] . k_row (h < G)
// from the key rows it holds: the G queries are the A operand of one more
// 32x32x16 MFMA chain per tile, the rows the B operand as for the projection.
template <int D>
__global__ __launch_bounds__(kDkvBlock) void dkv_score_mfma_kernel(
    const uint16_t* __restrict__ k, const uint16_t* __restrict__ v, const float* __restrict__ g,
    int N, int K, int r, int blocks_per_inst, float* __restrict__ out,
    const uint16_t* __restrict__ qdec, int G, float* __restrict__ dlog) {
  constexpr int KS = D / 16;
  __shared__ float sg[D * kDkvMaxR];
  __shared__ bf16x8_t sa[3][KS][kWave];   // [G^T head, G^T tail, decode queries][step][lane]
  const uint32_t lb = xcd_logical_block(blockIdx.x, gridDim.x);
  const int inst = (int)(lb / (uint32_t)blocks_per_inst);
  const int rb = (int)(lb % (uint32_t)blocks_per_inst);
  const int lane = threadIdx.x % kWave, wave = threadIdx.x / kWave, half = lane / 32;
  // G of this instance into LDS as [d][32], columns >= r zero
  const float* gi = g + (size_t)inst * D * r;
  for (int t = threadIdx.x; t < D * kDkvMaxR; t += kDkvBlock) {
    const int a = t / kDkvMaxR, b = t % kDkvMaxR;
    sg[t] = b < r ? gi[a * r + b] : 0.f;
  }
  __syncthreads();
  // A operands, the same for every wave: G^T (32 projection columns x D), head
  // and tail, and the decode queries (row = head, clamped), staged once per
  // block as per-lane fragments read at each step (in registers they would
  // take 96 VGPRs).  The contraction index is permuted identically in both
  // operands: lane half h, step ks holds elements [16*ks + 8*h, +8), so that
  // the two lanes of a row read 32 adjacent bytes in one load (with the
  // halves 128 bytes apart, every load touched 64 lines for 16 bytes each).
  const int col = lane % 32;
  for (int t = threadIdx.x; t < KS * kWave; t += kDkvBlock) {
    const int ks = t / kWave, l = t % kWave, c = l % 32, h = l / 32;
    bf16x8_t fh, fl;
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      __bf16 hi, lo;
      split_bf16(sg[(16 * ks + 8 * h + e) * kDkvMaxR + c], hi, lo);
      fh[e] = hi;
      fl[e] = lo;
    }
    sa[0][ks][l] = fh;
    sa[1][ks][l] = fl;
    if (dlog)
      sa[2][ks][l] = reinterpret_cast<const bf16x8_t*>(
          qdec + ((size_t)inst * G + min(c, G - 1)) * D + 8 * h)[2 * ks];
  }
  __syncthreads();
  const int rows = dlog ? N : K;
  const uint16_t* kinst = k + (size_t)inst * N * D;
  const uint16_t* vinst = v + (size_t)inst * N * D;
  float* oinst = out + (size_t)inst * K;
  const int row_base = rb * kDkvRowsPerBlock + wave * kDkvRowsPerWave;
  // tile t of this wave: rows row_base + 32 t + [0, 32); rows past K re-read
  // row K-1 and are not stored.  All 2*KS loads of a tile are issued before its
  // first MFMA (one wait per tile); the other waves of the SIMD cover it.
  auto load_tile = [&](int t, bf16x8_t (&kb)[KS], bf16x8_t (&vb)[KS]) {
    const int rr = min(row_base + t * 32 + col, rows - 1);
    const bf16x8_t* kr = reinterpret_cast<const bf16x8_t*>(kinst + (size_t)rr * D + 8 * half);
    const bf16x8_t* vr = reinterpret_cast<const bf16x8_t*>(vinst + (size_t)rr * D + 8 * half);
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
      kb[ks] = kr[2 * ks];
      vb[ks] = vr[2 * ks];
    }
  };
  auto tile_step = [&](int t, const bf16x8_t (&kb)[KS], const bf16x8_t (&vb)[KS]) {
    f32x16_t pk = f32x16_t{}, pv = f32x16_t{};
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
      const bf16x8_t ghi = sa[0][ks][lane], glo = sa[1][ks][lane];
      pk = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ghi, kb[ks], pk, 0, 0, 0);
      pv = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ghi, vb[ks], pv, 0, 0, 0);
      pk = __builtin_amdgcn_mfma_f32_32x32x16_bf16(glo, kb[ks], pk, 0, 0, 0);
      pv = __builtin_amdgcn_mfma_f32_32x32x16_bf16(glo, vb[ks], pv, 0, 0, 0);
    }
    // lane holds projection coordinates 8(e/4) + 4h + e%4 of row `col`
    float lk = 0.f, lv = 0.f;
#pragma unroll
    for (int e = 0; e < 16; ++e) {
      lk = __builtin_fmaf(pk[e], pk[e], lk);
      lv = __builtin_fmaf(pv[e], pv[e], lv);
    }
    lk += __shfl_xor(lk, 32, kWave);
    lv += __shfl_xor(lv, 32, kWave);
    const int row = row_base + t * 32 + col;
    if (half == 0 && row < K) oinst[row] = lk * lv;
    if (dlog) {
      f32x16_t pq = f32x16_t{};
#pragma unroll
      for (int ks = 0; ks < KS; ++ks)
        pq = __builtin_amdgcn_mfma_f32_32x32x16_bf16(sa[2][ks][lane], kb[ks], pq, 0, 0, 0);
      // lane holds head 8(e/4) + 4h + e%4 of row `col`
      if (row < N) {
#pragma unroll
        for (int e = 0; e < 16; ++e) {
          const int h = 8 * (e / 4) + 4 * half + e % 4;
          if (h < G) dlog[((size_t)inst * G + h) * N + row] = pq[e];
        }
      }
    }
  };
  const int nt = min(kDkvTilesPerWave, (rows - row_base + 31) / 32);
  for (int t = 0; t < nt; ++t) {
    bf16x8_t kb[KS], vb[KS];
    load_tile(t, kb, vb);
    __builtin_amdgcn_sched_barrier(0);
    tile_step(t, kb, vb);
  }
}

// fp32 caches: one thread per candidate row, G in LDS.
template <int D>
__global__ __launch_bounds__(kDkvBlock) void dkv_score_valu_kernel(
    const float* __restrict__ k, const float* __restrict__ v, const float* __restrict__ g, int N,
    int K, int r, float* __restrict__ out) {
  __shared__ float sg[D * kDkvMaxR];
  const int inst = blockIdx.y;
  const float* gi = g + (size_t)inst * D * r;
  for (int t = threadIdx.x; t < D * r; t += kDkvBlock) sg[t] = gi[t];
  __syncthreads();
  const int row = blockIdx.x * kDkvBlock + threadIdx.x;
  if (row >= K) return;
  const float* kr = k + ((size_t)inst * N + row) * D;
  const float* vr = v + ((size_t)inst * N + row) * D;
  float lk = 0.f, lv = 0.f;
  for (int b = 0; b < r; ++b) {
    float pk = 0.f, pv = 0.f;
    for (int a = 0; a < D; ++a) {
      pk = __builtin_fmaf(kr[a], sg[a * r + b], pk);
      pv = __builtin_fmaf(vr[a], sg[a * r + b], pv);
    }
    lk = __builtin_fmaf(pk, pk, lk);
    lv = __builtin_fmaf(pv, pv, lv);
  }
  out[(size_t)inst * K + row] = lk * lv;
}

}  // namespace

hipError_t launch_dkv_projection(int n_inst, uint32_t inst_base, int d, int r, uint64_t seed,
                                 uint32_t round, float* g, hipStream_t stream) {
  const size_t total = (size_t)n_inst * d * r;
  const unsigned grid = (unsigned)((total + kDkvBlock - 1) / kDkvBlock);
  hipLaunchKernelGGL(dkv_projection_kernel, dim3(grid), dim3(kDkvBlock), 0, stream, n_inst,
                     inst_base, d * r, r, (uint32_t)seed, (uint32_t)(seed >> 32), round, g);
  return hipGetLastError();
}

hipError_t launch_dkv_score(const void* k, const void* v, const float* g, int dtype, int n_inst,
                            int K, int B, int d, int r, float* out, const void* q_dec, int G,
                            float* dec_logits, hipStream_t stream) {
  const int N = K + B;
  if (dtype == VASE_BF16) {
    const int bpi = ((dec_logits ? N : K) + kDkvRowsPerBlock - 1) / kDkvRowsPerBlock;
    const uint16_t* qd = static_cast<const uint16_t*>(q_dec);
    const unsigned grid = (unsigned)(n_inst * bpi);
    const uint16_t* kk = static_cast<const uint16_t*>(k);
    const uint16_t* vv = static_cast<const uint16_t*>(v);
    if (d == 128)
      hipLaunchKernelGGL((dkv_score_mfma_kernel<128>), dim3(grid), dim3(kDkvBlock), 0, stream, kk,
                         vv, g, N, K, r, bpi, out, qd, G, dec_logits);
    else
      hipLaunchKernelGGL((dkv_score_mfma_kernel<64>), dim3(grid), dim3(kDkvBlock), 0, stream, kk,
                         vv, g, N, K, r, bpi, out, qd, G, dec_logits);
  } else {
    const dim3 grid((K + kDkvBlock - 1) / kDkvBlock, n_inst);
    const float* kk = static_cast<const float*>(k);
    const float* vv = static_cast<const float*>(v);
    if (d == 128)
      hipLaunchKernelGGL((dkv_score_valu_kernel<128>), grid, dim3(kDkvBlock), 0, stream, kk, vv, g,
                         N, K, r, out);
    else
      hipLaunchKernelGGL((dkv_score_valu_kernel<64>), grid, dim3(kDkvBlock), 0, stream, kk, vv, g,
                         N, K, r, out);
  }
  return hipGetLastError();
}

}  // namespace vase
