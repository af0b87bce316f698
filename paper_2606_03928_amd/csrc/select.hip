// select.hip -- VaSE-AttnV selection (Sec. 3.2 of the paper) on gfx950.
//
// One workgroup per head instance.  The instance's K scores live in LDS as
// 32-bit patterns (non-negative fp32 values order like their bit patterns), and
// both selections are exact radix selects (four 8-bit digit passes with an LDS
// histogram) followed by an index-ordered tie resolution, so the result is the
// unique answer under the total orders
//     reserve:  (Range desc, slot asc)        top N_v of [0, K)
//     evict:    (key   asc,  slot desc)       bottom B of C = [0, K) \ R_V
// The survivor map is an exclusive scan of the keep bitmask.
//
// The sampling noise E_i = -ln u_i is computed with a fixed sequence of IEEE
// binary32 operations (this translation unit is compiled with
// -ffp-contract=off), so it is bitwise reproducible on any IEEE machine that
// performs the same sequence.
#include "vase_internal.hpp"
#include "vase.h"

#pragma clang fp contract(off)

#include "rng.hpp"
#include "topk.hpp"

namespace vase {
namespace {

__global__ __launch_bounds__(kSelBlock) void select_kernel(
    const float* __restrict__ attn, const float* __restrict__ vrange, int K, int B, int Nv,
    uint32_t inst_base, uint32_t seed_lo, uint32_t seed_hi, uint32_t round, uint32_t flags,
    int32_t* __restrict__ src, float* __restrict__ keys_out, uint32_t* __restrict__ status) {
  extern __shared__ uint32_t lds[];
  __shared__ SelShared sh;
  const int N = K + B;
  const int nwK = ((K + 63) / 64) * 2;
  uint32_t* vals = lds;                 // [K]
  uint32_t* resv = vals + K;            // [nwK]
  uint32_t* evict = resv + nwK;         // [nwK]
  uint32_t* tie = evict + nwK;          // [nwN]
  const int inst = blockIdx.x;
  const int tid = threadIdx.x;
  const float* a = attn + (size_t)inst * K;
  const float* r = vrange + (size_t)inst * K;

  // inputs outside the contract (finite and >= 0): a bit pattern at or above
  // that of +inf is a NaN, an infinity or a negative number (-0 included)
  bool bad_attn = false, bad_value = false;

  // (1) R_V: top N_v Range values, ties to the lower slot.  Each thread issues
  // its loads before its LDS stores, so that they are in flight together.
  constexpr int kLoadU = 8;
  for (int i0 = tid; i0 < K; i0 += kLoadU * kSelBlock) {
    float x[kLoadU];
#pragma unroll
    for (int u = 0; u < kLoadU; ++u) {
      const int i = i0 + u * kSelBlock;
      x[u] = i < K ? r[i] : 0.f;
    }
#pragma unroll
    for (int u = 0; u < kLoadU; ++u) {
      const int i = i0 + u * kSelBlock;
      if (i < K) {
        vals[i] = __float_as_uint(x[u]);
        bad_value |= __float_as_uint(x[u]) >= 0x7f800000u;
      }
    }
  }
  __syncthreads();
  block_select_top(vals, nullptr, K, Nv, /*tie_low=*/true, resv, tie, sh);

  // (2) keys of the candidates C = [0, K) \ R_V, stored complemented so that the
  //     "largest" complemented value is the smallest key
  const uint32_t inst_id = inst_base + (uint32_t)inst;
  const bool det = (flags & VASE_DETERMINISTIC) != 0;
  for (int g = tid; g * 4 < K; g += kSelBlock) {
    uint4 x = make_uint4(0u, 0u, 0u, 0u);
    if (!det) x = philox4x32_10(make_uint4((uint32_t)g, inst_id, round, 0u), seed_lo, seed_hi);
    const uint32_t words[4] = {x.x, x.y, x.z, x.w};
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int i = 4 * g + j;
      if (i >= K) break;
      if (mask_bit(resv, i)) {
        vals[i] = 0u;  // excluded below
        if (keys_out) keys_out[(size_t)inst * K + i] = __uint_as_float(0x7fc00000u);
        continue;
      }
      const float w = a[i];
      bad_attn |= __float_as_uint(w) >= 0x7f800000u;
      const float key = det ? w : w / neg_log(uniform_from_word(words[j]));
      vals[i] = ~__float_as_uint(key);
      if (keys_out) keys_out[(size_t)inst * K + i] = key;
    }
  }
  __syncthreads();

  // (3) evict the B smallest keys of C, ties to the higher slot
  block_select_top(vals, resv, K, B, /*tie_low=*/false, evict, tie, sh);

  // (4) survivor map: slot i survives unless it is an evicted candidate; one
  //     32-slot word per thread, the block taking kSelBlock words at a time
  const int nw32 = (N + 31) / 32;
  int32_t* out = src + (size_t)inst * K;
  uint32_t run = 0;   // survivors in the words before this pass
  for (int w0 = 0; w0 < nw32; w0 += kSelBlock) {
    const int wd = w0 + tid;
    uint32_t keepw = 0, cnt = 0;
    if (wd < nw32) {
      const uint32_t ev = wd < nwK ? evict[wd] : 0u;
      keepw = ~ev;
      const int hi = N - 32 * wd;
      if (hi < 32) keepw &= (1u << hi) - 1u;
      cnt = __popc(keepw);
    }
    const uint32_t incl = wave_incl_scan(cnt);
    if (lane_id() == kWave - 1) sh.wsum[wave_id()] = incl;
    __syncthreads();
    uint32_t base = run + incl - cnt;
    uint32_t total = 0;
    for (uint32_t w = 0; w < (uint32_t)kSelWaves; ++w) {
      if (w < wave_id()) base += sh.wsum[w];
      total += sh.wsum[w];
    }
    while (keepw) {
      const uint32_t b = __ffs(keepw) - 1;
      keepw &= keepw - 1;
      if (base < (uint32_t)K) out[base] = 32 * wd + (int)b;
      ++base;
    }
    run += total;
    __syncthreads();   // sh.wsum is rewritten by the next pass
  }
  if (status) {
    block_status(status, bad_attn, VASE_STATUS_SELECT_ATTN);
    block_status(status, bad_value, VASE_STATUS_SELECT_VALUE);
  }
}

// Random reservation scores (the Appendix D ablation that reserves N_v random pairs):
// u_j from Philox4x32-10 with counter (j>>2, inst, round, 2), word j&3.
__global__ __launch_bounds__(256) void value_random_kernel(int K, uint32_t inst_base, uint32_t k0,
                                                          uint32_t k1, uint32_t round,
                                                          float* __restrict__ out) {
  const int inst = blockIdx.y;
  const int q4 = blockIdx.x * 256 + threadIdx.x;          // one Philox call per 4 slots
  if (4 * q4 >= K) return;
  const uint4 x = philox4x32_10(make_uint4((uint32_t)q4, inst_base + inst, round, 2u), k0, k1);
  const uint32_t w[4] = {x.x, x.y, x.z, x.w};
  float* o = out + (size_t)inst * K;
#pragma unroll
  for (int e = 0; e < 4; ++e)
    if (4 * q4 + e < K) o[4 * q4 + e] = uniform_from_word(w[e]);
}

}  // namespace

hipError_t launch_value_random(int n_inst, uint32_t inst_base, int K, uint64_t seed,
                               uint32_t round, float* vrange, hipStream_t stream) {
  const dim3 grid((K + 4 * 256 - 1) / (4 * 256), n_inst);
  hipLaunchKernelGGL(value_random_kernel, grid, dim3(256), 0, stream, K, inst_base,
                     (uint32_t)seed, (uint32_t)(seed >> 32), round, vrange);
  return hipGetLastError();
}

size_t select_lds_bytes(int K, int B) {
  const int N = K + B;
  const size_t nwK = (size_t)((K + 63) / 64) * 2;
  const size_t nwN = (size_t)((N + 63) / 64) * 2;
  return sizeof(uint32_t) * ((size_t)K + 2 * nwK + nwN);
}

hipError_t launch_select(const float* attn, const float* vrange, int n_inst, uint32_t inst_base,
                         int K, int B, int Nv, uint64_t seed, uint32_t round, uint32_t flags,
                         int32_t* src, float* keys, hipStream_t stream, uint32_t* status) {
  const size_t lds = select_lds_bytes(K, B);
  hipLaunchKernelGGL(select_kernel, dim3(n_inst), dim3(kSelBlock), lds, stream, attn, vrange, K,
                     B, Nv, inst_base, (uint32_t)seed, (uint32_t)(seed >> 32), round, flags, src,
                     keys, status);
  return hipGetLastError();
}

}  // namespace vase
