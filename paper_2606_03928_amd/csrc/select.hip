// select.hip -- VaSE-AttnV selection (Sec. 3.2 of the paper) on gfx950.
//
// One workgroup per head instance (four waves, eight at the largest K), the
// candidates [0, K) in registers.  Both selections are the exact k-th-largest
// searches of topk.hpp over 32-bit patterns (non-negative fp32 values order
// like their bit patterns) with an index-ordered tie resolution, so the result
// is the unique answer under the total orders
//     reserve:  (Range desc, slot asc)        top N_v of [0, K)
//     evict:    (key   asc,  slot desc)       bottom B of C = [0, K) \ R_V
// The survivor map is an exclusive scan of the per-thread keep counts.
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

template <int V, bool DET, int NWV>
__global__ __launch_bounds__(NWV * kWave) void select_kernel(
    const float* __restrict__ attn, const float* __restrict__ vrange, int K, int B, int Nv,
    uint32_t inst_base, uint32_t seed_lo, uint32_t seed_hi, uint32_t round,
    int32_t* __restrict__ src, float* __restrict__ keys_out, uint32_t* __restrict__ status) {
  constexpr int NW = (V + 31) / 32;
  constexpr int NT = NWV * kWave;
  __shared__ SelectShared<NWV> sh;
  const int inst = blockIdx.x;
  const int tid = threadIdx.x;
  const int s0 = V * tid;                              // this thread's first slot
  const int n_t = min(max(K - s0, 0), V);              // its slots below K
  uint32_t in_k[NW];
  slots_below<V>(K, in_k);
  // inputs outside the contract (finite and >= 0: a bit pattern at or above
  // that of +inf is a NaN, an infinity or a negative number, -0 included) only
  // set a status bit
  bool bad_attn = false, bad_value = false;

  // (1) R_V: top N_v Range values, ties to the lower slot
  uint32_t v[V];
  thread_load<V>(vrange + (size_t)inst * K + min(s0, K - 1), n_t, v);
#pragma unroll
  for (int i = 0; i < V; ++i) bad_value |= v[i] >= 0x7f800000u;
  uint32_t resv[NW];
  if (Nv > 0) {
    block_select_top_regs<V, NWV>(v, in_k, (uint32_t)Nv, /*tie_low=*/true, resv, sh);
  } else {
#pragma unroll
    for (int w = 0; w < NW; ++w) resv[w] = 0u;
  }

  // (2) keys of the candidates C = [0, K) \ R_V, complemented so that the
  //     largest pattern is the smallest key (a non-negative key's complement is
  //     never 0); Philox word i & 3 of counter (i >> 2, instance, round, 0)
  uint32_t cset[NW];
#pragma unroll
  for (int w = 0; w < NW; ++w) cset[w] = in_k[w] & ~resv[w];
  thread_load<V>(attn + (size_t)inst * K + min(s0, K - 1), n_t, v);
  const uint32_t inst_id = inst_base + (uint32_t)inst;
  float* ko = keys_out ? keys_out + (size_t)inst * K : nullptr;
#pragma unroll
  for (int q = 0; q < V / 4; ++q) {
    uint32_t cq[NW];
    opaque_words<NW>(cset, cq);
    uint4 x = make_uint4(0u, 0u, 0u, 0u);
    if (!DET) x = philox4x32_10(make_uint4((uint32_t)(s0 / 4 + q), inst_id, round, 0u), seed_lo, seed_hi);
    const uint32_t words[4] = {x.x, x.y, x.z, x.w};
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      // branch-free: every slot's key is formed, a non-candidate's dropped
      const int i = 4 * q + j;
      const uint32_t ci = (cq[i / 32] >> (i % 32)) & 1u;
      const float w = __uint_as_float(v[i]);
      bad_attn |= ci != 0u && v[i] >= 0x7f800000u;
      const float key = DET ? w : w / neg_log(uniform_from_word(words[j]));
      v[i] = ~__float_as_uint(key) & (0u - ci);
      if (ko && i < n_t) ko[s0 + i] = ci ? key : __uint_as_float(0x7fc00000u);
    }
  }

  // (3) evict the B smallest keys of C, ties to the higher slot
  uint32_t evict[NW];
  block_select_top_regs<V, NWV>(v, cset, (uint32_t)B, /*tie_low=*/false, evict, sh);

  // (4) survivor map: the kept candidate slots in slot order, then the B
  //     buffer slots [K, N)
  uint32_t keep[NW];
#pragma unroll
  for (int w = 0; w < NW; ++w) keep[w] = in_k[w] & ~evict[w];
  int32_t* out = src + (size_t)inst * K;
  block_list_slots<V, NWV>(keep, out, nullptr, sh);
  for (int b = tid; b < B; b += NT) out[K - B + b] = K + b;
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

// the selection keeps its candidates in registers: no dynamic LDS
size_t select_lds_bytes(int K, int B) {
  (void)K;
  (void)B;
  return 0;
}

hipError_t launch_select(const float* attn, const float* vrange, int n_inst, uint32_t inst_base,
                         int K, int B, int Nv, uint64_t seed, uint32_t round, uint32_t flags,
                         int32_t* src, float* keys, hipStream_t stream, uint32_t* status) {
  const bool det = (flags & VASE_DETERMINISTIC) != 0;
  const uint32_t k0 = (uint32_t)seed, k1 = (uint32_t)(seed >> 32);
  const size_t lds = select_lds_bytes(K, B);
  with_topk_layout(K, [&](auto v_, auto nw_) {
    constexpr int V = decltype(v_)::value, NWV = decltype(nw_)::value;
    if (det)
      hipLaunchKernelGGL((select_kernel<V, true, NWV>), dim3(n_inst), dim3(NWV * kWave), lds, stream,
                         attn, vrange, K, B, Nv, inst_base, k0, k1, round, src, keys, status);
    else
      hipLaunchKernelGGL((select_kernel<V, false, NWV>), dim3(n_inst), dim3(NWV * kWave), lds, stream,
                         attn, vrange, K, B, Nv, inst_base, k0, k1, round, src, keys, status);
  });
  return hipGetLastError();
}

}  // namespace vase
