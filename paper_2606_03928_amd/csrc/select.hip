// select.hip -- VaSE-AttnV selection (Sec. 3.2 of the paper) on gfx950.
//
// One workgroup per head instance (four waves, eight at the largest K).
// Thread t holds the slots [V*t, V*t + V) of the candidates [0, K) in registers as 32-bit patterns
// (non-negative fp32 values order like their bit patterns), and both
// selections are exact k-th-largest searches over those patterns followed by
// an index-ordered tie resolution, so the result is the unique answer under
// the total orders
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

// ---------------------------------------------------------------------------
// Selection with one workgroup per instance and the candidates in registers:
// thread t holds the V slots [V*t, V*t + V).  Both selections are exact
// k-th-largest searches over the 32-bit patterns that fix the threshold one bit
// at a time from the highest bit in which two candidates differ: a bit stays
// set when at least k candidates are at or above the threshold with it.  Each
// wave counts with ballots, the per-wave counts meet in LDS (double-buffered,
// one barrier per bit).  Ties at the threshold are taken in slot order from a
// block-wide prefix sum.
// ---------------------------------------------------------------------------
// NWV waves per workgroup: 4 (256 threads) up to K = 6144, 8 beyond
template <int NWV>
struct SelectShared {
  static constexpr int kWaves = NWV;
  uint32_t cnt[2][NWV];
  uint32_t red[2][NWV];
  uint32_t scan[NWV];
};

// Sum of x over the block (x uniform per wave), through the LDS row buf.
template <int NWV>
__device__ __forceinline__ uint32_t block_sum_waves(uint32_t x, uint32_t* buf) {
  if (lane_id() == 0) buf[wave_id()] = x;
  __syncthreads();
  uint32_t t = 0;
#pragma unroll
  for (int w = 0; w < NWV; ++w) t += buf[w];
  return t;
}

// Exclusive prefix sum of x over the block's threads, and the total.
template <int NWV>
__device__ __forceinline__ uint32_t block_excl_scan(uint32_t x, uint32_t& total, SelectShared<NWV>& sh) {
  const uint32_t incl = wave_incl_scan(x);
  if (lane_id() == kWave - 1) sh.scan[wave_id()] = incl;
  __syncthreads();
  uint32_t base = 0;
  total = 0;
#pragma unroll
  for (int w = 0; w < NWV; ++w) {
    const uint32_t c = sh.scan[w];
    base += (uint32_t)w < wave_id() ? c : 0u;
    total += c;
  }
  __syncthreads();   // sh.scan is reused
  return base + incl - x;
}

// Bit words of a thread that the compiler cannot see through, so that each
// loop re-extracts its bits instead of keeping a register per slot alive.
template <int NW>
__device__ __forceinline__ void opaque_words(const uint32_t (&in)[NW], uint32_t (&out)[NW]) {
#pragma unroll
  for (int w = 0; w < NW; ++w) {
    out[w] = in[w];
    asm volatile("" : "+v"(out[w]));
  }
}

// The k largest values among the block's candidates (cand bit i of a thread:
// its slot V*t + i takes part; every non-candidate value is 0), ties toward the
// lower slot (tie_low) or the higher slot; sel receives the thread's selection
// bits.  k >= 1, at least k candidates.
template <int V, int NWV>
__device__ void block_select_top_regs(const uint32_t (&v)[V], const uint32_t (&cand)[(V + 31) / 32],
                                      uint32_t k, bool tie_low, uint32_t (&sel)[(V + 31) / 32],
                                      SelectShared<NWV>& sh) {
  constexpr int NW = (V + 31) / 32;
  uint32_t cw[NW];
  opaque_words<NW>(cand, cw);
  uint32_t vand = 0xffffffffu, vor = 0u;
#pragma unroll
  for (int i = 0; i < V; ++i) {
    const uint32_t cm = 0u - ((cw[i / 32] >> (i % 32)) & 1u);
    vand &= v[i] | ~cm;
    vor |= v[i] & cm;
  }
#pragma unroll
  for (int o = kWave / 2; o >= 1; o >>= 1) {
    vand &= __shfl_xor(vand, o, kWave);
    vor |= __shfl_xor(vor, o, kWave);
  }
  if (lane_id() == 0) {
    sh.red[0][wave_id()] = vand;
    sh.red[1][wave_id()] = vor;
  }
  __syncthreads();
#pragma unroll
  for (int w = 0; w < NWV; ++w) {
    vand &= sh.red[0][w];
    vor |= sh.red[1][w];
  }
  vand = __builtin_amdgcn_readfirstlane(vand);
  vor = __builtin_amdgcn_readfirstlane(vor);
  const uint32_t diff = vand ^ vor;
  const int top = diff ? 32 - __clz(diff) : 0;
  uint32_t T = top >= 32 ? 0u : vand & ~((1u << top) - 1u);
  // T becomes the k-th largest candidate (non-candidates are 0 and never reach
  // a threshold with a bit set); the counts alternate between two LDS rows, so
  // one barrier per bit separates a row's writes from its reads and rewrites
  int par = 0;
  for (int b = top - 1; b >= 0; --b) {
    const uint32_t t = T | (1u << b);
    uint32_t cnt = 0;
#pragma unroll
    for (int i = 0; i < V; ++i) cnt += (uint32_t)__popcll(__ballot(v[i] >= t));
    if (lane_id() == 0) sh.cnt[par][wave_id()] = cnt;
    __syncthreads();
    uint32_t tot = 0;
#pragma unroll
    for (int w = 0; w < NWV; ++w) tot += sh.cnt[par][w];
    // the same in every lane: keep the threshold in a scalar register
    tot = __builtin_amdgcn_readfirstlane(tot);
    if (tot >= k) T = t;
    par ^= 1;
  }
  // every candidate above T, and `need` of those equal to T in slot order
  uint32_t gt_t = 0, eq_t = 0;
  opaque_words<NW>(cand, cw);
#pragma unroll
  for (int i = 0; i < V; ++i) {
    const uint32_t ci = (cw[i / 32] >> (i % 32)) & 1u;
    gt_t += ci & (v[i] > T ? 1u : 0u);
    eq_t += ci & (v[i] == T ? 1u : 0u);
  }
  uint32_t gt_w = gt_t;
#pragma unroll
  for (int o = kWave / 2; o >= 1; o >>= 1) gt_w += __shfl_xor(gt_w, o, kWave);
  __syncthreads();   // the last count row has been read by every wave
  const uint32_t gt = block_sum_waves<NWV>(gt_w, sh.cnt[0]);
  uint32_t eq_total;
  uint32_t r = block_excl_scan(eq_t, eq_total, sh);
  const uint32_t need = k - gt;
  const uint32_t lo = tie_low ? 0u : eq_total - need;
#pragma unroll
  for (int w = 0; w < NW; ++w) sel[w] = 0u;
  opaque_words<NW>(cand, cw);
#pragma unroll
  for (int i = 0; i < V; ++i) {
    const uint32_t ci = (cw[i / 32] >> (i % 32)) & 1u;
    const uint32_t gti = ci & (v[i] > T ? 1u : 0u);
    const uint32_t eqi = ci & (v[i] == T ? 1u : 0u);
    const uint32_t inr = r - lo < need ? 1u : 0u;     // lo <= r < lo + need
    sel[i / 32] |= (gti | (eqi & inr)) << (i % 32);
    r += eqi;
  }
}

// This thread's V slots of p (0 at and past n): a thread whose slots all lie
// below K loads them at fixed offsets from one base.
template <int V>
__device__ __forceinline__ void thread_load(const float* p, int n, uint32_t (&v)[V]) {
  if (n >= V) {
#pragma unroll
    for (int i = 0; i < V; ++i) v[i] = __float_as_uint(p[i]);
  } else {
#pragma unroll
    for (int i = 0; i < V; ++i) v[i] = i < n ? __float_as_uint(p[i]) : 0u;
  }
}

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
#pragma unroll
  for (int w = 0; w < NW; ++w) {
    const int lo = 32 * w, len = min(32, V - lo);
    const int c = min(max(n_t - lo, 0), len);
    in_k[w] = c >= 32 ? 0xffffffffu : (1u << c) - 1u;
  }
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
  uint32_t keep[NW], kc = 0;
#pragma unroll
  for (int w = 0; w < NW; ++w) {
    keep[w] = in_k[w] & ~evict[w];
    kc += __popc(keep[w]);
  }
  uint32_t total;
  uint32_t pos = block_excl_scan(kc, total, sh);
  int32_t* out = src + (size_t)inst * K;
  uint32_t kw[NW];
  opaque_words<NW>(keep, kw);
#pragma unroll
  for (int i = 0; i < V; ++i) {
    const uint32_t ki = (kw[i / 32] >> (i % 32)) & 1u;
    if (ki) out[pos] = s0 + i;
    pos += ki;
  }
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
#define VASE_SEL(V, NWV)                                                                          \
  if (det)                                                                                        \
    hipLaunchKernelGGL((select_kernel<V, true, NWV>), dim3(n_inst), dim3(NWV * kWave), lds,      \
                       stream, attn, vrange, K, B, Nv, inst_base, k0, k1, round, src, keys,      \
                       status);                                                                   \
  else                                                                                            \
    hipLaunchKernelGGL((select_kernel<V, false, NWV>), dim3(n_inst), dim3(NWV * kWave), lds,     \
                       stream, attn, vrange, K, B, Nv, inst_base, k0, k1, round, src, keys,      \
                       status)
  // slots per thread, a multiple of 4 (one Philox call per 4 slots): K over
  // 256 threads up to K = 6144, over 512 beyond
  if (K <= 8 * 256) {
    VASE_SEL(8, 4);
  } else if (K <= 16 * 256) {
    VASE_SEL(16, 4);
  } else if (K <= 24 * 256) {
    VASE_SEL(24, 4);
  } else {
    VASE_SEL(16, 8);
  }
#undef VASE_SEL
  return hipGetLastError();
}

}  // namespace vase
