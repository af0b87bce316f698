// topk.hpp -- block-wide exact top-k of one instance's K candidates held in
// registers, shared by the selection (Sec. 3.2 of the paper) and the
// quantiser's full-precision reserve.  gfx950.
//
// One workgroup of NWV waves per instance; thread t holds the V slots
// [V*t, V*t + V) as 32-bit patterns (non-negative fp32 values order like their
// bit patterns).  The k-th largest pattern is fixed one bit at a time from the
// highest bit in which two candidates differ: a bit stays set when at least k
// candidates are at or above the threshold with it.  Each wave counts with
// ballots, the per-wave counts meet in LDS (double-buffered, one barrier per
// bit), and the ties at the threshold are taken in slot order from a
// block-wide prefix sum, so the result is unique under (value desc, slot asc)
// or (value desc, slot desc).
#pragma once

#include "vase_internal.hpp"

#include <type_traits>

namespace vase {
namespace {

__device__ __forceinline__ uint32_t wave_id() { return threadIdx.x / kWave; }
__device__ __forceinline__ uint32_t lane_id() { return threadIdx.x % kWave; }

// Inclusive prefix sum over the 64 lanes of a wave.
__device__ __forceinline__ uint32_t wave_incl_scan(uint32_t x) {
  const uint32_t lane = lane_id();
#pragma unroll
  for (int o = 1; o < kWave; o <<= 1) {
    const uint32_t y = __shfl_up(x, o, kWave);
    if (lane >= (uint32_t)o) x += y;
  }
  return x;
}

// The thread layout for K candidates: V slots per thread, a multiple of 4 (the
// selection draws one Philox block per 4 slots), over four waves up to
// K = 6144 and eight beyond (K <= 8192).  f is called with
// std::integral_constant<int, V> and std::integral_constant<int, NWV>.
template <typename F>
void with_topk_layout(int K, F&& f) {
  static_assert(16 * 8 * kWave >= VASE_MAX_K, "the widest layout covers every K");
  using std::integral_constant;
  if (K <= 8 * 256)
    f(integral_constant<int, 8>{}, integral_constant<int, 4>{});
  else if (K <= 16 * 256)
    f(integral_constant<int, 16>{}, integral_constant<int, 4>{});
  else if (K <= 24 * 256)
    f(integral_constant<int, 24>{}, integral_constant<int, 4>{});
  else
    f(integral_constant<int, 16>{}, integral_constant<int, 8>{});
}

template <int NWV>
struct SelectShared {
  uint32_t cnt[2][NWV];
  uint32_t red[2][NWV];
  uint32_t scan[NWV];
};

// Bit words of this thread's slots below K.
template <int V>
__device__ __forceinline__ void slots_below(int K, uint32_t (&m)[(V + 31) / 32]) {
  const int n_t = min(max(K - V * (int)threadIdx.x, 0), V);
#pragma unroll
  for (int w = 0; w < (V + 31) / 32; ++w) {
    const int lo = 32 * w, len = min(32, V - lo);
    const int c = min(max(n_t - lo, 0), len);
    m[w] = c >= 32 ? 0xffffffffu : (1u << c) - 1u;
  }
}

// This thread's V slots of p (0 at and past n): a thread whose slots all lie
// below the end loads them at fixed offsets from one base.
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
// bits.  k >= 1, at least k candidates.  Called by the whole block.
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

// The slots of the thread's set bits m, written in ascending slot order to
// out[] at the positions of a block-wide scan (out[j] = j-th set slot of the
// block) and optionally to out2[] as well; returns the block's total.
template <int V, int NWV>
__device__ __forceinline__ uint32_t block_list_slots(const uint32_t (&m)[(V + 31) / 32], int32_t* out,
                                                     int32_t* out2, SelectShared<NWV>& sh) {
  constexpr int NW = (V + 31) / 32;
  uint32_t c = 0;
#pragma unroll
  for (int w = 0; w < NW; ++w) c += __popc(m[w]);
  uint32_t total;
  uint32_t pos = block_excl_scan(c, total, sh);
  uint32_t mw[NW];
  opaque_words<NW>(m, mw);
  const int s0 = V * (int)threadIdx.x;
#pragma unroll
  for (int i = 0; i < V; ++i) {
    const uint32_t bi = (mw[i / 32] >> (i % 32)) & 1u;
    if (bi) {
      out[pos] = s0 + i;
      if (out2) out2[pos] = s0 + i;
    }
    pos += bi;
  }
  return total;
}

}  // namespace
}  // namespace vase
