// topk.hpp -- block-wide exact top-k over uint32 keys held in LDS (radix passes
// of up to 8 bits below the bits all keys share, then the ties in slot order),
// used by the quantiser's full-precision reserve, and the wave scan helpers
// that the selection shares.  gfx950, blocks of kSelBlock threads.
#pragma once

#include "vase_internal.hpp"

namespace vase {
namespace {

constexpr int kSelBlock = 512;
constexpr int kSelWaves = kSelBlock / kWave;

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

__device__ __forceinline__ uint32_t wave_sum(uint32_t x) {
#pragma unroll
  for (int o = kWave / 2; o >= 1; o >>= 1) x += __shfl_xor(x, o, kWave);
  return x;
}

struct SelShared {
  uint32_t hist[256];
  uint32_t wsum[kSelWaves];
  uint32_t wand[kSelWaves];
  uint32_t wor[kSelWaves];
  uint32_t digit;
  uint32_t above;
  uint32_t n_eq;
};

__device__ __forceinline__ bool mask_bit(const uint32_t* m, int i) {
  return (m[i >> 5] >> (i & 31)) & 1u;
}

// Selects the k largest values of vals[0, n) (uint32 order) among the slots not
// excluded by `excl` (nullable bitmask), ties resolved toward the lower slot
// (tie_low) or the higher slot.  Writes the selection bitmask to sel[0, nw) and
// uses tie[0, nw) as scratch; nw = words covering n rounded up to 64 bits.
// Must be called by the whole block; ends with a barrier.
__device__ void block_select_top(const uint32_t* vals, const uint32_t* excl, int n, int k,
                                 bool tie_low, uint32_t* sel, uint32_t* tie, SelShared& sh) {
  const int tid = threadIdx.x;
  const int nw = ((n + 63) / 64) * 2;
  if (k <= 0) {
    for (int w = tid; w < nw; w += kSelBlock) sel[w] = 0u;
    __syncthreads();
    return;
  }
  // The bits that every candidate shares need no pass: the digits start at the
  // highest bit in which two candidates differ.  Scores of one instance share
  // their sign and most exponent bits, and a first digit taken there would put
  // nearly every candidate in one bin, whose LDS atomics serialise.
  uint32_t vand = 0xffffffffu, vor = 0u;
  for (int i = tid; i < n; i += kSelBlock) {
    if (excl && mask_bit(excl, i)) continue;
    vand &= vals[i];
    vor |= vals[i];
  }
#pragma unroll
  for (int o = kWave / 2; o >= 1; o >>= 1) {
    vand &= __shfl_xor(vand, o, kWave);
    vor |= __shfl_xor(vor, o, kWave);
  }
  if (lane_id() == 0) {
    sh.wand[wave_id()] = vand;
    sh.wor[wave_id()] = vor;
  }
  __syncthreads();
#pragma unroll
  for (int w = 0; w < kSelWaves; ++w) {
    vand &= sh.wand[w];
    vor |= sh.wor[w];
  }
  const uint32_t diff = vand ^ vor;
  int top = diff ? 32 - __clz(diff) : 0;          // bits [0, top) are undecided
  uint32_t pmask = top >= 32 ? 0u : ~((1u << top) - 1u);
  uint32_t prefix = vand & pmask;
  uint32_t krem = (uint32_t)k;
  while (top > 0) {
    const int width = top < 8 ? top : 8;
    const int shift = top - width;
    const uint32_t dmask = (1u << width) - 1u;
    for (int b = tid; b < 256; b += kSelBlock) sh.hist[b] = 0u;
    __syncthreads();
    for (int i = tid; i < n; i += kSelBlock) {
      if (excl && mask_bit(excl, i)) continue;
      const uint32_t v = vals[i];
      if ((v & pmask) == prefix) atomicAdd(&sh.hist[(v >> shift) & dmask], 1u);
    }
    __syncthreads();
    if (wave_id() == 0) {
      // lane L owns bins [4L, 4L+4); suffix counts from the top bin downwards
      const uint32_t lane = lane_id();
      const uint32_t c0 = sh.hist[4 * lane], c1 = sh.hist[4 * lane + 1];
      const uint32_t c2 = sh.hist[4 * lane + 2], c3 = sh.hist[4 * lane + 3];
      const uint32_t own = c0 + c1 + c2 + c3;
      // inclusive suffix sum: reverse the lane order and prefix-scan
      const uint32_t rev = __shfl(own, kWave - 1 - lane, kWave);
      const uint32_t rscan = wave_incl_scan(rev);
      const uint32_t suffix_incl = __shfl(rscan, kWave - 1 - lane, kWave);  // sum over lanes >= lane
      const uint32_t suffix_excl = suffix_incl - own;                          // lanes > lane
      if (suffix_excl < krem && suffix_incl >= krem) {
        uint32_t acc = suffix_excl;
        uint32_t d;
        if (acc + c3 >= krem) d = 4 * lane + 3;
        else if ((acc += c3) + c2 >= krem) d = 4 * lane + 2;
        else if ((acc += c2) + c1 >= krem) d = 4 * lane + 1;
        else { acc += c1; d = 4 * lane; }
        sh.digit = d;
        sh.above = acc;
      }
    }
    __syncthreads();
    const uint32_t d = sh.digit;
    krem -= sh.above;
    prefix |= d << shift;
    pmask |= dmask << shift;
    top = shift;
    __syncthreads();
  }
  const uint32_t T = prefix;
  const uint32_t need = krem;  // >= 1 elements equal to T still to take
  // mark v > T and v == T with wave ballots (64 consecutive slots per wave)
  for (int base = 0; base < n; base += kSelBlock) {
    const int i = base + tid;
    bool ok = i < n;
    if (ok && excl) ok = !mask_bit(excl, i);
    const uint32_t v = ok ? vals[i] : 0u;
    const uint64_t gt = __ballot(ok && v > T);
    const uint64_t eq = __ballot(ok && v == T);
    const int w0 = (base + (int)wave_id() * kWave) >> 5;
    if (lane_id() == 0 && w0 < nw) {
      sel[w0] = (uint32_t)gt;
      sel[w0 + 1] = (uint32_t)(gt >> 32);
      tie[w0] = (uint32_t)eq;
      tie[w0 + 1] = (uint32_t)(eq >> 32);
    }
  }
  __syncthreads();
  // ties: take `need` of them in slot order (ascending) or from the top (descending)
  if (wave_id() == 0) {
    uint32_t total = 0;
    for (int w = lane_id(); w < nw; w += kWave) total += __popc(tie[w]);
    total = wave_sum(total);
    if (total == need) {
      for (int w = lane_id(); w < nw; w += kWave) sel[w] |= tie[w];
    } else {
      const uint32_t lo = tie_low ? 0u : total - need;
      const uint32_t hi = lo + need;
      uint32_t run = 0;  // ties in words before this iteration's first word
      for (int w0 = 0; w0 < nw; w0 += kWave) {
        const int w = w0 + (int)lane_id();
        const uint32_t word = w < nw ? tie[w] : 0u;
        const uint32_t c = __popc(word);
        const uint32_t incl = wave_incl_scan(c);
        const uint32_t before = run + incl - c;
        if (w < nw && c > 0 && before < hi && before + c > lo) {
          uint32_t bits = word, r = before, take = 0;
          while (bits) {
            const uint32_t b = __ffs(bits) - 1;
            bits &= bits - 1;
            if (r >= lo && r < hi) take |= 1u << b;
            ++r;
          }
          sel[w] |= take;
        }
        run += __shfl(incl, kWave - 1, kWave);
      }
    }
  }
  __syncthreads();
}

}  // namespace
}  // namespace vase
