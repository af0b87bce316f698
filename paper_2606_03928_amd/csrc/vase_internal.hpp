// vase_internal.hpp -- device helpers and host launch declarations shared by the
// HIP translation units of libvase (gfx950 only).
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "vase.h"

namespace vase {

constexpr int kWave = 64;

// ---------------------------------------------------------------------------
// element access: bf16 is stored as raw uint16 bits
// ---------------------------------------------------------------------------
struct bf16_t {
  uint16_t bits;
};

__device__ __forceinline__ float to_f32(float x) { return x; }
__device__ __forceinline__ float to_f32(bf16_t x) { return __uint_as_float((uint32_t)x.bits << 16); }
__device__ __forceinline__ float bf16lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16hi(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }

// fp32 -> bf16, round to nearest even (finite inputs; NaN stays NaN).
__device__ __forceinline__ uint16_t f32_to_bf16_bits(float f) {
  uint32_t u = __float_as_uint(f);
  if ((u & 0x7fffffffu) > 0x7f800000u) return (uint16_t)((u >> 16) | 0x40u);
  u += 0x7fffu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}

template <typename T>
__device__ __forceinline__ void store_out(T* p, float v);
template <>
__device__ __forceinline__ void store_out<float>(float* p, float v) { *p = v; }
template <>
__device__ __forceinline__ void store_out<bf16_t>(bf16_t* p, float v) { p->bits = f32_to_bf16_bits(v); }

// Unpack 16 bytes of elements into fp32 (8 bf16 or 4 fp32 values).
template <typename T>
struct Vec16;
template <>
struct Vec16<bf16_t> {
  static constexpr int n = 8;
  __device__ __forceinline__ static void unpack(const uint4& w, float* out) {
    out[0] = bf16lo(w.x); out[1] = bf16hi(w.x);
    out[2] = bf16lo(w.y); out[3] = bf16hi(w.y);
    out[4] = bf16lo(w.z); out[5] = bf16hi(w.z);
    out[6] = bf16lo(w.w); out[7] = bf16hi(w.w);
  }
};
template <>
struct Vec16<float> {
  static constexpr int n = 4;
  __device__ __forceinline__ static void unpack(const uint4& w, float* out) {
    out[0] = __uint_as_float(w.x); out[1] = __uint_as_float(w.y);
    out[2] = __uint_as_float(w.z); out[3] = __uint_as_float(w.w);
  }
};

// ---------------------------------------------------------------------------
// sums over the lanes that hold one row (DPP butterflies; every lane of the
// row ends with the sum)
// ---------------------------------------------------------------------------
// x summed over the 16 lanes of a DPP row (butterfly: lane^1, lane^2, mirror
// within 8, mirror within 16); every lane of the row ends with the sum.
__device__ __forceinline__ float row16_sum(float x) {
  x += __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(x), 0xB1, 0xf, 0xf, false));
  x += __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(x), 0x4E, 0xf, 0xf, false));
  x += __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(x), 0x141, 0xf, 0xf, false));
  x += __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(x), 0x140, 0xf, 0xf, false));
  return x;
}
// the same over 8 lanes (lane^1, lane^2, mirror within 8)
__device__ __forceinline__ float row8_sum(float x) {
  x += __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(x), 0xB1, 0xf, 0xf, false));
  x += __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(x), 0x4E, 0xf, 0xf, false));
  x += __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(x), 0x141, 0xf, 0xf, false));
  return x;
}
// sum over the LANES consecutive lanes that hold one row (8, 16 or 32)
template <int LANES>
__device__ __forceinline__ float lanes_sum(float x) {
  static_assert(LANES == 8 || LANES == 16 || LANES == 32, "8, 16 or 32 lanes");
  if (LANES == 8) return row8_sum(x);
  x = row16_sum(x);
  if (LANES == 32) x += __shfl_xor(x, 16, kWave);
  return x;
}

// maximum over the LANES consecutive lanes that hold one row (8, 16 or 32)
template <int LANES>
__device__ __forceinline__ float lanes_max(float x) {
  static_assert(LANES == 8 || LANES == 16 || LANES == 32, "8, 16 or 32 lanes");
  x = fmaxf(x, __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(x), 0xB1, 0xf, 0xf, false)));
  x = fmaxf(x, __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(x), 0x4E, 0xf, 0xf, false)));
  x = fmaxf(x, __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(x), 0x141, 0xf, 0xf, false)));
  if (LANES >= 16)
    x = fmaxf(x, __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(x), 0x140, 0xf, 0xf, false)));
  if (LANES == 32) x = fmaxf(x, __shfl_xor(x, 16, kWave));
  return x;
}

// Value score of one row whose d = VEC * LANES elements are spread VEC per lane
// over LANES consecutive lanes: Range = max - min (Eq. 5), L2 = sqrt(sum v^2)
// or Var = (1/d) sum (v - mu)^2, two-pass (the variants of Appendix A).  Every
// lane of the row ends with it; the same operation order wherever it is used,
// so a row's score does not depend on which kernel computed it.
template <int VEC, int LANES>
__device__ __forceinline__ float row_value_score(const float (&f)[VEC], int kind) {
  constexpr float kInvD = 1.0f / (VEC * LANES);
  if (kind == VASE_VALUE_RANGE) {
    float mx = f[0], mn = f[0];
#pragma unroll
    for (int e = 1; e < VEC; ++e) {
      mx = fmaxf(mx, f[e]);
      mn = fminf(mn, f[e]);
    }
    return lanes_max<LANES>(mx) + lanes_max<LANES>(-mn);
  }
  if (kind == VASE_VALUE_L2) {
    float ss = 0.f;
#pragma unroll
    for (int e = 0; e < VEC; ++e) ss = __builtin_fmaf(f[e], f[e], ss);
    return __builtin_sqrtf(lanes_sum<LANES>(ss));
  }
  float s1 = 0.f;
#pragma unroll
  for (int e = 0; e < VEC; ++e) s1 += f[e];
  const float mu = lanes_sum<LANES>(s1) * kInvD;
  float ss = 0.f;
#pragma unroll
  for (int e = 0; e < VEC; ++e) ss = __builtin_fmaf(f[e] - mu, f[e] - mu, ss);
  return lanes_sum<LANES>(ss) * kInvD;
}

// A value row with a NaN or infinite element (checked per lane on its VEC elements).
template <int VEC>
__device__ __forceinline__ bool any_nonfinite(const float (&f)[VEC]) {
  bool bad = false;
#pragma unroll
  for (int e = 0; e < VEC; ++e) bad |= !(__builtin_fabsf(f[e]) <= 3.402823466e38f);
  return bad;
}

// OR `bit` into the caller's device status word (vase.h, VASE_STATUS_*) once per
// workgroup when any of its threads raised `flag`.  Every thread of the
// workgroup must reach the call: it synchronises the workgroup.
__device__ __forceinline__ void block_status(uint32_t* status, bool flag, uint32_t bit) {
  if (__syncthreads_or(flag) && threadIdx.x == 0) atomicOr(status, bit);
}

// ---------------------------------------------------------------------------
// XCD-aware block order.  MI355X dispatches consecutive workgroups round-robin
// over its 8 XCDs (each with a private L2).  Remapping the hardware block id
// gives every XCD one contiguous range of logical blocks, so neighbouring
// logical blocks (e.g. the key chunks of one head instance, which share its
// query window) run on the same XCD and share that L2.
// ---------------------------------------------------------------------------
constexpr int kNumXcd = 8;
__device__ __forceinline__ uint32_t xcd_logical_block(uint32_t hw_block, uint32_t n_blocks) {
  const uint32_t per = n_blocks / kNumXcd, rem = n_blocks % kNumXcd;
  const uint32_t xcd = hw_block % kNumXcd, slot = hw_block / kNumXcd;
  return xcd < rem ? xcd * (per + 1) + slot : rem * (per + 1) + (xcd - rem) * per + slot;
}

// ---------------------------------------------------------------------------
// host-side launchers (defined in the kernel translation units)
// ---------------------------------------------------------------------------
struct ScorePlan {
  int n_chunk1;     // slot ranges of the row-statistics pass (MFMA: ranges per instance)
  int n_chunk2;     // slot ranges of the probability pass
  int n_slab;       // query-row slabs (partial column sums per slab)
  int rows_per_slab;
  int waves;        // MFMA: waves per workgroup (64 query rows each)
  int split_keys;   // MFMA: slots per range (multiple of 32)
  bool mfma;
  bool pool_in_kernel;  // MFMA, one range and one slab per instance: no pool launch
  size_t off_part, off_lse, off_col, bytes;
};
ScorePlan score_plan(int dtype, int n_inst, int K, int B, int d, int G, int w);
// lse_win (nullable): [n_inst][G*w] natural-log LSE of each window row over
// the persistent slots [0, K); when given, row statistics cover [K, N) only
// ord (nullable, only with plan.pool_in_kernel): an order map; the kernel then
// pools over temporal ranks and writes attn and vrange by rank
// dec (bf16 only, no lse_win): with dec.out set, pass 1 also writes the decode
// queries' logits out[inst][g][t] = q[inst][g] . k[inst][t] (raw dot products,
// t < N, g < G <= 16) from the key rows it streams
struct DecLogits {
  const void* q = nullptr;   // [n_inst][G][d] bf16
  int G = 0;
  float* out = nullptr;      // [n_inst][G][N] fp32
};
// status (nullable): device word that collects VASE_STATUS_ROW_NORM (a window
// row's normaliser is not a positive finite number) and VASE_STATUS_VALUE_ROW
// (a value row read by this call has a NaN or infinite element)
hipError_t launch_score(const void* k, const void* v, const void* q, int dtype, int n_inst, int K,
                        int B, int d, int G, int w, int pool, int value_kind, const float* lse_win,
                        float* attn, float* vrange, void* ws, const ScorePlan& plan,
                        hipStream_t stream, const int32_t* ord = nullptr,
                        const DecLogits& dec = DecLogits(), uint32_t* status = nullptr);
// random reservation scores: vrange[i][j] = Philox uniform (purpose 2)
hipError_t launch_value_random(int n_inst, uint32_t inst_base, int K, uint64_t seed,
                               uint32_t round, float* vrange, hipStream_t stream);

// status (nullable): collects VASE_STATUS_SELECT_ATTN and VASE_STATUS_SELECT_VALUE
hipError_t launch_select(const float* attn, const float* vrange, int n_inst, uint32_t inst_base,
                         int K, int B, int Nv, uint64_t seed, uint32_t round, uint32_t flags,
                         int32_t* src, float* keys, hipStream_t stream, uint32_t* status = nullptr);
size_t select_lds_bytes(int K, int B);

struct CompactPlan {
  int n_part;       // destination ranges per instance
  int rows_per_part;
  size_t bytes;     // staging workspace
};
CompactPlan compact_plan(int dtype, int n_inst, int K, int B, int d);
hipError_t launch_compact(void* k, void* v, int dtype, int n_inst, int K, int B, int d,
                          const int32_t* src, void* ws, const CompactPlan& plan,
                          hipStream_t stream);

// Fused compaction + one decode step; only for plans with one part per instance
// and K <= kCompactDecodeMaxK (the survivor map is staged in LDS).
constexpr int kCompactDecodeMaxK = 16384;
// vrange (nullable): value score of kind value_kind of each compacted row [0, K)
hipError_t launch_compact_decode(void* k, void* v, int dtype, int n_inst, int K, int B, int d,
                                 const int32_t* src, const void* q, int G, void* out,
                                 int value_kind, float* vrange, hipStream_t stream);
// value scores (Range, L2 or Var) of rows [0, K) of a [n_inst][N][d] cache
hipError_t launch_value_rows(const void* v, int dtype, int n_inst, int N, int K, int d, int kind,
                             float* out, hipStream_t stream, uint32_t* status = nullptr);

struct DecodePlan {
  int n_split;      // key splits per instance
  int s1;           // splits over [0, n_persist); the rest cover [n_persist, n_valid)
  int rows_per_split;
  size_t bytes;     // partial (m, l, o) per split
};
DecodePlan decode_plan(int dtype, int n_inst, int K, int B, int d, int G, int n_valid,
                       int n_persist);
size_t decode_ws_bytes_max(int dtype, int n_inst, int K, int B, int d, int G);
// the library's own device scratch for the decode split partials (no caller
// workspace): its size, and its address on the current device (set up on the
// first call per device; every later call on that device returns the same one)
constexpr size_t kDecodeScratchBytes = (size_t)64 << 20;
hipError_t decode_scratch(void** ptr);
// lse (nullable): natural-log LSE over slots [0, n_persist) for each query head,
// written to lse[(inst * G + g) * lse_ld]
hipError_t launch_decode(const void* k, const void* v, const void* q, int dtype, int n_inst,
                         int K, int B, int d, int G, int n_valid, int n_persist, void* out,
                         float* lse, int lse_ld, void* ws, const DecodePlan& plan,
                         hipStream_t stream);
hipError_t launch_decode_append(void* k, void* v, const void* k_new, const void* v_new,
                                const void* q, void* q_win, int dtype, int n_inst, int K, int B,
                                int d, int G, int w, int pos, hipStream_t stream);

// The cache under an order map (ord[inst][t] = slot of temporal rank t < K).
// attn_out[t] = P-wide box filter over temporal ranks of attn_phys[ord[.]];
// vr_out[t] = vr_phys[ord[t]] when vr_phys is given.
hipError_t launch_order_scores(const float* attn_phys, const float* vr_phys, const int32_t* ord,
                               int n_inst, int K, int pool, float* attn_out, float* vr_out,
                               hipStream_t stream);
// Compaction under the order map (buffer rows into the evicted slots, new map
// into ord), fused with one decode step when q is given; K <= VASE_MAX_K.
// vrange_in (nullable, may equal vrange): the current candidates' value scores;
// survivors take theirs by rank and only the buffer rows are scored from V
hipError_t launch_compact_map(void* k, void* v, int dtype, int n_inst, int K, int B, int d,
                              const int32_t* src, int32_t* ord, const void* q, int G, void* out,
                              int value_kind, const float* vrange_in, float* vrange,
                              const float* dlog, hipStream_t stream);

// VaSE-DKV: per-instance Gaussian projections and the product score.
constexpr int kDkvMaxRank = 32;
hipError_t launch_dkv_projection(int n_inst, uint32_t inst_base, int d, int r, uint64_t seed,
                                 uint32_t round, float* g, hipStream_t stream);
hipError_t launch_dkv_score(const void* k, const void* v, const float* g, int dtype, int n_inst,
                            int K, int B, int d, int r, float* out, const void* q_dec, int G,
                            float* dec_logits, hipStream_t stream);

// Range-based per-token quantisation (Eq. 6) and its inverse, with a
// full-precision reserve of the N_v largest-Range rows.
hipError_t launch_quantize(const void* x, int dtype, int n_inst, int K, int B, int d, int bits,
                           int group, int Nv, uint8_t* codes, float* params, float* range,
                           float* mse, void* hp_rows, int32_t* hp_idx, hipStream_t stream);
hipError_t launch_dequantize(const uint8_t* codes, const float* params, const void* hp_rows,
                             const int32_t* hp_idx, int dtype, int n_inst, int K, int B, int d,
                             int bits, int group, int Nv, void* out, hipStream_t stream);

}  // namespace vase
