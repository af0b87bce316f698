// quant.hip -- Range-based per-token asymmetric quantisation of a cache (Eq. 6 of
// the paper, Sec. 4.3) with a full-precision reserve for the N_v rows of largest
// Range (the mixed-precision direction of Sec. 7), on gfx950.
//
// Per row and per group of GROUP elements:  z = min x,  Delta = Range / (2^b - 1),
// q_e = rint((x_e - z) / Delta) (ties to even; 0 when Delta = 0), clamped to
// [0, 2^b - 1];  x'_e = fma(q_e, Delta, z).  Codes of a row form a bit stream
// (code e at bits [e*b, e*b + b), little-endian in each byte); params hold
// (Delta, z) per group as fp32.
//
// The code of each element is decided by IEEE binary32 operations only (this
// translation unit is compiled without contraction).  The quotient is first
// formed as (x - z) * r with r the hardware reciprocal of Delta (within 1 ulp
// of 1/Delta), which lies within 3 ulp of the correctly rounded (x - z) / Delta;
// the quotient is at most 2^b - 1 <= 255, so 3 ulp are below 2^-13, and when
// the product is more than 2^-12 away from the nearest half-integer both round
// to the same integer.  Otherwise (or for a non-finite reciprocal) the element
// takes the IEEE divide.  The clamp to [0, 2^b - 1] needs no upper bound: with
// x - z <= Range (rounding is monotonic) the product stays below 2^b - 1/2.
//
// Layout: a row of D elements is spread over LPR = D*e/16 lanes, 16 bytes each;
// a group covers GROUP/VEC consecutive lanes, so its min and max are butterfly
// reductions over those lanes, and the row's Range two more levels up.
#include "vase_internal.hpp"
#include "vase.h"

#pragma clang fp contract(off)

#include "topk.hpp"

#include <type_traits>

namespace vase {
namespace {

constexpr int kQBlock = 256;
constexpr int kQRowsPerBlock = 64;

template <int LANES, bool MAX>
__device__ __forceinline__ float xor_reduce(float x, int from) {
  // reduce over lane bits [log2(from), log2(LANES)): from = 1 reduces LANES lanes
#pragma unroll
  for (int o = 1; o < LANES; o <<= 1) {
    if (o < from) continue;
    const float y = __shfl_xor(x, o, kWave);
    x = MAX ? fmaxf(x, y) : x + y;
  }
  return x;
}

template <int BYTES>
struct CodeStore;
template <>
struct CodeStore<1> {
  __device__ static void put(uint8_t* p, uint64_t c) { *p = (uint8_t)c; }
  __device__ static uint64_t get(const uint8_t* p) { return *p; }
};
template <>
struct CodeStore<2> {
  __device__ static void put(uint8_t* p, uint64_t c) { *reinterpret_cast<uint16_t*>(p) = (uint16_t)c; }
  __device__ static uint64_t get(const uint8_t* p) { return *reinterpret_cast<const uint16_t*>(p); }
};
template <>
struct CodeStore<4> {
  __device__ static void put(uint8_t* p, uint64_t c) { *reinterpret_cast<uint32_t*>(p) = (uint32_t)c; }
  __device__ static uint64_t get(const uint8_t* p) { return *reinterpret_cast<const uint32_t*>(p); }
};
template <>
struct CodeStore<8> {
  __device__ static void put(uint8_t* p, uint64_t c) {
    *reinterpret_cast<uint2*>(p) = make_uint2((uint32_t)c, (uint32_t)(c >> 32));
  }
  __device__ static uint64_t get(const uint8_t* p) {
    const uint2 w = *reinterpret_cast<const uint2*>(p);
    return (uint64_t)w.x | ((uint64_t)w.y << 32);
  }
};

// VEC fp32 values as 16 bytes of T (bf16: round to nearest even)
template <typename T>
__device__ __forceinline__ uint4 pack16(const float* r);
template <>
__device__ __forceinline__ uint4 pack16<float>(const float* r) {
  return make_uint4(__float_as_uint(r[0]), __float_as_uint(r[1]), __float_as_uint(r[2]),
                    __float_as_uint(r[3]));
}
template <>
__device__ __forceinline__ uint4 pack16<bf16_t>(const float* r) {
  uint32_t w[4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
    w[i] = (uint32_t)f32_to_bf16_bits(r[2 * i]) | ((uint32_t)f32_to_bf16_bits(r[2 * i + 1]) << 16);
  return make_uint4(w[0], w[1], w[2], w[3]);
}

// the code of one element (see the file comment for why the fast quotient is safe)
__device__ __forceinline__ float quant_code(float x, float z, float delta, float inv) {
  if (!(delta > 0.0f)) return 0.0f;
  const float t = x - z;
  float q = __builtin_rintf(t * inv);
  const float u = t * inv;
  if (!(__builtin_fabsf(u - q) <= 0.5f - 0x1p-12f)) q = __builtin_rintf(t / delta);
  return fmaxf(q, 0.0f);   // also maps a NaN (non-finite inputs) to 0
}

template <typename T, int D, int BITS, int GROUP>
__global__ __launch_bounds__(kQBlock) void quant_rows_kernel(
    const T* __restrict__ x, int N, int K, uint8_t* __restrict__ codes, float2* __restrict__ params,
    float* __restrict__ range_out, float* __restrict__ mse_out) {
  constexpr int VEC = Vec16<T>::n;
  constexpr int LPR = D / VEC;                 // lanes per row
  constexpr int LPG = GROUP / VEC;             // lanes per group
  constexpr int RPI = kQBlock / LPR;           // rows per block iteration
  constexpr int ITERS = kQRowsPerBlock / RPI;
  constexpr int CB = VEC * BITS / 8;           // code bytes per lane
  constexpr int NG = D / GROUP;
  static_assert(LPG >= 1 && LPG <= LPR && CB >= 1, "group must cover whole lanes");
  const float levels = (float)((1u << BITS) - 1u);
  constexpr float kRcpLevels = 1.0f / (float)((1u << BITS) - 1u);
  const int inst = blockIdx.y;
  const int seg = threadIdx.x % LPR;
  const int r_in = threadIdx.x / LPR;
  const int row0 = blockIdx.x * kQRowsPerBlock;
  const uint4* xb = reinterpret_cast<const uint4*>(x + (size_t)inst * N * D);

  uint4 w[ITERS];
#pragma unroll
  for (int it = 0; it < ITERS; ++it) {
    const int row = row0 + it * RPI + r_in;
    const int rr = row < K ? row : K - 1;
    w[it] = xb[(size_t)rr * LPR + seg];
  }
#pragma unroll
  for (int it = 0; it < ITERS; ++it) {
    const int row = row0 + it * RPI + r_in;
    float f[VEC];
    Vec16<T>::unpack(w[it], f);
    float mn = f[0], mx = f[0];
#pragma unroll
    for (int e = 1; e < VEC; ++e) {
      mn = fminf(mn, f[e]);
      mx = fmaxf(mx, f[e]);
    }
    const float gmn = -xor_reduce<LPG, true>(-mn, 1);
    const float gmx = xor_reduce<LPG, true>(mx, 1);
    // Delta = Range / levels, correctly rounded, from the product with the
    // rounded reciprocal and one fma correction: for the divisors 3, 15 and
    // 255 that is the IEEE quotient for every finite Range >= 0 (the host
    // tests check all of them); an infinite or NaN Range keeps the product
    const float range = gmx - gmn;
    const float q0 = range * kRcpLevels;
    const float qc = __builtin_fmaf(__builtin_fmaf(-q0, levels, range), kRcpLevels, q0);
    const float delta = q0 < INFINITY ? qc : q0;
    const float inv = __builtin_amdgcn_rcpf(delta);
    using Packed = typename std::conditional<VEC * BITS <= 32, uint32_t, uint64_t>::type;
    Packed packed = 0;
    float ss = 0.0f;
#pragma unroll
    for (int e = 0; e < VEC; ++e) {
      const float q = quant_code(f[e], gmn, delta, inv);
      packed |= (Packed)(uint32_t)q << (e * BITS);
      const float diff = f[e] - __builtin_fmaf(q, delta, gmn);
      ss = __builtin_fmaf(diff, diff, ss);
    }
    // the row's Range and squared error over all LPR lanes
    const float rmn = -xor_reduce<LPR, true>(-gmn, LPG);
    const float rmx = xor_reduce<LPR, true>(gmx, LPG);
    ss = xor_reduce<LPR, false>(ss, 1);
    if (row < K) {
      const size_t ri = (size_t)inst * K + row;
      CodeStore<CB>::put(codes + ri * (D * BITS / 8) + seg * CB, packed);
      if (seg % LPG == 0) params[ri * NG + seg / LPG] = make_float2(delta, gmn);
      if (seg == 0) {
        if (range_out) range_out[ri] = rmx - rmn;
        if (mse_out) mse_out[ri] = ss * (1.0f / D);
      }
    }
  }
}

template <typename T, int D, int BITS, int GROUP>
__global__ __launch_bounds__(kQBlock) void dequant_rows_kernel(
    const uint8_t* __restrict__ codes, const float2* __restrict__ params, int N, int K,
    T* __restrict__ out) {
  constexpr int VEC = Vec16<T>::n;
  constexpr int LPR = D / VEC;
  constexpr int LPG = GROUP / VEC;
  constexpr int RPI = kQBlock / LPR;
  constexpr int ITERS = kQRowsPerBlock / RPI;
  constexpr int CB = VEC * BITS / 8;
  constexpr int NG = D / GROUP;
  constexpr uint32_t kMask = (1u << BITS) - 1u;
  const int inst = blockIdx.y;
  const int seg = threadIdx.x % LPR;
  const int r_in = threadIdx.x / LPR;
  const int row0 = blockIdx.x * kQRowsPerBlock;
#pragma unroll
  for (int it = 0; it < ITERS; ++it) {
    const int row = row0 + it * RPI + r_in;
    if (row >= K) break;
    const size_t ri = (size_t)inst * K + row;
    const uint64_t packed = CodeStore<CB>::get(codes + ri * (D * BITS / 8) + seg * CB);
    const float2 p = params[ri * NG + seg / LPG];
    float r[VEC];
#pragma unroll
    for (int e = 0; e < VEC; ++e) {
      const float q = (float)((uint32_t)(packed >> (e * BITS)) & kMask);
      r[e] = __builtin_fmaf(q, p.x, p.y);
    }
    reinterpret_cast<uint4*>(out + ((size_t)inst * N + row) * D)[seg] = pack16<T>(r);
  }
}

// The N_v rows of largest Range (ties: lower slot) of each instance, listed in
// slot order in hp_idx, copied to hp_rows.  One workgroup per instance with
// the K Ranges in registers as bit patterns (Range >= 0, so they order like
// their values); the exact top-k search of topk.hpp.
template <typename T, int D, int V, int NWV>
__global__ __launch_bounds__(NWV * kWave) void quant_reserve_kernel(
    const float* __restrict__ range, int K, int Nv, const T* __restrict__ x, int N,
    T* __restrict__ hp_rows, int32_t* __restrict__ hp_idx) {
  constexpr int NW = (V + 31) / 32;
  constexpr int NT = NWV * kWave;
  extern __shared__ int32_t order[];   // [Nv] the selected slots, ascending
  __shared__ SelectShared<NWV> sh;
  const int inst = blockIdx.x;
  const int s0 = V * (int)threadIdx.x;
  const int n_t = min(max(K - s0, 0), V);
  uint32_t in_k[NW];
  slots_below<V>(K, in_k);
  uint32_t v[V];
  thread_load<V>(range + (size_t)inst * K + min(s0, K - 1), n_t, v);
  uint32_t sel[NW];
  block_select_top_regs<V, NWV>(v, in_k, (uint32_t)Nv, /*tie_low=*/true, sel, sh);
  block_list_slots<V, NWV>(sel, order, hp_idx + (size_t)inst * Nv, sh);
  __syncthreads();
  constexpr int kU4 = D * (int)sizeof(T) / 16;
  const uint4* xb = reinterpret_cast<const uint4*>(x + (size_t)inst * N * D);
  uint4* hb = reinterpret_cast<uint4*>(hp_rows + (size_t)inst * Nv * D);
  for (int t = threadIdx.x; t < Nv * kU4; t += NT) {
    const int s = order[t / kU4];
    hb[t] = xb[(size_t)s * kU4 + t % kU4];
  }
}

template <typename T, int D>
__global__ __launch_bounds__(256) void dequant_reserve_kernel(const T* __restrict__ hp_rows,
                                                             const int32_t* __restrict__ hp_idx,
                                                             int K, int Nv, int N,
                                                             T* __restrict__ out) {
  constexpr int kU4 = D * (int)sizeof(T) / 16;
  const int inst = blockIdx.x;
  const uint4* hb = reinterpret_cast<const uint4*>(hp_rows + (size_t)inst * Nv * D);
  uint4* ob = reinterpret_cast<uint4*>(out + (size_t)inst * N * D);
  for (int t = threadIdx.x; t < Nv * kU4; t += 256) {
    const int s = hp_idx[(size_t)inst * Nv + t / kU4];
    if (s >= 0 && s < K) ob[(size_t)s * kU4 + t % kU4] = hb[t];
  }
}

struct QuantArgs {
  const void* x;
  const uint8_t* codes_in;
  uint8_t* codes;
  const float* params_in;
  float* params;
  float* range;
  float* mse;
  const void* hp_in;
  void* hp;
  const int32_t* idx_in;
  int32_t* idx;
  void* out;
  int n_inst, N, K, Nv;
};

template <typename T, int D, int BITS, int GROUP>
hipError_t run_bg(const QuantArgs& a, bool quant, hipStream_t s) {
  const dim3 grid((a.K + kQRowsPerBlock - 1) / kQRowsPerBlock, a.n_inst);
  if (quant) {
    hipLaunchKernelGGL((quant_rows_kernel<T, D, BITS, GROUP>), grid, dim3(kQBlock), 0, s,
                       static_cast<const T*>(a.x), a.N, a.K, a.codes,
                       reinterpret_cast<float2*>(a.params), a.range, a.mse);
    if (a.Nv > 0) {
      const size_t lds = sizeof(int32_t) * (size_t)a.Nv;
      with_topk_layout(a.K, [&](auto v_, auto nw_) {
        constexpr int V = decltype(v_)::value, NWV = decltype(nw_)::value;
        hipLaunchKernelGGL((quant_reserve_kernel<T, D, V, NWV>), dim3(a.n_inst), dim3(NWV * kWave),
                           lds, s, a.range, a.K, a.Nv, static_cast<const T*>(a.x), a.N,
                           static_cast<T*>(a.hp), a.idx);
      });
    }
  } else {
    hipLaunchKernelGGL((dequant_rows_kernel<T, D, BITS, GROUP>), grid, dim3(kQBlock), 0, s,
                       a.codes_in, reinterpret_cast<const float2*>(a.params_in), a.N, a.K,
                       static_cast<T*>(a.out));
    if (a.Nv > 0) {
      hipLaunchKernelGGL((dequant_reserve_kernel<T, D>), dim3(a.n_inst), dim3(256), 0, s,
                         static_cast<const T*>(a.hp_in), a.idx_in, a.K, a.Nv, a.N,
                         static_cast<T*>(a.out));
    }
  }
  return hipGetLastError();
}

template <typename T, int D, int BITS>
hipError_t run_b(const QuantArgs& a, int group, bool quant, hipStream_t s) {
  switch (group) {
    case 32: return run_bg<T, D, BITS, 32>(a, quant, s);
    case 64: return run_bg<T, D, BITS, 64>(a, quant, s);
    case 128:
      if constexpr (D >= 128) return run_bg<T, D, BITS, 128>(a, quant, s);
      return hipErrorInvalidValue;
    default: return hipErrorInvalidValue;
  }
}

template <typename T, int D>
hipError_t run_d(const QuantArgs& a, int bits, int group, bool quant, hipStream_t s) {
  switch (bits) {
    case 2: return run_b<T, D, 2>(a, group, quant, s);
    case 4: return run_b<T, D, 4>(a, group, quant, s);
    case 8: return run_b<T, D, 8>(a, group, quant, s);
    default: return hipErrorInvalidValue;
  }
}

hipError_t run_quant(const QuantArgs& a, int dtype, int d, int bits, int group, bool quant,
                     hipStream_t s) {
  if (dtype == VASE_BF16) {
    if (d == 128) return run_d<bf16_t, 128>(a, bits, group, quant, s);
    if (d == 64) return run_d<bf16_t, 64>(a, bits, group, quant, s);
  } else {
    if (d == 128) return run_d<float, 128>(a, bits, group, quant, s);
    if (d == 64) return run_d<float, 64>(a, bits, group, quant, s);
  }
  return hipErrorInvalidValue;
}

}  // namespace

hipError_t launch_quantize(const void* x, int dtype, int n_inst, int K, int B, int d, int bits,
                           int group, int Nv, uint8_t* codes, float* params, float* range,
                           float* mse, void* hp_rows, int32_t* hp_idx, hipStream_t stream) {
  QuantArgs a{};
  a.x = x;
  a.codes = codes;
  a.params = params;
  a.range = range;
  a.mse = mse;
  a.hp = hp_rows;
  a.idx = hp_idx;
  a.n_inst = n_inst;
  a.N = K + B;
  a.K = K;
  a.Nv = Nv;
  return run_quant(a, dtype, d, bits, group, true, stream);
}

hipError_t launch_dequantize(const uint8_t* codes, const float* params, const void* hp_rows,
                             const int32_t* hp_idx, int dtype, int n_inst, int K, int B, int d,
                             int bits, int group, int Nv, void* out, hipStream_t stream) {
  QuantArgs a{};
  a.codes_in = codes;
  a.params_in = params;
  a.hp_in = hp_rows;
  a.idx_in = hp_idx;
  a.out = out;
  a.n_inst = n_inst;
  a.N = K + B;
  a.K = K;
  a.Nv = Nv;
  return run_quant(a, dtype, d, bits, group, false, stream);
}

}  // namespace vase
