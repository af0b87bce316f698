// peaks.hip -- measurement probes for the roofline denominators (built as
// libvase_peaks.so, loaded only by the benchmark; not part of the round).
//
// Each probe runs one kernel that saturates one unit of the chip, so that the
// benchmark can time it with events and report the measured peak beside the
// datasheet figure:
//   peaks_copy   a plain device copy, 16 bytes per thread per step (HBM read + write)
//   peaks_read   a read-only sum over a buffer (HBM read)
//   peaks_mfma   back-to-back v_mfma_f32_32x32x16_bf16 on register operands
//   peaks_exp2   independent chains of v_exp_f32 (the score's transcendental)
//   peaks_fma    independent chains of fp32 fma (plain VALU issue rate)
//   peaks_coexec MFMA and VALU work alone, and together (within each wave or
//                split over the two waves of a SIMD)
// Every kernel writes one value per thread into `out`, sized by the caller to
// the launched thread count, so that no work is optimised away.
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));

constexpr int kBlock = 256;

// U pieces of 16 bytes per thread and step, all loads issued before the stores
// so that each thread keeps U requests in flight
template <int U>
__global__ __launch_bounds__(kBlock) void copy_kernel(const uint4* __restrict__ src,
                                                      uint4* __restrict__ dst, size_t n16) {
  const size_t stride = (size_t)gridDim.x * kBlock;
  size_t i = (size_t)blockIdx.x * kBlock + threadIdx.x;
  for (; i + (U - 1) * stride < n16; i += U * stride) {
    uint4 x[U];
#pragma unroll
    for (int u = 0; u < U; ++u) x[u] = src[i + u * stride];
#pragma unroll
    for (int u = 0; u < U; ++u) dst[i + u * stride] = x[u];
  }
  for (; i < n16; i += stride) dst[i] = src[i];
}

template <int U>
__global__ __launch_bounds__(kBlock) void read_kernel(const uint4* __restrict__ src, size_t n16,
                                                      uint32_t* __restrict__ out) {
  const size_t stride = (size_t)gridDim.x * kBlock;
  uint32_t acc = 0;
  size_t i = (size_t)blockIdx.x * kBlock + threadIdx.x;
  for (; i + (U - 1) * stride < n16; i += U * stride) {
    uint4 x[U];
#pragma unroll
    for (int u = 0; u < U; ++u) x[u] = src[i + u * stride];
#pragma unroll
    for (int u = 0; u < U; ++u) acc ^= x[u].x ^ x[u].y ^ x[u].z ^ x[u].w;
  }
  for (; i < n16; i += stride) {
    const uint4 x = src[i];
    acc ^= x.x ^ x.y ^ x.z ^ x.w;
  }
  out[(size_t)blockIdx.x * kBlock + threadIdx.x] = acc;
}

// 4 independent accumulator chains per wave; the operands come from the thread
// id so that nothing folds at compile time
__global__ __launch_bounds__(kBlock) void mfma_kernel(int iters, float* __restrict__ out) {
  const int t = threadIdx.x;
  bf16x8_t a, b;
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    a[i] = (__bf16)(0.001f * (float)((t + i) & 7));
    b[i] = (__bf16)(0.002f * (float)((t * 3 + i) & 7));
  }
  f32x16_t acc[4] = {};
  for (int it = 0; it < iters; ++it) {
#pragma unroll
    for (int c = 0; c < 4; ++c) acc[c] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, acc[c], 0, 0, 0);
  }
  float s = 0.f;
#pragma unroll
  for (int c = 0; c < 4; ++c)
#pragma unroll
    for (int r = 0; r < 16; ++r) s += acc[c][r];
  out[(size_t)blockIdx.x * kBlock + t] = s;
}

// x <- 2^-x keeps every chain in [0.5, 1]: one v_exp_f32 per step (the
// negation is a source modifier)
__global__ __launch_bounds__(kBlock) void exp2_kernel(int iters, float* __restrict__ out) {
  float x[8];
#pragma unroll
  for (int c = 0; c < 8; ++c) x[c] = 0.1f * (float)((threadIdx.x + c) & 7);
  for (int it = 0; it < iters; ++it) {
#pragma unroll
    for (int c = 0; c < 8; ++c) x[c] = __builtin_amdgcn_exp2f(-x[c]);
  }
  float s = 0.f;
#pragma unroll
  for (int c = 0; c < 8; ++c) s += x[c];
  out[(size_t)blockIdx.x * kBlock + threadIdx.x] = s;
}

__global__ __launch_bounds__(kBlock) void fma_kernel(int iters, float m, float* __restrict__ out) {
  float x[8];
#pragma unroll
  for (int c = 0; c < 8; ++c) x[c] = 0.1f * (float)((threadIdx.x + c) & 7);
  for (int it = 0; it < iters; ++it) {
#pragma unroll
    for (int c = 0; c < 8; ++c) x[c] = __builtin_fmaf(x[c], m, 0.25f);
  }
  float s = 0.f;
#pragma unroll
  for (int c = 0; c < 8; ++c) s += x[c];
  out[(size_t)blockIdx.x * kBlock + threadIdx.x] = s;
}

// Co-execution of MFMA and VALU work.  Per loop step and wave: M pairs of
// v_mfma_f32_32x32x16_bf16 (two accumulator chains) and V groups of 8 x (fma,
// exp2, add) on registers, each group depending on the running sums (so nothing
// is hoisted).  ROLE 2: both kinds in every wave, interleaved; ROLE 1: even
// waves do 2M pairs and odd waves 2V groups (the same totals per wave pair).
// M = 0 or V = 0 measures one kind alone.
template <int ROLE, int M, int V>
__global__ __launch_bounds__(kBlock) void coexec_kernel(int iters, float* __restrict__ out) {
  const int t = threadIdx.x;
  const int wave = __builtin_amdgcn_readfirstlane(t / 64);
  bf16x8_t a, b;
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    a[i] = (__bf16)(0.001f * (float)((t + i) & 7));
    b[i] = (__bf16)(0.002f * (float)((t * 3 + i) & 7));
  }
  f32x16_t acc0 = {}, acc1 = {};
  float x[8], s[8];
#pragma unroll
  for (int c = 0; c < 8; ++c) {
    x[c] = 0.01f * (float)((t + c) & 7);
    s[c] = 0.f;
  }
  const int mp = ROLE == 2 ? M : ((wave & 1) == 0 ? 2 * M : 0);
  const int vg = ROLE == 2 ? V : ((wave & 1) == 1 ? 2 * V : 0);
  for (int it = 0; it < iters; ++it) {
    const int n = mp > vg ? mp : vg;
    for (int i = 0; i < n; ++i) {
      if (i < mp) {
        acc0 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, acc0, 0, 0, 0);
        acc1 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, acc1, 0, 0, 0);
      }
      // spread the VALU groups evenly over the MFMA pairs
      const bool grp = mp == 0 ? i < vg : (i * vg) / mp != ((i + 1) * vg) / mp;
      if (grp) {
#pragma unroll
        for (int c = 0; c < 8; ++c)
          s[c] += __builtin_amdgcn_exp2f(__builtin_fmaf(s[c], -1e-7f, x[c]));
      }
    }
  }
  float r = 0.f;
#pragma unroll
  for (int c = 0; c < 8; ++c) r += s[c];
#pragma unroll
  for (int i = 0; i < 16; ++i) r += acc0[i] + acc1[i];
  out[(size_t)blockIdx.x * kBlock + t] = r;
}

int done() { return hipGetLastError() == hipSuccess ? 0 : -4; }

}  // namespace

// All entry points enqueue on `stream` (a hipStream_t) and return 0, -1 for
// bad arguments or -4 for a failed launch.  `out` must hold blocks * 256
// elements.  Sizes are in 16-byte units (n16) or loop iterations per thread.
// unroll: 1, 4 or 8 pieces in flight per thread
extern "C" int peaks_copy(const void* src, void* dst, size_t n16, int blocks, int unroll,
                          void* stream) {
  if (!src || !dst || n16 == 0 || blocks < 1) return -1;
  const hipStream_t s = static_cast<hipStream_t>(stream);
  const uint4* a = static_cast<const uint4*>(src);
  uint4* b = static_cast<uint4*>(dst);
  if (unroll == 1) hipLaunchKernelGGL(copy_kernel<1>, dim3(blocks), dim3(kBlock), 0, s, a, b, n16);
  else if (unroll == 4) hipLaunchKernelGGL(copy_kernel<4>, dim3(blocks), dim3(kBlock), 0, s, a, b, n16);
  else if (unroll == 8) hipLaunchKernelGGL(copy_kernel<8>, dim3(blocks), dim3(kBlock), 0, s, a, b, n16);
  else return -1;
  return done();
}

extern "C" int peaks_read(const void* src, size_t n16, int blocks, int unroll, uint32_t* out,
                          void* stream) {
  if (!src || !out || n16 == 0 || blocks < 1) return -1;
  const hipStream_t s = static_cast<hipStream_t>(stream);
  const uint4* a = static_cast<const uint4*>(src);
  if (unroll == 1) hipLaunchKernelGGL(read_kernel<1>, dim3(blocks), dim3(kBlock), 0, s, a, n16, out);
  else if (unroll == 4) hipLaunchKernelGGL(read_kernel<4>, dim3(blocks), dim3(kBlock), 0, s, a, n16, out);
  else if (unroll == 8) hipLaunchKernelGGL(read_kernel<8>, dim3(blocks), dim3(kBlock), 0, s, a, n16, out);
  else return -1;
  return done();
}

// flops per launch: blocks * 4 waves * iters * 4 * 2 * 32 * 32 * 16
extern "C" int peaks_mfma(int blocks, int iters, float* out, void* stream) {
  if (!out || blocks < 1 || iters < 1) return -1;
  hipLaunchKernelGGL(mfma_kernel, dim3(blocks), dim3(kBlock), 0, static_cast<hipStream_t>(stream),
                     iters, out);
  return done();
}

// exp2 per launch: blocks * 256 * iters * 8
extern "C" int peaks_exp2(int blocks, int iters, float* out, void* stream) {
  if (!out || blocks < 1 || iters < 1) return -1;
  hipLaunchKernelGGL(exp2_kernel, dim3(blocks), dim3(kBlock), 0, static_cast<hipStream_t>(stream),
                     iters, out);
  return done();
}

// fma per launch: blocks * 256 * iters * 8
extern "C" int peaks_fma(int blocks, int iters, float* out, void* stream) {
  if (!out || blocks < 1 || iters < 1) return -1;
  hipLaunchKernelGGL(fma_kernel, dim3(blocks), dim3(kBlock), 0, static_cast<hipStream_t>(stream),
                     iters, 0.999f, out);
  return done();
}

// which: 0 MFMA alone (8 pairs), 1 VALU alone (4 groups), 2 both interleaved in
// every wave (8 pairs + 4 groups), 3 both split over even and odd waves
extern "C" int peaks_coexec(int which, int blocks, int iters, float* out, void* stream) {
  if (!out || blocks < 1 || iters < 1) return -1;
  const hipStream_t s = static_cast<hipStream_t>(stream);
  switch (which) {
    case 0: hipLaunchKernelGGL((coexec_kernel<2, 8, 0>), dim3(blocks), dim3(kBlock), 0, s, iters, out); break;
    case 1: hipLaunchKernelGGL((coexec_kernel<2, 0, 4>), dim3(blocks), dim3(kBlock), 0, s, iters, out); break;
    case 2: hipLaunchKernelGGL((coexec_kernel<2, 8, 4>), dim3(blocks), dim3(kBlock), 0, s, iters, out); break;
    case 3: hipLaunchKernelGGL((coexec_kernel<1, 8, 4>), dim3(blocks), dim3(kBlock), 0, s, iters, out); break;
    default: return -1;
  }
  return done();
}
