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
//   peaks_score_step  the score kernel's key-loop step on synthetic operands,
//                with and without its ring DMA, timed and clocked (shader
//                cycles over the 100 MHz reference counter)
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

// The score kernel's step: 8 waves per workgroup (2 per SIMD), per wave and
// step 16 v_mfma_f32_32x32x16_bf16 (two 32-row blocks x 8 depth steps) whose B
// operands are read from an 8-slot LDS ring with a wait per depth step, the
// epilogue (fma, exp2, add) of the previous step's 32 accumulator elements, and
// an s_barrier after every second step.  MEM 0 moves no data; MEM 1 and 2 add
// the kernel's ring refill, one 1 KB global->LDS DMA per wave and step (a
// 32-key chunk per workgroup step, fetched 6 steps ahead, waited for 3 steps
// ahead), from a 2 MiB window that stays in L2 (1) or from a 2 GiB streamed
// window (2, HBM).  EPI false leaves out the epilogue.  The operands are the
// caller's data (the A fragments and the initial ring from the first 2 MiB of
// `src`), since the MFMA's power draw, and so the clock the part sustains,
// depends on the operand bits; PAT replaces them by a few repeated small
// values (for comparison).
typedef __attribute__((address_space(3))) void lds_void_t;

template <int OFF>
__device__ __forceinline__ bf16x8_t ring_read(uint32_t addr) {
  bf16x8_t v;
  asm volatile("ds_read_b128 %0, %1 offset:%2" : "=v"(v) : "v"(addr), "i"(OFF));
  return v;
}

constexpr int kStepBlock = 512;
constexpr int kRingU4 = 512;          // 16-byte pieces per ring slot (8 KB)

template <int MEM, bool EPI>
struct StepBody {
  const bf16x8_t (&a)[2][8];
  const uint32_t (&ba)[8];
  f32x16_t (&acc)[2][2];
  float (&rs)[32];
  float (&l)[32];
  uint4* ring;
  const uint4* src;
  uint32_t off0, mask;
  int wave;
  float c;
  template <int U>
  __device__ __forceinline__ void step(int it) {
    if (MEM != 0) {
      // refill: piece (wave, lane) of the chunk 6 steps ahead
      const uint32_t o = (off0 + (uint32_t)(8 * it + U) * (uint32_t)kRingU4) & mask;
      __builtin_amdgcn_global_load_lds(
          static_cast<const void*>(reinterpret_cast<const char*>(src) + (size_t)o * 16u),
          (lds_void_t*)(ring + ((U + 6) % 8) * kRingU4 + wave * 64), 16, 0, 0);
    }
    bf16x8_t b[8];
#pragma unroll
    for (int k = 0; k < 8; ++k) b[k] = ring_read<((U + 1) % 8) * kRingU4 * 16>(ba[k]);
    acc[(U + 1) % 2][0] = f32x16_t{};
    acc[(U + 1) % 2][1] = f32x16_t{};
#pragma unroll
    for (int k = 0; k < 8; ++k) {
      asm volatile("s_waitcnt lgkmcnt(%1)" : "+v"(b[k]) : "i"(7 - k));
      acc[(U + 1) % 2][0] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[0][k], b[k], acc[(U + 1) % 2][0], 0, 0, 0);
      acc[(U + 1) % 2][1] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[1][k], b[k], acc[(U + 1) % 2][1], 0, 0, 0);
    }
    if (EPI) {
#pragma unroll
      for (int e = 0; e < 32; ++e)
        l[e] += __builtin_amdgcn_exp2f(__builtin_fmaf(acc[U % 2][e / 16][e % 16], c, -rs[e]));
    } else {
      asm volatile("" : : "v"(acc[U % 2][0]), "v"(acc[U % 2][1]));   // keep every MFMA
    }
    __builtin_amdgcn_sched_barrier(0);
    if (U % 2 == 1) {
      asm volatile("" ::: "memory");
      __builtin_amdgcn_s_waitcnt(0x0070 | 3);   // vmcnt(3) expcnt(7) lgkmcnt(0)
      __builtin_amdgcn_s_barrier();
      asm volatile("" ::: "memory");
    }
  }
};

template <int MEM, bool EPI, bool PAT>
__global__ __launch_bounds__(kStepBlock, 2) void score_step_kernel(const uint4* __restrict__ src,
                                                                   uint32_t mask, int iters, float c,
                                                                   float* __restrict__ out,
                                                                   unsigned long long* __restrict__ clk) {
  __shared__ uint4 ring[8 * kRingU4];   // 64 KB, as the score kernel's ring
  const unsigned long long c0 = __builtin_amdgcn_s_memtime();
  const unsigned long long r0 = __builtin_amdgcn_s_memrealtime();
  const int t = threadIdx.x, lane = t % 64;
  const int wave = __builtin_amdgcn_readfirstlane(t / 64);
  // the ring and the A fragments from the first 2 MiB of src (in the L2 window)
  const uint32_t w0 = ((uint32_t)blockIdx.x * 8u * kRingU4) & ((2u << 20) / 16u - 1u);
  for (int i = t; i < 8 * kRingU4; i += kStepBlock)
    ring[i] = PAT ? make_uint4(0x3c003c00u, 0x3c803c80u, 0x3d003d00u, 0x3d803d80u)
                  : src[(w0 + (uint32_t)i) & ((2u << 20) / 16u - 1u)];
  __syncthreads();
  bf16x8_t a[2][8];
#pragma unroll
  for (int f = 0; f < 2; ++f)
#pragma unroll
    for (int k = 0; k < 8; ++k) {
      if (PAT) {
#pragma unroll
        for (int i = 0; i < 8; ++i) a[f][k][i] = (__bf16)(0.001f * (float)((t + i + f + k) & 7));
      } else {
        a[f][k] = __builtin_bit_cast(bf16x8_t,
                                     src[(w0 + (uint32_t)(t * 16 + f * 8 + k)) & ((2u << 20) / 16u - 1u)]);
      }
    }
  // B-operand piece addresses of ring slot 0: lane l reads row l % 32, piece
  // 2k + l / 32, XOR-swizzled by the row's line as in the kernel (inside 8 KB)
  uint32_t ba[8];
#pragma unroll
  for (int k = 0; k < 8; ++k)
    ba[k] = (uint32_t)(uintptr_t)(const __attribute__((address_space(3))) uint4*)(
        ring + (lane % 32) * 16 + ((2 * k + lane / 32) ^ (lane % 16)));
  f32x16_t acc[2][2];
#pragma unroll
  for (int s = 0; s < 2; ++s) acc[s][0] = acc[s][1] = f32x16_t{};
  float rs[32], l[32];
#pragma unroll
  for (int i = 0; i < 32; ++i) { rs[i] = 0.01f * (float)((t + i) & 15); l[i] = 0.f; }
  // this workgroup's stream: consecutive 8 KB chunks, each wave one 1 KB piece
  const uint32_t off0 = (uint32_t)blockIdx.x * (uint32_t)(8 * iters) * (uint32_t)kRingU4 +
                        (uint32_t)(wave * 64 + lane);
  StepBody<MEM, EPI> sb{a, ba, acc, rs, l, ring, src, off0, mask, wave, c};
  for (int it = 0; it < iters; ++it) {
    sb.template step<0>(it); sb.template step<1>(it); sb.template step<2>(it); sb.template step<3>(it);
    sb.template step<4>(it); sb.template step<5>(it); sb.template step<6>(it); sb.template step<7>(it);
  }
  __builtin_amdgcn_s_waitcnt(0);   // trailing DMA
  float r = 0.f;
#pragma unroll
  for (int i = 0; i < 32; ++i) r += l[i];
#pragma unroll
  for (int s = 0; s < 2; ++s)
#pragma unroll
    for (int i = 0; i < 16; ++i) r += acc[s][0][i] + acc[s][1][i];
  out[(size_t)blockIdx.x * kStepBlock + t] = r;
  if (t == 0) {
    clk[2 * blockIdx.x] = __builtin_amdgcn_s_memtime() - c0;
    clk[2 * blockIdx.x + 1] = __builtin_amdgcn_s_memrealtime() - r0;
  }
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

// which: 0 no memory traffic, 1 DMA from L2, 2 DMA from HBM, 3 as 0 without the
// epilogue (MFMA, LDS reads and barriers only), 4 as 0 on patterned operands.
// 8 * iters steps per wave.
// `src` holds at least 2 GiB (it is read when which is 1 or 2); `out` holds
// blocks * 512 floats, `clk` blocks * 2 counters (shader clock and 100 MHz
// reference cycles of each workgroup).
extern "C" int peaks_score_step(int which, const void* src, size_t src_bytes, int blocks, int iters,
                                float* out, unsigned long long* clk, void* stream) {
  if (!out || !clk || !src || blocks < 1 || iters < 1 || which < 0 || which > 4) return -1;
  if (src_bytes < ((size_t)2 << 30)) return -1;
  // every chunk offset is masked into the window, so the DMA stays inside it
  const uint32_t mask = which == 1 ? (uint32_t)((2u << 20) / 16u - 1u) : (uint32_t)((2u << 30) / 16u - 1u);
  const hipStream_t s = static_cast<hipStream_t>(stream);
  const uint4* a = static_cast<const uint4*>(src);
  const float c = 0.1275f;
  switch (which) {
    case 0: hipLaunchKernelGGL((score_step_kernel<0, true, false>), dim3(blocks), dim3(kStepBlock), 0, s, a, mask, iters, c, out, clk); break;
    case 1: hipLaunchKernelGGL((score_step_kernel<1, true, false>), dim3(blocks), dim3(kStepBlock), 0, s, a, mask, iters, c, out, clk); break;
    case 2: hipLaunchKernelGGL((score_step_kernel<2, true, false>), dim3(blocks), dim3(kStepBlock), 0, s, a, mask, iters, c, out, clk); break;
    case 3: hipLaunchKernelGGL((score_step_kernel<0, false, false>), dim3(blocks), dim3(kStepBlock), 0, s, a, mask, iters, c, out, clk); break;
    default: hipLaunchKernelGGL((score_step_kernel<0, true, true>), dim3(blocks), dim3(kStepBlock), 0, s, a, mask, iters, c, out, clk); break;
  }
  return done();
}
