// rng_probe.hip -- test helper, not part of the library.  Evaluates the
// library's device random-number functions (paper_2606_03928_amd/csrc/rng.hpp)
// on caller-chosen inputs so that the GPU tests can compare them bit for bit
// with the oracle's independent implementation.  Built with the flags of the
// library's translation units that use rng.hpp (-ffp-contract=off, no packed
// fp32).
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "rng.hpp"

namespace {

// out[i] = neg_log(uniform_from_word((first + i) << 9)) for i < n: every u of the
// uniform map is an odd multiple of 2^-24 picked by the word's top 23 bits.
__global__ void neglog_words(float* __restrict__ out, uint32_t first, uint32_t n) {
  const uint32_t i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) out[i] = vase::neg_log(vase::uniform_from_word((first + i) << 9));
}

// out[i] = cos_2pi(uniform_from_word((first + i) << 9)) for i < n.
__global__ void cos2pi_words(float* __restrict__ out, uint32_t first, uint32_t n) {
  const uint32_t i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) out[i] = vase::cos_2pi(vase::uniform_from_word((first + i) << 9));
}

// Philox4x32-10 of counters (c0 + i, c1, c2, c3), key (k0, k1), into out[4 i .. 4 i + 3].
__global__ void philox_blocks(uint32_t* __restrict__ out, uint32_t c0, uint32_t c1, uint32_t c2,
                              uint32_t c3, uint32_t k0, uint32_t k1, uint32_t n) {
  const uint32_t i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= n) return;
  const uint4 x = vase::philox4x32_10(make_uint4(c0 + i, c1, c2, c3), k0, k1);
  out[4 * (size_t)i + 0] = x.x;
  out[4 * (size_t)i + 1] = x.y;
  out[4 * (size_t)i + 2] = x.z;
  out[4 * (size_t)i + 3] = x.w;
}

constexpr uint32_t kBlock = 256;

int finish() { return hipGetLastError() == hipSuccess ? 0 : -4; }

}  // namespace

// Each entry point enqueues one launch on `stream` (a hipStream_t) over device
// buffers the caller owns and returns 0, -1 for a null pointer or n = 0, or -4
// when the launch fails.
extern "C" int rngprobe_neglog(float* out, uint32_t first, uint32_t n, void* stream) {
  if (!out || n == 0) return -1;
  hipLaunchKernelGGL(neglog_words, dim3((n + kBlock - 1) / kBlock), dim3(kBlock), 0,
                     static_cast<hipStream_t>(stream), out, first, n);
  return finish();
}

extern "C" int rngprobe_cos2pi(float* out, uint32_t first, uint32_t n, void* stream) {
  if (!out || n == 0) return -1;
  hipLaunchKernelGGL(cos2pi_words, dim3((n + kBlock - 1) / kBlock), dim3(kBlock), 0,
                     static_cast<hipStream_t>(stream), out, first, n);
  return finish();
}

extern "C" int rngprobe_philox(uint32_t* out, uint32_t c0, uint32_t c1, uint32_t c2, uint32_t c3,
                               uint32_t k0, uint32_t k1, uint32_t n, void* stream) {
  if (!out || n == 0) return -1;
  hipLaunchKernelGGL(philox_blocks, dim3((n + kBlock - 1) / kBlock), dim3(kBlock), 0,
                     static_cast<hipStream_t>(stream), out, c0, c1, c2, c3, k0, k1, n);
  return finish();
}
