// Host driver for the sanitizer build of the C ABI (test infrastructure).
// libvase's host code is compiled with -fsanitize=address,undefined (device
// code unchanged); this program calls every entry point with arguments that
// the host-side validation must reject -- so no call reaches the device and no
// GPU is needed -- and vase_workspace_bytes over a sweep of shapes up to the
// largest accepted ones, where size arithmetic could overflow.  Prints "ok".
#include <cstdint>
#include <cstdio>
#include <cstdlib>

#include "vase.h"

#define EXPECT(x, code)                                                            \
  do {                                                                             \
    const int rc_ = (x);                                                           \
    if (rc_ != (code)) {                                                           \
      std::printf("FAIL %s -> %d (want %d)\n", #x, rc_, (int)(code));              \
      std::exit(1);                                                                \
    }                                                                              \
  } while (0)

int main() {
  void* f = reinterpret_cast<void*>(uintptr_t(1) << 20);   // aligned, never dereferenced
  void* m = reinterpret_cast<void*>((uintptr_t(1) << 20) + 4);
  float* ff = static_cast<float*>(f);
  int32_t* fi = static_cast<int32_t*>(f);
  int32_t* st2 = reinterpret_cast<int32_t*>((uintptr_t(1) << 20) + 2);
  const int E = VASE_ERR_INVALID_ARG;
  EXPECT(vase_score(nullptr, f, f, 0, 4, 256, 32, 128, 2, 16, 7, ff, ff, f, 1 << 30, nullptr, nullptr), E);
  EXPECT(vase_score(f, f, f, 0, 4, 256, 32, 96, 2, 16, 7, ff, ff, f, 1 << 30, nullptr, nullptr), E);
  EXPECT(vase_score(f, f, f, 0, 4, 256, 32, 128, 2, 16, 7, ff, ff, f, 1 << 30, st2, nullptr), E);
  EXPECT(vase_score(f, f, f, 0, 1 << 21, 256, 32, 128, 2, 16, 7, ff, ff, f, 1 << 30, nullptr, nullptr), E);
  EXPECT(vase_score(f, f, f, 0, 4, 1 << 24, 1, 128, 2, 16, 7, ff, ff, f, 1 << 30, nullptr, nullptr), E);
  EXPECT(vase_score(f, f, f, 0, 4, 256, 32, 128, 1 << 16, 2, 7, ff, ff, f, 1 << 30, nullptr, nullptr), E);
  EXPECT(vase_score_ex(f, f, f, 0, 4, 256, 32, 128, 2, 16, 7, 9, 1, 0, 0, ff, ff, f, 1 << 30, nullptr,
                       nullptr), E);
  EXPECT(vase_score_ex(f, f, m, 0, 4, 256, 32, 128, 2, 16, 7, 0, 1, 0, 0, ff, ff, f, 1 << 30, nullptr,
                       nullptr), E);
  EXPECT(vase_score_lse(f, f, f, nullptr, 0, 4, 256, 32, 128, 2, 16, 7, 0, 1, 0, 0, ff, ff, f, 1 << 30,
                        nullptr, nullptr), E);
  EXPECT(vase_score_map(f, f, f, nullptr, nullptr, 0, 4, 256, 32, 128, 2, 16, 7, 0, 1, 0, 0, ff, ff,
                        nullptr, nullptr, f, 1 << 30, nullptr, nullptr), E);
  EXPECT(vase_score_map(f, f, f, nullptr, fi, 0, 4, VASE_MAX_K + 32, 32, 128, 2, 16, 7, 0, 1, 0, 0,
                        ff, ff, nullptr, nullptr, f, 1 << 30, nullptr, nullptr), E);
  EXPECT(vase_score(f, f, f, 0, 4, 256, 32, 128, 2, 16, 7, ff, ff, nullptr, 0, nullptr, nullptr),
         VASE_ERR_WORKSPACE * (vase_workspace_bytes(VASE_OP_SCORE, 0, 4, 256, 32, 128, 2, 16) > 0) +
             0);
  EXPECT(vase_select(ff, ff, 4, 0, 256, 32, 225, 1, 0, 0, fi, nullptr, nullptr, nullptr), E);
  EXPECT(vase_select(ff, ff, 4, 0, VASE_MAX_K + 64, 32, 16, 1, 0, 0, fi, nullptr, nullptr, nullptr), E);
  EXPECT(vase_select(ff, ff, 4, 0, 256, 32, 16, 1, 0, 2, fi, nullptr, nullptr, nullptr), E);
  EXPECT(vase_select(ff, ff, 4, 0, 256, 32, 16, 1, 0, 0, fi, nullptr, st2, nullptr), E);
  EXPECT(vase_compact(f, f, 3, 4, 2048, 128, 128, fi, f, 1 << 30, nullptr), VASE_ERR_DTYPE);
  EXPECT(vase_compact(f, f, 0, 1, 2048, 128, 128, fi, nullptr, 0, nullptr), VASE_ERR_WORKSPACE);
  EXPECT(vase_decode_attn(f, f, f, 0, 4, 256, 32, 128, 9, 100, f, f, 1 << 30, nullptr), E);
  EXPECT(vase_decode_attn(f, f, f, 0, 4, 256, 32, 128, 4, 289, f, f, 1 << 30, nullptr), E);
  EXPECT(vase_decode_attn_lse(f, f, f, 0, 4, 256, 32, 128, 4, 100, 101, f, ff, f, 1 << 30, nullptr), E);
  EXPECT(vase_decode_step(f, f, f, f, f, 0, 4, 256, 32, 128, 4, 33, 0, f, ff, f, f, 1 << 30, nullptr), E);
  EXPECT(vase_decode_step(f, f, f, f, f, 0, 4, 256, 32, 128, 4, 16, 32, f, ff, f, f, 1 << 30, nullptr), E);
  EXPECT(vase_decode_step_noalloc(f, f, f, f, f, 1, 32768, 8192, 128, 128, 8, 128, 5, f, ff, f, nullptr),
         VASE_ERR_WORKSPACE);
  EXPECT(vase_decode_step_noalloc(f, f, f, f, m, 0, 4, 256, 32, 128, 4, 16, 0, f, ff, f, nullptr), E);
  EXPECT(vase_compact_decode(f, f, 0, 4, 256, 32, 128, fi, f, 0, f, f, 1 << 30, nullptr), E);
  EXPECT(vase_compact_decode_ex(f, f, 0, 4, 256, 32, 128, fi, f, 4, f, 3, ff, f, 1 << 30, nullptr), E);
  EXPECT(vase_compact_decode_map(f, f, 0, 4, 256, 32, 128, fi, fi, f, 4, nullptr, 0, nullptr, nullptr,
                                 nullptr, nullptr), E);
  EXPECT(vase_compact_decode_map(f, f, 1, 4, 256, 32, 128, fi, fi, f, 4, f, 0, nullptr, nullptr, ff,
                                 nullptr), VASE_ERR_DTYPE);
  EXPECT(vase_order_scores(ff, nullptr, fi, 4, 256, 4, ff, nullptr, nullptr), E);
  EXPECT(vase_dkv_projection(4, 0, 96, 20, 1, 0, ff, nullptr), E);
  EXPECT(vase_dkv_projection(4, 0, 128, 33, 1, 0, ff, nullptr), E);
  EXPECT(vase_dkv_score(f, f, ff, 0, 4, 256, 32, 128, 20, ff, f, 17, ff, nullptr), E);
  EXPECT(vase_quantize(f, 0, 4, 256, 32, 128, 3, 32, 0, static_cast<uint8_t*>(f), ff, ff, ff, f, fi,
                       nullptr), E);
  EXPECT(vase_dequantize(static_cast<uint8_t*>(f), ff, f, fi, 0, 4, 256, 32, 128, 4, 48, 0, f, nullptr), E);
  // workspace sizes over the accepted range (size_t arithmetic, no overflow)
  size_t acc = 0;
  const int insts[] = {1, 7, 512, 2304, 32768, 1 << 20};
  const int Ks[] = {1, 33, 4096, 8192};
  for (int op = 0; op <= 5; ++op)
    for (int n : insts)
      for (int K : Ks)
        for (int dt = 0; dt < 2; ++dt)
          acc += vase_workspace_bytes(op, dt, n, K, 128, 128, 8, 256) % 1000003;
  std::printf("%s\n", vase_status_str(VASE_ERR_HIP));
  std::printf("ok %zu\n", acc % 7);
  return 0;
}
