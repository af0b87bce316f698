// abi.hip -- the extern "C" entry points of libvase: host-side validation, workspace
// sizing and dispatch to the kernels.  Every argument is checked before the first
// HIP call, so an invalid call returns an error without touching the device.
#include "vase_internal.hpp"
#include "vase.h"

static_assert(VASE_DECODE_SCRATCH_BYTES == vase::kDecodeScratchBytes,
              "the header's scratch bound is the library's");

namespace {

constexpr int kVersion = (2 << 16) | 0;

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }
bool aligned4(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 3u) == 0; }

bool valid_dtype(int dtype) { return dtype == VASE_BF16 || dtype == VASE_F32; }
bool valid_d(int d) { return d == 64 || d == 128; }

// instance counts beyond this would overflow the launch grids or 32-bit slot math
constexpr long long kMaxInst = 1LL << 20;

int check_cache_shape(int n_inst, int K, int B, int d) {
  if (n_inst < 1 || n_inst > kMaxInst || K < 1 || B < 1 || !valid_d(d)) return VASE_ERR_INVALID_ARG;
  if ((long long)K + B > (1LL << 24)) return VASE_ERR_INVALID_ARG;
  return VASE_OK;
}

int hip_status(hipError_t e) { return e == hipSuccess ? VASE_OK : VASE_ERR_HIP; }

// vase_compact_decode runs one fused kernel (no workspace) when each instance
// fits one workgroup, else compaction then decode, which share the workspace
bool compact_decode_fused(int dtype, int n_inst, int K, int B, int d) {
  return vase::compact_plan(dtype, n_inst, K, B, d).n_part == 1 && K <= vase::kCompactDecodeMaxK;
}

size_t compact_decode_bytes(int dtype, int n_inst, int K, int B, int d, int G) {
  if (compact_decode_fused(dtype, n_inst, K, B, d)) return 0;
  const size_t a = vase::compact_plan(dtype, n_inst, K, B, d).bytes;
  const size_t b = vase::decode_plan(dtype, n_inst, K, B, d, G, K, K).bytes;
  return a > b ? a : b;
}

size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

// score under an order map: the score's own workspace, then the unpooled
// per-slot scores and value scores that order_scores puts into temporal order
size_t score_map_phys_offset(int dtype, int n_inst, int K, int B, int d, int G, int w) {
  return align256(vase::score_plan(dtype, n_inst, K, B, d, G, w).bytes);
}
size_t score_map_bytes(int dtype, int n_inst, int K, int B, int d, int G, int w) {
  const vase::ScorePlan pl = vase::score_plan(dtype, n_inst, K, B, d, G, w);
  if (pl.pool_in_kernel) return pl.bytes;   // the kernel pools through the map itself
  return score_map_phys_offset(dtype, n_inst, K, B, d, G, w) +
         2 * align256((size_t)n_inst * K * sizeof(float));
}

}  // namespace

extern "C" {

int vase_version(void) { return kVersion; }

const char* vase_status_str(int status) {
  switch (status) {
    case VASE_OK: return "ok";
    case VASE_ERR_INVALID_ARG: return "invalid argument";
    case VASE_ERR_DTYPE: return "unsupported dtype";
    case VASE_ERR_WORKSPACE: return "workspace too small";
    case VASE_ERR_HIP: return "HIP launch error";
    case VASE_ERR_UNSUPPORTED: return "unsupported shape";
    default: return "unknown status";
  }
}

size_t vase_workspace_bytes(int op, int dtype, int n_inst, int K, int B, int d, int G, int w) {
  if (!valid_dtype(dtype) || check_cache_shape(n_inst, K, B, d) != VASE_OK) return 0;
  switch (op) {
    case VASE_OP_SCORE:
      if (G < 1 || w < 1) return 0;
      return vase::score_plan(dtype, n_inst, K, B, d, G, w).bytes;
    case VASE_OP_SELECT:
      return 0;
    case VASE_OP_COMPACT:
      return vase::compact_plan(dtype, n_inst, K, B, d).bytes;
    case VASE_OP_COMPACT_DECODE:
      if (G < 1) return 0;
      return compact_decode_bytes(dtype, n_inst, K, B, d, G);
    case VASE_OP_SCORE_MAP:
      if (G < 1 || w < 1) return 0;
      return score_map_bytes(dtype, n_inst, K, B, d, G, w);
    case VASE_OP_DECODE: {
      if (G < 1) return 0;
      // the decode plan depends on n_valid and n_persist; size for the largest
      return vase::decode_ws_bytes_max(dtype, n_inst, K, B, d, G);
    }
    default:
      return 0;
  }
}

namespace {

int score_common(const void* k_cache, const void* v_cache, const void* q_win, const float* lse_win,
                 const int32_t* ord, int dtype, int n_inst, int K, int B, int d, int G, int w,
                 int pool, int value_kind, uint64_t seed, uint32_t round, uint32_t inst_base,
                 float* attn_out, float* vrange_out, void* ws, size_t ws_bytes,
                 int32_t* dev_status, void* stream, const void* q_dec = nullptr,
                 float* dec_logits = nullptr) {
  if (!k_cache || !v_cache || !q_win || !attn_out) return VASE_ERR_INVALID_ARG;
  if (!aligned4(dev_status)) return VASE_ERR_INVALID_ARG;
  uint32_t* status = reinterpret_cast<uint32_t*>(dev_status);
  if (value_kind < VASE_VALUE_RANGE || value_kind > VASE_VALUE_SKIP) return VASE_ERR_INVALID_ARG;
  if (!vrange_out && value_kind != VASE_VALUE_SKIP) return VASE_ERR_INVALID_ARG;
  if (!valid_dtype(dtype)) return VASE_ERR_DTYPE;
  int st = check_cache_shape(n_inst, K, B, d);
  if (st != VASE_OK) return st;
  if (G < 1 || w < 1 || (long long)G * w > (1 << 16)) return VASE_ERR_INVALID_ARG;
  if (pool < 1 || pool % 2 == 0 || pool > 255) return VASE_ERR_INVALID_ARG;
  if (!aligned16(k_cache) || !aligned16(v_cache) || !aligned16(q_win) || !aligned16(attn_out) ||
      (vrange_out && !aligned16(vrange_out)) || (lse_win && !aligned16(lse_win)))
    return VASE_ERR_INVALID_ARG;
  if (ord && (K > VASE_MAX_K || !aligned16(ord))) return VASE_ERR_INVALID_ARG;
  if ((q_dec == nullptr) != (dec_logits == nullptr)) return VASE_ERR_INVALID_ARG;
  if (dec_logits) {
    // the logits come from the MFMA pass over all N slots
    if (lse_win || G > 16 || !aligned16(q_dec) || !aligned16(dec_logits)) return VASE_ERR_INVALID_ARG;
    if (dtype != VASE_BF16) return VASE_ERR_DTYPE;
  }
  vase::DecLogits dec;
  dec.q = q_dec;
  dec.G = G;
  dec.out = dec_logits;
  const vase::ScorePlan plan = vase::score_plan(dtype, n_inst, K, B, d, G, w);
  const size_t need = ord ? score_map_bytes(dtype, n_inst, K, B, d, G, w) : plan.bytes;
  if (need > 0 && (!ws || ws_bytes < need || !aligned16(ws))) return VASE_ERR_WORKSPACE;
  const long long blocks = (long long)n_inst * plan.n_slab * (plan.n_chunk1 > plan.n_chunk2 ? plan.n_chunk1 : plan.n_chunk2);
  if (blocks > 0x7fffffffLL) return VASE_ERR_UNSUPPORTED;
  hipStream_t s = static_cast<hipStream_t>(stream);
  // under an order map: unpooled scores per physical slot into the workspace,
  // then pooled in temporal order; the value scores of the rows are permuted
  // the same way (random ones are drawn per temporal rank directly)
  const bool rows_scored = value_kind <= VASE_VALUE_VAR;
  if (ord && plan.pool_in_kernel) {
    // one workgroup holds each instance: it pools through the map itself
    hipError_t e = vase::launch_score(k_cache, v_cache, q_win, dtype, n_inst, K, B, d, G, w, pool,
                                      value_kind, lse_win, attn_out, vrange_out, ws, plan, s, ord,
                                      dec, status);
    if (e == hipSuccess && value_kind == VASE_VALUE_RANDOM)
      e = vase::launch_value_random(n_inst, inst_base, K, seed, round, vrange_out, s);
    return hip_status(e);
  }
  float* attn_k = attn_out;
  float* vr_k = vrange_out;
  if (ord) {
    char* phys = static_cast<char*>(ws) + score_map_phys_offset(dtype, n_inst, K, B, d, G, w);
    attn_k = reinterpret_cast<float*>(phys);
    if (rows_scored) vr_k = reinterpret_cast<float*>(phys + align256((size_t)n_inst * K * sizeof(float)));
  }
  hipError_t e = vase::launch_score(k_cache, v_cache, q_win, dtype, n_inst, K, B, d, G, w,
                                    ord ? 1 : pool, value_kind, lse_win, attn_k, vr_k, ws, plan, s,
                                    nullptr, dec, status);
  if (e == hipSuccess && value_kind == VASE_VALUE_RANDOM)
    e = vase::launch_value_random(n_inst, inst_base, K, seed, round, vrange_out, s);
  if (e == hipSuccess && ord)
    e = vase::launch_order_scores(attn_k, rows_scored ? vr_k : nullptr, ord, n_inst, K, pool,
                                  attn_out, vrange_out, s);
  return hip_status(e);
}

}  // namespace

int vase_score_ex(const void* k_cache, const void* v_cache, const void* q_win, int dtype,
                  int n_inst, int K, int B, int d, int G, int w, int pool, int value_kind,
                  uint64_t seed, uint32_t round, uint32_t inst_base, float* attn_out,
                  float* vrange_out, void* ws, size_t ws_bytes, int32_t* dev_status,
                  void* stream) {
  return score_common(k_cache, v_cache, q_win, nullptr, nullptr, dtype, n_inst, K, B, d, G, w,
                      pool, value_kind, seed, round, inst_base, attn_out, vrange_out, ws, ws_bytes,
                      dev_status, stream);
}

int vase_score_lse(const void* k_cache, const void* v_cache, const void* q_win,
                   const float* lse_win, int dtype, int n_inst, int K, int B, int d, int G, int w,
                   int pool, int value_kind, uint64_t seed, uint32_t round, uint32_t inst_base,
                   float* attn_out, float* vrange_out, void* ws, size_t ws_bytes,
                   int32_t* dev_status, void* stream) {
  if (!lse_win) return VASE_ERR_INVALID_ARG;
  return score_common(k_cache, v_cache, q_win, lse_win, nullptr, dtype, n_inst, K, B, d, G, w,
                      pool, value_kind, seed, round, inst_base, attn_out, vrange_out, ws, ws_bytes,
                      dev_status, stream);
}

int vase_score_map(const void* k_cache, const void* v_cache, const void* q_win,
                   const float* lse_win, const int32_t* ord, int dtype, int n_inst, int K, int B,
                   int d, int G, int w, int pool, int value_kind, uint64_t seed, uint32_t round,
                   uint32_t inst_base, float* attn_out, float* vrange_out, const void* q_dec,
                   float* dec_logits_out, void* ws, size_t ws_bytes, int32_t* dev_status,
                   void* stream) {
  if (!ord) return VASE_ERR_INVALID_ARG;
  return score_common(k_cache, v_cache, q_win, lse_win, ord, dtype, n_inst, K, B, d, G, w, pool,
                      value_kind, seed, round, inst_base, attn_out, vrange_out, ws, ws_bytes,
                      dev_status, stream, q_dec, dec_logits_out);
}

int vase_order_scores(const float* attn_phys, const float* vrange_phys, const int32_t* ord,
                      int n_inst, int K, int pool, float* attn_out, float* vrange_out,
                      void* stream) {
  if (!attn_phys || !ord || !attn_out || (vrange_phys && !vrange_out)) return VASE_ERR_INVALID_ARG;
  if (n_inst < 1 || n_inst > kMaxInst || K < 1 || K > VASE_MAX_K) return VASE_ERR_INVALID_ARG;
  if (pool < 1 || pool % 2 == 0 || pool > 255) return VASE_ERR_INVALID_ARG;
  if (!aligned16(attn_phys) || !aligned16(ord) || !aligned16(attn_out) ||
      (vrange_phys && (!aligned16(vrange_phys) || !aligned16(vrange_out))))
    return VASE_ERR_INVALID_ARG;
  return hip_status(vase::launch_order_scores(attn_phys, vrange_phys, ord, n_inst, K, pool,
                                              attn_out, vrange_phys ? vrange_out : nullptr,
                                              static_cast<hipStream_t>(stream)));
}

int vase_score(const void* k_cache, const void* v_cache, const void* q_win, int dtype, int n_inst,
               int K, int B, int d, int G, int w, int pool, float* attn_out, float* vrange_out,
               void* ws, size_t ws_bytes, int32_t* dev_status, void* stream) {
  return vase_score_ex(k_cache, v_cache, q_win, dtype, n_inst, K, B, d, G, w, pool,
                       VASE_VALUE_RANGE, 0, 0, 0, attn_out, vrange_out, ws, ws_bytes, dev_status,
                       stream);
}

int vase_select(const float* attn, const float* vrange, int n_inst, uint32_t inst_base, int K,
                int B, int Nv, uint64_t seed, uint32_t round, uint32_t flags, int32_t* src_out,
                float* keys_out, int32_t* dev_status, void* stream) {
  if (!attn || !vrange || !src_out) return VASE_ERR_INVALID_ARG;
  if (!aligned4(dev_status)) return VASE_ERR_INVALID_ARG;
  if (n_inst < 1 || n_inst > kMaxInst || K < 1 || K > VASE_MAX_K || B < 1 || Nv < 0 ||
      (long long)Nv + B > K)
    return VASE_ERR_INVALID_ARG;
  if ((flags & ~VASE_DETERMINISTIC) != 0u) return VASE_ERR_INVALID_ARG;
  if (!aligned16(attn) || !aligned16(vrange) || !aligned16(src_out) ||
      (keys_out && !aligned16(keys_out)))
    return VASE_ERR_INVALID_ARG;
  return hip_status(vase::launch_select(attn, vrange, n_inst, inst_base, K, B, Nv, seed, round,
                                        flags, src_out, keys_out,
                                        static_cast<hipStream_t>(stream),
                                        reinterpret_cast<uint32_t*>(dev_status)));
}

int vase_compact(void* k_cache, void* v_cache, int dtype, int n_inst, int K, int B, int d,
                 const int32_t* src, void* ws, size_t ws_bytes, void* stream) {
  if (!k_cache || !v_cache || !src) return VASE_ERR_INVALID_ARG;
  if (!valid_dtype(dtype)) return VASE_ERR_DTYPE;
  int st = check_cache_shape(n_inst, K, B, d);
  if (st != VASE_OK) return st;
  if (!aligned16(k_cache) || !aligned16(v_cache) || !aligned16(src)) return VASE_ERR_INVALID_ARG;
  const vase::CompactPlan plan = vase::compact_plan(dtype, n_inst, K, B, d);
  if (plan.bytes > 0 && (!ws || ws_bytes < plan.bytes || !aligned16(ws))) return VASE_ERR_WORKSPACE;
  return hip_status(vase::launch_compact(k_cache, v_cache, dtype, n_inst, K, B, d, src, ws, plan,
                                         static_cast<hipStream_t>(stream)));
}

namespace {

int decode_common(const void* k_cache, const void* v_cache, const void* q, int dtype, int n_inst,
                  int K, int B, int d, int G, int n_valid, int n_persist, void* out, float* lse,
                  int lse_ld, void* ws, size_t ws_bytes, hipStream_t s) {
  const vase::DecodePlan plan = vase::decode_plan(dtype, n_inst, K, B, d, G, n_valid, n_persist);
  if (plan.bytes > 0 && (!ws || ws_bytes < plan.bytes || !aligned16(ws))) return VASE_ERR_WORKSPACE;
  return hip_status(vase::launch_decode(k_cache, v_cache, q, dtype, n_inst, K, B, d, G, n_valid,
                                        n_persist, out, lse, lse_ld, ws, plan, s));
}

}  // namespace

int vase_decode_attn_lse(const void* k_cache, const void* v_cache, const void* q, int dtype,
                         int n_inst, int K, int B, int d, int G, int n_valid, int n_persist,
                         void* out, float* lse_out, void* ws, size_t ws_bytes, void* stream) {
  if (!k_cache || !v_cache || !q || !out) return VASE_ERR_INVALID_ARG;
  if (!valid_dtype(dtype)) return VASE_ERR_DTYPE;
  int st = check_cache_shape(n_inst, K, B, d);
  if (st != VASE_OK) return st;
  if (G < 1 || G > 8 || n_valid < 1 || n_valid > K + B) return VASE_ERR_INVALID_ARG;
  if (n_persist < 1 || n_persist > n_valid) return VASE_ERR_INVALID_ARG;
  if (!aligned16(k_cache) || !aligned16(v_cache) || !aligned16(q) || !aligned16(out))
    return VASE_ERR_INVALID_ARG;
  if (lse_out && !aligned16(lse_out)) return VASE_ERR_INVALID_ARG;
  return decode_common(k_cache, v_cache, q, dtype, n_inst, K, B, d, G, n_valid, n_persist, out,
                       lse_out, 1, ws, ws_bytes, static_cast<hipStream_t>(stream));
}

int vase_decode_attn(const void* k_cache, const void* v_cache, const void* q, int dtype, int n_inst,
                     int K, int B, int d, int G, int n_valid, void* out, void* ws, size_t ws_bytes,
                     void* stream) {
  return vase_decode_attn_lse(k_cache, v_cache, q, dtype, n_inst, K, B, d, G, n_valid, n_valid,
                              out, nullptr, ws, ws_bytes, stream);
}

int vase_decode_step(void* k_cache, void* v_cache, const void* k_new, const void* v_new,
                     const void* q, int dtype, int n_inst, int K, int B, int d, int G, int w,
                     int pos, void* q_win, float* lse_win, void* out, void* ws, size_t ws_bytes,
                     void* stream) {
  if (!k_cache || !v_cache || !k_new || !v_new || !q || !q_win || !lse_win || !out)
    return VASE_ERR_INVALID_ARG;
  if (!valid_dtype(dtype)) return VASE_ERR_DTYPE;
  int st = check_cache_shape(n_inst, K, B, d);
  if (st != VASE_OK) return st;
  if (G < 1 || G > 8 || w < 1 || w > B || pos < 0 || pos >= B) return VASE_ERR_INVALID_ARG;
  if (!aligned16(k_cache) || !aligned16(v_cache) || !aligned16(k_new) || !aligned16(v_new) ||
      !aligned16(q) || !aligned16(q_win) || !aligned16(lse_win) || !aligned16(out))
    return VASE_ERR_INVALID_ARG;
  const vase::DecodePlan plan = vase::decode_plan(dtype, n_inst, K, B, d, G, K + pos + 1, K);
  if (plan.bytes > 0 && (!ws || ws_bytes < plan.bytes || !aligned16(ws))) return VASE_ERR_WORKSPACE;
  hipStream_t s = static_cast<hipStream_t>(stream);
  const hipError_t e = vase::launch_decode_append(k_cache, v_cache, k_new, v_new, q, q_win, dtype,
                                                  n_inst, K, B, d, G, w, pos, s);
  if (e != hipSuccess) return VASE_ERR_HIP;
  return decode_common(k_cache, v_cache, q, dtype, n_inst, K, B, d, G, K + pos + 1, K, out,
                       lse_win + pos % w, w, ws, ws_bytes, s);
}

int vase_decode_step_noalloc(void* k_cache, void* v_cache, const void* k_new, const void* v_new,
                             const void* q, int dtype, int n_inst, int K, int B, int d, int G,
                             int w, int pos, void* q_win, float* lse_win, void* out,
                             void* stream) {
  if (!k_cache || !v_cache || !k_new || !v_new || !q || !q_win || !lse_win || !out)
    return VASE_ERR_INVALID_ARG;
  if (!valid_dtype(dtype)) return VASE_ERR_DTYPE;
  int st = check_cache_shape(n_inst, K, B, d);
  if (st != VASE_OK) return st;
  if (G < 1 || G > 8 || w < 1 || w > B || pos < 0 || pos >= B) return VASE_ERR_INVALID_ARG;
  if (!aligned16(k_cache) || !aligned16(v_cache) || !aligned16(k_new) || !aligned16(v_new) ||
      !aligned16(q) || !aligned16(q_win) || !aligned16(lse_win) || !aligned16(out))
    return VASE_ERR_INVALID_ARG;
  const vase::DecodePlan plan = vase::decode_plan(dtype, n_inst, K, B, d, G, K + pos + 1, K);
  if (plan.bytes > VASE_DECODE_SCRATCH_BYTES) return VASE_ERR_WORKSPACE;
  void* ws = nullptr;
  if (plan.bytes > 0 && vase::decode_scratch(&ws) != hipSuccess) return VASE_ERR_HIP;
  hipStream_t s = static_cast<hipStream_t>(stream);
  const hipError_t e = vase::launch_decode_append(k_cache, v_cache, k_new, v_new, q, q_win, dtype,
                                                  n_inst, K, B, d, G, w, pos, s);
  if (e != hipSuccess) return VASE_ERR_HIP;
  return decode_common(k_cache, v_cache, q, dtype, n_inst, K, B, d, G, K + pos + 1, K, out,
                       lse_win + pos % w, w, ws, plan.bytes, s);
}

int vase_compact_decode_ex(void* k_cache, void* v_cache, int dtype, int n_inst, int K, int B,
                           int d, const int32_t* src, const void* q, int G, void* out,
                           int value_kind, float* vrange_out, void* ws, size_t ws_bytes,
                           void* stream) {
  if (!k_cache || !v_cache || !src || !q || !out) return VASE_ERR_INVALID_ARG;
  if (vrange_out && (value_kind < VASE_VALUE_RANGE || value_kind > VASE_VALUE_VAR))
    return VASE_ERR_INVALID_ARG;
  if (!valid_dtype(dtype)) return VASE_ERR_DTYPE;
  int st = check_cache_shape(n_inst, K, B, d);
  if (st != VASE_OK) return st;
  if (G < 1 || G > 8) return VASE_ERR_INVALID_ARG;
  if (!aligned16(k_cache) || !aligned16(v_cache) || !aligned16(src) || !aligned16(q) ||
      !aligned16(out) || (vrange_out && !aligned16(vrange_out)))
    return VASE_ERR_INVALID_ARG;
  const vase::CompactPlan cp = vase::compact_plan(dtype, n_inst, K, B, d);
  const vase::DecodePlan dp = vase::decode_plan(dtype, n_inst, K, B, d, G, K, K);
  const size_t need = compact_decode_bytes(dtype, n_inst, K, B, d, G);
  if (need > 0 && (!ws || ws_bytes < need || !aligned16(ws))) return VASE_ERR_WORKSPACE;
  hipStream_t s = static_cast<hipStream_t>(stream);
  if (compact_decode_fused(dtype, n_inst, K, B, d)) {
    return hip_status(vase::launch_compact_decode(k_cache, v_cache, dtype, n_inst, K, B, d, src, q,
                                                  G, out, value_kind, vrange_out, s));
  }
  // instances split over several workgroups (or very long): compaction, the
  // compacted rows' value scores, then decode
  hipError_t e = vase::launch_compact(k_cache, v_cache, dtype, n_inst, K, B, d, src, ws, cp, s);
  if (e == hipSuccess && vrange_out)
    e = vase::launch_value_rows(v_cache, dtype, n_inst, K + B, K, d, value_kind, vrange_out, s);
  if (e != hipSuccess) return VASE_ERR_HIP;
  return hip_status(vase::launch_decode(k_cache, v_cache, q, dtype, n_inst, K, B, d, G, K, K, out,
                                        nullptr, 1, ws, dp, s));
}

int vase_compact_decode(void* k_cache, void* v_cache, int dtype, int n_inst, int K, int B, int d,
                        const int32_t* src, const void* q, int G, void* out, void* ws,
                        size_t ws_bytes, void* stream) {
  return vase_compact_decode_ex(k_cache, v_cache, dtype, n_inst, K, B, d, src, q, G, out,
                                VASE_VALUE_RANGE, nullptr, ws, ws_bytes, stream);
}

int vase_compact_decode_map(void* k_cache, void* v_cache, int dtype, int n_inst, int K, int B,
                            int d, const int32_t* src, int32_t* ord, const void* q, int G,
                            void* out, int value_kind, const float* vrange_in, float* vrange_out,
                            const float* dec_logits, void* stream) {
  if (!k_cache || !v_cache || !src || !ord) return VASE_ERR_INVALID_ARG;
  if (dec_logits) {
    // read by the MFMA decode (bf16)
    if (!q || !aligned16(dec_logits)) return VASE_ERR_INVALID_ARG;
    if (dtype != VASE_BF16) return VASE_ERR_DTYPE;
  }
  if ((q == nullptr) != (out == nullptr)) return VASE_ERR_INVALID_ARG;
  if (vrange_in && (!vrange_out || !aligned16(vrange_in))) return VASE_ERR_INVALID_ARG;
  if (vrange_out && (value_kind < VASE_VALUE_RANGE || value_kind > VASE_VALUE_VAR))
    return VASE_ERR_INVALID_ARG;
  if (!valid_dtype(dtype)) return VASE_ERR_DTYPE;
  int st = check_cache_shape(n_inst, K, B, d);
  if (st != VASE_OK) return st;
  if (K > VASE_MAX_K || B > K) return VASE_ERR_INVALID_ARG;
  if (q && (G < 1 || G > 8)) return VASE_ERR_INVALID_ARG;
  if (!aligned16(k_cache) || !aligned16(v_cache) || !aligned16(src) || !aligned16(ord) ||
      (q && (!aligned16(q) || !aligned16(out))) || (vrange_out && !aligned16(vrange_out)))
    return VASE_ERR_INVALID_ARG;
  return hip_status(vase::launch_compact_map(k_cache, v_cache, dtype, n_inst, K, B, d, src, ord, q,
                                             G, out, value_kind, vrange_in, vrange_out,
                                             dec_logits, static_cast<hipStream_t>(stream)));
}

int vase_dkv_projection(int n_inst, uint32_t inst_base, int d, int r, uint64_t seed,
                        uint32_t round, float* g_out, void* stream) {
  if (!g_out) return VASE_ERR_INVALID_ARG;
  if (n_inst < 1 || n_inst > kMaxInst || !valid_d(d) || r < 1 || r > vase::kDkvMaxRank)
    return VASE_ERR_INVALID_ARG;
  if (!aligned16(g_out)) return VASE_ERR_INVALID_ARG;
  return hip_status(vase::launch_dkv_projection(n_inst, inst_base, d, r, seed, round, g_out,
                                                static_cast<hipStream_t>(stream)));
}

int vase_dkv_score(const void* k_cache, const void* v_cache, const float* g, int dtype, int n_inst,
                   int K, int B, int d, int r, float* score_out, const void* q_dec, int G,
                   float* dec_logits_out, void* stream) {
  if (!k_cache || !v_cache || !g || !score_out) return VASE_ERR_INVALID_ARG;
  if ((q_dec == nullptr) != (dec_logits_out == nullptr)) return VASE_ERR_INVALID_ARG;
  if (!valid_dtype(dtype)) return VASE_ERR_DTYPE;
  int st = check_cache_shape(n_inst, K, B, d);
  if (st != VASE_OK) return st;
  if (r < 1 || r > vase::kDkvMaxRank) return VASE_ERR_INVALID_ARG;
  if (!aligned16(k_cache) || !aligned16(v_cache) || !aligned16(g) || !aligned16(score_out))
    return VASE_ERR_INVALID_ARG;
  if (dec_logits_out) {
    if (G < 1 || G > 16 || !aligned16(q_dec) || !aligned16(dec_logits_out))
      return VASE_ERR_INVALID_ARG;
    if (dtype != VASE_BF16) return VASE_ERR_DTYPE;
  }
  return hip_status(vase::launch_dkv_score(k_cache, v_cache, g, dtype, n_inst, K, B, d, r,
                                           score_out, q_dec, G, dec_logits_out,
                                           static_cast<hipStream_t>(stream)));
}

namespace {
bool valid_quant(int bits, int group, int d) {
  return (bits == 2 || bits == 4 || bits == 8) && (group == 32 || group == 64 || group == 128) &&
         group <= d;
}
}  // namespace

int vase_quantize(const void* x_cache, int dtype, int n_inst, int K, int B, int d, int bits,
                  int group, int Nv, uint8_t* codes_out, float* params_out, float* range_out,
                  float* mse_out, void* hp_rows_out, int32_t* hp_idx_out, void* stream) {
  if (!x_cache || !codes_out || !params_out) return VASE_ERR_INVALID_ARG;
  if (!valid_dtype(dtype)) return VASE_ERR_DTYPE;
  int st = check_cache_shape(n_inst, K, B, d);
  if (st != VASE_OK) return st;
  if (!valid_quant(bits, group, d) || Nv < 0 || Nv > K) return VASE_ERR_INVALID_ARG;
  if (Nv > 0 && (K > VASE_MAX_K || !range_out || !hp_rows_out || !hp_idx_out))
    return VASE_ERR_INVALID_ARG;
  if (!aligned16(x_cache) || !aligned16(codes_out) || !aligned16(params_out) ||
      (range_out && !aligned16(range_out)) || (mse_out && !aligned16(mse_out)) ||
      (hp_rows_out && !aligned16(hp_rows_out)) || (hp_idx_out && !aligned16(hp_idx_out)))
    return VASE_ERR_INVALID_ARG;
  return hip_status(vase::launch_quantize(x_cache, dtype, n_inst, K, B, d, bits, group, Nv,
                                          codes_out, params_out, range_out, mse_out, hp_rows_out,
                                          hp_idx_out, static_cast<hipStream_t>(stream)));
}

int vase_dequantize(const uint8_t* codes, const float* params, const void* hp_rows,
                    const int32_t* hp_idx, int dtype, int n_inst, int K, int B, int d, int bits,
                    int group, int Nv, void* out_cache, void* stream) {
  if (!codes || !params || !out_cache) return VASE_ERR_INVALID_ARG;
  if (!valid_dtype(dtype)) return VASE_ERR_DTYPE;
  int st = check_cache_shape(n_inst, K, B, d);
  if (st != VASE_OK) return st;
  if (!valid_quant(bits, group, d) || Nv < 0 || Nv > K) return VASE_ERR_INVALID_ARG;
  if (Nv > 0 && (!hp_rows || !hp_idx)) return VASE_ERR_INVALID_ARG;
  if (!aligned16(codes) || !aligned16(params) || !aligned16(out_cache) ||
      (hp_rows && !aligned16(hp_rows)) || (hp_idx && !aligned16(hp_idx)))
    return VASE_ERR_INVALID_ARG;
  return hip_status(vase::launch_dequantize(codes, params, hp_rows, hp_idx, dtype, n_inst, K, B,
                                            d, bits, group, Nv, out_cache,
                                            static_cast<hipStream_t>(stream)));
}

}  // extern "C"
