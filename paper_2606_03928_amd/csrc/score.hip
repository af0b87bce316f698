// score.hip -- pooled window-mean attention score and Range(v) on gfx950.
//
// abar_i = (1/R) sum_r exp(s_ri - lse_r),  s_ri = q_r . k_i / sqrt(d),  R = G*w rows,
// lse_r = log sum_{t<N} exp(s_rt) over all N slots (Eq. 1 rows inside Eq. 2),
// attn_i = (1/P) sum_{|j-i|<=P/2, 0<=j<K} abar_j,   vrange_i = max(v_i) - min(v_i) (Eq. 5).
//
// The row normaliser depends on every slot, so the scores are computed twice:
//   pass 1 (rows):  per key chunk, per row: max and sum of exp2 -> (m, l) partials
//   merge:          per row, fixed-order merge of the chunk partials -> lse2_r
//   pass 2 (cols):  per key chunk: p = exp2(s*c - lse2_r), column sums over rows
//   pool:           per slot: mean over slabs, /R, then the P-wide box filter
// All exponentials are base 2 with c = log2(e)/sqrt(d) folded in.  No floating
// point atomics are used; every reduction has a fixed order.
//
// bf16 caches use MFMA (v_mfma_f32_32x32x16_bf16): each wave of a 4-wave block
// keeps 64 keys of its instance resident in VGPRs as A operands (rows = keys)
// and the query window streams through LDS in 32-row blocks as B operands
// (columns = queries).  In the accumulator a lane holds 16 keys x 1 query per
// key block, so pass 1 reduces over keys inside the lane and pass 2 reduces
// over queries with a 5-step transpose-reduce across the 32 lanes of a half
// wave.  The contraction index d is permuted identically in both operands so
// that each lane loads a contiguous half row: lane half h, step ks holds
// elements [h*D/2 + 8*ks, +8).
// fp32 caches use a plain VALU path (one thread per row / per key).
#include "vase_internal.hpp"
#include "vase.h"

namespace vase {
namespace {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));

constexpr int kSBlock = 256;
constexpr int kKeysPerWave = 64;
constexpr int kKeysPerBlock = 256;  // 4 waves x 64 keys
constexpr int kMaxSlab = 512;       // query rows per workgroup in the MFMA passes
constexpr float kFloor = -3.0e38f;  // finite stand-in for an empty maximum
constexpr int kGenKeys = 32;        // VALU path: keys per chunk
constexpr int kGenRows = 32;        // VALU path: rows per staging step
constexpr int kGenBlock = 64;

__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }
__device__ __forceinline__ float fast_log2(float x) { return __builtin_amdgcn_logf(x); }

// ---------------------------------------------------------------------------
// MFMA building blocks
// ---------------------------------------------------------------------------
template <int D>
struct MfmaKeys {
  static constexpr int KS = D / 16;   // k-steps of 16
  bf16x8_t a[2][KS];                  // 2 key blocks of 32
};

// Load this wave's 64 keys (rows kbase .. kbase+63, clamped to nk-1) as A operands.
template <int D>
__device__ __forceinline__ void load_keys(MfmaKeys<D>& mk, const uint16_t* kinst, int kbase,
                                          int nk, int lane) {
  const int half = lane / 32;
#pragma unroll
  for (int kb = 0; kb < 2; ++kb) {
    int key = kbase + kb * 32 + (lane % 32);
    key = key < nk ? key : nk - 1;
    const bf16x8_t* row = reinterpret_cast<const bf16x8_t*>(kinst + (size_t)key * D + half * (D / 2));
#pragma unroll
    for (int ks = 0; ks < MfmaKeys<D>::KS; ++ks) mk.a[kb][ks] = row[ks];
  }
}

template <int D>
__device__ __forceinline__ void zero_keys(MfmaKeys<D>& mk) {
#pragma unroll
  for (int kb = 0; kb < 2; ++kb)
#pragma unroll
    for (int ks = 0; ks < MfmaKeys<D>::KS; ++ks) mk.a[kb][ks] = bf16x8_t{};
}

// LDS ring of 32-query-row tiles, row stride D + 8 elements (16-byte pad).
constexpr int kQRing = 4;
template <int D>
struct QTile {
  static constexpr int kStride = D + 8;
  static constexpr int kTile = 32 * kStride;
  uint16_t x[kQRing * kTile];
  __device__ __forceinline__ uint16_t* buf(int t) { return x + (t & (kQRing - 1)) * kTile; }
};

// Global -> registers for one 32-row query block (rows >= row_hi read as zero).
template <int D>
struct QStage {
  static constexpr int kPerRow = D / 8;                 // 16-byte pieces per row
  static constexpr int kRowsPerPass = kSBlock / kPerRow;
  static constexpr int kPasses = 32 / kRowsPerPass;
  uint4 r[kPasses];
  __device__ __forceinline__ void load(const uint16_t* qinst, int row0, int row_hi) {
    const int t = threadIdx.x;
#pragma unroll
    for (int p = 0; p < kPasses; ++p) {
      const int row = row0 + p * kRowsPerPass + t / kPerRow;
      r[p] = row < row_hi ? reinterpret_cast<const uint4*>(qinst + (size_t)row * D)[t % kPerRow]
                          : make_uint4(0u, 0u, 0u, 0u);
    }
  }
  __device__ __forceinline__ void store(uint16_t* tile) const {
    const int t = threadIdx.x;
#pragma unroll
    for (int p = 0; p < kPasses; ++p) {
      const int row = p * kRowsPerPass + t / kPerRow;
      *reinterpret_cast<uint4*>(tile + row * QTile<D>::kStride + (t % kPerRow) * 8) = r[p];
    }
  }
};

// acc[kb] = K_block(kb) x Q_tile^T for this wave's 64 keys and the tile's 32 queries.
template <int D>
__device__ __forceinline__ void mfma_tile(const MfmaKeys<D>& mk, const uint16_t* tile, int lane,
                                          f32x16_t acc[2]) {
  const int half = lane / 32;
  const uint16_t* brow = tile + (lane % 32) * QTile<D>::kStride + half * (D / 2);
  acc[0] = f32x16_t{};
  acc[1] = f32x16_t{};
#pragma unroll
  for (int ks = 0; ks < MfmaKeys<D>::KS; ++ks) {
    const bf16x8_t b = *reinterpret_cast<const bf16x8_t*>(brow + ks * 8);
    acc[0] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(mk.a[0][ks], b, acc[0], 0, 0, 0);
    acc[1] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(mk.a[1][ks], b, acc[1], 0, 0, 0);
  }
}

// key (relative to the wave's base) held by accumulator element (kb, r) of a lane
__device__ __forceinline__ int acc_key(int kb, int r, int half) {
  return kb * 32 + 8 * (r / 4) + 4 * half + (r % 4);
}

struct BlockMap {
  int inst, slab, chunk;
};
__device__ __forceinline__ BlockMap map_block(int n_slab, int n_chunk) {
  const uint32_t lb = xcd_logical_block(blockIdx.x, gridDim.x);
  BlockMap m;
  m.chunk = (int)(lb % (uint32_t)n_chunk);
  const uint32_t t = lb / (uint32_t)n_chunk;
  m.slab = (int)(t % (uint32_t)n_slab);
  m.inst = (int)(t / (uint32_t)n_slab);
  return m;
}

// ---------------------------------------------------------------------------
// Tile pipeline shared by both MFMA passes.  Query tiles of 32 rows cycle
// through a 4-deep LDS ring.  At step t a wave
//   * issues the global loads of tile t+3 into a register stage,
//   * issues the MFMAs of tile t+1 (ring slot t+1),
//   * runs the VALU epilogue of tile t (its accumulators were filled at step t-1),
//   * writes tile t+2 (loaded at step t-1) into ring slot t+2, then a barrier.
// So the matrix core and the vector ALU work on independent registers in the
// same basic block, and each global load has more than a full step to land.
// Slot t+2 last held tile t-2, whose MFMAs were issued at step t-3, before
// three barriers.  Past the last tile the MFMAs read a stale slot and the
// loads stage zero rows; those results are dropped.
// ---------------------------------------------------------------------------
template <int D, typename Pre, typename Epi>
__device__ __forceinline__ void run_tiles(const MfmaKeys<D>& mk, QTile<D>& qt,
                                          const uint16_t* qinst, int row_lo, int row_hi, int lane,
                                          Pre&& pre, Epi&& epi) {
  const int nrows = row_hi - row_lo;
  const int nqb = (nrows + 31) / 32;
  QStage<D> s0, s1;
  s0.load(qinst, row_lo, row_hi);
  s1.load(qinst, row_lo + 32, row_hi);
  s0.store(qt.buf(0));
  s1.store(qt.buf(1));
  s0.load(qinst, row_lo + 64, row_hi);          // tile 2, written at the end of step 0
  __syncthreads();
  f32x16_t a0[2], a1[2];
  mfma_tile<D>(mk, qt.buf(0), lane, a0);
  for (int t = 0; t < nqb; t += 2) {
    // ---- step t: load tile t+3 -> s1, MFMA tile t+1 -> a1, epilogue tile t, store tile t+2
    pre(t);
    s1.load(qinst, row_lo + (t + 3) * 32, row_hi);
    mfma_tile<D>(mk, qt.buf(t + 1), lane, a1);
    epi(t, a0);
    __builtin_amdgcn_sched_barrier(0);
    s0.store(qt.buf(t + 2));
    __syncthreads();
    if (t + 1 >= nqb) break;
    // ---- step t+1: load tile t+4 -> s0, MFMA tile t+2 -> a0, epilogue tile t+1, store t+3
    pre(t + 1);
    s0.load(qinst, row_lo + (t + 4) * 32, row_hi);
    mfma_tile<D>(mk, qt.buf(t + 2), lane, a0);
    epi(t + 1, a1);
    __builtin_amdgcn_sched_barrier(0);
    s1.store(qt.buf(t + 3));
    __syncthreads();
  }
}

// Range of the value rows [kbase, kbase+64) of one wave.  A row is D/8 lanes x
// 16 bytes, so one load covers 64/(D/8) rows; all loads are issued before the
// first reduction so their latencies overlap.
template <int D>
__device__ __forceinline__ void wave_range(const uint16_t* vinst, int kbase, int K, int lane,
                                           float* __restrict__ out) {
  constexpr int kLpr = D / 8;
  constexpr int kRpl = kWave / kLpr;
  constexpr int kGroups = kKeysPerWave / kRpl;
  const int seg = lane % kLpr;
  uint4 w[kGroups];
#pragma unroll
  for (int g = 0; g < kGroups; ++g) {
    const int row = kbase + g * kRpl + lane / kLpr;
    const int rr = row < K ? row : K - 1;
    w[g] = reinterpret_cast<const uint4*>(vinst + (size_t)rr * D)[seg];
  }
#pragma unroll
  for (int g = 0; g < kGroups; ++g) {
    float f[8];
    Vec16<bf16_t>::unpack(w[g], f);
    float mx = f[0], mn = f[0];
#pragma unroll
    for (int e = 1; e < 8; ++e) {
      mx = fmaxf(mx, f[e]);
      mn = fminf(mn, f[e]);
    }
#pragma unroll
    for (int off = 1; off < kLpr; off <<= 1) {
      mx = fmaxf(mx, __shfl_xor(mx, off, kWave));
      mn = fminf(mn, __shfl_xor(mn, off, kWave));
    }
    const int row = kbase + g * kRpl + lane / kLpr;
    if (row < K && seg == 0) out[row] = mx - mn;
  }
}

// ---------------------------------------------------------------------------
// pass 1 (MFMA): per-row (max, sum exp2) over one chunk of 256 slots, plus the
// Range of the chunk's candidate value rows (slab 0 only).
// part layout: [inst][chunk][R] float2 (m in log2 units, l)
// ---------------------------------------------------------------------------
template <int D, bool RAGGED>
__device__ __forceinline__ void score_rows_body(
    const uint16_t* __restrict__ k, const uint16_t* __restrict__ v, const uint16_t* __restrict__ q,
    int N, int K, int R, int n_chunk, int n_slab, int rows_per_slab, float c,
    float2* __restrict__ part, float* __restrict__ vrange, const BlockMap bm, QTile<D>& qt,
    float2* sstat) {
  const int lane = threadIdx.x % kWave, wave = threadIdx.x / kWave, half = lane / 32;
  const int row_lo = bm.slab * rows_per_slab;
  const int row_hi = min(R, row_lo + rows_per_slab);
  const int nrows = row_hi - row_lo;
  const int nqb = (nrows + 31) / 32;
  const int kbase = bm.chunk * kKeysPerBlock + wave * kKeysPerWave;
  const bool active = kbase < N;
  const uint16_t* kinst = k + (size_t)bm.inst * N * D;
  const uint16_t* vinst = v + (size_t)bm.inst * N * D;
  const uint16_t* qinst = q + (size_t)bm.inst * R * D;
  float* vr_inst = vrange + (size_t)bm.inst * K;
  const bool do_range = bm.slab == 0 && kbase < K;
  MfmaKeys<D> mk;
  if (active) load_keys<D>(mk, kinst, kbase, N, lane);
  else zero_keys<D>(mk);
  if (do_range) wave_range<D>(vinst, kbase, K, lane, vr_inst);

  auto pre = [](int) {};
  auto epi = [&](int t, f32x16_t (&acc)[2]) {
    if (RAGGED) {
#pragma unroll
      for (int kb = 0; kb < 2; ++kb)
#pragma unroll
        for (int r = 0; r < 16; ++r)
          acc[kb][r] = kbase + acc_key(kb, r, half) < N ? acc[kb][r] : -INFINITY;
    }
    float mx = kFloor;
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int r = 0; r < 16; ++r) mx = fmaxf(mx, acc[kb][r]);
    float mc = mx * c, lsum = 0.f;
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int r = 0; r < 16; ++r) lsum += fast_exp2(__builtin_fmaf(acc[kb][r], c, -mc));
    mc = active ? mc : kFloor * c;
    lsum = active ? lsum : 0.f;
    // merge with the other half wave (same query, the other 16 keys per block)
    const float m2 = __shfl_xor(mc, 32, kWave);
    const float l2 = __shfl_xor(lsum, 32, kWave);
    const float mm = fmaxf(mc, m2);
    const float ll = lsum * fast_exp2(mc - mm) + l2 * fast_exp2(m2 - mm);
    const int row = t * 32 + (lane % 32);
    if (half == 0 && row < nrows) sstat[wave * rows_per_slab + row] = make_float2(mm, ll);
  };
  run_tiles<D>(mk, qt, qinst, row_lo, row_hi, lane, pre, epi);

  // merge the four waves (fixed order) and write the chunk's partials
  for (int r = threadIdx.x; r < nrows; r += kSBlock) {
    const float2 s0 = sstat[r], s1 = sstat[rows_per_slab + r];
    const float2 s2 = sstat[2 * rows_per_slab + r], s3 = sstat[3 * rows_per_slab + r];
    const float mm = fmaxf(fmaxf(s0.x, s1.x), fmaxf(s2.x, s3.x));
    float ll = s0.y * fast_exp2(s0.x - mm);
    ll += s1.y * fast_exp2(s1.x - mm);
    ll += s2.y * fast_exp2(s2.x - mm);
    ll += s3.y * fast_exp2(s3.x - mm);
    part[((size_t)bm.inst * n_chunk + bm.chunk) * R + row_lo + r] = make_float2(mm, ll);
  }
}

template <int D>
__global__ __launch_bounds__(kSBlock, 2) void score_rows_mfma(
    const uint16_t* __restrict__ k, const uint16_t* __restrict__ v, const uint16_t* __restrict__ q,
    int N, int K, int R, int n_chunk, int n_slab, int rows_per_slab, float c,
    float2* __restrict__ part, float* __restrict__ vrange) {
  __shared__ QTile<D> qt;
  extern __shared__ float2 sstat[];   // [4][rows_per_slab]
  const BlockMap bm = map_block(n_slab, n_chunk);
  // only the last chunk of an instance holds slots past N; it masks them
  if ((bm.chunk + 1) * kKeysPerBlock > N)
    score_rows_body<D, true>(k, v, q, N, K, R, n_chunk, n_slab, rows_per_slab, c, part, vrange,
                             bm, qt, sstat);
  else
    score_rows_body<D, false>(k, v, q, N, K, R, n_chunk, n_slab, rows_per_slab, c, part, vrange,
                              bm, qt, sstat);
}

// ---------------------------------------------------------------------------
// pass 2 (MFMA): column sums of p = exp2(s*c - lse2_r) for one chunk of slots < K
// col layout: [inst][slab][K] float
// ---------------------------------------------------------------------------
template <int D>
__global__ __launch_bounds__(kSBlock, 2) void score_cols_mfma(
    const uint16_t* __restrict__ k, const uint16_t* __restrict__ q, int N, int K, int R,
    int n_chunk, int n_slab, int rows_per_slab, float c, const float* __restrict__ lse2,
    float* __restrict__ col) {
  __shared__ QTile<D> qt;
  extern __shared__ float s_lse[];     // [rows_per_slab rounded up to 32]
  const BlockMap bm = map_block(n_slab, n_chunk);
  const int lane = threadIdx.x % kWave, wave = threadIdx.x / kWave, half = lane / 32;
  const int row_lo = bm.slab * rows_per_slab;
  const int row_hi = min(R, row_lo + rows_per_slab);
  const int nrows = row_hi - row_lo;
  const int kbase = bm.chunk * kKeysPerBlock + wave * kKeysPerWave;
  const bool active = kbase < K;
  const uint16_t* kinst = k + (size_t)bm.inst * N * D;
  const uint16_t* qinst = q + (size_t)bm.inst * R * D;
  const float* lse_inst = lse2 + (size_t)bm.inst * R;
  const int nq32 = (nrows + 31) / 32 * 32;
  for (int r = threadIdx.x; r < nq32; r += kSBlock)
    s_lse[r] = r < nrows ? lse_inst[row_lo + r] : INFINITY;   // padded rows contribute 0

  MfmaKeys<D> mk;
  if (active) load_keys<D>(mk, kinst, kbase, K, lane);
  else zero_keys<D>(mk);
  float cs[32];
#pragma unroll
  for (int i = 0; i < 32; ++i) cs[i] = 0.f;

  auto pre = [](int) {};
  auto epi = [&](int t, f32x16_t (&acc)[2]) {
    const float lq = s_lse[t * 32 + (lane % 32)];
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int r = 0; r < 16; ++r)
        cs[kb * 16 + r] += fast_exp2(__builtin_fmaf(acc[kb][r], c, -lq));
  };
  // run_tiles starts with a barrier, which also publishes s_lse
  run_tiles<D>(mk, qt, qinst, row_lo, row_hi, lane, pre, epi);
  if (!active) return;
  // transpose-reduce over the 32 lanes of each half: lane j ends with value j
#pragma unroll
  for (int o = 16; o >= 1; o >>= 1) {
    const bool up = (lane & o) != 0;
#pragma unroll
    for (int i = 0; i < o; ++i) {
      const float send = up ? cs[i] : cs[i + o];
      const float keep = up ? cs[i + o] : cs[i];
      cs[i] = keep + __shfl_xor(send, o, kWave);
    }
  }
  const int j = lane % 32;
  const int key = kbase + acc_key(j / 16, j % 16, half);
  if (key < K) col[((size_t)bm.inst * n_slab + bm.slab) * K + key] = cs[0];
}

// ---------------------------------------------------------------------------
// VALU path (fp32 caches): one thread per row (pass 1) / per slot (pass 2)
// ---------------------------------------------------------------------------
template <typename T, int D>
__device__ __forceinline__ void stage_rows(float* dst, const T* src, int row0, int nrow_valid,
                                           int nrows) {
  for (int e = threadIdx.x; e < nrows * D; e += blockDim.x) {
    const int r = e / D, dd = e % D;
    dst[r * (D + 1) + dd] = r < nrow_valid ? to_f32(src[(size_t)(row0 + r) * D + dd]) : 0.f;
  }
}

template <typename T, int D>
__global__ __launch_bounds__(kGenBlock) void score_rows_valu(
    const T* __restrict__ k, const T* __restrict__ q, int N, int R, int n_chunk, float c,
    float2* __restrict__ part) {
  __shared__ float kt[kGenKeys * (D + 1)];
  __shared__ float qtile[kGenBlock * (D + 1)];
  const int chunk = blockIdx.x, rb = blockIdx.y, inst = blockIdx.z;
  const int key0 = chunk * kGenKeys;
  const int nk = min(kGenKeys, N - key0);
  const int row0 = rb * kGenBlock;
  const int nr = min(kGenBlock, R - row0);
  stage_rows<T, D>(kt, k + (size_t)inst * N * D, key0, nk, kGenKeys);
  stage_rows<T, D>(qtile, q + (size_t)inst * R * D, row0, nr, kGenBlock);
  __syncthreads();
  const int t = threadIdx.x;
  if (t >= nr) return;
  float m = kFloor, l = 0.f;
  for (int j = 0; j < nk; ++j) {
    float s = 0.f;
    for (int dd = 0; dd < D; ++dd) s = __builtin_fmaf(qtile[t * (D + 1) + dd], kt[j * (D + 1) + dd], s);
    const float x = s * c;
    const float mn = fmaxf(m, x);
    l = l * fast_exp2(m - mn) + fast_exp2(x - mn);
    m = mn;
  }
  part[((size_t)inst * n_chunk + chunk) * R + row0 + t] = make_float2(m, l);
}

template <typename T, int D>
__global__ __launch_bounds__(kGenBlock) void score_cols_valu(
    const T* __restrict__ k, const T* __restrict__ q, int N, int K, int R, float c,
    const float* __restrict__ lse2, float* __restrict__ col) {
  __shared__ float kt[kGenBlock * (D + 1)];
  __shared__ float qtile[kGenRows * (D + 1)];
  const int kb = blockIdx.x, inst = blockIdx.y;
  const int key0 = kb * kGenBlock;
  const int nk = min(kGenBlock, K - key0);
  stage_rows<T, D>(kt, k + (size_t)inst * N * D, key0, nk, kGenBlock);
  const int t = threadIdx.x;
  float acc = 0.f;
  for (int r0 = 0; r0 < R; r0 += kGenRows) {
    const int nr = min(kGenRows, R - r0);
    __syncthreads();
    stage_rows<T, D>(qtile, q + (size_t)inst * R * D, r0, nr, kGenRows);
    __syncthreads();
    for (int r = 0; r < nr; ++r) {
      float s = 0.f;
      for (int dd = 0; dd < D; ++dd) s = __builtin_fmaf(kt[t * (D + 1) + dd], qtile[r * (D + 1) + dd], s);
      acc += fast_exp2(__builtin_fmaf(s, c, -lse2[(size_t)inst * R + r0 + r]));
    }
  }
  if (t < nk) col[(size_t)inst * K + key0 + t] = acc;
}

// ---------------------------------------------------------------------------
// merge of the chunk partials: lse2_r = M + log2(sum_c l_c 2^(m_c - M))
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(kSBlock) void score_lse_kernel(const float2* __restrict__ part, int R,
                                                          int n_chunk, float* __restrict__ lse2) {
  const int inst = blockIdx.y;
  const int r = blockIdx.x * kSBlock + threadIdx.x;
  if (r >= R) return;
  const float2* p = part + (size_t)inst * n_chunk * R + r;
  float mm = p[0].x;
  for (int ch = 1; ch < n_chunk; ++ch) mm = fmaxf(mm, p[(size_t)ch * R].x);
  float ll = 0.f;
  for (int ch = 0; ch < n_chunk; ++ch) {
    const float2 v = p[(size_t)ch * R];
    ll += v.y * fast_exp2(v.x - mm);
  }
  lse2[(size_t)inst * R + r] = mm + fast_log2(ll);
}

// ---------------------------------------------------------------------------
// pooling: abar_j = (sum over slabs of col) / R ; attn_i = box filter / P
// ---------------------------------------------------------------------------
constexpr int kPoolTile = 256;
constexpr int kMaxHalo = 127;
__global__ __launch_bounds__(kSBlock) void score_pool_kernel(const float* __restrict__ col, int K,
                                                           int n_slab, int R, int pool,
                                                           float* __restrict__ attn) {
  __shared__ float tile[kPoolTile + 2 * kMaxHalo];
  const int inst = blockIdx.y;
  const int i0 = blockIdx.x * kPoolTile;
  const int h = pool / 2;
  const float fr = (float)R, fp = (float)pool;
  for (int t = threadIdx.x; t < kPoolTile + 2 * h; t += kSBlock) {
    const int j = i0 - h + t;
    float v = 0.f;
    if (j >= 0 && j < K) {
      float s = 0.f;
      for (int sl = 0; sl < n_slab; ++sl) s += col[((size_t)inst * n_slab + sl) * K + j];
      v = s / fr;
    }
    tile[t] = v;
  }
  __syncthreads();
  const int i = i0 + threadIdx.x;
  if (i >= K) return;
  float s = 0.f;
  for (int t = 0; t < pool; ++t) s += tile[threadIdx.x + t];
  attn[(size_t)inst * K + i] = s / fp;
}

// ---------------------------------------------------------------------------
// Range(v) = max - min over each of the K candidate value rows
// ---------------------------------------------------------------------------
template <typename T, int D>
__global__ __launch_bounds__(kSBlock) void vrange_kernel(const T* __restrict__ v, int N, int K,
                                                       float* __restrict__ out) {
  constexpr int VEC = Vec16<T>::n;
  constexpr int LPR = D / VEC;
  constexpr int RPB = kSBlock / LPR;
  const int inst = blockIdx.y;
  const int lane = threadIdx.x % kWave;
  const int row = blockIdx.x * RPB + threadIdx.x / LPR;
  const int seg = threadIdx.x % LPR;
  const bool ok = row < K;
  const int rr = ok ? row : K - 1;
  const uint4 w = reinterpret_cast<const uint4*>(v + ((size_t)inst * N + rr) * D)[seg];
  float f[VEC];
  Vec16<T>::unpack(w, f);
  float mx = f[0], mn = f[0];
#pragma unroll
  for (int e = 1; e < VEC; ++e) {
    mx = fmaxf(mx, f[e]);
    mn = fminf(mn, f[e]);
  }
#pragma unroll
  for (int off = 1; off < LPR; off <<= 1) {
    mx = fmaxf(mx, __shfl_xor(mx, off, kWave));
    mn = fminf(mn, __shfl_xor(mn, off, kWave));
  }
  (void)lane;
  if (ok && seg == 0) out[(size_t)inst * K + row] = mx - mn;
}

size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

template <typename T, int D>
void launch_valu(const void* k, const void* q, int n_inst, int N, int K, int R, float c,
                 const ScorePlan& pl, char* ws, hipStream_t stream) {
  float2* part = reinterpret_cast<float2*>(ws + pl.off_part);
  float* lse = reinterpret_cast<float*>(ws + pl.off_lse);
  float* col = reinterpret_cast<float*>(ws + pl.off_col);
  hipLaunchKernelGGL((score_rows_valu<T, D>), dim3(pl.n_chunk1, (R + kGenBlock - 1) / kGenBlock, n_inst),
                     dim3(kGenBlock), 0, stream, static_cast<const T*>(k), static_cast<const T*>(q),
                     N, R, pl.n_chunk1, c, part);
  hipLaunchKernelGGL(score_lse_kernel, dim3((R + kSBlock - 1) / kSBlock, n_inst), dim3(kSBlock), 0,
                     stream, part, R, pl.n_chunk1, lse);
  hipLaunchKernelGGL((score_cols_valu<T, D>), dim3((K + kGenBlock - 1) / kGenBlock, n_inst),
                     dim3(kGenBlock), 0, stream, static_cast<const T*>(k), static_cast<const T*>(q),
                     N, K, R, c, lse, col);
}

template <int D>
void launch_mfma(const void* k, const void* v, const void* q, int n_inst, int N, int K, int R,
                 float c, const ScorePlan& pl, char* ws, float* vrange, hipStream_t stream) {
  float2* part = reinterpret_cast<float2*>(ws + pl.off_part);
  float* lse = reinterpret_cast<float*>(ws + pl.off_lse);
  float* col = reinterpret_cast<float*>(ws + pl.off_col);
  const uint16_t* kk = static_cast<const uint16_t*>(k);
  const uint16_t* qq = static_cast<const uint16_t*>(q);
  const unsigned g1 = (unsigned)(n_inst * pl.n_slab * pl.n_chunk1);
  const size_t lds1 = sizeof(float2) * 4 * (size_t)pl.rows_per_slab;
  hipLaunchKernelGGL((score_rows_mfma<D>), dim3(g1), dim3(kSBlock), lds1, stream, kk,
                     static_cast<const uint16_t*>(v), qq, N, K, R, pl.n_chunk1, pl.n_slab,
                     pl.rows_per_slab, c, part, vrange);
  hipLaunchKernelGGL(score_lse_kernel, dim3((R + kSBlock - 1) / kSBlock, n_inst), dim3(kSBlock), 0,
                     stream, part, R, pl.n_chunk1, lse);
  const unsigned g2 = (unsigned)(n_inst * pl.n_slab * pl.n_chunk2);
  const size_t lds2 = sizeof(float) * (size_t)((pl.rows_per_slab + 31) / 32 * 32);
  hipLaunchKernelGGL((score_cols_mfma<D>), dim3(g2), dim3(kSBlock), lds2, stream, kk, qq, N, K,
                     R, pl.n_chunk2, pl.n_slab, pl.rows_per_slab, c, lse, col);
}

}  // namespace

ScorePlan score_plan(int dtype, int n_inst, int K, int B, int d, int G, int w) {
  ScorePlan pl{};
  const int N = K + B;
  const int R = G * w;
  pl.mfma = dtype == VASE_BF16;
  if (pl.mfma) {
    pl.n_chunk1 = (N + kKeysPerBlock - 1) / kKeysPerBlock;
    pl.n_chunk2 = (K + kKeysPerBlock - 1) / kKeysPerBlock;
    pl.n_slab = (R + kMaxSlab - 1) / kMaxSlab;
    int rps = (R + pl.n_slab - 1) / pl.n_slab;
    pl.rows_per_slab = (rps + 31) / 32 * 32;
  } else {
    pl.n_chunk1 = (N + kGenKeys - 1) / kGenKeys;
    pl.n_chunk2 = (K + kGenBlock - 1) / kGenBlock;
    pl.n_slab = 1;
    pl.rows_per_slab = R;
  }
  pl.off_part = 0;
  pl.off_lse = align256((size_t)n_inst * pl.n_chunk1 * R * sizeof(float2));
  pl.off_col = pl.off_lse + align256((size_t)n_inst * R * sizeof(float));
  pl.bytes = pl.off_col + align256((size_t)n_inst * pl.n_slab * K * sizeof(float));
  (void)d;
  return pl;
}

hipError_t launch_score(const void* k, const void* v, const void* q, int dtype, int n_inst, int K,
                        int B, int d, int G, int w, int pool, float* attn, float* vrange,
                        void* ws, const ScorePlan& pl, hipStream_t stream) {
  const int N = K + B;
  const int R = G * w;
  const float c = 1.4426950408889634f / sqrtf((float)d);
  char* wsb = static_cast<char*>(ws);
  if (dtype == VASE_BF16) {
    if (d == 128) launch_mfma<128>(k, v, q, n_inst, N, K, R, c, pl, wsb, vrange, stream);
    else launch_mfma<64>(k, v, q, n_inst, N, K, R, c, pl, wsb, vrange, stream);
  } else {
    if (d == 128) launch_valu<float, 128>(k, q, n_inst, N, K, R, c, pl, wsb, stream);
    else launch_valu<float, 64>(k, q, n_inst, N, K, R, c, pl, wsb, stream);
  }
  const float* col = reinterpret_cast<const float*>(wsb + pl.off_col);
  hipLaunchKernelGGL(score_pool_kernel, dim3((K + kPoolTile - 1) / kPoolTile, n_inst),
                     dim3(kSBlock), 0, stream, col, K, pl.n_slab, R, pool, attn);
  // Range over the K candidate value rows (fused into pass 1 on the MFMA path)
  if (dtype != VASE_BF16) {
    const int lpr = d * 4 / 16;
    const int rpb = kSBlock / lpr;
    const dim3 rg((K + rpb - 1) / rpb, n_inst);
    if (d == 128) hipLaunchKernelGGL((vrange_kernel<float, 128>), rg, dim3(kSBlock), 0, stream,
                                     static_cast<const float*>(v), N, K, vrange);
    else hipLaunchKernelGGL((vrange_kernel<float, 64>), rg, dim3(kSBlock), 0, stream,
                            static_cast<const float*>(v), N, K, vrange);
  }
  return hipGetLastError();
}

}  // namespace vase
