// score.hip -- pooled window-mean attention score and Range(v) on gfx950.
//
// abar_i = (1/R) sum_r exp(s_ri - lse_r),  s_ri = q_r . k_i / sqrt(d),  R = G*w rows,
// lse_r = log sum_{t<N} exp(s_rt) over all N slots (Eq. 1 rows inside Eq. 2),
// attn_i = (1/P) sum_{|j-i|<=P/2, 0<=j<K} abar_j,   vrange_i = max(v_i) - min(v_i) (Eq. 5).
//
// The row normaliser depends on every slot, so the scores are computed twice:
//   pass 1 (rows):  per row, the sum of exp2 over the slots -> lse2_r
//   pass 2 (cols):  p = exp2(s*c - lse2_r), column sums over rows
//   pool:           per slot: sum over row slabs, /R, then the P-wide box filter
// All exponentials are base 2 with c = log2(e)/sqrt(d) folded in.  No floating
// point atomics are used; every reduction has a fixed order.
// bf16 caches use MFMA (v_mfma_f32_32x32x16_bf16, described below); fp32 caches
// use a plain VALU path (one thread per row / per key) with Range as its own
// kernel.
#include "vase_internal.hpp"
#include "vase.h"

#include <type_traits>

namespace vase {
namespace {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));

constexpr int kSBlock = 256;
constexpr float kFloor = -3.0e38f;  // finite stand-in for an empty maximum
constexpr int kGenKeys = 32;        // VALU path: keys per chunk
constexpr int kGenRows = 32;        // VALU path: rows per staging step
constexpr int kGenBlock = 64;

__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }
__device__ __forceinline__ float fast_log2(float x) { return __builtin_amdgcn_logf(x); }
constexpr float kLog2e = 1.4426950408889634f;

// ---------------------------------------------------------------------------
// MFMA path (bf16), query-stationary.  A workgroup of W waves owns a slab of
// 64*W query rows of one instance and one range of its slots (the whole range
// when there are enough instances to fill the chip).  Each wave keeps its 64
// rows resident in VGPRs as A operands (two 32-row blocks); the slots stream
// through an LDS ring in chunks of 32 keys that all waves share as B operands
// (8 chunks deep, or 4 beside a 4-chunk ring of value rows when the pass
// scores them).  Accumulator element r of lane l holds (row 8(r/4) + 4h + r%4
// of a 32-row block, key l%32 of the chunk), h = l/32.
//
// The ring is filled by global->LDS DMA (global_load_lds_dwordx4) a ring's
// depth ahead of use, so the loads cost no VGPRs and their latency hides
// behind several chunks of MFMA work.  Completion is tracked with vmcnt by hand: the
// stream issues no other vector-memory operation, ring reads are explicit
// ds_read_b128 with their own lgkmcnt wait, and the barriers are plain
// s_barrier with the exact waits in front of them.  Column sums and Range
// collect in LDS and are written out after the stream.
//
// pass 1  m_f = midway between the largest and the smallest row maximum of a
//         32-row block over the first chunk (one offset per block, kept in a
//         scalar register); each lane sums exp2(s*c - m_f) over its keys, and
//         one transpose-reduce over the 32 lanes of a half wave gives l_r, so
//         lse2_r = m_f + log2 l_r.  That is exact while every row's sum lies in
//         [2^-90, FLT_MAX] (no term overflows, and the largest term of the row
//         is a normal number); otherwise the block computes the exact row
//         maxima and repeats the pass with one offset per row.  Attention-like
//         rows, whose maxima within a block differ by far less than 90
//         (base-2 units), never take that path.
// pass 2  p = exp2(s*c - lse2_r); each lane sums its 32 rows, one shuffle adds
//         the other half wave, and the W waves' sums meet in LDS in a fixed
//         order.  The same stream carries the value rows for Range (slab 0).
// With one range per instance both passes run in one kernel; otherwise pass 1
// writes (m_r, l_r) per range, a merge kernel forms lse2_r, and pass 2 runs
// as its own kernel.
// ---------------------------------------------------------------------------
typedef __attribute__((address_space(3))) void lds_void_t;

constexpr int kChunk = 32;         // keys per chunk
constexpr int kRingChunks = 8;     // LDS ring: 8 K chunks, or 4 K + 4 V chunks
constexpr int kMaxWaves = 8;
constexpr int kSlabRowsMax = 64 * kMaxWaves;
// slots per range: its column sums and Range (8 bytes per slot) share the 160
// KB of LDS with the ring (64 KB) and the row/column scratch (5 KB)
constexpr int kMaxSplitKeys = 11264;

template <int D>
struct QFrag {
  static constexpr int KS = D / 16;   // k-steps of 16
  bf16x8_t a[2][KS];
  // rows row_base + [0, 64); rows >= R read as zero.  The contraction index is
  // permuted identically in both operands: lane half h, step ks holds elements
  // [16*ks + 8*h, +8) of its row (piece 2*ks + h), so that the two lanes of a
  // row read 32 adjacent bytes in one load.
  __device__ __forceinline__ void load(const uint16_t* qinst, int row_base, int R, int lane) {
    const int half = lane / 32;
#pragma unroll
    for (int f = 0; f < 2; ++f) {
      const int row = row_base + f * 32 + lane % 32;
      const bool ok = row < R;
      const bf16x8_t* p =
          reinterpret_cast<const bf16x8_t*>(qinst + (size_t)(ok ? row : R - 1) * D + 8 * half);
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) {
        const bf16x8_t x = p[2 * ks];
        a[f][ks] = ok ? x : bf16x8_t{};
      }
    }
  }
};

// Layout of one 32-key chunk in LDS: 32 rows of D/8 16-byte pieces packed into
// 256-byte lines, the piece index XOR-swizzled by the line, so that the 16
// lanes of a B-operand read (16 rows, same piece) hit 16 bank groups.
template <int D>
struct ChunkLayout {
  static constexpr int kPieces = D / 8;
  static constexpr int kRowsPerLine = 16 / kPieces;
  static constexpr int kU4 = kChunk * kPieces;      // 16-byte pieces per chunk
  __device__ static __forceinline__ int off(int row, int p) {
    const int line = row / kRowsPerLine;
    const int lp = (row % kRowsPerLine) * kPieces + p;
    return line * 16 + (lp ^ (line & 15));
  }
  // inverse of off(): the (row, piece) stored at piece index idx
  __device__ static __forceinline__ void inv(int idx, int& row, int& p) {
    const int line = idx / 16;
    const int lp = (idx % 16) ^ (line & 15);
    row = line * kRowsPerLine + lp / kPieces;
    p = lp % kPieces;
  }
};

// DMA of one chunk (rows key0.., clamped to n_rows - 1) into an LDS slot.  The
// LDS side of global_load_lds is fixed (lane l of an instruction writes piece
// base + l), so each lane fetches the global piece that the swizzled layout
// puts there.  Per wave: kDma instructions (waves past the chunk issue none).
template <int D, int W>
struct ChunkDma {
  static constexpr int kU4 = ChunkLayout<D>::kU4;
  static constexpr int kDma = kU4 / (64 * W) > 0 ? kU4 / (64 * W) : 1;
  __device__ static __forceinline__ void issue(uint4* slot, const uint4* rows, int key0, int n_rows,
                                               int wave, int lane) {
#pragma unroll
    for (int i = 0; i < kDma; ++i) {
      const int base = (wave * kDma + i) * 64;
      if (kU4 % (64 * W) == 0 || base < kU4) {
        int row, p;
        ChunkLayout<D>::inv(base + lane, row, p);
        // byte offset from the instance's rows (an instance spans far less than
        // 4 GB), so the address is a uniform base plus one 32-bit lane offset
        const uint32_t key = (uint32_t)min(key0 + row, n_rows - 1);
        const uint32_t off = key * (uint32_t)(D * 2) + (uint32_t)p * 16u;
        __builtin_amdgcn_global_load_lds(
            static_cast<const void*>(reinterpret_cast<const char*>(rows) + off),
            (lds_void_t*)(slot + base), 16, 0, 0);
      }
    }
  }
};

// 16-byte LDS read that the compiler does not track (the ring is written by
// DMA, which the compiler would otherwise wait for in full before every read).
__device__ __forceinline__ bf16x8_t lds_read16(const uint4* p) {
  const uint32_t a = (uint32_t)(uintptr_t)(const __attribute__((address_space(3))) uint4*)p;
  bf16x8_t v;
  asm volatile("ds_read_b128 %0, %1" : "=v"(v) : "v"(a));
  return v;
}

// lds_read16 at a compile-time byte offset from a per-lane address (the
// instruction's 16-bit offset field), so that a ring slot known at compile
// time costs no address arithmetic.
template <int OFF>
__device__ __forceinline__ bf16x8_t lds_read16_at(uint32_t addr) {
  static_assert(OFF >= 0 && OFF < 65536, "ds_read offset field");
  bf16x8_t v;
  asm volatile("ds_read_b128 %0, %1 offset:%2" : "=v"(v) : "v"(addr), "i"(OFF));
  return v;
}

__device__ __forceinline__ uint32_t lds_addr(const void* p) {
  return (uint32_t)(uintptr_t)(const __attribute__((address_space(3))) void*)p;
}

// 4-byte LDS write, untracked for the same reason (the compiler cannot tell
// the dynamic LDS buffer from the DMA targets).  Barriers wait for it.
__device__ __forceinline__ void lds_write4(float* p, float x) {
  const uint32_t a = (uint32_t)(uintptr_t)(__attribute__((address_space(3))) float*)p;
  asm volatile("ds_write_b32 %0, %1" : : "v"(a), "v"(x) : "memory");
}

// Barrier with explicit waits: this wave's ring DMA down to `VM` outstanding
// instructions and all of its LDS operations done, then s_barrier.  Compiler
// barriers keep memory operations on their side.
template <int VM>
__device__ __forceinline__ void ring_barrier() {
  static_assert(VM >= 0 && VM < 16, "vmcnt field");
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_waitcnt(0x0070 | VM);   // vmcnt(VM) expcnt(7) lgkmcnt(0)
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
}

// The B operand pieces of one lane: LDS byte addresses of its KS pieces in
// ring slot 0 (the piece layout is the same in every slot).
template <int D>
struct BAddr {
  static constexpr int KS = D / 16;
  uint32_t a[KS];
  __device__ __forceinline__ BAddr(const uint4* ring, int lane) {
    const int row = lane % 32, half = lane / 32;
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) a[ks] = lds_addr(ring + ChunkLayout<D>::off(row, 2 * ks + half));
  }
};

// mfma_chunk for ring slot SLOT (a compile-time constant): the slot's offset
// goes into the LDS reads' offset field.
template <int D, int SLOT>
__device__ __forceinline__ void mfma_chunk_at(const QFrag<D>& qf, const BAddr<D>& ba,
                                              f32x16_t (&acc)[2]) {
  constexpr int KS = QFrag<D>::KS;
  constexpr int kSlotBytes = ChunkLayout<D>::kU4 * 16;
  bf16x8_t b[KS];
#pragma unroll
  for (int ks = 0; ks < KS; ++ks) b[ks] = lds_read16_at<SLOT * kSlotBytes>(ba.a[ks]);
  acc[0] = f32x16_t{};
  acc[1] = f32x16_t{};
  // LDS reads complete in order: depth step ks waits only for its own read
#pragma unroll
  for (int ks = 0; ks < KS; ++ks) {
    asm volatile("s_waitcnt lgkmcnt(%1)" : "+v"(b[ks]) : "i"(KS - 1 - ks));
    acc[0] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(qf.a[0][ks], b[ks], acc[0], 0, 0, 0);
    acc[1] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(qf.a[1][ks], b[ks], acc[1], 0, 0, 0);
  }
}

// acc[f] = Q_block(f) x K_chunk^T (32 rows x 32 keys each).
template <int D>
__device__ __forceinline__ void mfma_chunk(const QFrag<D>& qf, const uint4* slot, int lane,
                                           f32x16_t (&acc)[2]) {
  constexpr int KS = QFrag<D>::KS;
  const int row = lane % 32, half = lane / 32;
  bf16x8_t b[KS];
#pragma unroll
  for (int ks = 0; ks < KS; ++ks) b[ks] = lds_read16(slot + ChunkLayout<D>::off(row, 2 * ks + half));
  // the reads above are invisible to the compiler: wait for them here, tying
  // the registers so that no MFMA can be scheduled before the wait
  if constexpr (KS == 8)
    asm volatile("s_waitcnt lgkmcnt(0)" : "+v"(b[0]), "+v"(b[1]), "+v"(b[2]), "+v"(b[3]),
                 "+v"(b[4]), "+v"(b[5]), "+v"(b[6]), "+v"(b[7]));
  else
    asm volatile("s_waitcnt lgkmcnt(0)" : "+v"(b[0]), "+v"(b[1]), "+v"(b[2]), "+v"(b[3]));
  acc[0] = f32x16_t{};
  acc[1] = f32x16_t{};
#pragma unroll
  for (int ks = 0; ks < KS; ++ks) {
    acc[0] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(qf.a[0][ks], b[ks], acc[0], 0, 0, 0);
    acc[1] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(qf.a[1][ks], b[ks], acc[1], 0, 0, 0);
  }
}


// Value score of the rows of a chunk held in an LDS slot, into out[key - key_lo]
// for keys below hi: Range = max - min (Eq. 5), L2 = sqrt(sum v^2) or
// Var = mean (v - mu)^2 (Appendix A), over each row's D elements.
template <int D, int W>
__device__ __forceinline__ void chunk_value(const uint4* vslot, int key0, int key_lo, int hi,
                                            int kind, float* out, bool check, bool& bad) {
  constexpr int kPieces = D / 8;
  constexpr int kU4 = ChunkLayout<D>::kU4;
  constexpr int kPer = (kU4 + 64 * W - 1) / (64 * W);
#pragma unroll
  for (int i = 0; i < kPer; ++i) {
    const int pc = (int)threadIdx.x + i * 64 * W;   // consecutive lanes: consecutive pieces of a row
    const int pcc = pc < kU4 ? pc : kU4 - 1;
    const int row = pcc / kPieces;
    bf16x8_t w = lds_read16(vslot + ChunkLayout<D>::off(row, pcc % kPieces));
    asm volatile("s_waitcnt lgkmcnt(0)" : "+v"(w));
    float f[8];
    Vec16<bf16_t>::unpack(__builtin_bit_cast(uint4, w), f);
    const float val = row_value_score<8, kPieces>(f, kind);
    if (check) bad |= key0 + row < hi && any_nonfinite<8>(f);
    if (pc < kU4 && pc % kPieces == 0 && key0 + row < hi) lds_write4(out + (key0 + row - key_lo), val);
  }
}

// Transpose-reduce over the 32 lanes of each half wave: lane j ends with
// element j reduced (sum or max) over its half's lanes.
template <bool MAX>
__device__ __forceinline__ float treduce32(float (&v)[32], int lane) {
#pragma unroll
  for (int o = 16; o >= 1; o >>= 1) {
    // lanes with bit o set keep the upper half and send the lower; the swap is
    // done on the bits so that no element is picked by a lane-dependent index
    const uint32_t m = (lane & o) ? 0xffffffffu : 0u;
#pragma unroll
    for (int i = 0; i < o; ++i) {
      const uint32_t lo = __float_as_uint(v[i]), hi = __float_as_uint(v[i + o]);
      const uint32_t x = (lo ^ hi) & m;
      const float send = __uint_as_float(hi ^ x);
      const float keep = __uint_as_float(lo ^ x);
      const float got = __shfl_xor(send, o, kWave);
      v[i] = MAX ? fmaxf(keep, got) : keep + got;
    }
  }
  return v[0];
}

// slab row of element j (= 16 f + r) of a lane in half h of a wave
__device__ __forceinline__ int elem_row(int j, int half) {
  return (j / 16) * 32 + 8 * ((j % 16) / 4) + 4 * half + (j % 4);
}

// Decode-query logits of one chunk: q_dec[g] . k_key for the chunk's keys below
// hi and g < G, into dst[g * stride + key - base].  Two 16-key tiles of
// v_mfma_f32_16x16x32_bf16 with the keys as the A operand (lane l: key l % 16,
// depth [8(l/16), +8) of each 32-deep step) and the query rows as the B operand
// (column l % 16 = head, clamped to G - 1; those columns are dropped),
// accumulated over the depth steps in order, so that the logits are bit for
// bit those of a decode kernel that runs the same tiles from global memory.
// Lane l ends with keys 4(l/16) .. +3 of head l % 16.  TO_LDS: dst is LDS
// (written untracked, like the ring); else global memory.
typedef float df32x4_t __attribute__((ext_vector_type(4)));
template <int D, bool TO_LDS>
__device__ __forceinline__ void dec_logits_chunk(const uint4* slot, const uint4* qd, int G, int lane,
                                                 int key0, int hi, int base, float* dst,
                                                 int stride) {
  constexpr int KS = D / 32;
  constexpr int KP = D / 8;
  const int hm = lane % 16, hq = lane / 16;
  const int hc = min(hm, G - 1);
  if constexpr (D == 128 && TO_LDS) {
    // one 256-byte line per key row: piece p of row r sits at r*16 + (p ^ (r & 15)),
    // so depth step ks of tile t is at a per-lane base, a per-lane 64-byte step
    // (ks ^ (hm >> 2)) and a fixed 4 KB per tile (immediate offsets).  The lane
    // id is read here (volatile), so these addresses are formed at each call
    // instead of being kept live across the key loop, where they would spill.
    uint32_t ln;
    asm volatile("v_mbcnt_lo_u32_b32 %0, -1, 0\n\tv_mbcnt_hi_u32_b32 %0, -1, %0" : "=v"(ln));
    const int lm = (int)(ln % 16u), lq = (int)(ln / 16u);
    const int lc = min(lm, G - 1);
    const uint32_t bq = lds_addr(qd) + (uint32_t)(lc * KP + lq) * 16u;
    const uint32_t a0 = lds_addr(slot) + (uint32_t)(16 * lm + (lq ^ (lm & 3))) * 16u;
    uint32_t aa[KS];
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) aa[ks] = a0 + ((uint32_t)(ks ^ (lm >> 2)) << 6);
    bf16x8_t b[KS], a[KS];
    b[0] = lds_read16_at<0>(bq);
    b[1] = lds_read16_at<64>(bq);
    b[2] = lds_read16_at<128>(bq);
    b[3] = lds_read16_at<192>(bq);
    const bool full = key0 + kChunk <= hi && stride % 4 == 0;
    const int k4 = key0 + 4 * lq;
    float* p = dst + (size_t)lc * stride + (k4 - base);
#pragma unroll
    for (int t = 0; t < 2; ++t) {
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) a[ks] = t ? lds_read16_at<4096>(aa[ks]) : lds_read16_at<0>(aa[ks]);
      asm volatile("s_waitcnt lgkmcnt(0)" : "+v"(a[0]), "+v"(a[1]), "+v"(a[2]), "+v"(a[3]),
                   "+v"(b[0]), "+v"(b[1]), "+v"(b[2]), "+v"(b[3]));
      df32x4_t acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int ks = 0; ks < KS; ++ks)
        acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[ks], b[ks], acc, 0, 0, 0);
      if (lm < G) {
        if (full) {
          asm volatile("ds_write_b128 %0, %1 offset:%2" : : "v"(lds_addr(p)), "v"(acc), "i"(64 * t)
                       : "memory");
        } else {
#pragma unroll
          for (int i = 0; i < 4; ++i)
            if (k4 + 16 * t + i < hi) lds_write4(p + 16 * t + i, acc[i]);
        }
      }
    }
    return;
  }
  bf16x8_t b[KS];
#pragma unroll
  for (int ks = 0; ks < KS; ++ks) b[ks] = lds_read16(qd + hc * KP + 4 * ks + hq);
#pragma unroll
  for (int t = 0; t < 2; ++t) {
    bf16x8_t a[KS];
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) a[ks] = lds_read16(slot + ChunkLayout<D>::off(16 * t + hm, 4 * ks + hq));
    if constexpr (KS == 4)
      asm volatile("s_waitcnt lgkmcnt(0)" : "+v"(a[0]), "+v"(a[1]), "+v"(a[2]), "+v"(a[3]),
                   "+v"(b[0]), "+v"(b[1]), "+v"(b[2]), "+v"(b[3]));
    else
      asm volatile("s_waitcnt lgkmcnt(0)" : "+v"(a[0]), "+v"(a[1]), "+v"(b[0]), "+v"(b[1]));
    df32x4_t acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int ks = 0; ks < KS; ++ks)
      acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[ks], b[ks], acc, 0, 0, 0);
    if (hm < G) {
      const int key = key0 + 16 * t + 4 * hq;
      float* p = dst + (size_t)hm * stride + (key - base);
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        if (key + i < hi) {
          if (TO_LDS) lds_write4(p + i, acc[i]);
          else p[i] = acc[i];
        }
      }
    }
  }
}

enum ScoreMode { kPass1 = 0, kPass2 = 1, kFused = 2 };

// The ring and the stream state of one pass.  A pass that scores values (pass
// 2 with Range, L2 or Var) streams the V rows through a second ring of the
// same depth S = 4 beside the K ring; every other pass gives the whole LDS
// ring to K (S = 8), so its DMA runs further ahead.  Every chunk costs the
// same number of DMA instructions, which the vmcnt waits count.
template <int D, int W, bool WITH_V>
struct Stream {
  static constexpr int kU4 = ChunkLayout<D>::kU4;
  static constexpr int kPerChunk = ChunkDma<D, W>::kDma * (WITH_V ? 2 : 1);
  static constexpr int S = WITH_V ? kRingChunks / 2 : kRingChunks;   // ring depth in chunks
  uint4* kring;
  uint4* vring;
  const uint4* krows;
  const uint4* vrows;
  int key_lo, n_krows, n_vrows, wave, lane;
  __device__ __forceinline__ uint4* kslot(int ch) const { return kring + (ch % S) * kU4; }
  __device__ __forceinline__ uint4* vslot(int ch) const { return vring + (ch % S) * kU4; }
  __device__ __forceinline__ void fetch(int ch) const {
    const int key0 = key_lo + kChunk * ch;
    ChunkDma<D, W>::issue(kslot(ch), krows, key0, n_krows, wave, lane);
    if (WITH_V) ChunkDma<D, W>::issue(vslot(ch), vrows, key0, n_vrows, wave, lane);
  }
};

// Chunk pipeline over chunks [0, nc) with a ring of S chunks.  The first A
// chunks are fetched up front and chunk 0 goes through the MFMAs before the
// first step (init sees its products then); at step ch a wave
//   * fetches chunk ch+A into ring slot (ch+A)%S,
//   * runs side(ch+1) (value scores or decode logits of chunk ch+1, the
//     column-sum flush of an earlier chunk),
//   * issues the MFMAs of chunk ch+1 and the VALU epilogue of chunk ch (its
//     accumulators were filled at step ch-1) in one basic block,
//     (a wave whose rows all lie past the last window row skips both: it
//     only fetches and meets the other waves),
//   * after every step (S = 4, A = 4) or every odd step (S = 8, A = 6) waits
//     until its own DMA up to chunk ch+2 (S = 4) or ch+3 (S = 8) has landed and
//     meets the other waves.
// With S = 8 no wave can be more than one step ahead of another, so the slot
// (ch+6)%8 = (ch-2)%8 refilled at step ch was last read at step ch-3, and a
// barrier lies between any three consecutive steps; each barrier covers the
// chunks read in the two steps after it.  The loop is unrolled over the ring,
// so every slot and accumulator buffer is a compile-time constant.  Chunks
// past the end fetch clamped rows; their results are dropped.  The caller
// waits for the trailing DMA before the ring is used again.
template <int U, int S, typename F>
__device__ __forceinline__ bool ring_steps(F& step, int t) {
  if constexpr (U < S) {
    if (step(std::integral_constant<int, U>{}, t)) return true;
    return ring_steps<U + 1, S>(step, t);
  } else {
    return false;
  }
}

template <int D, typename St, typename Epi, typename Side, typename Init>
__device__ __forceinline__ void stream_chunks(const QFrag<D>& qf, const St& st, int nc, int lane,
                                              bool active, Epi&& epi, Side&& side, Init&& init) {
  constexpr int S = St::S;
  // an 8-deep ring meets after every other step: fetch 6 ahead, wait for 3 ahead
  constexpr bool kPair = S == 8;
  constexpr int kAhead = kPair ? S - 2 : S;
  constexpr int kWait = kPair ? 3 * St::kPerChunk : (S - 2) * St::kPerChunk;
  const BAddr<D> ba(st.kring, lane);
#pragma unroll
  for (int ch = 0; ch < kAhead; ++ch) st.fetch(ch);
  ring_barrier<kWait>();
  f32x16_t acc[2][2];
  side(0);
  if (active) {
    mfma_chunk_at<D, 0>(qf, ba, acc[0]);
    init(acc[0]);                       // sees chunk 0's products before its epilogue
  }
  ring_barrier<kWait>();
  auto step = [&](auto u_, int t) -> bool {
    constexpr int U = decltype(u_)::value;
    const int ch = t + U;
    st.fetch(ch + kAhead);
    side(ch + 1);
    if (active) {
      mfma_chunk_at<D, (U + 1) % S>(qf, ba, acc[(U + 1) % 2]);
      epi(ch, acc[U % 2]);
    }
    __builtin_amdgcn_sched_barrier(0);
    if (!kPair || U % 2 == 1) ring_barrier<kWait>();
    return ch + 1 >= nc;
  };
  for (int t = 0; t < nc; t += S)
    if (ring_steps<0, S>(step, t)) break;
}

// Plain loop (one chunk at a time) for the rarely taken exact path.
template <int D, typename St, typename Epi>
__device__ __forceinline__ void simple_chunks(const QFrag<D>& qf, const St& st, int nc, int lane,
                                              Epi&& epi) {
  for (int ch = 0; ch < nc; ++ch) {
    st.fetch(ch);
    ring_barrier<0>();
    f32x16_t a[2];
    mfma_chunk<D>(qf, st.kslot(ch), lane, a);
    epi(ch, a);
    ring_barrier<0>();
  }
}

// DL: decode-query logits of pass 1: 0 none, 1 staged in LDS and written after
// the pass, 2 written from the chunk loop (when they do not fit in LDS).
// PARTIAL: the last slab holds fewer than W waves' rows (its other waves only
// stream the keys); a separate instantiation, so that full slabs carry no test
template <int D, int W, int MODE, int DL, bool PARTIAL>
__global__ __launch_bounds__(64 * W, 2) void score_mfma_kernel(
    const uint4* __restrict__ k, const uint4* __restrict__ v, const uint16_t* __restrict__ q,
    int N, int K, int R, int n_slab, int n_split, int split_keys, float c, int pool, int value_kind,
    const float* __restrict__ lse_win, float2* __restrict__ part, const float* __restrict__ lse2,
    float* __restrict__ col, float* __restrict__ vrange, float* __restrict__ attn,
    const int32_t* __restrict__ ord, const uint4* __restrict__ qdec, int G_dec,
    float* __restrict__ dlog, int dl_stride, uint32_t* __restrict__ status) {
  constexpr int kU4 = ChunkLayout<D>::kU4;
  __shared__ uint4 ring[kRingChunks * kU4];
  __shared__ float rowbuf[W][2][32];
  __shared__ float colbuf[4][kChunk][W];   // [chunk % 4][column][wave]
  extern __shared__ float keybuf[];   // pass 2: [split_keys] column sums, then [split_keys] Range
  constexpr int KP = D / 8;
  const uint32_t lb = xcd_logical_block(blockIdx.x, gridDim.x);
  const int split = (int)(lb % (uint32_t)n_split);
  const uint32_t t0 = lb / (uint32_t)n_split;
  const int slab = (int)(t0 % (uint32_t)n_slab);
  const int inst = (int)(t0 / (uint32_t)n_slab);
  const int lane = threadIdx.x % kWave, half = lane / 32;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);   // uniform per wave
  const int j = lane % 32;
  const int row_base = slab * 64 * W + wave * 64;
  // waves whose 64 rows all lie past R (the last slab of a window that is not
  // a multiple of the slab) stream the keys with the others but score nothing;
  // the column sums take the first n_act waves' partial sums
  const bool active = !PARTIAL || row_base < R;
  const int n_act = PARTIAL ? min(W, (R - slab * 64 * W + 63) / 64) : W;
  const int key_lo = split * split_keys;
  const uint4* kinst = k + (size_t)inst * N * KP;
  QFrag<D> qf;
  qf.load(q + (size_t)inst * R * D, row_base, R, lane);
  float rs[32];   // per element: exact row maxima (exact path), then lse2 (pass 2)
  // data faults for the status word: a row normaliser that is not a positive
  // finite number (this lane's row), a value row with a non-finite element
  bool row_bad = false, v_bad = false;
  auto report = [&]() {
    if (status) {
      block_status(status, row_bad, VASE_STATUS_ROW_NORM);
      block_status(status, v_bad, VASE_STATUS_VALUE_ROW);
    }
  };

  if (MODE != kPass2) {
    // pass 1 covers this range's slots, or only the buffer [K, N) when the
    // persistent part of every row's normaliser is supplied (lse_win)
    const bool single = lse_win != nullptr;
    const int lo1 = single ? K : key_lo;
    const int hi1 = single ? N : min(N, key_lo + split_keys);
    const int nc1 = (hi1 - lo1 + kChunk - 1) / kChunk;
    const Stream<D, W, false> st{ring, ring, kinst, kinst, lo1, N, N, wave, lane};
    // decode-query logits of the streamed keys (slab 0 only).  The G_dec query
    // rows wait in the pass-2 scratch, which pass 1 does not use, and, when
    // dl_stride > 0, the logits too ([G_dec][dl_stride], written out after the
    // pass): a global store inside the chunk loop would be counted by the
    // vmcnt waits that pace the ring
    float* const dl = DL != 0 && slab == 0 ? dlog + (size_t)inst * G_dec * N : nullptr;
    uint4* const qd = reinterpret_cast<uint4*>(keybuf);
    float* const dls = keybuf + G_dec * KP * 4;
    if (dl) {
      for (int i = threadIdx.x; i < G_dec * KP; i += 64 * W) qd[i] = qdec[(size_t)inst * G_dec * KP + i];
    }
    // mb[f]: one offset per 32-row block, midway between the largest and the
    // smallest row maximum over the first chunk (rows >= R left out), taken
    // from chunk 0's products when the stream has computed them
    float mb[2] = {0.f, 0.f};
    auto init1 = [&](f32x16_t (&a)[2]) {
      const bool ok = lo1 + j < hi1;
      float t[32];
#pragma unroll
      for (int f = 0; f < 2; ++f)
#pragma unroll
        for (int r = 0; r < 16; ++r) t[f * 16 + r] = ok ? a[f][r] * c : -INFINITY;
      const float mj0 = treduce32<true>(t, lane);     // row max of element j over the chunk
      const bool rv = row_base + elem_row(j, half) < R;
      float hi = rv ? mj0 : -INFINITY, lo = rv ? mj0 : INFINITY;
#pragma unroll
      for (int o = 1; o <= 32; o <<= 1) {
        if (o == 16) continue;                        // lanes j and j^16 hold different blocks
        hi = fmaxf(hi, __shfl_xor(hi, o, kWave));
        lo = fminf(lo, __shfl_xor(lo, o, kWave));
      }
      const float mid = hi == -INFINITY ? 0.f : 0.5f * (hi + lo);
      mb[0] = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(mid), 0));
      mb[1] = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(mid), 16));
    };
    float l[32];
#pragma unroll
    for (int i = 0; i < 32; ++i) l[i] = 0.f;
    auto epi1 = [&](int ch, f32x16_t (&a)[2]) {
      const float okf = lo1 + kChunk * ch + j < hi1 ? 1.f : 0.f;
#pragma unroll
      for (int f = 0; f < 2; ++f)
#pragma unroll
        for (int r = 0; r < 16; ++r)
          l[f * 16 + r] = __builtin_fmaf(okf, fast_exp2(__builtin_fmaf(a[f][r], c, -mb[f])),
                                         l[f * 16 + r]);
    };
    auto side1 = [&](int ch) {
      if (DL != 0 && dl && ch < nc1 && wave == ch % W) {
        if constexpr (DL == 1)
          dec_logits_chunk<D, true>(st.kslot(ch), qd, G_dec, lane, lo1 + kChunk * ch, hi1, lo1,
                                    dls, dl_stride);
        else
          dec_logits_chunk<D, false>(st.kslot(ch), qd, G_dec, lane, lo1 + kChunk * ch, hi1, 0,
                                     dl, N);
      }
      // keep the logit tiles' registers apart from the chunk's MFMA operands
      if (DL != 0) __builtin_amdgcn_sched_barrier(0);
    };
    stream_chunks<D>(qf, st, nc1, lane, active, epi1, side1, init1);
    ring_barrier<0>();                                // trailing DMA landed
    if (DL == 1 && dl) {
      const int nk1 = hi1 - lo1;
      for (int i = threadIdx.x; i < G_dec * nk1; i += 64 * W) {
        const int g = i / nk1, t = i - g * nk1;
        dl[(size_t)g * N + lo1 + t] = dls[g * dl_stride + t];
      }
    }
    float lj = treduce32<false>(l, lane);
    float mj = j < 16 ? mb[0] : mb[1];
    const int row = row_base + elem_row(j, half);
    // Exact as long as every term stays finite and the largest term of each row
    // stays a normal number: sums in [2^-90, FLT_MAX] guarantee both.
    const bool bad = row < R && !(lj >= 0x1p-90f && lj <= 3.0e38f);
    if (__syncthreads_or(bad)) {
      // exact row maxima first, then the sums again with one offset per row
      float mx[32];
#pragma unroll
      for (int i = 0; i < 32; ++i) mx[i] = -INFINITY;
      auto epim = [&](int ch, f32x16_t (&a)[2]) {
        const bool ok = lo1 + kChunk * ch + j < hi1;
#pragma unroll
        for (int f = 0; f < 2; ++f)
#pragma unroll
          for (int r = 0; r < 16; ++r) mx[f * 16 + r] = ok ? fmaxf(mx[f * 16 + r], a[f][r] * c) : mx[f * 16 + r];
      };
      simple_chunks<D>(qf, st, nc1, lane, epim);
      rowbuf[wave][half][j] = treduce32<true>(mx, lane);
      __syncthreads();
#pragma unroll
      for (int i = 0; i < 32; ++i) {
        rs[i] = rowbuf[wave][half][i];
        l[i] = 0.f;
      }
      auto epix = [&](int ch, f32x16_t (&a)[2]) {
        const float okf = lo1 + kChunk * ch + j < hi1 ? 1.f : 0.f;
#pragma unroll
        for (int f = 0; f < 2; ++f)
#pragma unroll
          for (int r = 0; r < 16; ++r)
            l[f * 16 + r] = __builtin_fmaf(okf, fast_exp2(__builtin_fmaf(a[f][r], c, -rs[f * 16 + r])),
                                           l[f * 16 + r]);
      };
      simple_chunks<D>(qf, st, nc1, lane, epix);
      lj = treduce32<false>(l, lane);
      mj = rowbuf[wave][half][j];
    }
    if (MODE == kPass1) {
      if (row < R) part[((size_t)inst * n_split + split) * R + row] = make_float2(mj, lj);
      return;
    }
    __syncthreads();
    float l2 = mj + fast_log2(lj);
    if (single && row < R) {
      // add the supplied persistent part: log2(2^l2 + 2^(L log2 e))
      const float b = lse_win[(size_t)inst * R + row] * kLog2e;
      const float m = fmaxf(l2, b);
      l2 = m + fast_log2(fast_exp2(l2 - m) + fast_exp2(b - m));
    }
    row_bad = row < R && !(l2 > -INFINITY && l2 < INFINITY);
    rowbuf[wave][half][j] = row < R ? l2 : INFINITY;
    __syncthreads();
#pragma unroll
    for (int i = 0; i < 32; ++i) rs[i] = rowbuf[wave][half][i];
  } else {
#pragma unroll
    for (int i = 0; i < 32; ++i) {
      const int row = row_base + elem_row(i, half);
      rs[i] = row < R ? lse2[(size_t)inst * R + row] : INFINITY;   // padded rows give p = 0
    }
  }

  // ---- pass 2: column sums over the slab's rows for slots [key_lo, hi2)
  const int hi2 = min(K, key_lo + split_keys);
  if (hi2 <= key_lo) {
    report();
    return;
  }
  const int nc2 = (hi2 - key_lo + kChunk - 1) / kChunk;
  // value scores of the candidates: not for random reservation (drawn elsewhere)
  // nor when the caller supplies them
  const bool rng = slab == 0 && value_kind <= VASE_VALUE_VAR;
  float* colsum = keybuf;
  float* vr = keybuf + split_keys;
  // column sums of chunk ch over the W waves, fixed order; colbuf rotates over
  // four chunks.  With the value rows in the stream (a barrier after every
  // step) chunk ch is flushed at step ch+1; without them (a barrier after
  // every odd step) at step ch+2.  Either way the flush follows a barrier that
  // followed every wave's epilogue of ch, and a barrier separates it from the
  // epilogue of ch+4 that writes its buffer again
  auto flush = [&](int ch) {
    if (ch >= 0 && ch < nc2 && wave == ch % W && lane < kChunk) {
      // the W waves' sums of this column sit together: one or two 16-byte reads
      float cw[W];
#pragma unroll
      for (int w = 0; w < W; w += 4)
        *reinterpret_cast<float4*>(cw + w) = *reinterpret_cast<const float4*>(&colbuf[ch % 4][lane][w]);
      float sum = cw[0];
#pragma unroll
      for (int w = 1; w < W; ++w) sum += w < n_act ? cw[w] : 0.f;
      lds_write4(colsum + kChunk * ch + lane, sum);
    }
  };
  auto epi2 = [&](int ch, f32x16_t (&a)[2]) {
    // four partial sums, each seeded with its first term
    float p0 = fast_exp2(__builtin_fmaf(a[0][0], c, -rs[0]));
    float p1 = fast_exp2(__builtin_fmaf(a[0][1], c, -rs[1]));
    float p2 = fast_exp2(__builtin_fmaf(a[0][2], c, -rs[2]));
    float p3 = fast_exp2(__builtin_fmaf(a[0][3], c, -rs[3]));
#pragma unroll
    for (int f = 0; f < 2; ++f)
#pragma unroll
      for (int r = f == 0 ? 4 : 0; r < 16; r += 4) {
        const int e = f * 16 + r;
        p0 += fast_exp2(__builtin_fmaf(a[f][r], c, -rs[e]));
        p1 += fast_exp2(__builtin_fmaf(a[f][r + 1], c, -rs[e + 1]));
        p2 += fast_exp2(__builtin_fmaf(a[f][r + 2], c, -rs[e + 2]));
        p3 += fast_exp2(__builtin_fmaf(a[f][r + 3], c, -rs[e + 3]));
      }
    float cs = (p0 + p1) + (p2 + p3);
    cs += __shfl_xor(cs, 32, kWave);
    colbuf[ch % 4][j][wave] = cs;
  };
  if (rng) {
    // the value rows ride in the second half of the ring
    const Stream<D, W, true> st{ring, ring + (kRingChunks / 2) * kU4, kinst,
                                v + (size_t)inst * N * KP, key_lo, N, K, wave, lane};
    auto side2 = [&](int ch) {
      if (ch < nc2)
        chunk_value<D, W>(st.vslot(ch), key_lo + kChunk * ch, key_lo, hi2, value_kind, vr,
                          status != nullptr, v_bad);
      flush(ch - 2);
    };
    stream_chunks<D>(qf, st, nc2, lane, active, epi2, side2, [](f32x16_t (&)[2]) {});
  } else {
    const Stream<D, W, false> st{ring, ring, kinst, kinst, key_lo, N, N, wave, lane};
    stream_chunks<D>(qf, st, nc2, lane, active, epi2, [&](int ch) { flush(ch - 3); },
                     [](f32x16_t (&)[2]) {});
  }
  ring_barrier<0>();                                  // trailing DMA landed, last colbuf visible
  // the stream flushed chunks up to (last step + 1) - 2; flush the rest
  const int last_side = (nc2 - 1) + 1;                // side() of the final step
  for (int ch = max(last_side - (rng ? 1 : 2), 0); ch < nc2; ++ch) flush(ch);
  __syncthreads();
  float* vr_out = vrange + (size_t)inst * K;
  if (MODE == kFused && n_slab == 1) {
    // the workgroup holds every column sum of the instance: pool here, with
    // the same arithmetic as score_pool_kernel (mean over rows, then the
    // zero-padded box filter summed in slot order, then / P).  Under an order
    // map the filter runs over temporal ranks: rank t is slot ord[t], and the
    // outputs are indexed by rank (the map is staged in the idle ring).
    const float fr = (float)R, fp = (float)pool;
    const int h = pool / 2;
    float* attn_out = attn + (size_t)inst * K;
    int* slot_of = reinterpret_cast<int*>(ring);
    if (ord) {
      for (int i = threadIdx.x; i < K; i += 64 * W)
        slot_of[i] = min(max(ord[(size_t)inst * K + i], 0), K - 1);
      __syncthreads();
    }
    for (int i = threadIdx.x; i < K; i += 64 * W) {
      float sum = 0.f;
      for (int t = 0; t < pool; ++t) {
        const int jj = i - h + t;
        sum += (jj >= 0 && jj < K) ? colsum[ord ? slot_of[jj] : jj] / fr : 0.f;
      }
      attn_out[i] = sum / fp;
      if (rng) vr_out[i] = vr[ord ? slot_of[i] : i];
    }
    report();
    return;
  }
  float* col_out = col + ((size_t)inst * n_slab + slab) * K;
  for (int i = threadIdx.x; i < hi2 - key_lo; i += 64 * W) {
    col_out[key_lo + i] = colsum[i];
    if (rng) vr_out[key_lo + i] = vr[i];
  }
  report();
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
    const T* __restrict__ k, const T* __restrict__ q, int N, int R, int n_chunk, int key_base,
    float c, float2* __restrict__ part) {
  __shared__ float kt[kGenKeys * (D + 1)];
  __shared__ float qtile[kGenBlock * (D + 1)];
  const int chunk = blockIdx.x, rb = blockIdx.y, inst = blockIdx.z;
  const int key0 = key_base + chunk * kGenKeys;
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
// (plus, when lse_win is given, its persistent part: lse2_r <- log2(2^lse2_r + 2^(L_r log2 e))).
// Returns false when lse2_r is not finite (the normaliser is 0, infinite or NaN).
__device__ __forceinline__ bool score_lse_row(const float2* __restrict__ part, int R, int n_chunk,
                                              const float* __restrict__ lse_win,
                                              float* __restrict__ lse2, int inst, int r) {
  const float2* p = part + (size_t)inst * n_chunk * R + r;
  float mm = p[0].x;
  for (int ch = 1; ch < n_chunk; ++ch) mm = fmaxf(mm, p[(size_t)ch * R].x);
  float ll = 0.f;
  for (int ch = 0; ch < n_chunk; ++ch) {
    const float2 v = p[(size_t)ch * R];
    ll += v.y * fast_exp2(v.x - mm);
  }
  float l2 = mm + fast_log2(ll);
  if (lse_win) {
    const float b = lse_win[(size_t)inst * R + r] * kLog2e;
    const float m = fmaxf(l2, b);
    l2 = m + fast_log2(fast_exp2(l2 - m) + fast_exp2(b - m));
  }
  lse2[(size_t)inst * R + r] = l2;
  return l2 > -INFINITY && l2 < INFINITY;
}

__global__ __launch_bounds__(kSBlock) void score_lse_kernel(const float2* __restrict__ part, int R,
                                                          int n_chunk, const float* __restrict__ lse_win,
                                                          float* __restrict__ lse2,
                                                          uint32_t* __restrict__ status) {
  const int inst = blockIdx.y;
  const int r = blockIdx.x * kSBlock + threadIdx.x;
  bool bad = false;
  if (r < R) bad = !score_lse_row(part, R, n_chunk, lse_win, lse2, inst, r);
  if (status) block_status(status, bad, VASE_STATUS_ROW_NORM);
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
// value score of each of the K candidate value rows (fp32 caches): Range,
// L2 or Var as in chunk_value
// ---------------------------------------------------------------------------

template <typename T, int D>
__global__ __launch_bounds__(kSBlock) void value_kernel(const T* __restrict__ v, int N, int K,
                                                      int kind, float* __restrict__ out,
                                                      uint32_t* __restrict__ status) {
  constexpr int VEC = Vec16<T>::n;
  constexpr int LPR = D / VEC;
  constexpr int RPB = kSBlock / LPR;
  const int inst = blockIdx.y;
  const int row = blockIdx.x * RPB + threadIdx.x / LPR;
  const int seg = threadIdx.x % LPR;
  const bool ok = row < K;
  const int rr = ok ? row : K - 1;
  const uint4 w = reinterpret_cast<const uint4*>(v + ((size_t)inst * N + rr) * D)[seg];
  float f[VEC];
  Vec16<T>::unpack(w, f);
  const float val = row_value_score<VEC, LPR>(f, kind);
  if (ok && seg == 0) out[(size_t)inst * K + row] = val;
  if (status) block_status(status, ok && any_nonfinite<VEC>(f), VASE_STATUS_VALUE_ROW);
}

size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

template <typename T, int D>
void launch_valu(const void* k, const void* q, int n_inst, int N, int K, int R, float c,
                 const float* lse_win, const ScorePlan& pl, char* ws, hipStream_t stream,
                 uint32_t* status) {
  float2* part = reinterpret_cast<float2*>(ws + pl.off_part);
  float* lse = reinterpret_cast<float*>(ws + pl.off_lse);
  float* col = reinterpret_cast<float*>(ws + pl.off_col);
  // row statistics over all N slots, or over the buffer only when lse_win is given
  const int key_base = lse_win ? K : 0;
  const int n_chunk = (N - key_base + kGenKeys - 1) / kGenKeys;
  hipLaunchKernelGGL((score_rows_valu<T, D>), dim3(n_chunk, (R + kGenBlock - 1) / kGenBlock, n_inst),
                     dim3(kGenBlock), 0, stream, static_cast<const T*>(k), static_cast<const T*>(q),
                     N, R, n_chunk, key_base, c, part);
  hipLaunchKernelGGL(score_lse_kernel, dim3((R + kSBlock - 1) / kSBlock, n_inst), dim3(kSBlock), 0,
                     stream, part, R, n_chunk, lse_win, lse, status);
  hipLaunchKernelGGL((score_cols_valu<T, D>), dim3((K + kGenBlock - 1) / kGenBlock, n_inst),
                     dim3(kGenBlock), 0, stream, static_cast<const T*>(k), static_cast<const T*>(q),
                     N, K, R, c, lse, col);
}

template <int D, int W, bool P>
void launch_mfma_w(const void* k, const void* v, const void* q, int n_inst, int N, int K, int R,
                   float c, int pool, int kind, const float* lse_win, const ScorePlan& pl, char* ws,
                   float* vrange, float* attn, const int32_t* ord, const DecLogits& dec,
                   hipStream_t stream, uint32_t* status) {
  const uint4* qd = static_cast<const uint4*>(dec.q);
  // pass 1 stages the decode queries, and the logits when they fit, in the
  // dynamic LDS that pass 2 uses
  const int dl_keys = ((pl.n_chunk1 == 1 ? N : pl.split_keys) + 3) / 4 * 4;   // 16-byte rows
  constexpr size_t kStaticLds = (size_t)kRingChunks * ChunkLayout<D>::kU4 * 16 + W * 2 * 32 * 4 +
                                4 * kChunk * W * 4;
  constexpr size_t kLdsCap = 160 * 1024 - kStaticLds - 1024;
  const size_t q_lds = (size_t)dec.G * D * 2;
  const int dl_stride =
      dec.out && q_lds + (size_t)dec.G * dl_keys * 4 <= kLdsCap && !lse_win ? dl_keys : 0;
  const size_t dec_lds = dec.out ? q_lds + (size_t)dec.G * dl_stride * 4 : 0;
  const int dl_mode = !dec.out ? 0 : dl_stride > 0 ? 1 : 2;
  float2* part = reinterpret_cast<float2*>(ws + pl.off_part);
  float* lse = reinterpret_cast<float*>(ws + pl.off_lse);
  float* col = reinterpret_cast<float*>(ws + pl.off_col);
  const uint4* kk = static_cast<const uint4*>(k);
  const uint4* vv = static_cast<const uint4*>(v);
  const uint16_t* qq = static_cast<const uint16_t*>(q);
  const unsigned grid = (unsigned)(n_inst * pl.n_slab * pl.n_chunk1);
  const size_t keybuf = 2 * sizeof(float) * (size_t)pl.split_keys;
  if (pl.n_chunk1 == 1) {
    auto fused = dl_mode == 0 ? score_mfma_kernel<D, W, kFused, 0, P>
                 : dl_mode == 1 ? score_mfma_kernel<D, W, kFused, 1, P>
                                : score_mfma_kernel<D, W, kFused, 2, P>;
    hipLaunchKernelGGL(fused, dim3(grid), dim3(64 * W), keybuf > dec_lds ? keybuf : dec_lds,
                       stream, kk, vv, qq, N, K, R, pl.n_slab, 1, pl.split_keys, c, pool, kind,
                       lse_win, part, lse, col, vrange, attn, ord, qd, dec.G, dec.out, dl_stride,
                       status);
    return;
  }
  // pass 1: every slot range, or one range over the buffer [K, N) when the
  // persistent part of each row's normaliser is supplied
  const int n1 = lse_win ? 1 : pl.n_chunk1;
  const int keys1 = lse_win ? (N - K + kChunk - 1) / kChunk * kChunk : pl.split_keys;
  auto pass1 = dl_mode == 0 ? score_mfma_kernel<D, W, kPass1, 0, P>
               : dl_mode == 1 ? score_mfma_kernel<D, W, kPass1, 1, P>
                              : score_mfma_kernel<D, W, kPass1, 2, P>;
  hipLaunchKernelGGL(pass1, dim3((unsigned)(n_inst * pl.n_slab * n1)), dim3(64 * W), dec_lds,
                     stream, kk, vv, qq, N, K, R, pl.n_slab, n1, keys1, c, pool, kind, lse_win,
                     part, lse, col, vrange, attn, nullptr, qd, dec.G, dec.out, dl_stride, nullptr);
  hipLaunchKernelGGL(score_lse_kernel, dim3((R + kSBlock - 1) / kSBlock, n_inst), dim3(kSBlock), 0,
                     stream, part, R, n1, lse_win, lse, status);
  hipLaunchKernelGGL((score_mfma_kernel<D, W, kPass2, 0, P>), dim3(grid), dim3(64 * W), keybuf, stream,
                     kk, vv, qq, N, K, R, pl.n_slab, pl.n_chunk1, pl.split_keys, c, pool, kind,
                     nullptr, part, lse, col, vrange, attn, nullptr, nullptr, 0, nullptr, 0, status);
}

template <int D>
void launch_mfma(const void* k, const void* v, const void* q, int n_inst, int N, int K, int R,
                 float c, int pool, int kind, const float* lse_win, const ScorePlan& pl, char* ws,
                 float* vrange, float* attn, const int32_t* ord, const DecLogits& dec,
                 hipStream_t stream, uint32_t* status) {
  // some waves of the last slab hold no window row
  const bool partial = pl.n_slab * pl.rows_per_slab - R >= 64;
#define VASE_MFMA_W(W, P)                                                                          \
  launch_mfma_w<D, W, P>(k, v, q, n_inst, N, K, R, c, pool, kind, lse_win, pl, ws, vrange, attn, \
                         ord, dec, stream, status)
  if (pl.waves == 4) {
    if (partial) VASE_MFMA_W(4, true);
    else VASE_MFMA_W(4, false);
  } else {
    if (partial) VASE_MFMA_W(8, true);
    else VASE_MFMA_W(8, false);
  }
#undef VASE_MFMA_W
}

}  // namespace

ScorePlan score_plan(int dtype, int n_inst, int K, int B, int d, int G, int w) {
  ScorePlan pl{};
  const int N = K + B;
  const int R = G * w;
  pl.mfma = dtype == VASE_BF16;
  if (pl.mfma) {
    // slabs of at most 512 rows; 4 or 8 waves of 64 rows per slab
    pl.n_slab = (R + kSlabRowsMax - 1) / kSlabRowsMax;
    const int need = (R + 64 * pl.n_slab - 1) / (64 * pl.n_slab);
    pl.waves = need <= 4 ? 4 : 8;
    pl.rows_per_slab = 64 * pl.waves;
    pl.n_slab = (R + pl.rows_per_slab - 1) / pl.rows_per_slab;
    // one slot range per (instance, slab) when that alone gives >= 512 workgroups
    // and the range's column sums fit in LDS; otherwise split the slots so that
    // about 1024 workgroups run
    const long long base = (long long)n_inst * pl.n_slab;
    int n_split = (N + kMaxSplitKeys - 1) / kMaxSplitKeys;
    if (base < 512) {
      const long long want = (1024 + base - 1) / base;
      const int max_split = (N + kChunk - 1) / kChunk;
      const int more = (int)(want < max_split ? want : max_split);
      n_split = more > n_split ? more : n_split;
    }
    const int per = (N + n_split - 1) / n_split;
    pl.split_keys = (per + kChunk - 1) / kChunk * kChunk;
    pl.n_chunk1 = (N + pl.split_keys - 1) / pl.split_keys;
    pl.n_chunk2 = pl.n_chunk1;
  } else {
    pl.n_chunk1 = (N + kGenKeys - 1) / kGenKeys;
    pl.n_chunk2 = (K + kGenBlock - 1) / kGenBlock;
    pl.n_slab = 1;
    pl.rows_per_slab = R;
    pl.waves = 0;
    pl.split_keys = 0;
  }
  pl.off_part = 0;
  // the fused MFMA kernel needs no row partials, and pools by itself when one
  // workgroup holds the instance's every row
  const bool fused = pl.mfma && pl.n_chunk1 == 1;
  pl.pool_in_kernel = fused && pl.n_slab == 1;
  pl.off_lse = fused ? 0 : align256((size_t)n_inst * pl.n_chunk1 * R * sizeof(float2));
  const size_t lse_bytes = fused ? 0 : align256((size_t)n_inst * R * sizeof(float));
  pl.off_col = pl.off_lse + lse_bytes;
  pl.bytes = pl.pool_in_kernel ? 0 : pl.off_col + align256((size_t)n_inst * pl.n_slab * K * sizeof(float));
  (void)d;
  return pl;
}

hipError_t launch_value_rows(const void* v, int dtype, int n_inst, int N, int K, int d, int kind,
                             float* out, hipStream_t stream, uint32_t* status) {
  const int lpr = d * (dtype == VASE_BF16 ? 2 : 4) / 16;
  const int rpb = kSBlock / lpr;
  const dim3 rg((K + rpb - 1) / rpb, n_inst);
  if (dtype == VASE_BF16) {
    if (d == 128) hipLaunchKernelGGL((value_kernel<bf16_t, 128>), rg, dim3(kSBlock), 0, stream,
                                     static_cast<const bf16_t*>(v), N, K, kind, out, status);
    else hipLaunchKernelGGL((value_kernel<bf16_t, 64>), rg, dim3(kSBlock), 0, stream,
                            static_cast<const bf16_t*>(v), N, K, kind, out, status);
  } else {
    if (d == 128) hipLaunchKernelGGL((value_kernel<float, 128>), rg, dim3(kSBlock), 0, stream,
                                     static_cast<const float*>(v), N, K, kind, out, status);
    else hipLaunchKernelGGL((value_kernel<float, 64>), rg, dim3(kSBlock), 0, stream,
                            static_cast<const float*>(v), N, K, kind, out, status);
  }
  return hipGetLastError();
}

hipError_t launch_score(const void* k, const void* v, const void* q, int dtype, int n_inst, int K,
                        int B, int d, int G, int w, int pool, int value_kind, const float* lse_win,
                        float* attn, float* vrange, void* ws, const ScorePlan& pl,
                        hipStream_t stream, const int32_t* ord, const DecLogits& dec,
                        uint32_t* status) {
  const int N = K + B;
  const int R = G * w;
  const float c = 1.4426950408889634f / sqrtf((float)d);
  char* wsb = static_cast<char*>(ws);
  if (dtype == VASE_BF16) {
    if (d == 128)
      launch_mfma<128>(k, v, q, n_inst, N, K, R, c, pool, value_kind, lse_win, pl, wsb, vrange,
                       attn, ord, dec, stream, status);
    else
      launch_mfma<64>(k, v, q, n_inst, N, K, R, c, pool, value_kind, lse_win, pl, wsb, vrange,
                      attn, ord, dec, stream, status);
  } else {
    if (d == 128) launch_valu<float, 128>(k, q, n_inst, N, K, R, c, lse_win, pl, wsb, stream, status);
    else launch_valu<float, 64>(k, q, n_inst, N, K, R, c, lse_win, pl, wsb, stream, status);
  }
  const float* col = reinterpret_cast<const float*>(wsb + pl.off_col);
  if (!pl.pool_in_kernel) {
    hipLaunchKernelGGL(score_pool_kernel, dim3((K + kPoolTile - 1) / kPoolTile, n_inst),
                       dim3(kSBlock), 0, stream, col, K, pl.n_slab, R, pool, attn);
  }
  // value score of the K candidate rows (fused into pass 2 on the MFMA path;
  // random reservation scores are drawn by the caller of this function)
  if (dtype != VASE_BF16 && value_kind <= VASE_VALUE_VAR) {
    const int lpr = d * 4 / 16;
    const int rpb = kSBlock / lpr;
    const dim3 rg((K + rpb - 1) / rpb, n_inst);
    if (d == 128) hipLaunchKernelGGL((value_kernel<float, 128>), rg, dim3(kSBlock), 0, stream,
                                     static_cast<const float*>(v), N, K, value_kind, vrange, status);
    else hipLaunchKernelGGL((value_kernel<float, 64>), rg, dim3(kSBlock), 0, stream,
                            static_cast<const float*>(v), N, K, value_kind, vrange, status);
  }
  return hipGetLastError();
}

}  // namespace vase
