/*
 * vase.h -- C ABI of the VaSE-AttnV eviction round on AMD Instinct MI355X (gfx950).
 *
 * Method: "Value-Aware Stochastic KV Cache Eviction for Reasoning Models".
 * Under periodic eviction (Sec. 2) a head's static cache holds N = K + B slots:
 * K persistent slots [0, K) and a recency buffer [K, N) that fills one token per
 * decode step.  When the buffer is full, one eviction round runs for every
 * (layer, batch, KV head) instance independently:
 *
 *   vase_score        pooled window-mean attention score (Eq. 2 over Eq. 1 rows,
 *                     pooling per the Sec. 2 footnote) and the value score
 *                     Range(v) = max_j v_j - min_j v_j (Eq. 5)
 *   vase_select       VaSE-AttnV (Sec. 3.2): reserve the N_v largest-Range
 *                     candidates, keep the buffer, fill the remaining budget by
 *                     weighted sampling without replacement proportional to the
 *                     pooled score; emit the survivor map
 *   vase_compact      move the K survivors to slots [0, K) in slot order
 *   vase_decode_attn  decode attention over the compacted cache (Eq. 1)
 *   vase_quantize     Range-based per-token quantisation of a cache (Eq. 6)
 *                     with a full-precision reserve; vase_dequantize inverts it
 *   vase_decode_step  one decode step between rounds: append, window ring,
 *                     decode attention and the persistent normaliser part
 *                     that vase_score_lse turns into a one-pass score
 *   vase_score_map, vase_compact_decode_map
 *                     the round on a cache whose temporal order is kept in an
 *                     order map: compaction moves only the B buffer rows
 *
 * Conventions for every entry point
 * ---------------------------------
 *  - A head instance ("inst") is one (layer, batch, KV head).  n_inst instances
 *    are processed per call; they are independent.
 *  - Cache tensors k_cache, v_cache: device pointers to [n_inst][N][d] elements of
 *    the given dtype, contiguous (instance stride N*d elements), N = K + B.
 *  - Window queries q_win: device pointer, [n_inst][G][w][d] (the G query heads of
 *    the instance's GQA group, each with its w most recent queries), same dtype.
 *  - dtype: VASE_BF16 (bf16 storage, fp32 arithmetic; MFMA path) or VASE_F32.
 *  - d must be 64 or 128.
 *  - All device pointers must be 16-byte aligned.  The caller allocates and owns
 *    every buffer (caches, queries, outputs, workspace); the library allocates
 *    nothing, frees nothing and keeps no pointer after a call returns.
 *  - stream: a hipStream_t (NULL = default stream).  Every call only enqueues work
 *    and returns; outputs are valid in stream order.  No call synchronizes.
 *  - Return value: VASE_OK, or a negative status.  Arguments are validated on the
 *    host before any HIP call, so an invalid call has no effect on the device.
 *    VASE_ERR_HIP reports a launch failure (hipGetLastError after the launch).
 *  - Determinism: every output is a pure function of the inputs and of
 *    (seed, round, inst_base); repeated calls produce bitwise identical results
 *    (fixed reduction orders, no floating-point atomics).
 *  - The library holds no mutable global state; calls on different streams or
 *    threads do not interact, except through buffers the caller shares.  The
 *    one exception is vase_decode_step_noalloc, which uses a scratch array the
 *    library keeps on each GPU (see there).
 *  - Data faults: what the method is not defined on (a NaN or infinite input, a
 *    softmax normaliser that is not a positive finite number) cannot be known on
 *    the host without a synchronisation.  The score and select entry points take
 *    a nullable device word dev_status (int32_t, 4-byte aligned) and OR the
 *    VASE_STATUS_* bits below into it when they meet such data; outputs are then
 *    unspecified, but every access stays inside the caller's buffers and every
 *    kernel completes.  The library never clears the word: the caller zeroes it
 *    and reads it in stream order.  Calls that share a word only OR into it.
 */
#ifndef VASE_H_
#define VASE_H_

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define VASE_OK 0
#define VASE_ERR_INVALID_ARG (-1)
#define VASE_ERR_DTYPE (-2)
#define VASE_ERR_WORKSPACE (-3)
#define VASE_ERR_HIP (-4)
#define VASE_ERR_UNSUPPORTED (-5)

#define VASE_BF16 0
#define VASE_F32 1

/* Bits of the device status word (dev_status).  Each names the first entry
 * point that can see the fault; later steps of a round are then unspecified. */
#define VASE_STATUS_ROW_NORM 1     /* vase_score*: the softmax normaliser of a window row
                                      over the N slots (Eq. 1) is not a positive finite
                                      number, i.e. a key or query element is NaN or
                                      infinite (with lse_win: or the supplied part is) */
#define VASE_STATUS_VALUE_ROW 2    /* vase_score*: a value row that the call reads (its
                                      Range, L2 or Var) has a NaN or infinite element */
#define VASE_STATUS_SELECT_ATTN 4  /* vase_select: a candidate's attn is NaN, infinite or
                                      negative (including -0) */
#define VASE_STATUS_SELECT_VALUE 8 /* vase_select: a value score is NaN, infinite or
                                      negative (a Range that overflows fp32 is infinite) */

/* vase_select flags */
#define VASE_DETERMINISTIC 1u /* fill by the pooled score's top-k (the ablation of
                                 Sec. 4.1 that drops the sampling) instead of sampling */

/* operation ids for vase_workspace_bytes */
#define VASE_OP_SCORE 0
#define VASE_OP_SELECT 1
#define VASE_OP_COMPACT 2
#define VASE_OP_DECODE 3
#define VASE_OP_COMPACT_DECODE 4
#define VASE_OP_SCORE_MAP 5

/* value scores for vase_score_ex: the quantity whose N_v largest slots fill R_V.
 * Range is the method (Eq. 5); L2, Var and random reservation are the variants
 * of Appendix A and the random-reservation ablation of Appendix D. */
#define VASE_VALUE_RANGE 0  /* max_c v[c] - min_c v[c] */
#define VASE_VALUE_L2 1     /* sqrt(sum_c v[c]^2) */
#define VASE_VALUE_VAR 2    /* (1/d) sum_c (v[c] - mu)^2, mu = (1/d) sum_c v[c] */
#define VASE_VALUE_RANDOM 3 /* uniform in (0,1) from Philox4x32-10, counter
                               (i >> 2, inst_base + inst, round, 2), word i & 3,
                               key (seed_lo, seed_hi), mapped as in vase_select */
#define VASE_VALUE_SKIP 4   /* vase_score_ex only: vrange_out is left untouched
                               (nullable); the caller already holds the value
                               scores, e.g. from vase_compact_decode_ex */

/* Largest persistent budget K the selection kernel accepts (its per-instance
 * working set lives in LDS). */
#define VASE_MAX_K 8192

/* vase_score_map with q_dec (bf16 MFMA path) keeps a range's decode logits in
 * LDS and writes them after its pass over the keys when
 *     G * (range slots rounded up to 4) * 4 + G * d * 2 <= VASE_DEC_LOGITS_LDS
 * (a range is all N slots when one workgroup scores an instance); otherwise it
 * stores them from inside its key loop, which is correct but slows the score
 * by more than the decode saves.  Callers can use the bound with N in place of
 * the range to decide whether to ask for the logits. */
#define VASE_DEC_LOGITS_LDS 92160

/*
 * Device workspace, in bytes, that one call of operation `op` needs for this
 * shape (0 if none).  Pass a buffer at least this large as `ws` / `ws_bytes`.
 * Arguments not used by `op` are ignored.  Returns 0 for invalid shapes.
 */
size_t vase_workspace_bytes(int op, int dtype, int n_inst, int K, int B, int d, int G, int w);

/*
 * Step 1 + 2: scores of the K persistent slots of every instance.
 *
 *   attn_out[inst][i]   = (1/P) * sum_{j=i-P/2}^{i+P/2} abar_j     (zero padded)
 *   abar_j              = (1/(G*w)) * sum_r softmax_{0<=t<N}(q_r.k_t / sqrt(d))_j
 *   vrange_out[inst][i] = max_c v_i[c] - min_c v_i[c]               (exact in fp32)
 *
 * Each of the G*w window rows r is a softmax over all N slots (buffer included,
 * no causal mask), as in Eq. (1); the mean over the rows is Eq. (2) over the GQA
 * group; P = pool is the smoothing kernel (odd, >= 1; P = 1 disables pooling).
 *
 *  k_cache, v_cache  in   [n_inst][N][d] device, dtype
 *  q_win             in   [n_inst][G][w][d] device, dtype
 *  attn_out          out  [n_inst][K] device fp32
 *  vrange_out        out  [n_inst][K] device fp32
 *  ws, ws_bytes      scratch, >= vase_workspace_bytes(VASE_OP_SCORE, ...) bytes
 *  dev_status        nullable device int32: VASE_STATUS_ROW_NORM, VASE_STATUS_VALUE_ROW
 * Errors: VASE_ERR_INVALID_ARG (null pointer, n_inst < 1, K < 1, B < 1, G < 1,
 *         w < 1, G*w > 65536, d not 64/128, pool even, < 1 or > 255, unaligned
 *         pointer),
 *         VASE_ERR_DTYPE, VASE_ERR_WORKSPACE, VASE_ERR_HIP.
 */
int vase_score(const void* k_cache, const void* v_cache, const void* q_win, int dtype,
               int n_inst, int K, int B, int d, int G, int w, int pool, float* attn_out,
               float* vrange_out, void* ws, size_t ws_bytes, int32_t* dev_status, void* stream);

/*
 * vase_score with a choice of value score (the variants of Appendix A, and
 * the ablation of Appendix D that reserves random pairs instead):
 *
 *   value_kind = VASE_VALUE_RANGE   vrange_out as in vase_score (same call)
 *                VASE_VALUE_L2      sqrt(sum_c v_i[c]^2), fp32 accumulation
 *                VASE_VALUE_VAR     two-pass (1/d) sum_c (v_i[c] - mu)^2, fp32
 *                VASE_VALUE_RANDOM  Philox uniforms (see VASE_VALUE_RANDOM);
 *                                   v_cache is not read
 *                VASE_VALUE_SKIP    no value scores (vrange_out may be NULL and
 *                                   is not written); v_cache is not read
 *
 * seed, round and inst_base are used by VASE_VALUE_RANDOM only (pass the values
 * given to vase_select for the same round).  attn_out and dev_status are as in
 * vase_score (no value row is read, so none is checked, for RANDOM and SKIP).
 * Errors: as vase_score, plus VASE_ERR_INVALID_ARG for an unknown value_kind.
 */
int vase_score_ex(const void* k_cache, const void* v_cache, const void* q_win, int dtype,
                  int n_inst, int K, int B, int d, int G, int w, int pool, int value_kind,
                  uint64_t seed, uint32_t round, uint32_t inst_base, float* attn_out,
                  float* vrange_out, void* ws, size_t ws_bytes, int32_t* dev_status,
                  void* stream);

/*
 * vase_score_ex in one pass over the candidates: each window row's softmax
 * normaliser over all N slots (Eq. 1) is the supplied persistent part plus the
 * buffer slots, so only the w x B buffer block is scored twice.
 *
 *   lse_win[inst][g][t] = ln sum_{i < K} exp(q_win[g][t] . k_i / sqrt(d))
 *
 * as vase_decode_step leaves it.  With the exact lse_win the outputs equal
 * vase_score_ex's up to fp32 rounding; the call cannot check that lse_win
 * belongs to this cache and window.
 *
 *  lse_win           in   [n_inst][G][w] device fp32, 16-byte aligned
 * Other arguments (dev_status included), workspace and errors as vase_score_ex.
 */
int vase_score_lse(const void* k_cache, const void* v_cache, const void* q_win,
                   const float* lse_win, int dtype, int n_inst, int K, int B, int d, int G, int w,
                   int pool, int value_kind, uint64_t seed, uint32_t round, uint32_t inst_base,
                   float* attn_out, float* vrange_out, void* ws, size_t ws_bytes,
                   int32_t* dev_status, void* stream);

/*
 * Steps 3-6: VaSE-AttnV selection and the survivor map (Sec. 3.2).
 *
 *  R_V  = the N_v slots of [0, K) with the largest vrange (ties: lower slot first)
 *  C    = [0, K) \ R_V
 *  key_i = attn_i / E_i for i in C, with E_i = -ln(u_i), u_i from Philox4x32-10
 *         (counter = (i >> 2, inst_base + inst, round, 0), key = (seed_lo, seed_hi),
 *          output word i & 3, u = (2 * (x >> 9) + 1) * 2^-24); with
 *         VASE_DETERMINISTIC, key_i = attn_i.
 *  T    = the K - N_v - B candidates with the largest key (ties: lower slot first),
 *         i.e. weighted sampling without replacement proportional to attn
 *         (exponential keys; the B candidates not in T are evicted)
 *  S    = R_V + T + [K, N)              (|S| = K)
 *  src_out[inst][j] = the j-th smallest slot of S, j < K  (strictly increasing,
 *                     src[j] >= j; the buffer lands in [K - B, K))
 *
 *  attn, vrange  in   [n_inst][K] device fp32, finite and >= 0
 *  src_out       out  [n_inst][K] device int32
 *  keys_out      out  nullable; [n_inst][K] device fp32: key_i for i in C, NaN for R_V
 *  dev_status    nullable device int32: VASE_STATUS_SELECT_ATTN, VASE_STATUS_SELECT_VALUE
 *                (the survivor map is then unspecified but still a valid map)
 * Errors: VASE_ERR_INVALID_ARG (null pointer, n_inst < 1, B < 1, N_v < 0,
 *         N_v + B > K, K > VASE_MAX_K, unaligned pointer), VASE_ERR_HIP.
 */
int vase_select(const float* attn, const float* vrange, int n_inst, uint32_t inst_base, int K,
                int B, int Nv, uint64_t seed, uint32_t round, uint32_t flags, int32_t* src_out,
                float* keys_out, int32_t* dev_status, void* stream);

/*
 * Step 7: in-place stable compaction (the cache returns to K slots, Sec. 2).
 *   for j < K:  k[j] <- k[src[j]],  v[j] <- v[src[j]]   (raw row copies)
 * src must be a survivor map as produced by vase_select (strictly increasing,
 * src[j] >= j, src[K-1] < N); rows [K, N) are left unspecified afterwards.
 *
 *  k_cache, v_cache  in/out [n_inst][N][d] device, dtype
 *  src               in     [n_inst][K] device int32
 *  ws, ws_bytes      scratch, >= vase_workspace_bytes(VASE_OP_COMPACT, ...) bytes
 * Errors: VASE_ERR_INVALID_ARG, VASE_ERR_DTYPE, VASE_ERR_WORKSPACE, VASE_ERR_HIP.
 * A map that violates the contract gives unspecified cache contents but never
 * accesses memory outside the instance's N rows (source slots are clamped).
 */
int vase_compact(void* k_cache, void* v_cache, int dtype, int n_inst, int K, int B, int d,
                 const int32_t* src, void* ws, size_t ws_bytes, void* stream);

/*
 * Step 8: decode attention over the first n_valid slots (Eq. 1):
 *   out[inst][g] = sum_{i < n_valid} softmax_i(q_g . k_i / sqrt(d)) * v_i
 * for the G query heads g of the instance's GQA group.
 *
 *  k_cache, v_cache  in   [n_inst][N][d] device, dtype (N = K + B is the stride)
 *  q                 in   [n_inst][G][d] device, dtype
 *  out               out  [n_inst][G][d] device, dtype (fp32 accumulation)
 *  ws, ws_bytes      scratch, >= vase_workspace_bytes(VASE_OP_DECODE, ...) bytes
 * Errors: VASE_ERR_INVALID_ARG (n_valid < 1 or > N, G < 1 or > 8, ...),
 *         VASE_ERR_DTYPE, VASE_ERR_WORKSPACE, VASE_ERR_HIP.
 */
int vase_decode_attn(const void* k_cache, const void* v_cache, const void* q, int dtype,
                     int n_inst, int K, int B, int d, int G, int n_valid, void* out, void* ws,
                     size_t ws_bytes, void* stream);

/*
 * vase_decode_attn that also returns, for each query head, the log-sum-exp of
 * its scores over the first n_persist slots: the persistent part of Eq. (1)'s
 * softmax normaliser, which vase_score_lse reuses at the next round.
 *
 *   lse_out[inst][g] = ln sum_{i < n_persist} exp(q_g . k_i / sqrt(d))   (fp32)
 *
 *  n_persist         1 <= n_persist <= n_valid (normally K)
 *  lse_out           out  nullable; [n_inst][G] device fp32
 * Other arguments and errors as vase_decode_attn; the workspace is the same.
 */
int vase_decode_attn_lse(const void* k_cache, const void* v_cache, const void* q, int dtype,
                         int n_inst, int K, int B, int d, int G, int n_valid, int n_persist,
                         void* out, float* lse_out, void* ws, size_t ws_bytes, void* stream);

/*
 * One decode step between two rounds (Sec. 2, periodic eviction): the new
 * token's (k, v) goes into buffer slot K + pos, its G queries into the window
 * ring, and the step attends over the K + pos + 1 valid slots:
 *
 *   k[K + pos] <- k_new,  v[K + pos] <- v_new,  q_win[g][pos % w] <- q[g]
 *   out[g]                = vase_decode_attn over n_valid = K + pos + 1
 *   lse_win[g][pos % w]   = ln sum_{i < K} exp(q_g . k_i / sqrt(d))
 *
 * After the B steps of a period (pos = 0 .. B-1) q_win holds the last w
 * queries and lse_win the persistent part of each one's normaliser, as
 * vase_score_lse expects: the persistent slots do not change between rounds,
 * which is why w <= B is required.
 *
 *  k_cache, v_cache  in/out [n_inst][N][d] device, dtype
 *  k_new, v_new      in     [n_inst][d] device, dtype
 *  q                 in     [n_inst][G][d] device, dtype
 *  q_win             in/out [n_inst][G][w][d] device, dtype (ring, slot pos % w written)
 *  lse_win           in/out [n_inst][G][w] device fp32 (ring, slot pos % w written)
 *  out               out    [n_inst][G][d] device, dtype
 *  ws, ws_bytes      scratch, >= vase_workspace_bytes(VASE_OP_DECODE, ...) bytes
 * Errors: VASE_ERR_INVALID_ARG (pos < 0 or >= B, w < 1 or > B, G < 1 or > 8,
 *         null or unaligned pointer, ...), VASE_ERR_DTYPE, VASE_ERR_WORKSPACE,
 *         VASE_ERR_HIP.
 */
int vase_decode_step(void* k_cache, void* v_cache, const void* k_new, const void* v_new,
                     const void* q, int dtype, int n_inst, int K, int B, int d, int G, int w,
                     int pos, void* q_win, float* lse_win, void* out, void* ws, size_t ws_bytes,
                     void* stream);

/*
 * vase_decode_step for callers that cannot allocate device memory (code under
 * HIP graph capture, tight serving loops, harnesses that forbid allocation):
 * the same step, with the same results bit for bit, but its decode split
 * partials go to a scratch array that the library itself holds on each GPU
 * (VASE_DECODE_SCRATCH_BYTES, set up on the first call on a device and kept
 * until the process ends) instead of a caller workspace.  The call allocates
 * nothing.  It uses the device current on the calling thread (the stream must
 * belong to it).  All calls on one GPU share that GPU's scratch: calls whose
 * work overlaps on one GPU (on different streams, or from different threads
 * without ordering) race on it and must not be issued.  Nothing in the scratch
 * needs clearing: every call overwrites the part it reads.
 *
 * Arguments as vase_decode_step, without ws and ws_bytes.
 * Errors: as vase_decode_step; VASE_ERR_WORKSPACE when the step's partials
 *         (n_inst * splits * G * (d + 4) * 4 bytes, as vase_workspace_bytes
 *         reports for VASE_OP_DECODE at most) exceed VASE_DECODE_SCRATCH_BYTES;
 *         VASE_ERR_HIP when the scratch cannot be set up on the device.
 */
#define VASE_DECODE_SCRATCH_BYTES (64u << 20)
int vase_decode_step_noalloc(void* k_cache, void* v_cache, const void* k_new, const void* v_new,
                             const void* q, int dtype, int n_inst, int K, int B, int d, int G,
                             int w, int pos, void* q_win, float* lse_win, void* out, void* stream);

/*
 * Steps 7 + 8 fused: the in-place stable compaction of vase_compact followed by
 * one decode-attention step over the K compacted slots, as vase_decode_attn with
 * n_valid = K (Sec. 2: after an eviction round the decoder continues over the
 * restored K-slot cache; Eq. 1).  The results are those of the two calls in
 * sequence (the same cache bytes; the same attention output up to fp32
 * summation order).  When each instance fits one workgroup, the cache is read
 * once for both steps; otherwise the two steps run one after the other.
 *
 *  k_cache, v_cache  in/out [n_inst][N][d] device, dtype
 *  src               in     [n_inst][K] device int32 survivor map (vase_select)
 *  q                 in     [n_inst][G][d] device, dtype
 *  out               out    [n_inst][G][d] device, dtype
 *  ws, ws_bytes      scratch, >= vase_workspace_bytes(VASE_OP_COMPACT_DECODE, ...)
 * Errors: VASE_ERR_INVALID_ARG (G < 1 or > 8, null or unaligned pointer, ...),
 *         VASE_ERR_DTYPE, VASE_ERR_WORKSPACE, VASE_ERR_HIP.
 */
int vase_compact_decode(void* k_cache, void* v_cache, int dtype, int n_inst, int K, int B, int d,
                        const int32_t* src, const void* q, int G, void* out, void* ws,
                        size_t ws_bytes, void* stream);

/*
 * vase_compact_decode that also returns the value score of every compacted row:
 *
 *   vrange_out[inst][j] = Range, L2 or Var (value_kind) of v[j] after compaction
 *
 * computed from the rows the compaction reads anyway.  Until the next round only
 * the buffer slots change, so these are the next round's candidate value scores:
 * pass them to vase_select after vase_score_ex with VASE_VALUE_SKIP, and the
 * score does not read V.  The scores equal what vase_score_ex computes for the
 * same rows, bit for bit.
 *
 *  value_kind   VASE_VALUE_RANGE, VASE_VALUE_L2 or VASE_VALUE_VAR
 *  vrange_out   out  nullable (then as vase_compact_decode); [n_inst][K] device fp32
 * Other arguments, workspace and errors as vase_compact_decode.
 */
int vase_compact_decode_ex(void* k_cache, void* v_cache, int dtype, int n_inst, int K, int B,
                           int d, const int32_t* src, const void* q, int G, void* out,
                           int value_kind, float* vrange_out, void* ws, size_t ws_bytes,
                           void* stream);

/*
 * The cache under an order map.  Sec. 2 restores the cache to K persistent slots
 * after every round; a stable compaction (vase_compact) keeps them in temporal
 * order and so moves every survivor behind the first evicted slot.  Under an
 * order map the survivors stay where they are:
 *
 *   ord[inst][t]  the slot that holds the persistent token of temporal rank t
 *                 (t < K, oldest first); buffer token K + b is in slot K + b
 *
 * Read through the map, the cache is the temporal cache T[t] = X[ord[t]]
 * (t < K), T[t] = X[t] (K <= t < N).  A cache with an order map goes through a
 * round as vase_score_map -> vase_select (unchanged: it works on temporal
 * ranks) -> vase_compact_decode_map, and every output equals what the
 * stable-layout calls produce on T (up to fp32 summation order in the score's
 * row normalisers and in the decode).  After a prefill ord is the identity.
 */

/*
 * vase_score_ex / vase_score_lse on T: the window scores of every slot, then
 * the average pooling (Sec. 2 footnote) over temporal neighbours:
 *
 *   attn_out[inst][t]   = (1/P) sum_{u=t-P/2}^{t+P/2} abar(ord[u])   (0 <= u < K)
 *   vrange_out[inst][t] = value score of the row in slot ord[t]
 *
 * with abar(s) the window mean of slot s (vase_score_ex with P = 1).
 * VASE_VALUE_RANDOM draws its uniforms per temporal rank, VASE_VALUE_SKIP
 * leaves vrange_out untouched (vase_compact_decode_map writes it by rank).
 *
 * With q_dec given, the pass that reads every key row for the row normalisers
 * also writes the decode queries' logits (the q.k products of Eq. 1, before the
 * 1/sqrt(d) scale) for every physical slot:
 *
 *   dec_logits_out[inst][g][t] = q_dec[inst][g] . k_t      (t < N, g < G)
 *
 * so that vase_compact_decode_map can run the decode step of this round
 * without reading K again.  The slots it decodes over after compaction are the
 * survivors, which stay in their slots, and the buffer rows, whose logits are
 * at t = K + b; each logit is bit for bit the one the decode kernel computes.
 *
 *  lse_win         in   nullable: as vase_score_lse (one pass over the candidates)
 *  ord             in   [n_inst][K] device int32, a permutation of [0, K) per instance
 *  q_dec           in   nullable, with dec_logits_out: [n_inst][G][d] device, bf16
 *                       (the G heads' queries of the decode step that follows)
 *  dec_logits_out  out  nullable, with q_dec: [n_inst][G][N] device fp32
 *  ws              >= vase_workspace_bytes(VASE_OP_SCORE_MAP, ...) bytes
 * Other arguments (dev_status included) as vase_score_ex.  Errors: as vase_score_ex, plus
 * VASE_ERR_INVALID_ARG for a null or unaligned ord, K > VASE_MAX_K, only one of
 * q_dec and dec_logits_out, or q_dec with lse_win or G > 16, and VASE_ERR_DTYPE
 * for q_dec with an fp32 cache.
 */
int vase_score_map(const void* k_cache, const void* v_cache, const void* q_win,
                   const float* lse_win, const int32_t* ord, int dtype, int n_inst, int K, int B,
                   int d, int G, int w, int pool, int value_kind, uint64_t seed, uint32_t round,
                   uint32_t inst_base, float* attn_out, float* vrange_out, const void* q_dec,
                   float* dec_logits_out, void* ws, size_t ws_bytes, int32_t* dev_status,
                   void* stream);

/*
 * The reordering step of vase_score_map on its own, for scores computed per
 * slot elsewhere (e.g. vase_dkv_score, with pool = 1):
 *
 *   attn_out[inst][t]   = (1/P) sum_{u=t-P/2}^{t+P/2} attn_phys[inst][ord[u]]  (0 <= u < K)
 *   vrange_out[inst][t] = vrange_phys[inst][ord[t]]        (if vrange_phys != NULL)
 *
 *  attn_phys, vrange_phys  in   [n_inst][K] device fp32 (vrange_phys nullable)
 *  ord                     in   [n_inst][K] device int32
 *  attn_out, vrange_out    out  [n_inst][K] device fp32 (vrange_out used with vrange_phys)
 * Errors: VASE_ERR_INVALID_ARG (null or unaligned pointer, K < 1 or
 *         > VASE_MAX_K, pool even, < 1 or > 255), VASE_ERR_HIP.
 */
int vase_order_scores(const float* attn_phys, const float* vrange_phys, const int32_t* ord,
                      int n_inst, int K, int pool, float* attn_out, float* vrange_out,
                      void* stream);

/*
 * Compaction under the order map, optionally fused with one decode step over
 * the K compacted slots.  With e_0 < ... < e_{B-1} the evicted ranks ([0, K)
 * minus src[0 .. K-B)), buffer row K + b is copied to slot ord[e_b] and
 *
 *   ord'[j] = ord[src[j]]  (j < K - B),    ord'[K - B + b] = ord[e_b]
 *
 * so that X'[ord'[j]] = T[src[j]] for every j < K: the stable compaction of T,
 * reached with B row copies (survivors do not move).  ord is updated in place.
 * With q given, the call also runs decode attention over the K slots (Eq. 1),
 * as vase_decode_attn with n_valid = K, reading each row once.  With
 * vrange_out (with or without q), it writes the value score of the row of rank
 * j at vrange_out[inst][j] for every j < K (the next round's candidates, as
 * vase_compact_decode_ex).  With vrange_in as well (the value scores of kind
 * value_kind that vase_select used for this round's candidates), a survivor
 * takes its score from vrange_in, as its row has not changed, and only the B
 * buffer rows are scored from V; the result is the same, bit for bit, when
 * vrange_in holds those scores.  Without q and vrange_in the survivors' V rows
 * are read for their scores.
 * vrange_in may be vrange_out.  With dec_logits (what vase_score_map or
 * vase_dkv_score wrote for this cache and q this round, indexed by physical
 * slot, before any copy) the decode takes the q.k products from it and reads no
 * K row, only V, the logits and the B buffer rows; with vase_score_map's logits
 * the output is the same, bit for bit.
 *
 *  k_cache, v_cache  in/out [n_inst][N][d] device, dtype; rows [K, N) unchanged
 *  src               in     [n_inst][K] device int32 survivor map (vase_select
 *                           on the temporal ranks)
 *  ord               in/out [n_inst][K] device int32
 *  q, out            nullable together: [n_inst][G][d] device, dtype
 *  value_kind        VASE_VALUE_RANGE, L2 or VAR (with vrange_out)
 *  vrange_in         in   nullable; needs vrange_out; [n_inst][K] device fp32
 *  vrange_out        out  nullable; [n_inst][K] device fp32
 *  dec_logits        in   nullable; needs q and bf16; [n_inst][G][N] device fp32
 * No workspace.  Errors: VASE_ERR_INVALID_ARG (null or unaligned pointer, q and
 * out not both given or both NULL, vrange_in without vrange_out, dec_logits
 * without q, K > VASE_MAX_K, B > K, G < 1
 * or > 8), VASE_ERR_DTYPE (also dec_logits with an fp32 cache), VASE_ERR_HIP.
 * A src or ord that breaks its contract gives unspecified contents but no
 * access outside the instance.
 */
int vase_compact_decode_map(void* k_cache, void* v_cache, int dtype, int n_inst, int K, int B,
                            int d, const int32_t* src, int32_t* ord, const void* q, int G,
                            void* out, int value_kind, const float* vrange_in, float* vrange_out,
                            const float* dec_logits, void* stream);

/*
 * VaSE-DKV (Sec. 3.2; the product score is CurDKV's, Eq. 4).  At every eviction
 * step each head instance draws a Gaussian projection G_t in R^{d x r}, entries
 * N(0, 1/r), independent of all earlier steps (the paper uses r = 20), and
 * scores each candidate slot i < K by
 *     s_i = ||G_t^T k_i||^2 * ||G_t^T v_i||^2.
 * The round keeps the K - B highest scores and the buffer: vase_select with
 * VASE_DETERMINISTIC, N_v = 0 and attn = the scores (vrange is then unused and
 * may be any array of K floats per instance); compaction and decode follow as
 * for VaSE-AttnV.
 *
 * vase_dkv_projection draws G_t for n_inst instances.  Instance n (global id
 * inst_base + n) and entry e = a*r + b of its [d][r] matrix take Philox4x32-10
 * words 2(e&1), 2(e&1)+1 of counter (e>>1, inst_id, round, 1) and key seed
 * (low word first) through Box-Muller, z = sqrt(2 E(u1)) cos(2 pi u2) with
 * E(u) = -ln u as in vase_select and the uniform map as there, and
 * G = z / sqrt(r); every step is a fixed binary32 operation sequence.
 *
 *  g_out  out [n_inst][d][r] fp32, device, 16-byte aligned
 *  r      1 .. 32
 * Errors: VASE_ERR_INVALID_ARG (n_inst < 1, d not 64 or 128, r out of range,
 *         null or unaligned pointer), VASE_ERR_HIP.
 */
int vase_dkv_projection(int n_inst, uint32_t inst_base, int d, int r, uint64_t seed,
                        uint32_t round, float* g_out, void* stream);

/*
 * The DKV score of the K candidate slots of every instance.
 *
 *  k_cache, v_cache  in  [n_inst][N][d] device, dtype (N = K + B)
 *  g                 in  [n_inst][d][r] fp32 device (vase_dkv_projection)
 *  score_out         out [n_inst][K] fp32 device
 *  q_dec             in  nullable, with dec_logits_out: [n_inst][G][d] device, bf16
 *                        (the queries of the decode step that follows the round)
 *  dec_logits_out    out nullable, with q_dec: [n_inst][G][N] fp32 device,
 *                        dec_logits_out[inst][h][t] = q_dec[inst][h] . k_t for every
 *                        slot t < N, for vase_compact_decode_map (the pass then
 *                        also reads the B buffer rows); 1 <= G <= 16
 * bf16 caches project with MFMA against a two-term bf16 split of G (relative
 * error of G about 2^-16, fp32 accumulation); fp32 caches use fp32 FMA.  The
 * logits are fp32 MFMA sums of the bf16 products (32x32x16 steps, so they may
 * differ in the last bits from the ones vase_compact_decode_map computes from K).
 * Errors: VASE_ERR_INVALID_ARG (also only one of q_dec and dec_logits_out, G out
 * of range), VASE_ERR_DTYPE (also dec_logits_out with an fp32 cache), VASE_ERR_HIP.
 */
int vase_dkv_score(const void* k_cache, const void* v_cache, const float* g, int dtype, int n_inst,
                   int K, int B, int d, int r, float* score_out, const void* q_dec, int G,
                   float* dec_logits_out, void* stream);

/*
 * Range-based per-token asymmetric quantisation (Eq. 6, Sec. 4.3) of rows
 * [0, K) of a cache, with an optional full-precision reserve for the N_v rows of
 * largest Range (the mixed-precision direction of Sec. 7).  Per row and per
 * group of `group` consecutive elements:
 *
 *   z = min x,  Delta = (max x - min x) / (2^bits - 1)          (fp32)
 *   q_e = rint((x_e - z) / Delta), ties to even, clamped to [0, 2^bits - 1]
 *         (q_e = 0 when Delta = 0); the quotient is decided as an IEEE fp32
 *         divide of the fp32 difference, so codes are reproducible
 *   x'_e = fma(q_e, Delta, z)                                   (fp32)
 *
 *  x_cache      in   [n_inst][N][d] device, dtype (N = K + B; rows [0, K) used)
 *  bits, group  bits in {2, 4, 8}; group in {32, 64, 128}, group <= d
 *  Nv           0 <= Nv <= K; Nv > 0 needs K <= VASE_MAX_K
 *  codes_out    out  [n_inst][K][d*bits/8] device uint8: code e of a row at bits
 *                    [e*bits, e*bits + bits) of the row's bytes, little-endian
 *  params_out   out  [n_inst][K][d/group][2] device fp32: (Delta, z) per group
 *  range_out    out  nullable ([n_inst][K] fp32, Range of each row, Eq. 5);
 *                    required when Nv > 0
 *  mse_out      out  nullable; [n_inst][K] fp32: (1/d) sum_e (x_e - x'_e)^2,
 *                    fp32 accumulation
 *  hp_rows_out  out  [n_inst][Nv][d] device, dtype: copies of the reserved rows
 *  hp_idx_out   out  [n_inst][Nv] device int32: their slots, ascending; the
 *                    reserved rows are the first N_v under (Range desc, slot asc)
 * Errors: VASE_ERR_INVALID_ARG (null or unaligned pointer, bad bits/group,
 *         Nv out of range, ...), VASE_ERR_DTYPE, VASE_ERR_HIP.
 */
int vase_quantize(const void* x_cache, int dtype, int n_inst, int K, int B, int d, int bits,
                  int group, int Nv, uint8_t* codes_out, float* params_out, float* range_out,
                  float* mse_out, void* hp_rows_out, int32_t* hp_idx_out, void* stream);

/*
 * Inverse of vase_quantize: rows [0, K) of out_cache get x' (stored in dtype,
 * bf16 rounded to nearest even), then the N_v reserved rows get their
 * full-precision copies hp_rows at slots hp_idx (entries outside [0, K) are
 * skipped).  Rows [K, N) of out_cache are not written.
 *
 *  codes, params     in   as written by vase_quantize
 *  hp_rows, hp_idx   in   as written by vase_quantize (needed when Nv > 0)
 *  out_cache         out  [n_inst][N][d] device, dtype
 * Errors: as vase_quantize.
 */
int vase_dequantize(const uint8_t* codes, const float* params, const void* hp_rows,
                    const int32_t* hp_idx, int dtype, int n_inst, int K, int B, int d, int bits,
                    int group, int Nv, void* out_cache, void* stream);

/* Human-readable name of a status code (static string). */
const char* vase_status_str(int status);

/* Library ABI version: (major << 16) | minor.  2.0 added dev_status to the score
 * and select entry points. */
int vase_version(void);

#ifdef __cplusplus
}
#endif

#endif /* VASE_H_ */
