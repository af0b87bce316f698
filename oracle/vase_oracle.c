/*
 * vase_oracle.c -- plain, slow CPU oracle for one VaSE-AttnV eviction round.
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing in the product path may link, load or
 * call this file: only the tests, the smoke check and the CPU-baseline leg of
 * the benchmark do.  It shares no source with the HIP library.
 *
 * Every real-valued quantity is computed in double from inputs that were
 * upcast exactly from their storage type (bf16 or fp32).  Results are rounded
 * to fp32 only where the round hands a value to the next step (the pooled
 * attention score, the Range score, the selection key).  Loops follow the
 * order in which the paper states the definitions; there is no blocking, no
 * fusion and no reordering beyond what a definition itself allows.
 *
 * Paper: "Value-Aware Stochastic KV Cache Eviction for Reasoning Models".
 *   Eq. (1)   decode attention over the N cached pairs          (Sec. 2)
 *   periodic eviction with budget K and buffer B                (Sec. 2)
 *   Eq. (2)   SnapKV window-mean attention score + pooling      (Sec. 2, footnote)
 *   Eq. (5)   Range(v) = max_j v_j - min_j v_j                  (Sec. 3.1)
 *   VaSE-AttnV: reserve the N_v largest-Range slots, fill the rest of the
 *   budget by sampling proportional to the pooled score         (Sec. 3.2)
 *   VaSE-DKV: CurDKV's product of key and value projection norms (Eq. 4)
 *   under a Gaussian projection drawn afresh at every eviction step, then a
 *   deterministic top-(K-B)                                     (Sec. 3.2)
 *
 * Readings of points the paper leaves open (all listed in the design notes):
 *   - each window row is a softmax over all N = K + B slots (non-causal);
 *   - the score is the mean over all G*w rows of the GQA group's window;
 *   - pooling: odd kernel P, stride 1, zero padded, always divided by P,
 *     over the K candidate slots in slot order;
 *   - sampling is successive weighted sampling without replacement, realised
 *     with exponential keys  key_i = w_i / E_i,  E_i ~ Exp(1)
 *     (Efraimidis & Spirakis, Inf. Proc. Lett. 97(5), 2006);
 *   - E_i = -ln(u_i) with u_i from Philox4x32-10 (Salmon et al., SC'11),
 *     counter (i>>2, inst, round, purpose), key (seed_lo, seed_hi), word i&3;
 *   - ties: Range descending then slot ascending; key descending then slot
 *     ascending;
 *   - compaction keeps the temporal (slot) order of the survivors; under an
 *     order map (vo_order_compact) the same temporal cache is reached by
 *     leaving survivors in place and filling the evicted slots with the buffer.
 *
 * Build: gcc -O2 -fopenmp -ffp-contract=off -fPIC -shared (no -ffast-math:
 * the fp32 selection arithmetic must be IEEE round-to-nearest-even).
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#define VO_OK 0
#define VO_ERR_ARG (-1)
#define VO_ERR_NOMEM (-2)
#define VO_ERR_BUDGET (-3)

#define VO_FLAG_DETERMINISTIC 1u

/* ------------------------------------------------------------------------ */
/* Philox4x32-10 (Salmon, Moraes, Dror, Shaw, SC'11).  Ten rounds of the    */
/* 4x32 bijection; the two multipliers and the two Weyl key increments are  */
/* the constants published with the generator.                              */
/* ------------------------------------------------------------------------ */
static void philox_round(uint32_t c[4], const uint32_t k[2])
{
    const uint64_t p0 = (uint64_t)0xD2511F53u * (uint64_t)c[0];
    const uint64_t p1 = (uint64_t)0xCD9E8D57u * (uint64_t)c[2];
    const uint32_t hi0 = (uint32_t)(p0 >> 32), lo0 = (uint32_t)p0;
    const uint32_t hi1 = (uint32_t)(p1 >> 32), lo1 = (uint32_t)p1;
    const uint32_t n0 = hi1 ^ c[1] ^ k[0];
    const uint32_t n1 = lo1;
    const uint32_t n2 = hi0 ^ c[3] ^ k[1];
    const uint32_t n3 = lo0;
    c[0] = n0; c[1] = n1; c[2] = n2; c[3] = n3;
}

void vo_philox4x32_10(const uint32_t ctr[4], const uint32_t key[2], uint32_t out[4])
{
    uint32_t c[4] = {ctr[0], ctr[1], ctr[2], ctr[3]};
    uint32_t k[2] = {key[0], key[1]};
    for (int r = 0; r < 10; ++r) {
        philox_round(c, k);
        k[0] += 0x9E3779B9u;
        k[1] += 0xBB67AE85u;
    }
    memcpy(out, c, sizeof c);
}

/* One 32-bit word -> a uniform in (0,1): the top 23 bits select one of the
 * 2^23 odd multiples of 2^-24, all exactly representable in fp32. */
float vo_uniform(uint32_t x)
{
    return (float)(2u * (x >> 9) + 1u) * 0x1p-24f;
}

/* E = -ln(u) in fp32 with a fixed IEEE operation sequence (textbook method:
 * Cody-Waite reduction to m in [sqrt(1/2), sqrt(2)] and the odd atanh series
 *   ln m = 2f + 2f z (1/3 + z/5 + z^2/7 + z^3/9),  f = (m-1)/(m+1), z = f^2,
 * as in Muller, "Elementary Functions", ch. 11).  Every step is one IEEE
 * binary32 operation rounded to nearest-even, so any IEEE implementation of
 * the same sequence returns the same bits. */
float vo_neglog(float u)
{
    uint32_t bits;
    memcpy(&bits, &u, 4);
    int e = (int)((bits >> 23) & 0xffu) - 127;
    uint32_t mb = (bits & 0x007fffffu) | 0x3f800000u;   /* m in [1,2) */
    if (mb > 0x3fb504f3u) {                               /* m > sqrt(2) */
        mb -= 0x00800000u;                                /* m /= 2      */
        e += 1;
    }
    float m;
    memcpy(&m, &mb, 4);
    const float num = m - 1.0f;            /* exact (Sterbenz) */
    const float den = m + 1.0f;
    const float f = num / den;
    const float z = f * f;
    float p = fmaf(0x1.c71c72p-4f /* 1/9 */, z, 0x1.24924ap-3f /* 1/7 */);
    p = fmaf(p, z, 0x1.99999ap-3f /* 1/5 */);
    p = fmaf(p, z, 0x1.555556p-2f /* 1/3 */);
    const float f2 = f * 2.0f;                 /* exact */
    const float t = z * p;
    const float lnm = fmaf(f2, t, f2);         /* 2f + 2f*z*p' */
    const float fe = (float)e;
    const float lo = fe * 0x1.7f7d1cp-20f;    /* e * (ln2 - LN2_HI)      */
    const float s = lo + lnm;
    const float hi = fe * 0x1.62e400p-1f;     /* e * LN2_HI, exact       */
    const float r = hi + s;
    return -r;
}

/* neglog over an array (for exhaustive checks of the scalar routine). */
void vo_neglog_n(const float* u, float* out, int64_t n)
{
    for (int64_t i = 0; i < n; ++i) out[i] = vo_neglog(u[i]);
}

/* ------------------------------------------------------------------------ */
/* Value-score variants of the ablations (Appendix A: L2, Range, Var) and   */
/* random reservation (Appendix D: N_v slots reserved for random pairs).     */
/*   L2(v)  = sqrt(sum_j v_j^2)                                              */
/*   Var(v) = (1/d) sum_j (v_j - mu)^2,  mu = (1/d) sum_j v_j                */
/*   random: u_i from Philox4x32-10 with purpose word 2, counter             */
/*           (i>>2, inst, round, 2), word i&3, the uniform map above, so    */
/*           the top N_v of u is a uniformly random N_v-subset.             */
/* ------------------------------------------------------------------------ */
#define VO_VALUE_RANGE 0
#define VO_VALUE_L2 1
#define VO_VALUE_VAR 2
#define VO_VALUE_RANDOM 3

int vo_vrange(const double* v, int n_inst, int N, int K, int d, float* out);

int vo_value_score(const double* v, int n_inst, uint32_t inst_base, int N, int K, int d, int kind,
                   uint64_t seed, uint32_t round, float* out)
{
    if (!out || n_inst < 0 || K < 1 || N < K || d < 1 || kind < 0 || kind > 3) return VO_ERR_ARG;
    if (kind != VO_VALUE_RANDOM && !v) return VO_ERR_ARG;
    if (kind == VO_VALUE_RANGE) return vo_vrange(v, n_inst, N, K, d, out);
#pragma omp parallel for schedule(static)
    for (int inst = 0; inst < n_inst; ++inst) {
        for (int i = 0; i < K; ++i) {
            double x;
            if (kind == VO_VALUE_RANDOM) {
                const uint32_t ctr[4] = {(uint32_t)i >> 2, inst_base + (uint32_t)inst, round, 2u};
                const uint32_t key[2] = {(uint32_t)seed, (uint32_t)(seed >> 32)};
                uint32_t w[4];
                vo_philox4x32_10(ctr, key, w);
                x = (double)vo_uniform(w[i & 3]);
            } else {
                const double* row = v + ((size_t)inst * N + i) * d;
                if (kind == VO_VALUE_L2) {
                    double ss = 0.0;
                    for (int j = 0; j < d; ++j) ss += row[j] * row[j];
                    x = sqrt(ss);
                } else {
                    double mu = 0.0;
                    for (int j = 0; j < d; ++j) mu += row[j];
                    mu /= d;
                    double ss = 0.0;
                    for (int j = 0; j < d; ++j) ss += (row[j] - mu) * (row[j] - mu);
                    x = ss / d;
                }
            }
            out[(size_t)inst * K + i] = (float)x;
        }
    }
    return VO_OK;
}

/* ------------------------------------------------------------------------ */
/* VaSE-DKV (Sec. 3.2 with the product score of Eq. 4).  At every eviction  */
/* step each head instance draws G_t in R^{d x r} with entries N(0, 1/r),   */
/* independent of earlier steps, and scores candidate i by                   */
/*   s_i = ||G_t^T k_i||^2 * ||G_t^T v_i||^2.                                */
/* Survivors are the K-B highest scores (vo_select in deterministic mode,   */
/* N_v = 0).  Readings: one G_t per (instance, step); the Gaussians come    */
/* from Philox4x32-10 with purpose word 1 through Box-Muller:               */
/*   entry e = a*r + b of G[a][b] takes words 2(e&1), 2(e&1)+1 of           */
/*   Philox(counter (e>>1, inst, round, 1), key (seed_lo, seed_hi)),        */
/*   z = sqrt(2 E(u1)) * cos(2 pi u2),  G = z / sqrt(r)  (all fp32).        */
/* ------------------------------------------------------------------------ */

/* cos(2 pi u), u in (0,1), in fp32 with a fixed operation sequence: the
 * quadrant comes from u itself (t = 4u and f = t - floor(t) are exact), then
 * the Taylor series of cos(pi f / 2) and sin(pi f / 2) in f, both truncated
 * after the f^14 / f^15 terms (remainders below 2e-10), by Horner with fma. */
float vo_cos2pi(float u)
{
    const float t = 4.0f * u;
    const float qf = floorf(t);
    const float f = t - qf;
    const int q = (int)qf & 3;
    const float z = f * f;
    /* (-1)^k (pi/2)^(2k) / (2k)!,  k = 7 .. 0 */
    float c = -0x1.b6e250p-28f;
    c = fmaf(c, z, 0x1.f9d38ap-22f);
    c = fmaf(c, z, -0x1.a6d1f2p-16f);
    c = fmaf(c, z, 0x1.e1f506p-11f);
    c = fmaf(c, z, -0x1.55d3c8p-6f);
    c = fmaf(c, z, 0x1.03c1f0p-2f);
    c = fmaf(c, z, -0x1.3bd3ccp+0f);
    c = fmaf(c, z, 1.0f);
    /* (-1)^k (pi/2)^(2k+1) / (2k+1)!,  k = 7 .. 0, times f */
    float sn = -0x1.6fadbap-31f;
    sn = fmaf(sn, z, 0x1.e8f434p-25f);
    sn = fmaf(sn, z, -0x1.e30750p-19f);
    sn = fmaf(sn, z, 0x1.507834p-13f);
    sn = fmaf(sn, z, -0x1.32d2ccp-8f);
    sn = fmaf(sn, z, 0x1.466bc6p-4f);
    sn = fmaf(sn, z, -0x1.4abbcep-1f);
    sn = fmaf(sn, z, 0x1.921fb6p+0f);
    sn = sn * f;
    /* cos(q pi/2 + theta) */
    return q == 0 ? c : (q == 1 ? -sn : (q == 2 ? -c : sn));
}

/* G_t of one instance: [d][r] fp32, row-major. */
void vo_dkv_gaussian(uint64_t seed, uint32_t inst_id, uint32_t round, int d, int r, float* g)
{
    const uint32_t key[2] = {(uint32_t)seed, (uint32_t)(seed >> 32)};
    const float scale = 1.0f / sqrtf((float)r);
    for (int e = 0; e < d * r; ++e) {
        const uint32_t ctr[4] = {(uint32_t)e >> 1, inst_id, round, 1u};
        uint32_t x[4];
        vo_philox4x32_10(ctr, key, x);
        const float u1 = vo_uniform(x[2 * (e & 1)]);
        const float u2 = vo_uniform(x[2 * (e & 1) + 1]);
        const float rad = sqrtf(2.0f * vo_neglog(u1));
        const float z = rad * vo_cos2pi(u2);
        g[e] = z * scale;
    }
}

/* Product score for given projections: k, v [n_inst][N][d] (exact upcasts),
 * g [n_inst][d][r] (fp32), out [n_inst][K] fp32.  Double accumulation. */
int vo_dkv_score_g(const double* k, const double* v, const float* g, int n_inst, int N, int K,
                   int d, int r, float* out)
{
    if (!k || !v || !g || !out || n_inst < 0 || K < 1 || N < K || d < 1 || r < 1)
        return VO_ERR_ARG;
    #pragma omp parallel for schedule(dynamic)
    for (int n = 0; n < n_inst; ++n) {
        const float* gi = g + (size_t)n * d * r;
        for (int i = 0; i < K; ++i) {
            const double* ki = k + ((size_t)n * N + i) * d;
            const double* vi = v + ((size_t)n * N + i) * d;
            double lk = 0.0, lv = 0.0;
            for (int b = 0; b < r; ++b) {
                double pk = 0.0, pv = 0.0;
                for (int a = 0; a < d; ++a) {
                    pk += ki[a] * (double)gi[a * r + b];
                    pv += vi[a] * (double)gi[a * r + b];
                }
                lk += pk * pk;
                lv += pv * pv;
            }
            out[(size_t)n * K + i] = (float)(lk * lv);
        }
    }
    return VO_OK;
}

/* The DKV score of one round: draws G_t per instance, then vo_dkv_score_g. */
int vo_dkv_score(const double* k, const double* v, int n_inst, uint32_t inst_base, int N, int K,
                 int d, int r, uint64_t seed, uint32_t round, float* out)
{
    if (n_inst < 0 || d < 1 || r < 1) return VO_ERR_ARG;
    float* g = (float*)malloc(sizeof(float) * (size_t)(n_inst > 0 ? n_inst : 1) * d * r);
    if (!g) return VO_ERR_NOMEM;
    for (int n = 0; n < n_inst; ++n)
        vo_dkv_gaussian(seed, inst_base + (uint32_t)n, round, d, r, g + (size_t)n * d * r);
    const int rc = vo_dkv_score_g(k, v, g, n_inst, N, K, d, r, out);
    free(g);
    return rc;
}

/* ------------------------------------------------------------------------ */
/* Step 1: pooled SnapKV score (Eq. 1 inside Eq. 2, pooling per footnote).  */
/* q: [n_inst][R][d] (R = G*w window rows of the group), k: [n_inst][N][d]  */
/* attn_out: [n_inst][K] fp32.  abar_out (nullable): [n_inst][N] double,    */
/* the unpooled mean over rows for every slot (buffer slots included).      */
/* ------------------------------------------------------------------------ */
int vo_score(const double* q, const double* k, int n_inst, int R, int N, int K, int d,
             int pool, float* attn_out, double* abar_out)
{
    if (!q || !k || !attn_out || n_inst < 0 || R < 1 || K < 1 || N < K || d < 1 ||
        pool < 1 || (pool % 2) == 0)
        return VO_ERR_ARG;
    const double scale = 1.0 / sqrt((double)d);
    int err = VO_OK;
#pragma omp parallel for schedule(dynamic, 1)
    for (int inst = 0; inst < n_inst; ++inst) {
        const double* qi = q + (size_t)inst * R * d;
        const double* ki = k + (size_t)inst * N * d;
        double* s = (double*)malloc(sizeof(double) * (size_t)N);
        double* abar = (double*)calloc((size_t)N, sizeof(double));
        if (!s || !abar) {
            free(s); free(abar);
#pragma omp atomic write
            err = VO_ERR_NOMEM;
            continue;
        }
        for (int r = 0; r < R; ++r) {
            const double* qr = qi + (size_t)r * d;
            /* s_ri = q_r . k_i / sqrt(d) for every cached slot (Eq. 1) */
            for (int i = 0; i < N; ++i) {
                double acc = 0.0;
                for (int j = 0; j < d; ++j) acc += qr[j] * ki[(size_t)i * d + j];
                s[i] = acc * scale;
            }
            double mx = s[0];
            for (int i = 1; i < N; ++i) if (s[i] > mx) mx = s[i];
            double l = 0.0;
            for (int i = 0; i < N; ++i) l += exp(s[i] - mx);
            /* alpha_i^(r) = softmax over all N slots; mean over rows */
            for (int i = 0; i < N; ++i) abar[i] += exp(s[i] - mx) / l;
        }
        for (int i = 0; i < N; ++i) abar[i] /= (double)R;
        if (abar_out) memcpy(abar_out + (size_t)inst * N, abar, sizeof(double) * (size_t)N);
        /* average pooling over the K candidates, zero padded, divided by P */
        const int h = pool / 2;
        for (int i = 0; i < K; ++i) {
            double acc = 0.0;
            for (int j = i - h; j <= i + h; ++j)
                if (j >= 0 && j < K) acc += abar[j];
            attn_out[(size_t)inst * K + i] = (float)(acc / (double)pool);
        }
        free(s);
        free(abar);
    }
    return err;
}

/* Step 2: Range(v) = max_j v_j - min_j v_j for the K candidate slots (Eq. 5). */
int vo_vrange(const double* v, int n_inst, int N, int K, int d, float* out)
{
    if (!v || !out || n_inst < 0 || K < 1 || N < K || d < 1) return VO_ERR_ARG;
#pragma omp parallel for schedule(static)
    for (int inst = 0; inst < n_inst; ++inst) {
        for (int i = 0; i < K; ++i) {
            const double* row = v + ((size_t)inst * N + i) * d;
            double mx = row[0], mn = row[0];
            for (int j = 1; j < d; ++j) {
                if (row[j] > mx) mx = row[j];
                if (row[j] < mn) mn = row[j];
            }
            out[(size_t)inst * K + i] = (float)(mx - mn);
        }
    }
    return VO_OK;
}

/* ------------------------------------------------------------------------ */
/* Steps 3-6: reservation, stochastic fill and the survivor map.            */
/* ------------------------------------------------------------------------ */
typedef struct { float v; int32_t i; } vo_pair;

/* larger value first; equal values: lower slot first */
static int cmp_desc_then_slot(const void* a, const void* b)
{
    const vo_pair* x = (const vo_pair*)a;
    const vo_pair* y = (const vo_pair*)b;
    if (x->v > y->v) return -1;
    if (x->v < y->v) return 1;
    return (x->i < y->i) ? -1 : (x->i > y->i);
}

/* The selection noise of one candidate slot: E_i = -ln(u_i). */
float vo_noise(uint64_t seed, uint32_t inst_id, uint32_t round, uint32_t purpose, int32_t slot)
{
    const uint32_t ctr[4] = {(uint32_t)slot >> 2, inst_id, round, purpose};
    const uint32_t key[2] = {(uint32_t)seed, (uint32_t)(seed >> 32)};
    uint32_t x[4];
    vo_philox4x32_10(ctr, key, x);
    return vo_neglog(vo_uniform(x[slot & 3]));
}

/*
 * attn, vrange: [n_inst][K] fp32.  src_out: [n_inst][K] int32, src[j] = old
 * slot that lands in new slot j.  keys_out (nullable): [n_inst][K] fp32
 * selection key of each slot (NaN for reserved slots).  Returns VO_OK, or
 * VO_ERR_BUDGET if an instance would not end with exactly K slots.
 */
int vo_select(const float* attn, const float* vrange, int n_inst, uint32_t inst_base, int K,
              int B, int Nv, uint64_t seed, uint32_t round, uint32_t flags, int32_t* src_out,
              float* keys_out)
{
    if (!attn || !vrange || !src_out || n_inst < 0 || K < 1 || B < 1 || Nv < 0 ||
        Nv + B > K)
        return VO_ERR_ARG;
    const int N = K + B;
    int err = VO_OK;
#pragma omp parallel for schedule(dynamic, 4)
    for (int inst = 0; inst < n_inst; ++inst) {
        const float* a = attn + (size_t)inst * K;
        const float* r = vrange + (size_t)inst * K;
        const uint32_t inst_id = inst_base + (uint32_t)inst;
        vo_pair* byrange = (vo_pair*)malloc(sizeof(vo_pair) * (size_t)K);
        vo_pair* cand = (vo_pair*)malloc(sizeof(vo_pair) * (size_t)K);
        unsigned char* keep = (unsigned char*)calloc((size_t)N, 1);
        if (!byrange || !cand || !keep) {
            free(byrange); free(cand); free(keep);
#pragma omp atomic write
            err = VO_ERR_NOMEM;
            continue;
        }
        /* R_V: the N_v candidates with the largest Range (Sec. 3.2) */
        for (int i = 0; i < K; ++i) { byrange[i].v = r[i]; byrange[i].i = i; }
        qsort(byrange, (size_t)K, sizeof(vo_pair), cmp_desc_then_slot);
        for (int t = 0; t < Nv; ++t) keep[byrange[t].i] = 1;
        /* R_B: the buffer [K, N) is always kept (Sec. 2) */
        for (int i = K; i < N; ++i) keep[i] = 1;
        /* C = [K] \ R_V; each candidate gets key = attn_i / E_i */
        int nc = 0;
        for (int i = 0; i < K; ++i) {
            if (keep[i]) {
                if (keys_out) keys_out[(size_t)inst * K + i] = NAN;
                continue;
            }
            float key;
            if (flags & VO_FLAG_DETERMINISTIC) {
                key = a[i];
            } else {
                const float E = vo_noise(seed, inst_id, round, 0u, i);
                key = a[i] / E;
            }
            if (keys_out) keys_out[(size_t)inst * K + i] = key;
            cand[nc].v = key;
            cand[nc].i = i;
            ++nc;
        }
        /* fill the remaining K - |R| slots with the largest keys */
        const int m = K - Nv - B;
        qsort(cand, (size_t)nc, sizeof(vo_pair), cmp_desc_then_slot);
        for (int t = 0; t < m; ++t) keep[cand[t].i] = 1;
        /* survivor map: kept slots in increasing slot order */
        int j = 0;
        for (int i = 0; i < N; ++i)
            if (keep[i]) {
                if (j < K) src_out[(size_t)inst * K + j] = i;
                ++j;
            }
        if (j != K || nc - m != B) {
#pragma omp atomic write
            err = VO_ERR_BUDGET;
        }
        free(byrange);
        free(cand);
        free(keep);
    }
    return err;
}

/* Step 7: K'[j] = K[src[j]], V'[j] = V[src[j]] for j < K; raw row copies.
 * Reads every source row before writing, so it is correct in place. */
int vo_compact(void* k, void* v, const int32_t* src, int n_inst, int N, int K, size_t row_bytes)
{
    if (!k || !v || !src || n_inst < 0 || K < 1 || N < K || row_bytes == 0) return VO_ERR_ARG;
    int err = VO_OK;
#pragma omp parallel for schedule(static)
    for (int inst = 0; inst < n_inst; ++inst) {
        unsigned char* kb = (unsigned char*)k + (size_t)inst * N * row_bytes;
        unsigned char* vb = (unsigned char*)v + (size_t)inst * N * row_bytes;
        unsigned char* tk = (unsigned char*)malloc((size_t)K * row_bytes);
        unsigned char* tv = (unsigned char*)malloc((size_t)K * row_bytes);
        if (!tk || !tv) {
            free(tk); free(tv);
#pragma omp atomic write
            err = VO_ERR_NOMEM;
            continue;
        }
        for (int j = 0; j < K; ++j) {
            const int s = src[(size_t)inst * K + j];
            if (s < 0 || s >= N) {
#pragma omp atomic write
                err = VO_ERR_ARG;
                continue;
            }
            memcpy(tk + (size_t)j * row_bytes, kb + (size_t)s * row_bytes, row_bytes);
            memcpy(tv + (size_t)j * row_bytes, vb + (size_t)s * row_bytes, row_bytes);
        }
        memcpy(kb, tk, (size_t)K * row_bytes);
        memcpy(vb, tv, (size_t)K * row_bytes);
        free(tk);
        free(tv);
    }
    return err;
}

/* Step 7 under an order map.  The cache returns to K persistent slots (Sec. 2)
 * without moving the survivors: ord[t] is the physical slot of the persistent
 * token of temporal rank t (t < K, oldest first) and the buffer token K + b sits
 * in slot K + b.  Read through the map, the cache is the temporal cache
 *   T[t] = X[ord[t]] (t < K),  T[t] = X[t] (K <= t < N),
 * and the round's survivor map src (vo_select, over temporal ranks) keeps
 * T'[j] = T[src[j]].  Here the survivors stay where they are and the B buffer
 * rows move into the B slots that the evicted tokens leave:
 *   e_0 < e_1 < ... < e_{B-1}  the evicted ranks, [0, K) minus src[0 .. K-B)
 *   moves_out[b] = ord[e_b]    the slot that buffer row K + b is copied to
 *   ord_out[j]   = ord[src[j]] for j < K - B,   ord_out[K - B + b] = ord[e_b]
 * so that X'[ord_out[j]] = T'[j] for every j < K: the same temporal cache as
 * the stable compaction, with B row copies instead of up to K.
 * ord, ord_out: [n_inst][K]; src: [n_inst][K]; moves_out: [n_inst][B]. */
int vo_order_compact(const int32_t* ord, const int32_t* src, int n_inst, int K, int B,
                     int32_t* ord_out, int32_t* moves_out)
{
    if (!ord || !src || !ord_out || !moves_out || n_inst < 0 || B < 1 || K < B) return VO_ERR_ARG;
    int err = VO_OK;
    const int M = K - B;   /* survivors among the K candidates */
    for (int inst = 0; inst < n_inst; ++inst) {
        const int32_t* o = ord + (size_t)inst * K;
        const int32_t* s = src + (size_t)inst * K;
        int32_t* on = ord_out + (size_t)inst * K;
        int32_t* mv = moves_out + (size_t)inst * B;
        unsigned char* kept = (unsigned char*)calloc((size_t)K, 1);
        if (!kept) return VO_ERR_NOMEM;
        for (int j = 0; j < M; ++j) {
            if (s[j] < 0 || s[j] >= K || (j > 0 && s[j] <= s[j - 1]) || o[s[j]] < 0 ||
                o[s[j]] >= K) { err = VO_ERR_ARG; break; }
            kept[s[j]] = 1;
            on[j] = o[s[j]];
        }
        for (int j = M; j < K && err == VO_OK; ++j)
            if (s[j] != K + (j - M)) err = VO_ERR_ARG;    /* the buffer, in order */
        int b = 0;
        for (int t = 0; t < K && err == VO_OK; ++t) {
            if (kept[t]) continue;
            if (b >= B) { err = VO_ERR_ARG; break; }
            mv[b] = o[t];
            on[M + b] = o[t];
            ++b;
        }
        if (err == VO_OK && b != B) err = VO_ERR_ARG;
        free(kept);
        if (err != VO_OK) return err;
    }
    return err;
}

/* Step 8: decode attention, Eq. (1), over the first n_valid slots.
 * q: [n_inst][G][d]; k, v: [n_inst][N][d]; out: [n_inst][G][d] double. */
int vo_decode(const double* q, const double* k, const double* v, int n_inst, int N,
              int n_valid, int G, int d, double* out)
{
    if (!q || !k || !v || !out || n_inst < 0 || n_valid < 1 || n_valid > N || G < 1 || d < 1)
        return VO_ERR_ARG;
    const double scale = 1.0 / sqrt((double)d);
    int err = VO_OK;
#pragma omp parallel for schedule(static)
    for (int inst = 0; inst < n_inst; ++inst) {
        double* s = (double*)malloc(sizeof(double) * (size_t)n_valid);
        if (!s) {
#pragma omp atomic write
            err = VO_ERR_NOMEM;
            continue;
        }
        const double* ki = k + (size_t)inst * N * d;
        const double* vi = v + (size_t)inst * N * d;
        for (int g = 0; g < G; ++g) {
            const double* qg = q + ((size_t)inst * G + g) * d;
            double* o = out + ((size_t)inst * G + g) * d;
            for (int i = 0; i < n_valid; ++i) {
                double acc = 0.0;
                for (int j = 0; j < d; ++j) acc += qg[j] * ki[(size_t)i * d + j];
                s[i] = acc * scale;
            }
            double mx = s[0];
            for (int i = 1; i < n_valid; ++i) if (s[i] > mx) mx = s[i];
            double l = 0.0;
            for (int i = 0; i < n_valid; ++i) l += exp(s[i] - mx);
            for (int j = 0; j < d; ++j) o[j] = 0.0;
            for (int i = 0; i < n_valid; ++i) {
                const double p = exp(s[i] - mx) / l;
                for (int j = 0; j < d; ++j) o[j] += p * vi[(size_t)i * d + j];
            }
        }
        free(s);
    }
    return err;
}

/* ------------------------------------------------------------------------ */
/* Decode-side integration.  Between two rounds the persistent slots [0, K)  */
/* do not change: each decode step only appends to the buffer.  The step    */
/* that produces a window query already runs Eq. (1) for it over [0, K), so  */
/* it can hand the round the log of that part of the softmax normaliser,    */
/*   L_r = ln sum_{i < K} exp(q_r . k_i / sqrt(d)),                          */
/* and the round completes each row's normaliser with the buffer slots only. */
/* ------------------------------------------------------------------------ */

/* lse_out[inst][g] = ln sum_{i < n_persist} exp(q_g . k_i / sqrt(d)), the
 * normaliser of Eq. (1) restricted to the persistent slots, in double. */
int vo_decode_lse(const double* q, const double* k, int n_inst, int N, int n_persist, int G,
                  int d, double* lse_out)
{
    if (!q || !k || !lse_out || n_inst < 0 || n_persist < 1 || n_persist > N || G < 1 || d < 1)
        return VO_ERR_ARG;
    const double scale = 1.0 / sqrt((double)d);
    int err = VO_OK;
#pragma omp parallel for schedule(static)
    for (int inst = 0; inst < n_inst; ++inst) {
        double* s = (double*)malloc(sizeof(double) * (size_t)n_persist);
        if (!s) {
#pragma omp atomic write
            err = VO_ERR_NOMEM;
            continue;
        }
        const double* ki = k + (size_t)inst * N * d;
        for (int g = 0; g < G; ++g) {
            const double* qg = q + ((size_t)inst * G + g) * d;
            for (int i = 0; i < n_persist; ++i) {
                double acc = 0.0;
                for (int j = 0; j < d; ++j) acc += qg[j] * ki[(size_t)i * d + j];
                s[i] = acc * scale;
            }
            double mx = s[0];
            for (int i = 1; i < n_persist; ++i) if (s[i] > mx) mx = s[i];
            double l = 0.0;
            for (int i = 0; i < n_persist; ++i) l += exp(s[i] - mx);
            lse_out[(size_t)inst * G + g] = mx + log(l);
        }
        free(s);
    }
    return err;
}

/* Step 1 with the persistent part of each row's normaliser supplied:
 * lse_win[inst][r] = L_r as above.  Row r's softmax over all N slots is
 *   p_ri = exp(s_ri) / (exp(L_r) + sum_{K <= i < N} exp(s_ri)),
 * then the window mean and pooling exactly as in vo_score.  When L_r is the
 * true value this is vo_score's result. */
int vo_score_lse(const double* q, const double* k, const double* lse_win, int n_inst, int R, int N,
                 int K, int d, int pool, float* attn_out)
{
    if (!q || !k || !lse_win || !attn_out || n_inst < 0 || R < 1 || K < 1 || N < K || d < 1 ||
        pool < 1 || (pool % 2) == 0)
        return VO_ERR_ARG;
    const double scale = 1.0 / sqrt((double)d);
    int err = VO_OK;
#pragma omp parallel for schedule(dynamic, 1)
    for (int inst = 0; inst < n_inst; ++inst) {
        const double* qi = q + (size_t)inst * R * d;
        const double* ki = k + (size_t)inst * N * d;
        double* s = (double*)malloc(sizeof(double) * (size_t)N);
        double* abar = (double*)calloc((size_t)K, sizeof(double));
        if (!s || !abar) {
            free(s); free(abar);
#pragma omp atomic write
            err = VO_ERR_NOMEM;
            continue;
        }
        for (int r = 0; r < R; ++r) {
            const double* qr = qi + (size_t)r * d;
            for (int i = 0; i < N; ++i) {
                double acc = 0.0;
                for (int j = 0; j < d; ++j) acc += qr[j] * ki[(size_t)i * d + j];
                s[i] = acc * scale;
            }
            /* normaliser: the supplied persistent part plus the buffer slots */
            const double lp = lse_win[(size_t)inst * R + r];
            double mx = lp;
            for (int i = K; i < N; ++i) if (s[i] > mx) mx = s[i];
            double l = exp(lp - mx);
            for (int i = K; i < N; ++i) l += exp(s[i] - mx);
            for (int i = 0; i < K; ++i) abar[i] += exp(s[i] - mx) / l;
        }
        for (int i = 0; i < K; ++i) abar[i] /= (double)R;
        const int h = pool / 2;
        for (int i = 0; i < K; ++i) {
            double acc = 0.0;
            for (int j = i - h; j <= i + h; ++j)
                if (j >= 0 && j < K) acc += abar[j];
            attn_out[(size_t)inst * K + i] = (float)(acc / (double)pool);
        }
        free(s);
        free(abar);
    }
    return err;
}

/* ------------------------------------------------------------------------ */
/* Range-based per-token asymmetric quantisation (Eq. 6, Sec. 4.3) with the  */
/* mixed-precision reservation suggested in Sec. 7: the N_v rows with the    */
/* largest Range stay in full precision, the rest are stored as b-bit codes. */
/*                                                                           */
/* Per token (row) and per group of g consecutive elements:                  */
/*   z = min x,  Delta = (max x - min x) / (2^b - 1),                        */
/*   q_e = round((x_e - z) / Delta)  (nearest, ties to even; 0 if Delta = 0) */
/*   x'_e = q_e * Delta + z                                                  */
/* Readings: every step that decides a code is one fp32 operation (the      */
/* subtraction, the IEEE divides, rint), so the codes are reproducible; the  */
/* reconstruction is one fp32 fma.  Codes of one row form a bit stream, code */
/* e at bits [e*b, e*b + b), little-endian within each byte.                 */
/* ------------------------------------------------------------------------ */

/* fp32 -> bf16 bits, round to nearest even (finite inputs) */
static uint16_t vo_f32_to_bf16(float f)
{
    uint32_t u;
    memcpy(&u, &f, 4);
    if ((u & 0x7fffffffu) > 0x7f800000u) return (uint16_t)((u >> 16) | 0x40u);
    u += 0x7fffu + ((u >> 16) & 1u);
    return (uint16_t)(u >> 16);
}

/* x: [n_inst][N][d] (rows [0, K) quantised); codes: [n_inst][K][d*bits/8];
 * params: [n_inst][K][d/group][2] = (Delta, z); range_out, mse_out: [n_inst][K]
 * (nullable); hp_idx: [n_inst][Nv] reserved slots in ascending order (nullable
 * when Nv = 0).  mse = (1/d) sum_e (x_e - x'_e)^2 with x' in fp32. */
int vo_quantize(const double* x, int n_inst, int N, int K, int d, int bits, int group, int Nv,
                uint8_t* codes, float* params, float* range_out, float* mse_out, int32_t* hp_idx)
{
    if (!x || !codes || !params || n_inst < 0 || K < 1 || N < K || d < 1 ||
        !(bits == 2 || bits == 4 || bits == 8) || group < 1 || d % group != 0 ||
        (d * bits) % 8 != 0 || Nv < 0 || Nv > K || (Nv > 0 && !hp_idx))
        return VO_ERR_ARG;
    const int row_bytes = d * bits / 8;
    const int ng = d / group;
    const float levels = (float)((1u << bits) - 1u);
    int err = VO_OK;
#pragma omp parallel for schedule(static)
    for (int inst = 0; inst < n_inst; ++inst) {
        vo_pair* byrange = (vo_pair*)malloc(sizeof(vo_pair) * (size_t)K);
        if (!byrange) {
#pragma omp atomic write
            err = VO_ERR_NOMEM;
            continue;
        }
        for (int i = 0; i < K; ++i) {
            const double* row = x + ((size_t)inst * N + i) * d;
            uint8_t* cb = codes + ((size_t)inst * K + i) * row_bytes;
            memset(cb, 0, (size_t)row_bytes);
            double se = 0.0;
            float rmax = (float)row[0], rmin = (float)row[0];
            for (int gi = 0; gi < ng; ++gi) {
                const double* xg = row + gi * group;
                float mn = (float)xg[0], mx = (float)xg[0];
                for (int e = 1; e < group; ++e) {
                    const float v = (float)xg[e];
                    if (v < mn) mn = v;
                    if (v > mx) mx = v;
                }
                if (mn < rmin) rmin = mn;
                if (mx > rmax) rmax = mx;
                const float range = mx - mn;
                const float delta = range / levels;
                float* pp = params + (((size_t)inst * K + i) * ng + gi) * 2;
                pp[0] = delta;
                pp[1] = mn;
                for (int e = 0; e < group; ++e) {
                    const float v = (float)xg[e];
                    float q = 0.0f;
                    if (delta > 0.0f) {
                        q = rintf((v - mn) / delta);
                        if (!(q >= 0.0f)) q = 0.0f;      /* also a NaN quotient (Range overflow) */
                        if (q > levels) q = levels;
                    }
                    const int bit = (gi * group + e) * bits;
                    cb[bit >> 3] |= (uint8_t)((uint32_t)q << (bit & 7));
                    const float xr = fmaf(q, delta, mn);
                    se += ((double)v - (double)xr) * ((double)v - (double)xr);
                }
            }
            if (mse_out) mse_out[(size_t)inst * K + i] = (float)(se / d);
            const float rg = rmax - rmin;      /* Range(x), Eq. (5) */
            if (range_out) range_out[(size_t)inst * K + i] = rg;
            byrange[i].v = rg;
            byrange[i].i = i;
        }
        if (Nv > 0) {
            /* the N_v largest Ranges (ties: lower slot), listed in slot order */
            qsort(byrange, (size_t)K, sizeof(vo_pair), cmp_desc_then_slot);
            int32_t* hp = hp_idx + (size_t)inst * Nv;
            for (int t = 0; t < Nv; ++t) hp[t] = byrange[t].i;
            for (int a = 1; a < Nv; ++a)           /* insertion sort, ascending */
                for (int b = a; b > 0 && hp[b - 1] > hp[b]; --b) {
                    const int32_t tmp = hp[b]; hp[b] = hp[b - 1]; hp[b - 1] = tmp;
                }
        }
        free(byrange);
    }
    return err;
}

/* Inverse: out rows [0, K) of [n_inst][N][d] get x'_e = fma(q_e, Delta, z)
 * (fp32) stored in the output type (out_bf16: round to nearest even), except
 * the reserved rows hp_idx, which take the full-precision rows hp_rows
 * ([n_inst][Nv][d], raw bytes of the output type). */
int vo_dequantize(const uint8_t* codes, const float* params, const void* hp_rows,
                  const int32_t* hp_idx, int n_inst, int N, int K, int d, int bits, int group,
                  int Nv, int out_bf16, void* out)
{
    if (!codes || !params || !out || n_inst < 0 || K < 1 || N < K || d < 1 ||
        !(bits == 2 || bits == 4 || bits == 8) || group < 1 || d % group != 0 || Nv < 0 ||
        Nv > K || (Nv > 0 && (!hp_rows || !hp_idx)))
        return VO_ERR_ARG;
    const int row_bytes = d * bits / 8;
    const int ng = d / group;
    const size_t es = out_bf16 ? 2 : 4;
    const uint32_t mask = (1u << bits) - 1u;
#pragma omp parallel for schedule(static)
    for (int inst = 0; inst < n_inst; ++inst) {
        for (int i = 0; i < K; ++i) {
            const uint8_t* cb = codes + ((size_t)inst * K + i) * row_bytes;
            uint8_t* orow = (uint8_t*)out + ((size_t)inst * N + i) * d * es;
            for (int e = 0; e < d; ++e) {
                const int gi = e / group;
                const float* pp = params + (((size_t)inst * K + i) * ng + gi) * 2;
                const int bit = e * bits;
                const float q = (float)((cb[bit >> 3] >> (bit & 7)) & mask);
                const float xr = fmaf(q, pp[0], pp[1]);
                if (out_bf16) {
                    const uint16_t h = vo_f32_to_bf16(xr);
                    memcpy(orow + e * 2, &h, 2);
                } else {
                    memcpy(orow + e * 4, &xr, 4);
                }
            }
        }
        for (int t = 0; t < Nv; ++t) {
            const int32_t i = hp_idx[(size_t)inst * Nv + t];
            if (i < 0 || i >= K) continue;
            memcpy((uint8_t*)out + ((size_t)inst * N + i) * d * es,
                   (const uint8_t*)hp_rows + ((size_t)inst * Nv + t) * d * es, (size_t)d * es);
        }
    }
    return VO_OK;
}
