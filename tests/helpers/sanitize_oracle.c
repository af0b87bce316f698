/* Host driver for the sanitizer build of the oracle (test infrastructure).
 * Compiled together with oracle/vase_oracle.c under -fsanitize=address,undefined;
 * runs every oracle entry point on small seeded inputs, with ragged shapes and
 * the boundary cases (B = K - N_v, N_v = 0, P = 1, n_valid = N, one instance),
 * so that an out-of-bounds access, a use of freed memory or undefined integer
 * or shift behaviour in the oracle stops the run.  Prints "ok" and exits 0. */
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

int vo_score(const double* q, const double* k, int n_inst, int R, int N, int K, int d, int pool,
             float* attn_out, double* abar_out);
int vo_score_lse(const double* q, const double* k, const double* lse_win, int n_inst, int R, int N,
                 int K, int d, int pool, float* attn_out);
int vo_vrange(const double* v, int n_inst, int N, int K, int d, float* out);
int vo_value_score(const double* v, int n_inst, uint32_t inst_base, int N, int K, int d, int kind,
                   uint64_t seed, uint32_t round, float* out);
int vo_select(const float* attn, const float* vrange, int n_inst, uint32_t inst_base, int K, int B,
              int Nv, uint64_t seed, uint32_t round, uint32_t flags, int32_t* src_out,
              float* keys_out);
int vo_compact(void* k, void* v, const int32_t* src, int n_inst, int N, int K, size_t row_bytes);
int vo_order_compact(const int32_t* ord, const int32_t* src, int n_inst, int K, int B,
                     int32_t* ord_out, int32_t* moves_out);
int vo_decode(const double* q, const double* k, const double* v, int n_inst, int N, int n_valid,
              int G, int d, double* out);
int vo_decode_lse(const double* q, const double* k, int n_inst, int N, int n_persist, int G, int d,
                  double* lse_out);
int vo_dkv_score(const double* k, const double* v, int n_inst, uint32_t inst_base, int N, int K,
                 int d, int r, uint64_t seed, uint32_t round, float* out);
int vo_quantize(const double* x, int n_inst, int N, int K, int d, int bits, int group, int Nv,
                uint8_t* codes, float* params, float* range_out, float* mse_out, int32_t* hp_idx);
int vo_dequantize(const uint8_t* codes, const float* params, const void* hp_rows,
                  const int32_t* hp_idx, int n_inst, int N, int K, int d, int bits, int group,
                  int Nv, int out_bf16, void* out);
void vo_neglog_n(const float* u, float* out, int64_t n);

static uint64_t rng = 88172645463325252ull;
static double gauss(void) {
    /* xorshift64 + Box-Muller; inputs only, no method arithmetic */
    rng ^= rng << 13; rng ^= rng >> 7; rng ^= rng << 17;
    double u1 = ((rng >> 11) + 0.5) * (1.0 / 9007199254740992.0);
    rng ^= rng << 13; rng ^= rng >> 7; rng ^= rng << 17;
    double u2 = ((rng >> 11) + 0.5) * (1.0 / 9007199254740992.0);
    return sqrt(-2.0 * log(u1)) * cos(6.283185307179586 * u2);
}
static double* randn(size_t n) {
    double* p = malloc(n * sizeof(double));
    for (size_t i = 0; i < n; ++i) p[i] = gauss();
    return p;
}
#define CHECK(x) do { int rc_ = (x); if (rc_ != 0) { printf("FAIL %s -> %d\n", #x, rc_); exit(1); } } while (0)

static void round_case(int n, int G, int w, int K, int B, int d, int Nv, int pool) {
    const int N = K + B, R = G * w;
    double* q = randn((size_t)n * R * d);
    double* k = randn((size_t)n * N * d);
    double* v = randn((size_t)n * N * d);
    double* qd = randn((size_t)n * G * d);
    float* attn = malloc(sizeof(float) * n * K);
    double* abar = malloc(sizeof(double) * n * N);
    float* vr = malloc(sizeof(float) * n * K);
    int32_t* src = malloc(sizeof(int32_t) * n * K);
    float* keys = malloc(sizeof(float) * n * K);
    CHECK(vo_score(q, k, n, R, N, K, d, pool, attn, abar));
    CHECK(vo_vrange(v, n, N, K, d, vr));
    for (int kind = 0; kind < 4; ++kind) CHECK(vo_value_score(v, n, 7, N, K, d, kind, 5, 3, vr));
    CHECK(vo_vrange(v, n, N, K, d, vr));
    CHECK(vo_select(attn, vr, n, 0, K, B, Nv, 0x123456789abcdefull, 9, 0, src, keys));
    CHECK(vo_select(attn, vr, n, 0, K, B, Nv, 1, 2, 1, src, NULL));
    double* lse = malloc(sizeof(double) * n * R);
    CHECK(vo_decode_lse(q, k, n, N, K, R, d, lse));
    CHECK(vo_score_lse(q, k, lse, n, R, N, K, d, pool, attn));
    int32_t* ord = malloc(sizeof(int32_t) * n * K);
    int32_t* ord2 = malloc(sizeof(int32_t) * n * K);
    int32_t* moves = malloc(sizeof(int32_t) * n * B);
    for (int i = 0; i < n; ++i)
        for (int t = 0; t < K; ++t) ord[(size_t)i * K + t] = K - 1 - t;
    CHECK(vo_order_compact(ord, src, n, K, B, ord2, moves));
    CHECK(vo_compact(k, v, src, n, N, K, sizeof(double) * d));
    double* out = malloc(sizeof(double) * n * G * d);
    CHECK(vo_decode(qd, k, v, n, N, K, G, d, out));
    CHECK(vo_decode(qd, k, v, n, N, N, G, d, out));
    CHECK(vo_dkv_score(k, v, n, 3, N, K, d, 20, 11, 2, attn));
    free(q); free(k); free(v); free(qd); free(attn); free(abar); free(vr); free(src); free(keys);
    free(lse); free(ord); free(ord2); free(moves); free(out);
}

static void quant_case(int n, int K, int B, int d, int bits, int group, int Nv) {
    const int N = K + B;
    double* x = randn((size_t)n * N * d);
    uint8_t* codes = malloc((size_t)n * K * d * bits / 8);
    float* params = malloc(sizeof(float) * n * K * (d / group) * 2);
    float* range = malloc(sizeof(float) * n * K);
    float* mse = malloc(sizeof(float) * n * K);
    int32_t* hp_idx = malloc(sizeof(int32_t) * (n * Nv + 1));
    float* hp = malloc(sizeof(float) * ((size_t)n * Nv * d + 1));
    float* out = malloc(sizeof(float) * n * N * d);
    CHECK(vo_quantize(x, n, N, K, d, bits, group, Nv, codes, params, range, mse, hp_idx));
    CHECK(vo_dequantize(codes, params, hp, hp_idx, n, N, K, d, bits, group, Nv, 0, out));
    free(x); free(codes); free(params); free(range); free(mse); free(hp_idx); free(hp); free(out);
}

int main(void) {
    round_case(2, 2, 8, 128, 32, 64, 8, 7);        /* the tiny configuration */
    round_case(3, 4, 5, 200, 23, 64, 0, 1);        /* ragged, no reservation, no pooling */
    round_case(1, 5, 3, 96, 40, 128, 56, 31);      /* B = K - N_v: nothing sampled */
    round_case(2, 1, 1, 64, 1, 64, 63, 3);         /* B = 1, N_v + B = K */
    quant_case(2, 100, 8, 64, 4, 32, 10);
    quant_case(1, 64, 4, 128, 2, 128, 0);
    quant_case(1, 33, 3, 64, 8, 64, 33);
    float u[1024], e[1024];
    for (int i = 0; i < 1024; ++i) u[i] = (float)((2.0 * (i * 8191 % 8388608) + 1.0) / 16777216.0);
    vo_neglog_n(u, e, 1024);
    printf("ok\n");
    return 0;
}
