/*
 * oracle_sanitize_main.c -- a driver that runs the oracle's pins on tiny inputs
 * in one process, so that the oracle can be built with the address and
 * undefined-behaviour sanitizers (tests/test_oracle_sanitize.py).  Exits 0
 * when every check holds; a sanitizer finding aborts the process.
 */
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

double oracle_fp16_value(uint16_t h);
uint16_t oracle_fp16_round_up(double s);
double oracle_bf16_value(uint16_t b);
uint16_t oracle_bf16_round(double v);
int oracle_quantize(const float* w, int64_t ld_w, int R, int K, int bits, int group, uint8_t* q,
                    uint16_t* s16, uint16_t* z16);
void oracle_dequant(const uint8_t* q, const uint16_t* s16, const uint16_t* z16, int R, int K,
                    int group, double* w_hat);
int oracle_pack(const uint8_t* q, int R, int K, int bits, uint32_t* words);
int oracle_unpack(const uint32_t* words, int R, int K, int bits, uint8_t* q);
float oracle_cexp(float x);
int oracle_route(const uint16_t* x, int T, int d, const float* Wr, const float* bias, int E,
                 int k, float* logits, int32_t* ids, float* w);
int oracle_permute(const int32_t* ids, int T, int E, int k, int S, int32_t* offsets,
                   int32_t* perm, int32_t* inv);
int oracle_switch(const int32_t* hdr, int n_slots, int E, int R, const int32_t* slots_on,
                  int n_on, int32_t* row_slot);
void oracle_expert_ffn(const double* Wg, const double* Wu, const double* Wd, int f, int d,
                       const uint16_t* x, const int32_t* rows, int n, int round_h, double* o);
void oracle_combine(const double* o, const int32_t* inv, const float* w, int T, int k, int S,
                    int d, double* y);

static int failures = 0;
#define CHECK(c, ...)                                   \
  do {                                                  \
    if (!(c)) {                                         \
      fprintf(stderr, "FAIL %s:%d: ", __FILE__, __LINE__); \
      fprintf(stderr, __VA_ARGS__);                     \
      fprintf(stderr, "\n");                            \
      failures++;                                       \
    }                                                   \
  } while (0)

/* xorshift64* -- the driver's own inputs */
static uint64_t rs = 0x9E3779B97F4A7C15ull;
static uint64_t rnd(void) {
  rs ^= rs >> 12;
  rs ^= rs << 25;
  rs ^= rs >> 27;
  return rs * 2685821657736338717ull;
}
static double unif(void) { return (double)(rnd() >> 11) / 9007199254740992.0; }
static double gauss(void) {
  double u = unif() + 1e-300, v = unif();
  return sqrt(-2.0 * log(u)) * cos(6.283185307179586 * v);
}

static void check_fp16_round_up(void) {
  for (int i = 0; i < 2000; i++) {
    double s = ldexp(0.5 + unif(), (int)(rnd() % 40) - 30);
    uint16_t h = oracle_fp16_round_up(s);
    if (h == 0x7C00) continue;
    CHECK(oracle_fp16_value(h) >= s, "round up below s");
    if (h > 1) CHECK(oracle_fp16_value((uint16_t)(h - 1)) < s, "not the smallest fp16 >= s");
  }
}

static void check_quantize_pack(void) {
  const int bitsv[5] = {2, 3, 4, 6, 8};
  const int R = 6, K = 256, g = 128, G = K / g;
  float* w = malloc(sizeof(float) * R * K);
  uint8_t* q = malloc(R * K);
  uint8_t* q2 = malloc(R * K);
  uint8_t* qin = malloc(R * K);
  uint16_t s16[6 * 2], z16[6 * 2], sin[6 * 2];
  int zin[6 * 2];
  double* wh = malloc(sizeof(double) * R * K);
  uint32_t* words = malloc(sizeof(uint32_t) * R * K * 8 / 32);
  for (int bi = 0; bi < 5; bi++) {
    const int b = bitsv[bi], qmax = (1 << b) - 1;
    /* exact recovery: w = s (q - z) with codes 0 and qmax present */
    for (int r = 0; r < R; r++)
      for (int j = 0; j < G; j++) {
        sin[r * G + j] = oracle_fp16_round_up(ldexp(1.0 + unif(), -10 - (int)(rnd() % 4)));
        zin[r * G + j] = (int)(rnd() % (uint64_t)(qmax + 1));
        for (int i = 0; i < g; i++) qin[r * K + j * g + i] = (uint8_t)(rnd() % (uint64_t)(qmax + 1));
        qin[r * K + j * g + (int)(rnd() % g)] = 0;
        int p;
        do p = (int)(rnd() % g); while (qin[r * K + j * g + p] == 0);
        qin[r * K + j * g + p] = (uint8_t)qmax;
        for (int i = 0; i < g; i++)
          w[r * K + j * g + i] = (float)(oracle_fp16_value(sin[r * G + j]) *
                                         ((double)qin[r * K + j * g + i] - zin[r * G + j]));
      }
    CHECK(oracle_quantize(w, K, R, K, b, g, q, s16, z16) == 0, "quantize status");
    CHECK(memcmp(q, qin, R * K) == 0, "exact recovery of codes at %d bits", b);
    for (int i = 0; i < R * G; i++) {
      CHECK(s16[i] == sin[i], "exact recovery of scale at %d bits", b);
      CHECK(oracle_fp16_value(z16[i]) == zin[i], "exact recovery of zero at %d bits", b);
    }
    /* error bound on random weights */
    for (int i = 0; i < R * K; i++) w[i] = (float)(0.02 * gauss());
    CHECK(oracle_quantize(w, K, R, K, b, g, q, s16, z16) == 0, "quantize status");
    oracle_dequant(q, s16, z16, R, K, g, wh);
    for (int r = 0; r < R; r++)
      for (int c = 0; c < K; c++)
        CHECK(fabs((double)w[r * K + c] - wh[r * K + c]) <= oracle_fp16_value(s16[r * G + c / g]) / 2,
              "|w - w_hat| > s/2 at %d bits", b);
    /* pack / unpack round trip */
    CHECK(oracle_pack(q, R, K, b, words) == 0, "pack status");
    CHECK(oracle_unpack(words, R, K, b, q2) == 0, "unpack status");
    CHECK(memcmp(q, q2, R * K) == 0, "pack round trip at %d bits", b);
  }
  free(w); free(q); free(q2); free(qin); free(wh); free(words);
}

static void check_cexp(void) {
  for (int i = 0; i <= 20000; i++) {
    float x = (float)(-80.0 * i / 20000.0);
    double ref = exp((double)x), v = oracle_cexp(x);
    CHECK(fabs(v - ref) <= 2.0 * ldexp(1.0, ilogb(ref) - 23), "cexp(%g) off by more than 2 ulp", x);
  }
}

static void check_layer(void) {
  enum { T = 9, d = 64, f = 64, E = 4, k = 2, S = 1 };
  uint16_t x[T * d];
  float Wr[E * d], logits[T * E], tw[T * k];
  int32_t ids[T * k], off[E + S + 1], perm[T * (k + S)], inv[T * (k + S)];
  for (int i = 0; i < T * d; i++) x[i] = oracle_bf16_round(gauss());
  for (int i = 0; i < E * d; i++) Wr[i] = (float)(0.1 * gauss());
  CHECK(oracle_route(x, T, d, Wr, NULL, E, k, logits, ids, tw) == 0, "route status");
  for (int t = 0; t < T; t++) {
    double sw = 0;
    for (int j = 0; j < k; j++) {
      sw += tw[t * k + j];
      if (j) CHECK(logits[t * E + ids[t * k + j - 1]] >= logits[t * E + ids[t * k + j]], "top-k order");
    }
    CHECK(fabs(sw - 1.0) <= 2.0 * k * ldexp(1.0, -24), "weights sum to 1");
  }
  CHECK(oracle_permute(ids, T, E, k, S, off, perm, inv) == 0, "permute status");
  CHECK(off[E + S] == T * (k + S), "segments cover every row");
  for (int t = 0; t < T; t++)
    for (int j = 0; j < k + S; j++) CHECK(perm[inv[t * (k + S) + j]] == t, "inverse permutation");
  /* switch: a slot list and a duplicated one */
  int32_t hdr[6] = {0, 1, 2, 3, 0, 1}, on[2] = {0, 1}, dup[2] = {0, 2}, row_slot[E * 8];
  CHECK(oracle_switch(hdr, 3, E, 8, on, 2, row_slot) == 0, "switch status");
  CHECK(row_slot[1] == 0 && row_slot[2 * 8 + 3] == 1 && row_slot[0] == -1, "switch table");
  CHECK(oracle_switch(hdr, 3, E, 8, dup, 2, row_slot) != 0, "two slots naming one row");
  /* expert FFN and combine against a direct loop */
  double* W = malloc(sizeof(double) * 3 * f * d * (E + S));
  double* o = malloc(sizeof(double) * T * (k + S) * d);
  double y[T * d];
  for (int i = 0; i < 3 * f * d * (E + S); i++) W[i] = 0.05 * gauss();
  for (int e = 0; e < E + S; e++) {
    const double* Wg = W + (size_t)e * 3 * f * d;
    int n = off[e + 1] - off[e];
    oracle_expert_ffn(Wg, Wg + f * d, Wg + 2 * f * d, f, d, x, perm + off[e], n, 0, o + (size_t)off[e] * d);
    for (int p = off[e]; p < off[e + 1]; p++) {
      double h[f];
      for (int i = 0; i < f; i++) {
        double gg = 0, uu = 0;
        for (int c = 0; c < d; c++) {
          gg += Wg[i * d + c] * oracle_bf16_value(x[perm[p] * d + c]);
          uu += Wg[f * d + i * d + c] * oracle_bf16_value(x[perm[p] * d + c]);
        }
        h[i] = gg / (1.0 + exp(-gg)) * uu;
      }
      for (int c = 0; c < d; c++) {
        double acc = 0;
        for (int i = 0; i < f; i++) acc += Wg[2 * f * d + c * f + i] * h[i];
        CHECK(fabs(acc - o[(size_t)p * d + c]) <= 1e-12 * (1.0 + fabs(acc)), "expert FFN");
      }
    }
  }
  oracle_combine(o, inv, tw, T, k, S, d, y);
  for (int t = 0; t < T; t++)
    for (int c = 0; c < d; c++) {
      double acc = 0;
      for (int j = 0; j < k; j++) acc += tw[t * k + j] * o[(size_t)inv[t * (k + S) + j] * d + c];
      acc += o[(size_t)inv[t * (k + S) + k] * d + c];
      CHECK(fabs(acc - y[t * d + c]) <= 1e-12 * (1.0 + fabs(acc)), "combine");
    }
  free(W);
  free(o);
}

int main(void) {
  check_fp16_round_up();
  check_quantize_pack();
  check_cexp();
  check_layer();
  if (failures) {
    fprintf(stderr, "%d checks failed\n", failures);
    return 1;
  }
  printf("oracle pins under the sanitizers: ok\n");
  return 0;
}
