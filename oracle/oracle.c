/*
 * oracle.c -- plain, slow CPU reference of the mixed-precision MoE expert-FFN
 * hot path of DynaMo (arXiv 2503.21135).
 *
 * TEST INFRASTRUCTURE ONLY.  This file is compiled with gcc alone (no HIP),
 * shares no code with the GPU library, and is called only by the tests, the
 * smoke check and the CPU-baseline leg of the benchmark.  The product path
 * never calls it.
 *
 * Every function states the passage of the paper, or the reading of it, that
 * it follows.  Floating point is IEEE binary64 unless a step is defined in
 * fp32 (the router, whose integer decision both sides must take in the same
 * precision) or on a 16-bit format (the fp16 scale, the bf16 hidden
 * activation).  Build flags: -O2 -ffp-contract=off, no fast-math.
 *
 * Pins: every function here is checked by the -m "not gpu" tests against
 * closed forms, invariants, special cases that reduce to a library routine,
 * or brute force.  See the header comment of the tests for the list.
 */
#include <math.h>
#ifdef _OPENMP
#include <omp.h>
#endif
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#define ORC_OK 0
#define ORC_ERR_ARG (-1)
#define ORC_ERR_BITS (-2)
#define ORC_ERR_SLOT (-5)
#define ORC_ERR_RANGE (-6)

/* Threads the OpenMP loops below use. */
int oracle_num_threads(void) {
#ifdef _OPENMP
  return omp_get_max_threads();
#else
  return 1;
#endif
}

/* Sets the threads of later OpenMP loops (n >= 1); for timing only. */
void oracle_set_num_threads(int n) {
#ifdef _OPENMP
  if (n >= 1) omp_set_num_threads(n);
#else
  (void)n;
#endif
}

/* ------------------------------------------------------------------------ */
/* 16-bit float formats, written from the IEEE 754 definitions.             */
/* ------------------------------------------------------------------------ */

/* Value of an IEEE binary16 bit pattern. */
double oracle_fp16_value(uint16_t h) {
  int sign = h >> 15, ex = (h >> 10) & 31, man = h & 1023;
  double v;
  if (ex == 0)
    v = ldexp((double)man, -24);
  else if (ex == 31)
    v = man ? NAN : INFINITY;
  else
    v = ldexp((double)(1024 + man), ex - 25);
  return sign ? -v : v;
}

/*
 * The smallest binary16 value >= s, for s > 0 (returns the +inf pattern when
 * it exceeds 65504).  Arithmetic form: with s in [2^E, 2^(E+1)), the binary16
 * grid there has spacing 2^(E-10) (2^-24 below the normal range), so the
 * answer is ceil(s / spacing) * spacing.
 */
uint16_t oracle_fp16_round_up(double s) {
  int e;
  frexp(s, &e);
  int E = e - 1; /* s in [2^E, 2^(E+1)) */
  if (E < -14) {
    double k = ceil(ldexp(s, 24)); /* multiples of 2^-24; k <= 1024 */
    return (uint16_t)k;            /* k = 1024 is the pattern of 2^-14 */
  }
  double k = ceil(s / ldexp(1.0, E - 10)); /* in [1024, 2048] */
  if (k >= 2048.0) {
    k = 1024.0;
    E += 1;
  }
  if (E > 15) return 0x7C00;
  return (uint16_t)(((E + 15) << 10) | ((int)k - 1024));
}

/* binary16 pattern of a small non-negative integer (exact). */
static uint16_t fp16_of_int(int z) {
  if (z == 0) return 0;
  int E = 0;
  while ((z >> (E + 1)) != 0) E++;
  return (uint16_t)(((E + 15) << 10) | ((z << (10 - E)) - 1024));
}

/* Value of a bfloat16 bit pattern: the top half of a binary32. */
double oracle_bf16_value(uint16_t b) {
  uint32_t u = (uint32_t)b << 16;
  float f;
  memcpy(&f, &u, 4);
  return (double)f;
}

/* Nearest bfloat16 to v, ties to even (one rounding from binary64). */
uint16_t oracle_bf16_round(double v) {
  float f;
  uint32_t u;
  if (v == 0.0 || !isfinite(v)) {
    f = (float)v;
    memcpy(&u, &f, 4);
    return (uint16_t)(u >> 16);
  }
  int e;
  frexp(v, &e);
  int E = e - 1;
  if (E < -126) E = -126; /* bf16 subnormal spacing 2^-133 */
  double ulp = ldexp(1.0, E - 7);
  double q = rint(v / ulp); /* 8 significant bits, ties to even */
  f = (float)(q * ulp);     /* exact, or +-inf past the range */
  memcpy(&u, &f, 4);
  return (uint16_t)(u >> 16);
}

/*
 * The unquantized 16-bit reference weights (the "FP16 model" the paper's
 * speedup is measured against, Sec. VI-C, kept here in bfloat16 like the
 * activations): each fp32 weight rounded to the nearest bfloat16, as binary64.
 */
void oracle_bf16_weights(const float* w, int64_t n, double* out) {
#pragma omp parallel for schedule(static)
  for (int64_t i = 0; i < n; i++) out[i] = oracle_bf16_value(oracle_bf16_round((double)w[i]));
}

/* ------------------------------------------------------------------------ */
/* Quantization (Sec. IV-A: expert-level mixed precision, uniform quantizer)  */
/* ------------------------------------------------------------------------ */

/*
 * Asymmetric uniform quantization of rows of w, group by group along K.
 * The paper fixes only "uniform quantization" at the expert's precision
 * (Sec. IV-A); the reading used here: the range [mn, mx] always contains 0,
 * the scale is the binary64 quotient (mx - mn)/(2^b - 1) rounded up to
 * binary16 so that the grid spans the range, the zero point is the integer
 * rint(-mn/s16), codes are rint(w/s16) + z clamped to [0, 2^b - 1].
 *
 *   w   [R][ld_w] fp32;  q [R][K] codes;  s16, z16 [R][K/group] fp16 patterns.
 * Returns ORC_ERR_RANGE when a scale overflows binary16 (its group is still
 * written, with an infinite scale).
 */
int oracle_quantize(const float* w, int64_t ld_w, int R, int K, int bits,
                    int group, uint8_t* q, uint16_t* s16, uint16_t* z16) {
  if (!(bits == 2 || bits == 3 || bits == 4 || bits == 6 || bits == 8)) return ORC_ERR_BITS;
  if (R < 0 || K <= 0 || group <= 0 || K % group) return ORC_ERR_ARG;
  const int qmax = (1 << bits) - 1;
  const int G = K / group;
  int status = ORC_OK;
#pragma omp parallel for schedule(static) reduction(min : status)
  for (int r = 0; r < R; r++) {
    for (int j = 0; j < G; j++) {
      const float* wg = w + (int64_t)r * ld_w + (int64_t)j * group;
      double mn = 0.0, mx = 0.0;
      for (int i = 0; i < group; i++) {
        double v = (double)wg[i];
        if (v < mn) mn = v;
        if (v > mx) mx = v;
      }
      double s = (mx - mn) / (double)qmax;
      uint16_t sb = (s == 0.0) ? (uint16_t)0x3C00 : oracle_fp16_round_up(s);
      if (sb == 0x7C00) status = ORC_ERR_RANGE;
      double sf = oracle_fp16_value(sb);
      int z = (int)rint(-mn / sf);
      if (z < 0) z = 0; /* -0.0 and the overflow case */
      s16[(int64_t)r * G + j] = sb;
      z16[(int64_t)r * G + j] = fp16_of_int(z);
      for (int i = 0; i < group; i++) {
        double t = rint((double)wg[i] / sf) + (double)z;
        if (t < 0.0) t = 0.0;
        if (t > (double)qmax) t = (double)qmax;
        q[(int64_t)r * K + (int64_t)j * group + i] = (uint8_t)t;
      }
    }
  }
  return status;
}

/* Dequantized weight s16 * (q - z) for every element (exact in binary64). */
void oracle_dequant(const uint8_t* q, const uint16_t* s16, const uint16_t* z16,
                    int R, int K, int group, double* w_hat) {
  const int G = K / group;
#pragma omp parallel for schedule(static)
  for (int r = 0; r < R; r++)
    for (int c = 0; c < K; c++) {
      int j = c / group;
      double sf = oracle_fp16_value(s16[(int64_t)r * G + j]);
      double z = oracle_fp16_value(z16[(int64_t)r * G + j]);
      w_hat[(int64_t)r * K + c] = sf * ((double)q[(int64_t)r * K + c] - z);
    }
}

/* ------------------------------------------------------------------------ */
/* Packing (Sec. V-B: several low-bit codes in one 32-bit word)              */
/* ------------------------------------------------------------------------ */

/* Bit position of local code i inside a word of the b-bit half-split order:
 * even codes fill the low half-word, odd codes the high half-word. */
static int halfsplit_pos(int i, int b) { return (i >> 1) * b + 16 * (i & 1); }

/* Pack codes q[R][K] into words[R][K*bits/32] in the layout the library's
 * header defines. */
int oracle_pack(const uint8_t* q, int R, int K, int bits, uint32_t* words) {
  if (!(bits == 2 || bits == 3 || bits == 4 || bits == 6 || bits == 8)) return ORC_ERR_BITS;
  if (K % 32) return ORC_ERR_ARG;
  const int W = K * bits / 32;
  for (int r = 0; r < R; r++) {
    const uint8_t* qr = q + (int64_t)r * K;
    uint32_t* wr = words + (int64_t)r * W;
    memset(wr, 0, sizeof(uint32_t) * W);
    if (bits == 6) {
      /* per block of 32 codes: bits 0..3 of code i in word i/8 (4-bit
       * order), bits 4..5 in word 4 + i/16 (2-bit order) */
      for (int blk = 0; blk < K / 32; blk++)
        for (int i = 0; i < 32; i++) {
          uint32_t code = qr[blk * 32 + i];
          wr[6 * blk + (i >> 3)] |= (code & 15u) << halfsplit_pos(i & 7, 4);
          wr[6 * blk + 4 + (i >> 4)] |= (code >> 4) << halfsplit_pos(i & 15, 2);
        }
    } else if (bits != 3) {
      const int per = 32 / bits;
      for (int c = 0; c < K; c++)
        wr[c / per] |= (uint32_t)qr[c] << halfsplit_pos(c % per, bits);
    } else {
      for (int blk = 0; blk < K / 32; blk++) {
        for (int i = 0; i < 32; i++) {
          uint32_t code = qr[blk * 32 + i];
          wr[3 * blk + (i >> 4)] |= (code & 3u) << halfsplit_pos(i & 15, 2);
          wr[3 * blk + 2] |= ((code >> 2) & 1u) << halfsplit_pos(i, 1);
        }
      }
    }
  }
  return ORC_OK;
}

/* Inverse of oracle_pack. */
int oracle_unpack(const uint32_t* words, int R, int K, int bits, uint8_t* q) {
  if (!(bits == 2 || bits == 3 || bits == 4 || bits == 6 || bits == 8)) return ORC_ERR_BITS;
  if (K % 32) return ORC_ERR_ARG;
  const int W = K * bits / 32;
  for (int r = 0; r < R; r++) {
    const uint32_t* wr = words + (int64_t)r * W;
    uint8_t* qr = q + (int64_t)r * K;
    if (bits == 6) {
      for (int blk = 0; blk < K / 32; blk++)
        for (int i = 0; i < 32; i++) {
          uint32_t lo = (wr[6 * blk + (i >> 3)] >> halfsplit_pos(i & 7, 4)) & 15u;
          uint32_t hi = (wr[6 * blk + 4 + (i >> 4)] >> halfsplit_pos(i & 15, 2)) & 3u;
          qr[blk * 32 + i] = (uint8_t)(lo | (hi << 4));
        }
    } else if (bits != 3) {
      const int per = 32 / bits;
      const uint32_t mask = (1u << bits) - 1u;
      for (int c = 0; c < K; c++)
        qr[c] = (uint8_t)((wr[c / per] >> halfsplit_pos(c % per, bits)) & mask);
    } else {
      for (int blk = 0; blk < K / 32; blk++)
        for (int i = 0; i < 32; i++) {
          uint32_t lo = (wr[3 * blk + (i >> 4)] >> halfsplit_pos(i & 15, 2)) & 3u;
          uint32_t hi = (wr[3 * blk + 2] >> halfsplit_pos(i, 1)) & 1u;
          qr[blk * 32 + i] = (uint8_t)(lo | (hi << 2));
        }
    }
  }
  return ORC_OK;
}

/* ------------------------------------------------------------------------ */
/* Router (Sec. II-A: a fixed number of experts selected per token)           */
/* ------------------------------------------------------------------------ */

/*
 * Exponential for x <= 0, defined so that both implementations produce the
 * same fp32 bits: 0 below -80; n = rint(x * fl(log2 e)); r = x - n ln2 by a
 * Cody-Waite reduction with ln2 = LN2_HI + LN2_LO, LN2_HI = 2839/4096 (ln2 to
 * 12 significant bits, so n*LN2_HI is exact for |n| < 2^12) and LN2_LO its
 * fp32 remainder; e^r by the degree-7 Taylor polynomial with coefficients
 * fl(1/i!) evaluated by Horner's rule in fmaf; result scaled by 2^n.
 */
float oracle_cexp(float x) {
  if (x < -80.0f) return 0.0f;
  const float log2e = (float)1.4426950408889634;
  const float ln2_hi = 2839.0f / 4096.0f;
  const float ln2_lo = (float)(0.69314718055994531 - 2839.0 / 4096.0);
  float n = rintf(x * log2e);
  float r = fmaf(-n, ln2_hi, x);
  r = fmaf(-n, ln2_lo, r);
  double fact = 1.0;
  float c[8];
  for (int i = 0; i < 8; i++) {
    if (i > 0) fact *= (double)i;
    c[i] = (float)(1.0 / fact);
  }
  float p = c[7];
  for (int i = 6; i >= 0; i--) p = fmaf(p, r, c[i]);
  return ldexpf(p, (int)n);
}

/* A logit as the top-k order sees it: NaN in the place of -inf. */
static float rank_key(float v) { return isnan(v) ? -INFINITY : v; }

/*
 * Router logits, top-k and combine weights.  The summation order of the
 * logit is fixed (the paper is silent; both implementations follow it so the
 * top-k decision is taken on identical fp32 values): 64 partial sums, partial
 * l accumulates fmaf over columns l, l+64, ... in increasing order, then a
 * halving tree partial[l] += partial[l+off], off = 32..1; then + bias.
 * Top-k by (logit descending, index ascending); weights are the softmax over
 * the k selected logits (weights sum to 1).  The order is total over numbers
 * only, so a NaN logit takes the place of -inf in the selection and in the
 * softmax: the k picks are always k distinct experts.
 *
 *   x [T][d] bf16 patterns; Wr [E][d]; bias [E] or NULL;
 *   logits [T][E] (output, may be NULL); ids [T][k]; w [T][k].
 */
int oracle_route(const uint16_t* x, int T, int d, const float* Wr,
                 const float* bias, int E, int k, float* logits, int32_t* ids,
                 float* w) {
  if (T < 0 || d <= 0 || d % 64 || E <= 0 || k < 1 || k > E) return ORC_ERR_ARG;
  float* lg_all = (float*)malloc(sizeof(float) * (size_t)(T > 0 ? T : 1) * E);
  if (!lg_all) return ORC_ERR_ARG;
#pragma omp parallel for schedule(static)
  for (int t = 0; t < T; t++) {
    float* lg = lg_all + (int64_t)t * E;
    for (int e = 0; e < E; e++) {
      float acc[64];
      for (int l = 0; l < 64; l++) acc[l] = 0.0f;
      for (int c = 0; c < d; c++) {
        float xv = (float)oracle_bf16_value(x[(int64_t)t * d + c]);
        acc[c % 64] = fmaf(xv, Wr[(int64_t)e * d + c], acc[c % 64]);
      }
      for (int off = 32; off >= 1; off >>= 1)
        for (int l = 0; l < off; l++) acc[l] = acc[l] + acc[l + off];
      lg[e] = bias ? acc[0] + bias[e] : acc[0];
    }
    /* selection of the k best, ties to the lower index */
    int32_t* id = ids + (int64_t)t * k;
    for (int j = 0; j < k; j++) {
      int best = -1;
      for (int e = 0; e < E; e++) {
        int taken = 0;
        for (int i = 0; i < j; i++)
          if (id[i] == e) taken = 1;
        if (taken) continue;
        if (best < 0 || rank_key(lg[e]) > rank_key(lg[best])) best = e;
      }
      id[j] = best;
    }
    float ex[64];
    float m = rank_key(lg[id[0]]);
    float S = 0.0f;
    for (int j = 0; j < k; j++) {
      ex[j] = oracle_cexp(rank_key(lg[id[j]]) - m);
      S = S + ex[j];
    }
    for (int j = 0; j < k; j++) w[(int64_t)t * k + j] = ex[j] / S;
  }
  if (logits) memcpy(logits, lg_all, sizeof(float) * (size_t)T * E);
  free(lg_all);
  return ORC_OK;
}

/*
 * Token permutation into per-expert segments: segment e lists the tokens that
 * selected e in increasing token order; shared segment s lists all tokens.
 * offsets [E+S+1], perm [T*(k+S)], inv [T][k+S].
 */
int oracle_permute(const int32_t* ids, int T, int E, int k, int S,
                   int32_t* offsets, int32_t* perm, int32_t* inv) {
  if (T < 0 || E <= 0 || k < 1 || k > E || S < 0) return ORC_ERR_ARG;
  int32_t* cursor = (int32_t*)calloc((size_t)E + 1, sizeof(int32_t));
  if (!cursor) return ORC_ERR_ARG;
  for (int t = 0; t < T; t++)
    for (int j = 0; j < k; j++) {
      int e = ids[(int64_t)t * k + j];
      if (e < 0 || e >= E) {
        free(cursor);
        return ORC_ERR_ARG;
      }
      for (int i = 0; i < j; i++)
        if (ids[(int64_t)t * k + i] == e) {
          free(cursor);
          return ORC_ERR_ARG;
        }
      cursor[e]++;
    }
  offsets[0] = 0;
  for (int e = 0; e < E; e++) offsets[e + 1] = offsets[e] + cursor[e];
  for (int s = 0; s < S; s++) offsets[E + s + 1] = offsets[E + s] + T;
  for (int e = 0; e < E; e++) cursor[e] = offsets[e];
  for (int t = 0; t < T; t++)
    for (int j = 0; j < k; j++) {
      int e = ids[(int64_t)t * k + j];
      int p = cursor[e]++;
      perm[p] = t;
      inv[(int64_t)t * (k + S) + j] = p;
    }
  for (int s = 0; s < S; s++)
    for (int t = 0; t < T; t++) {
      int p = offsets[E + s] + t;
      perm[p] = t;
      inv[(int64_t)t * (k + S) + k + s] = p;
    }
  free(cursor);
  return ORC_OK;
}

/* ------------------------------------------------------------------------ */
/* Channel switch (Sec. IV-B replacement by index match; Sec. V-A headers)    */
/* ------------------------------------------------------------------------ */

/*
 * row_slot[E][R] = -1 everywhere, then row_slot[hdr expert][hdr row] = s for
 * each slot s listed.  Rejects slots out of range, repeated slots and two
 * slots naming the same row.
 */
int oracle_switch(const int32_t* hdr, int n_slots, int E, int R,
                  const int32_t* slots_on, int n_on, int32_t* row_slot) {
  if (n_on < 0 || n_on > n_slots) return ORC_ERR_SLOT;
  for (int64_t i = 0; i < (int64_t)E * R; i++) row_slot[i] = -1;
  for (int i = 0; i < n_on; i++) {
    int s = slots_on[i];
    if (s < 0 || s >= n_slots) return ORC_ERR_SLOT;
    int e = hdr[2 * s], r = hdr[2 * s + 1];
    if (e < 0 || e >= E || r < 0 || r >= R) return ORC_ERR_SLOT;
    if (row_slot[(int64_t)e * R + r] != -1) return ORC_ERR_SLOT;
    row_slot[(int64_t)e * R + r] = s;
  }
  return ORC_OK;
}

/* ------------------------------------------------------------------------ */
/* Expert FFN and combine                                                    */
/* ------------------------------------------------------------------------ */

/*
 * SiLU-gated expert FFN (the paper never writes the expert FFN out; the
 * evaluated MoE models use this form) on effective dequantized weights
 * Wg, Wu [f][d], Wd [d][f] (binary64):
 *   g = Wg x, u = Wu x, h = silu(g) u, o = Wd h.
 * round_h != 0 rounds h to bfloat16 (round to nearest even) before the down
 * projection: the paper feeds 16-bit activations to the matrix cores
 * (Sec. V-B), bf16 on this hardware.  Accumulation in binary64.
 *   x [T][d] bf16 patterns; rows[n] token indices; o [n][d].
 */
void oracle_expert_ffn(const double* Wg, const double* Wu, const double* Wd,
                       int f, int d, const uint16_t* x, const int32_t* rows,
                       int n, int round_h, double* o) {
#pragma omp parallel for schedule(dynamic, 1)
  for (int i = 0; i < n; i++) {
    double* xv = (double*)malloc(sizeof(double) * d);
    double* hv = (double*)malloc(sizeof(double) * f);
    const uint16_t* xr = x + (int64_t)rows[i] * d;
    for (int c = 0; c < d; c++) xv[c] = oracle_bf16_value(xr[c]);
    for (int j = 0; j < f; j++) {
      double g = 0.0, u = 0.0;
      const double* wg = Wg + (int64_t)j * d;
      const double* wu = Wu + (int64_t)j * d;
      for (int c = 0; c < d; c++) {
        g += wg[c] * xv[c];
        u += wu[c] * xv[c];
      }
      double h = g / (1.0 + exp(-g)) * u;
      if (round_h) h = oracle_bf16_value(oracle_bf16_round(h));
      hv[j] = h;
    }
    for (int c = 0; c < d; c++) {
      double acc = 0.0;
      const double* wd = Wd + (int64_t)c * f;
      for (int j = 0; j < f; j++) acc += wd[j] * hv[j];
      o[(int64_t)i * d + c] = acc;
    }
    free(xv);
    free(hv);
  }
}

/*
 * Un-permute and combine: y[t] = sum_j w[t][j] o[inv[t][j]] + sum_s
 * o[inv[t][k+s]] (shared experts with weight 1), binary64.
 */
void oracle_combine(const double* o, const int32_t* inv, const float* w, int T,
                    int k, int S, int d, double* y) {
#pragma omp parallel for schedule(static)
  for (int t = 0; t < T; t++)
    for (int c = 0; c < d; c++) {
      double acc = 0.0;
      for (int j = 0; j < k; j++)
        acc += (double)w[(int64_t)t * k + j] *
               o[(int64_t)inv[(int64_t)t * (k + S) + j] * d + c];
      for (int s = 0; s < S; s++)
        acc += o[(int64_t)inv[(int64_t)t * (k + S) + k + s] * d + c];
      y[(int64_t)t * d + c] = acc;
    }
}
