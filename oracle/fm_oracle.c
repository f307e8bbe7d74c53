/*
 * fm_oracle.c -- plain, slow CPU oracle for low-precision evaluation of a
 * bilinear fast matrix multiplication scheme.
 *
 * TEST INFRASTRUCTURE ONLY.  Only the test suite, the smoke check and the
 * benchmark's CPU-baseline leg may load this file's library.  The product
 * path (the HIP library) never calls, links or executes anything here, and
 * this file shares no code, header, table or helper with it.
 *
 * What it computes follows the paper:
 *   - the bilinear form, eq. (1) of Sec. 2.1: block sums of A and of B, R
 *     block products M_r, and the reconstruction C_ij = sum_r w_{r,ij} M_r;
 *   - the FP8 schedule of App. B (criteria and operands paragraph): block sums
 *     rounded to FP8 (e4m3) before multiplying, products and their
 *     combination carried out in fp32;
 *   - the error measure of App. B / App. F: relative error in the Frobenius
 *     norm against a float64 reference.
 *   - the finer scale granularity of App. B.1's synthetic matrices: one scale
 *     per row of each block sum of A and per column of each block sum of B.
 * Choices the paper leaves open (combination order, one scale per whole
 * block-sum tensor by default, exact block-product accumulation rounded once
 * to fp32) are the readings listed in the design notes; each function states
 * its own.
 *
 * Arithmetic rules, so that every step can be checked by eye:
 *   - fp32 steps use C float arithmetic (SSE, round-to-nearest-even,
 *     subnormals kept); fused multiply-adds are explicit fmaf() calls and the
 *     file is compiled with -ffp-contract=off so no other contraction occurs;
 *   - block products are accumulated exactly in integers and rounded once.
 */
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

/* Host allocation that ends the process with a message when it fails (the  */
/* oracle's buffers are test-sized; a failure is a broken test set-up).      */
static void* orc_alloc(size_t n) {
  void* p = malloc(n ? n : 1);
  if (!p) {
    fprintf(stderr, "oracle: out of host memory (%zu bytes)\n", n);
    abort();
  }
  return p;
}

/* ------------------------------------------------------------------------ */
/* FP8 formats (OCP 8-bit floating point: E4M3FN and E5M2).                  */
/* The paper rounds block sums to e4m3 (App. B); E5M2 is the second operand  */
/* format of the Laderman workload.                                          */
/* ------------------------------------------------------------------------ */

#define ORC_E4M3 0
#define ORC_E5M2 1

typedef struct {
  int exp_bits, man_bits, bias;
  double max_finite;  /* largest finite magnitude */
} fp8_format;

static fp8_format fmt_of(int fmt) {
  fp8_format f;
  if (fmt == ORC_E4M3) {
    f.exp_bits = 4; f.man_bits = 3; f.bias = 7; f.max_finite = 448.0;
  } else {
    f.exp_bits = 5; f.man_bits = 2; f.bias = 15; f.max_finite = 57344.0;
  }
  return f;
}

double orc_fp8_max(int fmt) { return fmt_of(fmt).max_finite; }

/* Value of an 8-bit code, by the format's definition.  NaN codes give NaN;
 * E5M2 infinities give +-inf. */
double orc_fp8_decode(uint8_t code, int fmt) {
  fp8_format f = fmt_of(fmt);
  int sign = code >> 7;
  int e = (code >> f.man_bits) & ((1 << f.exp_bits) - 1);
  int m = code & ((1 << f.man_bits) - 1);
  double v;
  if (fmt == ORC_E4M3 && e == 15 && m == 7) return NAN;
  if (fmt == ORC_E5M2 && e == 31) return m ? NAN : (sign ? -INFINITY : INFINITY);
  if (e == 0) /* subnormal: m * 2^(1 - bias - man_bits) */
    v = ldexp((double)m, 1 - f.bias - f.man_bits);
  else
    v = ldexp(1.0 + (double)m / (double)(1 << f.man_bits), e - f.bias);
  return sign ? -v : v;
}

/* Encode an fp32 value: round to the nearest representable value, ties to
 * the even significand, and saturate finite overflow to the largest finite
 * value ("satfinite").  NaN maps to the format's NaN code, infinities
 * saturate.  Works in double, where every step below is exact. */
uint8_t orc_fp8_encode(float x, int fmt) {
  fp8_format f = fmt_of(fmt);
  uint8_t sign = signbit(x) ? 0x80 : 0x00;
  double a = fabs((double)x);
  if (isnan(x)) return (uint8_t)(fmt == ORC_E4M3 ? 0x7F : 0x7E) | sign;
  double min_normal = ldexp(1.0, 1 - f.bias);
  double quantum; /* spacing of representable values around a */
  if (a < min_normal) {
    quantum = ldexp(1.0, 1 - f.bias - f.man_bits);
  } else {
    int e2;
    frexp(a, &e2); /* a = frac * 2^e2, frac in [0.5, 1) => binade 2^(e2-1) */
    quantum = ldexp(1.0, e2 - 1 - f.man_bits);
  }
  double n = a / quantum; /* exact: power-of-two divisor */
  double fl = floor(n);
  double rem = n - fl;
  double k;
  if (rem > 0.5) k = fl + 1.0;
  else if (rem < 0.5) k = fl;
  else k = (fmod(fl, 2.0) == 0.0) ? fl : fl + 1.0; /* tie: even multiple */
  double v = k * quantum;
  if (v > f.max_finite || isinf(x)) v = f.max_finite;
  /* bit pattern of v */
  if (v == 0.0) return sign;
  if (v < min_normal) {
    int m = (int)(v / ldexp(1.0, 1 - f.bias - f.man_bits));
    return sign | (uint8_t)m;
  }
  int e2;
  double fr = frexp(v, &e2); /* v = fr * 2^e2 */
  int e = e2 - 1 + f.bias;
  int m = (int)((fr * 2.0 - 1.0) * (double)(1 << f.man_bits));
  return sign | (uint8_t)(e << f.man_bits) | (uint8_t)m;
}

void orc_fp8_encode_array(const float* x, int64_t n, int fmt, uint8_t* out) {
  for (int64_t i = 0; i < n; ++i) out[i] = orc_fp8_encode(x[i], fmt);
}

void orc_fp8_decode_array(const uint8_t* c, int64_t n, int fmt, double* out) {
  for (int64_t i = 0; i < n; ++i) out[i] = orc_fp8_decode(c[i], fmt);
}

/* ------------------------------------------------------------------------ */
/* Block sums, eq. (1): T[x][y] = sum over blocks (p,q) with c[p*gc+q] != 0, */
/* in ascending row-major (p,q) order, of c * X_pq[x][y].                    */
/* X is rows x cols row-major, split into a gr x gc grid of contiguous       */
/* blocks of size (rows/gr) x (cols/gc).  The accumulator starts at +0.0f    */
/* and every step is one fmaf.  For A this is sum_{i,l} u_{r,il} A_il; for B */
/* it is sum_{l,j} v_{r,lj} B_lj, with T left in B's own orientation.        */
/* ------------------------------------------------------------------------ */
void orc_block_sum(const float* X, int rows, int cols, int gr, int gc,
                   const float* c, float* T) {
  int br = rows / gr, bc = cols / gc;
  int64_t n = (int64_t)br * bc;
  for (int64_t e = 0; e < n; ++e) T[e] = 0.0f;
  /* block by block, so every entry sees the nonzero coefficients in the   */
  /* order stated above; rows of T are independent                         */
  for (int p = 0; p < gr; ++p)
    for (int q = 0; q < gc; ++q) {
      float u = c[p * gc + q];
      if (u == 0.0f) continue;
#pragma omp parallel for schedule(static)
      for (int x = 0; x < br; ++x) {
        const float* src = X + (int64_t)(p * br + x) * cols + (int64_t)q * bc;
        float* dst = T + (int64_t)x * bc;
        for (int y = 0; y < bc; ++y) dst[y] = fmaf(u, src[y], dst[y]);
      }
    }
}

/* ------------------------------------------------------------------------ */
/* One scale per block-sum tensor.  amax = max |T|; if amax == 0 the scale   */
/* is 1 (an all-zero tensor, as the paper's quantizer sets d = 1 for an      */
/* all-zero group, App. D); otherwise r = FMAX/amax and d = amax/FMAX, each  */
/* one correctly rounded fp32 division.  Codes: encode(x * r), one fp32      */
/* multiplication then FP8 rounding.  Returns d, writes r to *r_out.         */
/* ------------------------------------------------------------------------ */
/* The scale rule for one group of values with largest magnitude amax. */
static float scale_from_amax(float amax, int fmt, float* r_out) {
  float fmax = (float)fmt_of(fmt).max_finite;
  if (amax == 0.0f) { *r_out = 1.0f; return 1.0f; }
  *r_out = fmax / amax;
  return amax / fmax;
}

float orc_tensor_scale(const float* T, int64_t n, int fmt, float* r_out) {
  float amax = 0.0f;
  /* the largest magnitude does not depend on the order it is searched in */
#pragma omp parallel for reduction(max : amax) schedule(static) if (n > 65536)
  for (int64_t i = 0; i < n; ++i) {
    float a = fabsf(T[i]);
    if (a > amax) amax = a;
  }
  return scale_from_amax(amax, fmt, r_out);
}

float orc_quantize_tensor(const float* T, int64_t n, int fmt, uint8_t* codes) {
  float r;
  float d = orc_tensor_scale(T, n, fmt, &r);
#pragma omp parallel for schedule(static) if (n > 65536)
  for (int64_t i = 0; i < n; ++i) {
    float y = T[i] * r;
    codes[i] = orc_fp8_encode(y, fmt);
  }
  return d;
}

/* ------------------------------------------------------------------------ */
/* Finer scale granularity (App. B.1, the synthetic-matrix form): one scale  */
/* for every row of a block sum of A and for every column of a block sum of  */
/* B, each with the same rule as a whole tensor.  T is rows x cols           */
/* row-major (B's block sums in B's orientation, bk x bc).                   */
/* ------------------------------------------------------------------------ */
void orc_quantize_rows(const float* T, int rows, int cols, int fmt, uint8_t* codes, float* d) {
  for (int x = 0; x < rows; ++x) {
    const float* t = T + (int64_t)x * cols;
    float r;
    d[x] = orc_tensor_scale(t, cols, fmt, &r);
    for (int y = 0; y < cols; ++y) codes[(int64_t)x * cols + y] = orc_fp8_encode(t[y] * r, fmt);
  }
}

void orc_quantize_cols(const float* T, int rows, int cols, int fmt, uint8_t* codes, float* d) {
  for (int z = 0; z < cols; ++z) {
    float amax = 0.0f;
    for (int y = 0; y < rows; ++y) {
      float a = fabsf(T[(int64_t)y * cols + z]);
      if (a > amax) amax = a;
    }
    float r;
    d[z] = scale_from_amax(amax, fmt, &r);
    for (int y = 0; y < rows; ++y)
      codes[(int64_t)y * cols + z] = orc_fp8_encode(T[(int64_t)y * cols + z] * r, fmt);
  }
}

/* ------------------------------------------------------------------------ */
/* Group scales (App. B.1, the models' schedule): the block sums of A get a  */
/* scale for every 128 consecutive entries of a row; those of B are first    */
/* rounded to bf16 and get a scale for every 128 x 128 block.  Each scale    */
/* follows the tensor rule on its group.  T is rows x cols row-major (B's    */
/* block sums in B's orientation, bk x bc).  d is group-major:               */
/* A: d[kg * rows + x]; B: d[kg * (cols / 128) + zb].                        */
/* ------------------------------------------------------------------------ */
#define ORC_GROUP 128

/* fp32 -> nearest bf16 (ties to even), returned as the fp32 it equals. */
float orc_bf16_round(float x) {
  uint32_t u;
  memcpy(&u, &x, 4);
  if ((u & 0x7f800000u) == 0x7f800000u) { /* Inf, NaN: truncate, keep NaN */
    uint32_t t = u & 0xffff0000u;
    if ((u & 0x007fffffu) && !(t & 0x007fffffu)) t |= 0x00400000u;
    memcpy(&x, &t, 4);
    return x;
  }
  uint32_t lsb = (u >> 16) & 1u;
  u = (u + 0x7fffu + lsb) & 0xffff0000u;
  memcpy(&x, &u, 4);
  return x;
}

void orc_quantize_row_groups(const float* T, int rows, int cols, int fmt, uint8_t* codes,
                             float* d) {
  int ng = cols / ORC_GROUP;
  for (int x = 0; x < rows; ++x)
    for (int kg = 0; kg < ng; ++kg) {
      const float* t = T + (int64_t)x * cols + (int64_t)kg * ORC_GROUP;
      float r;
      d[(int64_t)kg * rows + x] = orc_tensor_scale(t, ORC_GROUP, fmt, &r);
      for (int y = 0; y < ORC_GROUP; ++y)
        codes[(int64_t)x * cols + (int64_t)kg * ORC_GROUP + y] = orc_fp8_encode(t[y] * r, fmt);
    }
}

void orc_quantize_bf16_blocks(const float* T, int rows, int cols, int fmt, uint8_t* codes,
                              float* d) {
  int nkg = rows / ORC_GROUP, nzb = cols / ORC_GROUP;
  float* t = (float*)orc_alloc(sizeof(float) * (size_t)rows * cols);
  for (int64_t i = 0; i < (int64_t)rows * cols; ++i) t[i] = orc_bf16_round(T[i]);
  for (int kg = 0; kg < nkg; ++kg)
    for (int zb = 0; zb < nzb; ++zb) {
      float amax = 0.0f;
      for (int y = kg * ORC_GROUP; y < (kg + 1) * ORC_GROUP; ++y)
        for (int z = zb * ORC_GROUP; z < (zb + 1) * ORC_GROUP; ++z) {
          float a = fabsf(t[(int64_t)y * cols + z]);
          if (a > amax) amax = a;
        }
      float r;
      d[(int64_t)kg * nzb + zb] = scale_from_amax(amax, fmt, &r);
      for (int y = kg * ORC_GROUP; y < (kg + 1) * ORC_GROUP; ++y)
        for (int z = zb * ORC_GROUP; z < (zb + 1) * ORC_GROUP; ++z)
          codes[(int64_t)y * cols + z] = orc_fp8_encode(t[(int64_t)y * cols + z] * r, fmt);
    }
  free(t);
}

/* ------------------------------------------------------------------------ */
/* Block product M = (Tq * Sq) scaled: the FP8 values are multiples of the   */
/* format's smallest subnormal q0 (2^-9 for E4M3, 2^-16 for E5M2), so every  */
/* value is an integer times q0 and every product an integer times q0^2.    */
/* The sum over the inner index is formed exactly in a 128-bit integer and   */
/* rounded once to fp32; then M = (M * dT) * dS, two fp32 multiplications.   */
/* Tq is br x bk (row-major), Sq is bk x bc (row-major, B's orientation).    */
/* ------------------------------------------------------------------------ */
static int64_t code_to_int(uint8_t c, int fmt) {
  fp8_format f = fmt_of(fmt);
  double v = orc_fp8_decode(c, fmt);
  return (int64_t)ldexp(v, f.bias + f.man_bits - 1); /* exact */
}

static float exact_sum_to_float(__int128 s, int fmt) {
  fp8_format f = fmt_of(fmt);
  /* value = s * 2^(-2*(bias+man_bits-1)); (float)s is correctly rounded and
   * the power-of-two scaling is exact (results stay far from fp32's
   * subnormal and overflow ranges at every supported inner length). */
  float fs = (float)s;
  return ldexpf(fs, -2 * (f.bias + f.man_bits - 1));
}

void orc_block_product(const uint8_t* Tq, const uint8_t* Sq, float dT, float dS,
                       int br, int bc, int bk, int fmt, float* Mout) {
  int64_t* ti = (int64_t*)orc_alloc(sizeof(int64_t) * (size_t)br * bk);
  int64_t* sti = (int64_t*)orc_alloc(sizeof(int64_t) * (size_t)bc * bk); /* Sq^T */
  for (int64_t i = 0; i < (int64_t)br * bk; ++i) ti[i] = code_to_int(Tq[i], fmt);
  for (int y = 0; y < bk; ++y)
    for (int z = 0; z < bc; ++z)
      sti[(int64_t)z * bk + y] = code_to_int(Sq[(int64_t)y * bc + z], fmt);
#pragma omp parallel for schedule(static)
  for (int x = 0; x < br; ++x) {
    for (int z = 0; z < bc; ++z) {
      const int64_t* a = ti + (int64_t)x * bk;
      const int64_t* b = sti + (int64_t)z * bk;
      __int128 s = 0;
      for (int y = 0; y < bk; ++y) s += (__int128)a[y] * b[y];
      float m = exact_sum_to_float(s, fmt);
      m = m * dT;
      m = m * dS;
      Mout[(int64_t)x * bc + z] = m;
    }
  }
  free(ti);
  free(sti);
}

/* The block product with a scale per row of Tq (dT[x]) and per column of   */
/* Sq (dS[z]): M[x][z] = (exact sum rounded once * dT[x]) * dS[z].           */
void orc_block_product_rc(const uint8_t* Tq, const uint8_t* Sq, const float* dT,
                          const float* dS, int br, int bc, int bk, int fmt, float* Mout) {
  orc_block_product(Tq, Sq, 1.0f, 1.0f, br, bc, bk, fmt, Mout); /* exact sums, x1 x1 */
  for (int x = 0; x < br; ++x)
    for (int z = 0; z < bc; ++z) {
      float m = Mout[(int64_t)x * bc + z];
      m = m * dT[x];
      m = m * dS[z];
      Mout[(int64_t)x * bc + z] = m;
    }
}

/* The block product with group scales: for every group kg of 128 inner     */
/* indices, the exact sum P rounded once to fp32 is added as                  */
/* acc = fmaf(P, fl(dT[kg][x] * dS[kg][z / 128]), acc) from +0 in ascending   */
/* kg; the product is returned rounded to bf16 (held as fp32).               */
void orc_block_product_groups_acc(const uint8_t* Tq, const uint8_t* Sq, const float* dT,
                                  const float* dS, int br, int bc, int bk, int fmt, int bf16_out,
                                  float* Mout);
void orc_block_product_groups(const uint8_t* Tq, const uint8_t* Sq, const float* dT,
                              const float* dS, int br, int bc, int bk, int fmt, float* Mout) {
  orc_block_product_groups_acc(Tq, Sq, dT, dS, br, bc, bk, fmt, 1, Mout);
}

/* The same with the fp32 accumulator itself returned when bf16_out is 0. */
void orc_block_product_groups_acc(const uint8_t* Tq, const uint8_t* Sq, const float* dT,
                                  const float* dS, int br, int bc, int bk, int fmt, int bf16_out,
                                  float* Mout) {
  int ng = bk / ORC_GROUP, nzb = bc / ORC_GROUP;
  int64_t* ti = (int64_t*)orc_alloc(sizeof(int64_t) * (size_t)br * bk);
  int64_t* sti = (int64_t*)orc_alloc(sizeof(int64_t) * (size_t)bc * bk); /* Sq^T */
  for (int64_t i = 0; i < (int64_t)br * bk; ++i) ti[i] = code_to_int(Tq[i], fmt);
  for (int y = 0; y < bk; ++y)
    for (int z = 0; z < bc; ++z)
      sti[(int64_t)z * bk + y] = code_to_int(Sq[(int64_t)y * bc + z], fmt);
#pragma omp parallel for schedule(static)
  for (int x = 0; x < br; ++x) {
    for (int z = 0; z < bc; ++z) {
      const int64_t* a = ti + (int64_t)x * bk;
      const int64_t* b = sti + (int64_t)z * bk;
      float acc = 0.0f;
      for (int kg = 0; kg < ng; ++kg) {
        __int128 sum = 0;
        for (int y = kg * ORC_GROUP; y < (kg + 1) * ORC_GROUP; ++y) sum += (__int128)a[y] * b[y];
        float P = exact_sum_to_float(sum, fmt);
        float sc = dT[(int64_t)kg * br + x] * dS[(int64_t)kg * nzb + z / ORC_GROUP];
        acc = fmaf(P, sc, acc);
      }
      Mout[(int64_t)x * bc + z] = bf16_out ? orc_bf16_round(acc) : acc;
    }
  }
  free(ti);
  free(sti);
}

/* The same block product at selected positions (xs[t], zs[t]) only. */
void orc_block_product_at(const uint8_t* Tq, const uint8_t* Sq, float dT, float dS,
                          int br, int bc, int bk, int fmt, const int* xs,
                          const int* zs, int npos, float* out) {
  (void)br;
  for (int t = 0; t < npos; ++t) {
    __int128 s = 0;
    for (int y = 0; y < bk; ++y)
      s += (__int128)code_to_int(Tq[(int64_t)xs[t] * bk + y], fmt) *
           code_to_int(Sq[(int64_t)y * bc + zs[t]], fmt);
    float m = exact_sum_to_float(s, fmt);
    m = m * dT;
    m = m * dS;
    out[t] = m;
  }
}

/* ------------------------------------------------------------------------ */
/* Reconstruction, eq. (1): C_ij = sum_r w_{r,ij} M_r, over r ascending with */
/* w != 0, from +0.0f, one fmaf per term.  Mr holds R blocks br x bc; W is   */
/* R x (gm*gn); C is (gm*br) x (gn*bc) row-major.                            */
/* ------------------------------------------------------------------------ */
void orc_reconstruct(const float* Mr, const float* W, int R, int gm, int gn,
                     int br, int bc, float* C) {
  int64_t bsz = (int64_t)br * bc;
  int N = gn * bc;
#pragma omp parallel for schedule(static)
  for (int i = 0; i < gm; ++i)
    for (int j = 0; j < gn; ++j)
      for (int x = 0; x < br; ++x)
        for (int z = 0; z < bc; ++z) {
          float acc = 0.0f;
          for (int r = 0; r < R; ++r) {
            float w = W[(int64_t)r * gm * gn + i * gn + j];
            if (w == 0.0f) continue;
            acc = fmaf(w, Mr[r * bsz + (int64_t)x * bc + z], acc);
          }
          C[(int64_t)(i * br + x) * N + (j * bc + z)] = acc;
        }
}

/* ------------------------------------------------------------------------ */
/* float64 reference C = A B from the fp32 operands (App. F: a float64       */
/* reference), sum over the inner index in ascending order.                  */
/* ------------------------------------------------------------------------ */
void orc_reference_f64(const float* A, const float* B, int M, int N, int K,
                       double* C) {
#pragma omp parallel for schedule(static)
  for (int i = 0; i < M; ++i) {
    double* row = C + (int64_t)i * N;
    for (int j = 0; j < N; ++j) row[j] = 0.0;
    for (int k = 0; k < K; ++k) {
      double a = (double)A[(int64_t)i * K + k];
      const float* brow = B + (int64_t)k * N;
      for (int j = 0; j < N; ++j) row[j] += a * (double)brow[j];
    }
  }
}

/* One entry of the float64 reference. */
double orc_reference_f64_at(const float* A, const float* B, int N, int K, int i,
                            int j) {
  double s = 0.0;
  for (int k = 0; k < K; ++k)
    s += (double)A[(int64_t)i * K + k] * (double)B[(int64_t)k * N + j];
  return s;
}

/* ------------------------------------------------------------------------ */
/* Squared Frobenius norms for the relative error (App. B, App. F):          */
/* err_sq = sum (C - Cref)^2, ref_sq = sum Cref^2, in float64.               */
/* ------------------------------------------------------------------------ */
void orc_error_sums(const float* C, const double* Cref, int64_t n,
                    double* err_sq, double* ref_sq) {
  double e = 0.0, r = 0.0;
  for (int64_t i = 0; i < n; ++i) {
    double d = (double)C[i] - Cref[i];
    e += d * d;
    r += Cref[i] * Cref[i];
  }
  *err_sq = e;
  *ref_sq = r;
}

/* ------------------------------------------------------------------------ */
/* The whole schedule for one scheme, eq. (1) with FP8 block sums:           */
/*   for each product r: block sums of A and B (orc_block_sum), one scale   */
/*   per tensor and FP8 codes (orc_quantize_tensor), the scaled block       */
/*   product (orc_block_product); then the reconstruction.                  */
/* U is R x (gm*gk), V is R x (gk*gn), W is R x (gm*gn), all fp32, grid     */
/* indices row-major.  Optional outputs (NULL to skip): Tq (R x br x bk),   */
/* dT (R), Sq (R x bk x bc, B's orientation), dS (R), Mr (R x br x bc).     */
/* ------------------------------------------------------------------------ */
int orc_lowp_matmul(const float* A, const float* B, int M, int N, int K,
                    int gm, int gk, int gn, int R, const float* U,
                    const float* V, const float* W, int fmt, float* C,
                    uint8_t* Tq_out, float* dT_out, uint8_t* Sq_out,
                    float* dS_out, float* Mr_out) {
  if (M % gm || K % gk || N % gn) return -1;
  int br = M / gm, bk = K / gk, bc = N / gn;
  int64_t tsz = (int64_t)br * bk, ssz = (int64_t)bk * bc, msz = (int64_t)br * bc;
  float* T = (float*)orc_alloc(sizeof(float) * (size_t)(tsz > ssz ? tsz : ssz));
  uint8_t* tq = (uint8_t*)orc_alloc((size_t)tsz);
  uint8_t* sq = (uint8_t*)orc_alloc((size_t)ssz);
  float* Mr = Mr_out ? Mr_out : (float*)orc_alloc(sizeof(float) * (size_t)(msz * R));
  for (int r = 0; r < R; ++r) {
    orc_block_sum(A, M, K, gm, gk, U + (int64_t)r * gm * gk, T);
    float dT = orc_quantize_tensor(T, tsz, fmt, tq);
    orc_block_sum(B, K, N, gk, gn, V + (int64_t)r * gk * gn, T);
    float dS = orc_quantize_tensor(T, ssz, fmt, sq);
    if (Tq_out) memcpy(Tq_out + r * tsz, tq, (size_t)tsz);
    if (Sq_out) memcpy(Sq_out + r * ssz, sq, (size_t)ssz);
    if (dT_out) dT_out[r] = dT;
    if (dS_out) dS_out[r] = dS;
    orc_block_product(tq, sq, dT, dS, br, bc, bk, fmt, Mr + r * msz);
  }
  orc_reconstruct(Mr, W, R, gm, gn, br, bc, C);
  if (!Mr_out) free(Mr);
  free(T);
  free(tq);
  free(sq);
  return 0;
}

/* The whole schedule with a choice of scale granularity: scale_mode 0 is   */
/* one scale per block-sum tensor (orc_lowp_matmul), 1 is one per row of     */
/* each A-side block sum and one per column of each B-side block sum, 2 the  */
/* group scales (1 x 128 on A's block sums, 128 x 128 on B's bf16-rounded    */
/* ones, products returned in bf16).  Scale outputs hold R values (mode 0),  */
/* R x br and R x bc (mode 1), or R x (bk/128) x br and                      */
/* R x (bk/128) x (bc/128) (mode 2).                                          */
int orc_lowp_matmul_sm(const float* A, const float* B, int M, int N, int K,
                       int gm, int gk, int gn, int R, const float* U,
                       const float* V, const float* W, int fmt, int scale_mode,
                       float* C, uint8_t* Tq_out, float* dT_out, uint8_t* Sq_out,
                       float* dS_out, float* Mr_out) {
  if (scale_mode == 0)
    return orc_lowp_matmul(A, B, M, N, K, gm, gk, gn, R, U, V, W, fmt, C, Tq_out, dT_out,
                           Sq_out, dS_out, Mr_out);
  if (scale_mode != 1 && scale_mode != 2) return -2;
  if (R < 1 || M % gm || K % gk || N % gn) return -1;
  int br = M / gm, bk = K / gk, bc = N / gn;
  if (scale_mode == 2 && (bk % ORC_GROUP || bc % ORC_GROUP)) return -1;
  /* scales per product: mode 1 br and bc; mode 2 (bk/128) br and (bk/128) (bc/128) */
  int64_t nta = scale_mode == 1 ? br : (int64_t)(bk / ORC_GROUP) * br;
  int64_t nsb = scale_mode == 1 ? bc : (int64_t)(bk / ORC_GROUP) * (bc / ORC_GROUP);
  int64_t tsz = (int64_t)br * bk, ssz = (int64_t)bk * bc, msz = (int64_t)br * bc;
  float* T = (float*)orc_alloc(sizeof(float) * (size_t)(tsz > ssz ? tsz : ssz));
  uint8_t* tq = (uint8_t*)orc_alloc((size_t)tsz);
  uint8_t* sq = (uint8_t*)orc_alloc((size_t)ssz);
  float* dT = (float*)orc_alloc(sizeof(float) * (size_t)nta);
  float* dS = (float*)orc_alloc(sizeof(float) * (size_t)nsb);
  float* Mr = Mr_out ? Mr_out : (float*)orc_alloc(sizeof(float) * (size_t)(msz * R));
  for (int r = 0; r < R; ++r) {
    orc_block_sum(A, M, K, gm, gk, U + (int64_t)r * gm * gk, T);
    if (scale_mode == 1) orc_quantize_rows(T, br, bk, fmt, tq, dT);
    else orc_quantize_row_groups(T, br, bk, fmt, tq, dT);
    orc_block_sum(B, K, N, gk, gn, V + (int64_t)r * gk * gn, T);
    if (scale_mode == 1) orc_quantize_cols(T, bk, bc, fmt, sq, dS);
    else orc_quantize_bf16_blocks(T, bk, bc, fmt, sq, dS);
    if (Tq_out) memcpy(Tq_out + r * tsz, tq, (size_t)tsz);
    if (Sq_out) memcpy(Sq_out + r * ssz, sq, (size_t)ssz);
    if (dT_out) memcpy(dT_out + (int64_t)r * nta, dT, sizeof(float) * (size_t)nta);
    if (dS_out) memcpy(dS_out + (int64_t)r * nsb, dS, sizeof(float) * (size_t)nsb);
    if (scale_mode == 1) orc_block_product_rc(tq, sq, dT, dS, br, bc, bk, fmt, Mr + r * msz);
    else orc_block_product_groups(tq, sq, dT, dS, br, bc, bk, fmt, Mr + r * msz);
  }
  orc_reconstruct(Mr, W, R, gm, gn, br, bc, C);
  if (!Mr_out) free(Mr);
  free(T);
  free(tq);
  free(sq);
  free(dT);
  free(dS);
  return 0;
}

/* Quantized operands only (block sums, scales and codes) for one side:     */
/* X rows x cols, grid gr x gc, R coefficient rows.  codes: R x (rows/gr) x */
/* (cols/gc) in X's orientation; d: R scales.                               */
void orc_form_operands(const float* X, int rows, int cols, int gr, int gc, int R,
                       const float* coef, int fmt, uint8_t* codes, float* d) {
  int64_t sz = (int64_t)(rows / gr) * (cols / gc);
  float* T = (float*)orc_alloc(sizeof(float) * (size_t)sz);
  for (int r = 0; r < R; ++r) {
    orc_block_sum(X, rows, cols, gr, gc, coef + (int64_t)r * gr * gc, T);
    d[r] = orc_quantize_tensor(T, sz, fmt, codes + r * sz);
  }
  free(T);
}

/* The same with a choice of scale granularity: scale_mode 1 gives one scale */
/* per row of each block sum (side 0, A) or per column (side 1, B); d holds  */
/* R x (rows/gr) or R x (cols/gc) values.  scale_mode 2: the group scales   */
/* (side 0: 1 x 128 groups, d R x (bc/128) x br; side 1: bf16 rounding then */
/* 128 x 128 blocks, d R x (br/128) x (bc/128)).                             */
void orc_form_operands_sm(const float* X, int rows, int cols, int gr, int gc, int R,
                          const float* coef, int fmt, int scale_mode, int side,
                          uint8_t* codes, float* d) {
  if (scale_mode == 0) {
    orc_form_operands(X, rows, cols, gr, gc, R, coef, fmt, codes, d);
    return;
  }
  int br = rows / gr, bc = cols / gc;
  int64_t sz = (int64_t)br * bc;
  float* T = (float*)orc_alloc(sizeof(float) * (size_t)sz);
  /* mode 2 scales per product: A (bc/128) br, B (br/128) (bc/128) */
  int64_t nd = scale_mode == 1 ? (side == 0 ? br : bc)
                               : (side == 0 ? (int64_t)(bc / ORC_GROUP) * br
                                            : (int64_t)(br / ORC_GROUP) * (bc / ORC_GROUP));
  for (int r = 0; r < R; ++r) {
    orc_block_sum(X, rows, cols, gr, gc, coef + (int64_t)r * gr * gc, T);
    if (scale_mode == 1 && side == 0)
      orc_quantize_rows(T, br, bc, fmt, codes + r * sz, d + r * nd);
    else if (scale_mode == 1)
      orc_quantize_cols(T, br, bc, fmt, codes + r * sz, d + r * nd);
    else if (side == 0)
      orc_quantize_row_groups(T, br, bc, fmt, codes + r * sz, d + r * nd);
    else
      orc_quantize_bf16_blocks(T, br, bc, fmt, codes + r * sz, d + r * nd);
  }
  free(T);
}

/* ======================================================================== */
/* Integer codes and the classical int8 operator at a quantization           */
/* specification (Sec. 2.2; App. D, the specification of the model runs):   */
/* groups of g consecutive entries along the inner dimension; one scale per  */
/* row of A and per column of B in every group, d = max|x| / b (one          */
/* correctly rounded fp32 division; d = 1 for an all-zero group); code =     */
/* x / d (one fp32 division) rounded to the nearest integer, ties to even,   */
/* with no clipping.  Codes are held in int8 (|code| <= b <= 127).           */
/* ======================================================================== */
static int8_t int_code(float x, float d) {
  float y = x / d;
  return (int8_t)lrintf(y); /* current rounding mode: nearest, ties to even */
}

/* A: M x K row-major; codes M x K; d: M x (K/g), d[t*(K/g) + gi]. */
void orc_int8_quantize_a(const float* A, int M, int K, int g, int b, int8_t* codes, float* d) {
  int ng = K / g;
  for (int t = 0; t < M; ++t)
    for (int gi = 0; gi < ng; ++gi) {
      const float* x = A + (int64_t)t * K + (int64_t)gi * g;
      float amax = 0.0f;
      for (int k = 0; k < g; ++k) {
        float a = fabsf(x[k]);
        if (a > amax) amax = a;
      }
      float s = amax == 0.0f ? 1.0f : amax / (float)b;
      d[(int64_t)t * ng + gi] = s;
      for (int k = 0; k < g; ++k) codes[(int64_t)t * K + (int64_t)gi * g + k] = int_code(x[k], s);
    }
}

/* B: K x N row-major; codes K x N; d: (K/g) x N, d[gi*N + j]. */
void orc_int8_quantize_b(const float* B, int K, int N, int g, int b, int8_t* codes, float* d) {
  int ng = K / g;
  for (int j = 0; j < N; ++j)
    for (int gi = 0; gi < ng; ++gi) {
      float amax = 0.0f;
      for (int k = 0; k < g; ++k) {
        float a = fabsf(B[(int64_t)(gi * g + k) * N + j]);
        if (a > amax) amax = a;
      }
      float s = amax == 0.0f ? 1.0f : amax / (float)b;
      d[(int64_t)gi * N + j] = s;
      for (int k = 0; k < g; ++k) {
        int64_t at = (int64_t)(gi * g + k) * N + j;
        codes[at] = int_code(B[at], s);
      }
    }
}

/* One group's exact integer product of the codes, P[t][j] (int64). */
void orc_int8_group_product(const int8_t* Ac, const int8_t* Bc, int M, int N, int K, int g,
                            int gi, int64_t* P) {
  for (int t = 0; t < M; ++t)
    for (int j = 0; j < N; ++j) {
      int64_t s = 0;
      for (int k = gi * g; k < (gi + 1) * g; ++k)
        s += (int64_t)Ac[(int64_t)t * K + k] * Bc[(int64_t)k * N + j];
      P[(int64_t)t * N + j] = s;
    }
}

/* The output side of the specification: out starts at +0; for each group in */
/* ascending order, out += (fl32(P) * dA) * dB, each step one fp32 operation. */
static void rescale_accumulate(const double* P, const float* dA, const float* dB, int M, int N,
                               int ng, int gi, float* out) {
  for (int t = 0; t < M; ++t)
    for (int j = 0; j < N; ++j) {
      float p = (float)P[(int64_t)t * N + j];
      float v = p * dA[(int64_t)t * ng + gi];
      v = v * dB[(int64_t)gi * N + j];
      out[(int64_t)t * N + j] = out[(int64_t)t * N + j] + v;
    }
}

void orc_int8_classical(const int8_t* Ac, const float* dA, const int8_t* Bc, const float* dB,
                        int M, int N, int K, int g, float* out) {
  int ng = K / g;
  int64_t* P = (int64_t*)orc_alloc(sizeof(int64_t) * (size_t)M * N);
  double* Pd = (double*)orc_alloc(sizeof(double) * (size_t)M * N);
  for (int64_t i = 0; i < (int64_t)M * N; ++i) out[i] = 0.0f;
  for (int gi = 0; gi < ng; ++gi) {
    orc_int8_group_product(Ac, Bc, M, N, K, g, gi, P);
    for (int64_t i = 0; i < (int64_t)M * N; ++i) Pd[i] = (double)P[i];
    rescale_accumulate(Pd, dA, dB, M, N, ng, gi, out);
  }
  free(P);
  free(Pd);
}

/* ------------------------------------------------------------------------ */
/* Fast realization of one group's integer product (Sec. 4.2, Prop. 1): the */
/* group is covered by calls of gk*h consecutive inner indices; each call   */
/* takes all M rows and N columns, split into gm x gk blocks of A's codes   */
/* (M/gm x h) and gk x gn blocks of B's codes (h x N/gn), and evaluates     */
/* eq. (1) with the given integer coefficients: block sums, R block         */
/* products, combination; the calls' results are added.  All arithmetic is  */
/* exact (int64); viol[0] counts block-sum entries outside [-127, 127]      */
/* (condition (i)), viol[1] products or partial sums, in the order formed,  */
/* outside int32 (condition (ii)).  With round_fp8 = 1 every block-sum      */
/* entry is first rounded to E4M3 (nearest even, saturating), and products  */
/* and sums are carried in float64 (exact at these magnitudes).             */
/* P receives the group product (M x N, as float64).                        */
/* ------------------------------------------------------------------------ */
void orc_int8_group_product_fast(const int8_t* Ac, const int8_t* Bc, int M, int N, int K, int g,
                                 int gi, int h, int gm, int gk, int gn, int R, const float* U,
                                 const float* V, const float* W, int round_fp8, double* P,
                                 int64_t* viol) {
  const int br = M / gm, bc = N / gn;
  const int64_t lim = (int64_t)1 << 31;
  double* T = (double*)orc_alloc(sizeof(double) * (size_t)br * h);
  double* S = (double*)orc_alloc(sizeof(double) * (size_t)h * bc);
  double* Mr = (double*)orc_alloc(sizeof(double) * (size_t)R * br * bc);
  for (int64_t i = 0; i < (int64_t)M * N; ++i) P[i] = 0.0;
  for (int k0 = gi * g; k0 < (gi + 1) * g; k0 += gk * h) { /* one call */
    for (int r = 0; r < R; ++r) {
      /* block sums of codes, ascending row-major grid order */
      for (int x = 0; x < br; ++x)
        for (int y = 0; y < h; ++y) {
          double acc = 0.0;
          for (int p = 0; p < gm; ++p)
            for (int q = 0; q < gk; ++q) {
              double u = U[(int64_t)r * gm * gk + p * gk + q];
              if (u == 0.0) continue;
              acc += u * Ac[(int64_t)(p * br + x) * K + k0 + q * h + y];
            }
          if (fabs(acc) > 127.0) ++viol[0];
          T[(int64_t)x * h + y] = round_fp8 ? orc_fp8_decode(orc_fp8_encode((float)acc, 0), 0) : acc;
        }
      for (int y = 0; y < h; ++y)
        for (int z = 0; z < bc; ++z) {
          double acc = 0.0;
          for (int p = 0; p < gk; ++p)
            for (int q = 0; q < gn; ++q) {
              double v = V[(int64_t)r * gk * gn + p * gn + q];
              if (v == 0.0) continue;
              acc += v * Bc[(int64_t)(k0 + p * h + y) * N + q * bc + z];
            }
          if (fabs(acc) > 127.0) ++viol[0];
          S[(int64_t)y * bc + z] = round_fp8 ? orc_fp8_decode(orc_fp8_encode((float)acc, 0), 0) : acc;
        }
      /* block product */
      for (int x = 0; x < br; ++x)
        for (int z = 0; z < bc; ++z) {
          double s = 0.0;
          for (int y = 0; y < h; ++y) {
            s += T[(int64_t)x * h + y] * S[(int64_t)y * bc + z];
            if (fabs(s) >= (double)lim) ++viol[1];
          }
          Mr[((int64_t)r * br + x) * bc + z] = s;
        }
    }
    /* combination, ascending r; added to the group's running sum */
    for (int i = 0; i < gm; ++i)
      for (int j = 0; j < gn; ++j)
        for (int x = 0; x < br; ++x)
          for (int z = 0; z < bc; ++z) {
            double c = 0.0;
            for (int r = 0; r < R; ++r) {
              double w = W[(int64_t)r * gm * gn + i * gn + j];
              if (w == 0.0) continue;
              c += w * Mr[((int64_t)r * br + x) * bc + z];
              if (fabs(c) >= (double)lim) ++viol[1];
            }
            double* pp = P + (int64_t)(i * br + x) * N + j * bc + z;
            *pp += c;
            if (fabs(*pp) >= (double)lim) ++viol[1];
          }
  }
  free(T);
  free(S);
  free(Mr);
}

/* The fast realization's output: the group products of the calls, then the */
/* classical operator's rescaling and fp32 order.  Returns 0, or -1 if the  */
/* tiling does not fit (M, N, g divisibility).                              */
int orc_int8_fast(const int8_t* Ac, const float* dA, const int8_t* Bc, const float* dB, int M,
                  int N, int K, int g, int h, int gm, int gk, int gn, int R, const float* U,
                  const float* V, const float* W, float* out, int64_t* viol) {
  if (M % gm || N % gn || K % g || g % (gk * h)) return -1;
  int ng = K / g;
  double* P = (double*)orc_alloc(sizeof(double) * (size_t)M * N);
  for (int64_t i = 0; i < (int64_t)M * N; ++i) out[i] = 0.0f;
  for (int gi = 0; gi < ng; ++gi) {
    orc_int8_group_product_fast(Ac, Bc, M, N, K, g, gi, h, gm, gk, gn, R, U, V, W, 0, P, viol);
    rescale_accumulate(P, dA, dB, M, N, ng, gi, out);
  }
  free(P);
  return 0;
}

/* ------------------------------------------------ the overflow correction */
/* Sec. 4.3 (eq. (2)) and App. D (the corrected computation's certificate):  */
/* a block sum of codes s, exact in a wide integer type, splits as           */
/* s = s0 + 256 q with q = floor((s + 128) / 256) and s0 = s - 256 q, so      */
/* s0 lies in [-128, 127]; then  s_A s_B = A0 B0 + 256 (R_A B0 + A0 R_B)      */
/* + 256^2 R_A R_B  with every multiplicand an int8 value.                  */
void orc_int8_split(int64_t s, int64_t* s0, int64_t* q) {
  int64_t t = s + 128;
  int64_t f = t >= 0 ? t / 256 : -((-t + 255) / 256); /* floor division */
  *q = f;
  *s0 = s - 256 * f;
}

/* One group's product with the correction: per call and product r, the     */
/* exact block sums are split, the block product is formed as the four       */
/* terms of eq. (2) (each an integer matrix product), and the output blocks  */
/* combine the products with the weights W.                                  */
/*   stats[0]: max over output entries and calls of the sum of the absolute  */
/*             values of every weighted scalar term (bounds every partial    */
/*             sum, in any order);                                           */
/*   stats[1]: split parts outside s0 in [-128, 127], |q| <= 2 (count);     */
/*   stats[2]: block sums whose q is nonzero (the overflows, count);         */
/*   counts[0]: multiplications of the A0 B0 products;                       */
/*   counts[1]: the correction's multiplications counting only nonzero       */
/*              entries of R_A and R_B (R_A B0: each nonzero of R_A times a   */
/*              row of B0; A0 R_B: a column of A0 times each nonzero of R_B;  */
/*              R_A R_B: the pairs of nonzeros that meet);                   */
/*   counts[2]: the correction's multiplications as dense products over the  */
/*              rows of R_A and the columns of R_B holding a nonzero entry.  */
void orc_int8_group_product_corrected(const int8_t* Ac, const int8_t* Bc, int M, int N, int K,
                                      int g, int gi, int h, int gm, int gk, int gn, int R,
                                      const float* U, const float* V, const float* W, double* P,
                                      double* stats, double* counts) {
  const int br = M / gm, bc = N / gn;
  int64_t* A0 = (int64_t*)orc_alloc(sizeof(int64_t) * (size_t)br * h);
  int64_t* RA = (int64_t*)orc_alloc(sizeof(int64_t) * (size_t)br * h);
  int64_t* B0 = (int64_t*)orc_alloc(sizeof(int64_t) * (size_t)h * bc);
  int64_t* RB = (int64_t*)orc_alloc(sizeof(int64_t) * (size_t)h * bc);
  int64_t* Mr = (int64_t*)orc_alloc(sizeof(int64_t) * (size_t)R * br * bc);
  double* Mabs = (double*)orc_alloc(sizeof(double) * (size_t)R * br * bc);
  for (int64_t i = 0; i < (int64_t)M * N; ++i) P[i] = 0.0;
  for (int k0 = gi * g; k0 < (gi + 1) * g; k0 += gk * h) { /* one call */
    for (int r = 0; r < R; ++r) {
      for (int x = 0; x < br; ++x)
        for (int y = 0; y < h; ++y) {
          int64_t acc = 0;
          for (int p = 0; p < gm; ++p)
            for (int q = 0; q < gk; ++q) {
              int64_t u = (int64_t)U[(int64_t)r * gm * gk + p * gk + q];
              if (u == 0) continue;
              acc += u * Ac[(int64_t)(p * br + x) * K + k0 + q * h + y];
            }
          int64_t s0, qq;
          orc_int8_split(acc, &s0, &qq);
          if (s0 < -128 || s0 > 127 || qq < -2 || qq > 2) stats[1] += 1;
          if (qq != 0) stats[2] += 1;
          A0[(int64_t)x * h + y] = s0;
          RA[(int64_t)x * h + y] = qq;
        }
      for (int y = 0; y < h; ++y)
        for (int z = 0; z < bc; ++z) {
          int64_t acc = 0;
          for (int p = 0; p < gk; ++p)
            for (int q = 0; q < gn; ++q) {
              int64_t v = (int64_t)V[(int64_t)r * gk * gn + p * gn + q];
              if (v == 0) continue;
              acc += v * Bc[(int64_t)(k0 + p * h + y) * N + q * bc + z];
            }
          int64_t s0, qq;
          orc_int8_split(acc, &s0, &qq);
          if (s0 < -128 || s0 > 127 || qq < -2 || qq > 2) stats[1] += 1;
          if (qq != 0) stats[2] += 1;
          B0[(int64_t)y * bc + z] = s0;
          RB[(int64_t)y * bc + z] = qq;
        }
      /* the block product as the four terms of eq. (2) */
      for (int x = 0; x < br; ++x)
        for (int z = 0; z < bc; ++z) {
          int64_t t00 = 0, t10 = 0, t01 = 0, t11 = 0;
          double ab = 0.0;
          for (int y = 0; y < h; ++y) {
            int64_t a0 = A0[(int64_t)x * h + y], ra = RA[(int64_t)x * h + y];
            int64_t b0 = B0[(int64_t)y * bc + z], rb = RB[(int64_t)y * bc + z];
            t00 += a0 * b0;
            t10 += ra * b0;
            t01 += a0 * rb;
            t11 += ra * rb;
            ab += (double)llabs(a0 * b0) + 256.0 * (double)llabs(ra * b0) +
                  256.0 * (double)llabs(a0 * rb) + 65536.0 * (double)llabs(ra * rb);
          }
          Mr[((int64_t)r * br + x) * bc + z] = t00 + 256 * (t10 + t01) + 65536 * t11;
          Mabs[((int64_t)r * br + x) * bc + z] = ab;
        }
      /* multiplication counts of this product */
      counts[0] += (double)br * bc * h;
      int64_t nnzA = 0, nnzB = 0, rowsA = 0, colsB = 0;
      double pairs = 0.0;
      for (int x = 0; x < br; ++x) {
        int any = 0;
        for (int y = 0; y < h; ++y)
          if (RA[(int64_t)x * h + y]) ++nnzA, any = 1;
        rowsA += any;
      }
      for (int z = 0; z < bc; ++z) {
        int any = 0;
        for (int y = 0; y < h; ++y)
          if (RB[(int64_t)y * bc + z]) ++nnzB, any = 1;
        colsB += any;
      }
      for (int y = 0; y < h; ++y) {
        int64_t ca = 0, cb = 0;
        for (int x = 0; x < br; ++x) ca += RA[(int64_t)x * h + y] != 0;
        for (int z = 0; z < bc; ++z) cb += RB[(int64_t)y * bc + z] != 0;
        pairs += (double)ca * cb;
      }
      counts[1] += (double)nnzA * bc + (double)br * nnzB + pairs;
      counts[2] += (double)rowsA * h * bc + (double)br * h * colsB + (double)rowsA * h * colsB;
    }
    /* combination, ascending r; added to the group's running sum */
    for (int i = 0; i < gm; ++i)
      for (int j = 0; j < gn; ++j)
        for (int x = 0; x < br; ++x)
          for (int z = 0; z < bc; ++z) {
            int64_t c = 0;
            double cabs = 0.0;
            for (int r = 0; r < R; ++r) {
              int64_t w = (int64_t)W[(int64_t)r * gm * gn + i * gn + j];
              if (w == 0) continue;
              c += w * Mr[((int64_t)r * br + x) * bc + z];
              cabs += (double)llabs(w) * Mabs[((int64_t)r * br + x) * bc + z];
            }
            if (cabs > stats[0]) stats[0] = cabs;
            P[(int64_t)(i * br + x) * N + j * bc + z] += (double)c;
          }
  }
  free(A0);
  free(RA);
  free(B0);
  free(RB);
  free(Mr);
  free(Mabs);
}

/* The corrected realization's output: group products as above, then the    */
/* classical operator's rescaling and fp32 order.  Returns 0, or -1 if the   */
/* tiling does not fit.                                                      */
int orc_int8_fast_corrected(const int8_t* Ac, const float* dA, const int8_t* Bc, const float* dB,
                            int M, int N, int K, int g, int h, int gm, int gk, int gn, int R,
                            const float* U, const float* V, const float* W, float* out,
                            double* stats, double* counts) {
  if (M % gm || N % gn || K % g || g % (gk * h)) return -1;
  int ng = K / g;
  double* P = (double*)orc_alloc(sizeof(double) * (size_t)M * N);
  for (int64_t i = 0; i < (int64_t)M * N; ++i) out[i] = 0.0f;
  for (int gi = 0; gi < ng; ++gi) {
    orc_int8_group_product_corrected(Ac, Bc, M, N, K, g, gi, h, gm, gk, gn, R, U, V, W, P, stats,
                                     counts);
    rescale_accumulate(P, dA, dB, M, N, ng, gi, out);
  }
  free(P);
  return 0;
}

/* ======================================================================== */
/* Repairs (App. C, the repair rules), options of the group-scale schedule. */
/* ======================================================================== */

/* Exponent k of the outside row scale d_t = 2^k, k = ceil(log2(max(RMS(x_t), */
/* 1e-3))), RMS over the full row.  The sum of squares is formed in float64   */
/* in a fixed order: partial sums over the residues of the index mod 64, in   */
/* ascending index, combined pairwise as v[l] + v[l ^ off] for off = 32, 16, */
/* ..., 1; then m2 = sum / K (one float64 division).  k is the least integer */
/* with 4^k >= m2 (so 2^k >= RMS), found exactly from m2's binary exponent,  */
/* and at least -9 (2^-9 is the least power of two >= 1e-3).  A non-finite  */
/* row gets k = 0.                                                           */
int orc_row_exponent(const float* x, int K) {
  double v[64];
  for (int l = 0; l < 64; ++l) v[l] = 0.0;
  for (int i = 0; i < K; ++i) v[i & 63] += (double)x[i] * (double)x[i];
  for (int off = 32; off >= 1; off >>= 1) {
    double w[64];
    for (int l = 0; l < 64; ++l) w[l] = v[l] + v[l ^ off];
    memcpy(v, w, sizeof v);
  }
  double m2 = v[0] / (double)K;
  if (!isfinite(m2)) return 0;
  if (m2 == 0.0) return -9;
  int e;
  double fr = frexp(m2, &e); /* m2 = fr 2^e, fr in [0.5, 1) */
  int c = fr == 0.5 ? e - 1 : e; /* ceil(log2 m2) */
  int k = c >= 0 ? (c + 1) / 2 : -((-c) / 2); /* ceil(c / 2) */
  return k < -9 ? -9 : k;
}

/* Joint rounding of one position of B's block sums (the repair rules): for   */
/* every product r, s[r] is the bf16 block-sum entry, q[r] and d[r] its       */
/* block's scales.  The candidates are the two codes whose values bracket     */
/* y = s q (one fp32 multiply) -- the nearest (the ordinary rounding) and its */
/* neighbour on the other side of y (none when y is a code value, or beyond   */
/* the largest finite one) -- valued fl(dec(code) d); the start is the one    */
/* whose value is nearer s (fp32 distances fl(value - s); on equal distances  */
/* the nearest-even code).  With e_r = fl(value - s[r]) and g = H e (g_r =    */
/* fmaf over s ascending from +0), sweep r = 0..R-1:                          */
/* delta = fl(alt value - current value), change = fl(fl(fl(2 delta) g_r) +  */
/* fl(fl(delta delta) H_rr)); if change < 0 the alternative is taken,        */
/* e_r = fl(new value - s[r]) and g_t = fmaf(H_tr, delta, g_t) for every t   */
/* ascending.  Stop after a sweep with no change or after max_sweeps.        */
/* Returns the number of sweeps made.                                         */
static uint8_t code_step(uint8_t c, int up, int fmt) {
  /* the neighbouring code one step larger (up) or smaller in magnitude,    */
  /* 0xff when none (beyond the largest finite or below zero)              */
  uint8_t mag = c & 0x7f, sign = c & 0x80;
  uint8_t maxmag = (uint8_t)(fmt == ORC_E4M3 ? 0x7e : 0x7b);
  if (up) return mag >= maxmag ? 0xff : (uint8_t)(sign | (mag + 1));
  return mag == 0 ? 0xff : (uint8_t)(sign | (mag - 1));
}

int orc_joint_round_position(const float* s, const float* q, const float* d, const float* H,
                             int R, int fmt, int max_sweeps, uint8_t* codes) {
  uint8_t cur[512], alt[512];
  float e[512], g[512], val[512], aval[512];
  if (R > 512) return -1;
  for (int r = 0; r < R; ++r) {
    float y = s[r] * q[r];
    uint8_t c = orc_fp8_encode(y, fmt);
    double dv = orc_fp8_decode(c, fmt);
    uint8_t a = 0xff;
    if (dv != (double)y) {
      /* the neighbour on the other side of y, in magnitude */
      int away = fabs((double)y) > fabs(dv); /* y beyond the code: step up */
      a = code_step(c, away, fmt);
      if (a != 0xff && (c & 0x7f) == 0) a = (uint8_t)((y < 0 ? 0x80 : 0x00) | (a & 0x7f));
    }
    cur[r] = c;
    alt[r] = a;
    val[r] = (float)dv * d[r];
    aval[r] = a == 0xff ? 0.0f : (float)orc_fp8_decode(a, fmt) * d[r];
    e[r] = val[r] - s[r];
    if (a != 0xff) {
      /* start at the candidate whose value is nearer s (fp32 distances; on */
      /* equal distances the nearest-even code)                            */
      float ea = aval[r] - s[r];
      if (fabsf(ea) < fabsf(e[r])) {
        cur[r] = a;
        alt[r] = c;
        float tv = val[r];
        val[r] = aval[r];
        aval[r] = tv;
        e[r] = ea;
      }
    }
  }
  for (int r = 0; r < R; ++r) {
    float acc = 0.0f;
    for (int t = 0; t < R; ++t) acc = fmaf(H[(int64_t)r * R + t], e[t], acc);
    g[r] = acc;
  }
  int sweeps = 0;
  for (int sw = 0; sw < max_sweeps; ++sw) {
    ++sweeps;
    int changed = 0;
    for (int r = 0; r < R; ++r) {
      if (alt[r] == 0xff) continue;
      float delta = aval[r] - val[r];
      float two = 2.0f * delta;
      float lin = two * g[r];
      float sq = delta * delta;
      float quad = sq * H[(int64_t)r * R + r];
      float change = lin + quad;
      if (change < 0.0f) {
        uint8_t tc = cur[r];
        cur[r] = alt[r];
        alt[r] = tc;
        float tv = val[r];
        val[r] = aval[r];
        aval[r] = tv;
        e[r] = val[r] - s[r];
        for (int t = 0; t < R; ++t) g[t] = fmaf(H[(int64_t)t * R + r], delta, g[t]);
        changed = 1;
      }
    }
    if (!changed) break;
  }
  for (int r = 0; r < R; ++r) codes[r] = cur[r];
  return sweeps;
}

/* H_rs = <w_r, w_s> <u_r, u_s> from the fp32 coefficient tables: each inner */
/* product in float64 over ascending index, their product rounded once to   */
/* fp32.  U is R x nu, W is R x nw.                                          */
void orc_repair_gram(const float* U, const float* W, int R, int nu, int nw, float* H) {
  for (int r = 0; r < R; ++r)
    for (int t = 0; t < R; ++t) {
      double uu = 0.0, ww = 0.0;
      for (int i = 0; i < nu; ++i) uu += (double)U[(int64_t)r * nu + i] * U[(int64_t)t * nu + i];
      for (int i = 0; i < nw; ++i) ww += (double)W[(int64_t)r * nw + i] * W[(int64_t)t * nw + i];
      H[(int64_t)r * R + t] = (float)(ww * uu);
    }
}

/* Scales of B's bf16 block sums in 128 x 128 blocks, as                   */
/* orc_quantize_bf16_blocks computes them: q[kg * nzb + zb], d[...] .        */
static void bf16_block_scales(const float* Tb, int rows, int cols, int fmt, float* q, float* d) {
  int nkg = rows / ORC_GROUP, nzb = cols / ORC_GROUP;
  for (int kg = 0; kg < nkg; ++kg)
    for (int zb = 0; zb < nzb; ++zb) {
      float amax = 0.0f;
      for (int y = kg * ORC_GROUP; y < (kg + 1) * ORC_GROUP; ++y)
        for (int z = zb * ORC_GROUP; z < (zb + 1) * ORC_GROUP; ++z) {
          float a = fabsf(Tb[(int64_t)y * cols + z]);
          if (a > amax) amax = a;
        }
      float r;
      d[(int64_t)kg * nzb + zb] = scale_from_amax(amax, fmt, &r);
      q[(int64_t)kg * nzb + zb] = r;
    }
}

/* The group-scale schedule with repairs (flags: 1 = outside power-of-two   */
/* row scaling of A, 2 = joint rounding of B's block sums, 12 sweeps at     */
/* most).  Row scaling: A's row t is multiplied by 2^-k_t (exact) before    */
/* the block sums and C's row t by 2^k_t after the reconstruction.  Joint   */
/* rounding replaces the nearest-code rounding of B's bf16 block sums; the  */
/* block scales are those of the ordinary schedule.  Outputs as             */
/* orc_lowp_matmul_sm (mode 2), plus the row exponents (M ints) if asked.   */
#define ORC_REPAIR_SWEEPS 12
int orc_lowp_matmul_repaired(const float* A, const float* B, int M, int N, int K, int gm, int gk,
                             int gn, int R, const float* U, const float* V, const float* W,
                             int fmt, int flags, float* C, uint8_t* Tq_out, float* dT_out,
                             uint8_t* Sq_out, float* dS_out, float* Mr_out, int* rowexp_out) {
  if (M % gm || K % gk || N % gn) return -1;
  int br = M / gm, bk = K / gk, bc = N / gn;
  if (bk % ORC_GROUP || bc % ORC_GROUP) return -1;
  int nkg = bk / ORC_GROUP, nzb = bc / ORC_GROUP;
  int64_t nta = (int64_t)nkg * br, nsb = (int64_t)nkg * nzb;
  int64_t tsz = (int64_t)br * bk, ssz = (int64_t)bk * bc, msz = (int64_t)br * bc;
  /* row scaling */
  int* kx = (int*)orc_alloc(sizeof(int) * (size_t)M);
  const float* Ause = A;
  float* As = NULL;
  for (int t = 0; t < M; ++t) kx[t] = (flags & 1) ? orc_row_exponent(A + (int64_t)t * K, K) : 0;
  if (flags & 1) {
    As = (float*)orc_alloc(sizeof(float) * (size_t)M * K);
    for (int t = 0; t < M; ++t) {
      float f = ldexpf(1.0f, -kx[t]);
      for (int i = 0; i < K; ++i) As[(int64_t)t * K + i] = A[(int64_t)t * K + i] * f;
    }
    Ause = As;
  }
  if (rowexp_out) memcpy(rowexp_out, kx, sizeof(int) * (size_t)M);
  /* B side for every product first: joint rounding looks across r */
  float* S = (float*)orc_alloc(sizeof(float) * (size_t)ssz);
  float* Sb = (float*)orc_alloc(sizeof(float) * (size_t)(ssz * R));
  float* qS = (float*)orc_alloc(sizeof(float) * (size_t)(nsb * R));
  float* dS = (float*)orc_alloc(sizeof(float) * (size_t)(nsb * R));
  uint8_t* sq = (uint8_t*)orc_alloc((size_t)(ssz * R));
  for (int r = 0; r < R; ++r) {
    orc_block_sum(B, K, N, gk, gn, V + (int64_t)r * gk * gn, S);
    for (int64_t i = 0; i < ssz; ++i) Sb[r * ssz + i] = orc_bf16_round(S[i]);
    bf16_block_scales(Sb + r * ssz, bk, bc, fmt, qS + r * nsb, dS + r * nsb);
    for (int y = 0; y < bk; ++y)
      for (int z = 0; z < bc; ++z) {
        int64_t blk = (int64_t)(y / ORC_GROUP) * nzb + z / ORC_GROUP;
        sq[r * ssz + (int64_t)y * bc + z] =
            orc_fp8_encode(Sb[r * ssz + (int64_t)y * bc + z] * qS[r * nsb + blk], fmt);
      }
  }
  if (flags & 2) {
    float* H = (float*)orc_alloc(sizeof(float) * (size_t)R * R);
    orc_repair_gram(U, W, R, gm * gk, gm * gn, H);
    float* sv = (float*)orc_alloc(sizeof(float) * (size_t)R * 3);
    float *qv = sv + R, *dv = sv + 2 * R;
    uint8_t* cv = (uint8_t*)orc_alloc((size_t)R);
    for (int y = 0; y < bk; ++y)
      for (int z = 0; z < bc; ++z) {
        int64_t pos = (int64_t)y * bc + z;
        int64_t blk = (int64_t)(y / ORC_GROUP) * nzb + z / ORC_GROUP;
        for (int r = 0; r < R; ++r) {
          sv[r] = Sb[r * ssz + pos];
          qv[r] = qS[r * nsb + blk];
          dv[r] = dS[r * nsb + blk];
        }
        orc_joint_round_position(sv, qv, dv, H, R, fmt, ORC_REPAIR_SWEEPS, cv);
        for (int r = 0; r < R; ++r) sq[r * ssz + pos] = cv[r];
      }
    free(H);
    free(sv);
    free(cv);
  }
  /* A side, products, reconstruction */
  float* T = (float*)orc_alloc(sizeof(float) * (size_t)tsz);
  uint8_t* tq = (uint8_t*)orc_alloc((size_t)tsz);
  float* dT = (float*)orc_alloc(sizeof(float) * (size_t)nta);
  float* Mr = Mr_out ? Mr_out : (float*)orc_alloc(sizeof(float) * (size_t)(msz * R));
  for (int r = 0; r < R; ++r) {
    orc_block_sum(Ause, M, K, gm, gk, U + (int64_t)r * gm * gk, T);
    orc_quantize_row_groups(T, br, bk, fmt, tq, dT);
    if (Tq_out) memcpy(Tq_out + r * tsz, tq, (size_t)tsz);
    if (dT_out) memcpy(dT_out + (int64_t)r * nta, dT, sizeof(float) * (size_t)nta);
    orc_block_product_groups(tq, sq + r * ssz, dT, dS + r * nsb, br, bc, bk, fmt, Mr + r * msz);
  }
  if (Sq_out) memcpy(Sq_out, sq, (size_t)(ssz * R));
  if (dS_out) memcpy(dS_out, dS, sizeof(float) * (size_t)(nsb * R));
  orc_reconstruct(Mr, W, R, gm, gn, br, bc, C);
  if (flags & 1)
    for (int t = 0; t < M; ++t) {
      float f = ldexpf(1.0f, kx[t]);
      for (int j = 0; j < N; ++j) C[(int64_t)t * N + j] = C[(int64_t)t * N + j] * f;
    }
  if (!Mr_out) free(Mr);
  free(T);
  free(tq);
  free(dT);
  free(S);
  free(Sb);
  free(qS);
  free(dS);
  free(sq);
  free(As);
  free(kx);
  return 0;
}
