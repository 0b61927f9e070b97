/*
 * pot_oracle.c -- plain, slow CPU oracle for power-of-two-key decode attention
 * ("Shift-Accumulate Attention", arXiv 2609.09208).
 *
 * TEST INFRASTRUCTURE ONLY. Only the test suite, the smoke check and the
 * benchmark's CPU-baseline leg may load or run this file. It shares no code,
 * header, table or constant generator with the GPU library: every layout and
 * constant below is re-derived here from the paper and from the written cache
 * layout contract (row = (b*Hkv + h)*t_cap + t; sign/exponent nibbles, element
 * 2i in the low nibble of byte i, nibble = neg<<3 | e, e = 7 is zero; k
 * mantissa bit-planes of 64 bits).
 *
 * Style: scalar loops, fp64 where the paper leaves the precision open, no
 * blocking, no fusion, no SIMD. Build with -O2 -ffp-contract=off so that every
 * fp32 operation written below is one correctly rounded IEEE operation.
 *
 * Every function returns 0 on success and a negative code when an invariant of
 * the method is violated (e.g. a right shift would be needed, eq. exact).
 *
 * Parity pins: see tests/test_oracle_*.py. Nothing here is "parity unpinned"
 * except where a comment says so.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#define DIM 64
#define EXP_MAX 6            /* E: b = 4 bits = 1 sign + 3 exponent bits (Sec. II-A) */
#define ZERO_FIELD 7         /* e = E + 1 reserved for the exact zero (Sec. II-A) */
#define QMAX 127             /* symmetric INT8 query (Sec. II-A, bound of Sec. II-C) */

/* fp32 value of log2(e) rounded to nearest (0x3FB8AA3B). Written as the
 * decimal expansion of that float. */
static const float LOG2E_F32 = 1.44269502162933349609375f;

/* ---------------------------------------------------------------------- */
/* IEEE 754 binary16 conversions, written from the format definition.      */

float oracle_half_to_float(uint16_t h) {
  int sign = (h >> 15) & 1;
  int ex = (h >> 10) & 31;
  int man = h & 1023;
  double v;
  if (ex == 0)
    v = ldexp((double)man, -24); /* subnormal: man * 2^-24 */
  else if (ex == 31)
    v = man ? NAN : INFINITY;
  else
    v = ldexp((double)(man + 1024), ex - 25); /* (1 + man/1024) 2^(ex-15) */
  return (float)(sign ? -v : v);
}

/* Round a float to the nearest binary16 (ties to even). */
uint16_t oracle_float_to_half(float xf) {
  double x = (double)xf;
  uint16_t sign = signbit(x) ? 0x8000 : 0;
  double a = fabs(x);
  if (isnan(x)) return (uint16_t)(sign | 0x7E00);
  if (a >= 65520.0) return (uint16_t)(sign | 0x7C00); /* rounds past 65504 */
  if (a < ldexp(1.0, -14)) {
    /* subnormal range: integer multiple of 2^-24, exact in fp64 */
    double n = rint(a * 16777216.0);
    return (uint16_t)(sign | (uint16_t)n); /* n == 1024 is the smallest normal */
  }
  int ex;
  frexp(a, &ex); /* a = f 2^ex, f in [0.5, 1) */
  int e_unb = ex - 1;
  double mant = rint((ldexp(a, -e_unb) - 1.0) * 1024.0);
  uint32_t bits = (uint32_t)((e_unb + 15) << 10) + (uint32_t)mant; /* carry ok */
  return (uint16_t)(sign | bits);
}

/* ---------------------------------------------------------------------- */
/* Hadamard rotation (Sec. I-A QuaRot, Sec. V-A): orthonormal H/8 with H the */
/* 64x64 Sylvester matrix, H[i][j] = (-1)^popcount(i & j).                    */

static int sylvester_sign(int i, int j) {
  int v = i & j, c = 0;
  while (v) {
    c += v & 1;
    v >>= 1;
  }
  return (c & 1) ? -1 : 1;
}

/* Keys: fp16 inputs. Every fp16 value is an integer multiple of 2^-24 below
 * 2^16, so a signed sum of 64 of them is exact in fp64 in any order; the
 * rotated key is that exact value divided by 8, rounded once to fp32. */
static void rotate_key_row(const float* k, float* out) {
  for (int i = 0; i < DIM; ++i) {
    double s = 0.0;
    for (int j = 0; j < DIM; ++j) s += sylvester_sign(i, j) * (double)k[j];
    out[i] = (float)(s / 8.0);
  }
}

/* Rotated fp32 keys for n rows of fp16 bit patterns (exposed for the pins). */
void oracle_rotate_keys(const uint16_t* k_fp16, int64_t n_rows, float* out) {
  for (int64_t r = 0; r < n_rows; ++r) {
    float kf[DIM];
    for (int m = 0; m < DIM; ++m) kf[m] = oracle_half_to_float(k_fp16[r * DIM + m]);
    rotate_key_row(kf, out + r * DIM);
  }
}

/* Queries: fp32 inputs, where a dense fp64 sum is not exact in general. The
 * rotation is defined as the radix-2 fast Walsh-Hadamard transform in fp64,
 * stages of span 1, 2, 4, ..., 32 each mapping (a, b) -> (a + b, a - b), then
 * division by 8 and one rounding to fp32 (the reading recorded for this
 * build). tests pin it against the exact rational H q. */
void oracle_fwht_query(const float* q, float* out) {
  double v[DIM];
  for (int i = 0; i < DIM; ++i) v[i] = (double)q[i];
  for (int h = 1; h < DIM; h <<= 1) {
    for (int i = 0; i < DIM; i += 2 * h) {
      for (int j = i; j < i + h; ++j) {
        double a = v[j], b = v[j + h];
        v[j] = a + b;
        v[j + h] = a - b;
      }
    }
  }
  for (int i = 0; i < DIM; ++i) out[i] = (float)(v[i] / 8.0);
}

/* ---------------------------------------------------------------------- */
/* Query quantisation (Sec. II-A: INT8 with a per-vector step Delta_i).      */
/* amax = max |q'|; Delta = fl32(amax/127); q^ = clamp(rne(fl32(q' *        */
/* fl32(127/amax))), -127, 127); amax = 0 gives Delta = 0 and q^ = 0.       */

static void quantize_vector(const float* qv, int8_t* qhat, float* delta) {
  float amax = 0.0f;
  for (int m = 0; m < DIM; ++m) {
    float a = fabsf(qv[m]);
    if (a > amax) amax = a;
  }
  if (amax == 0.0f) {
    for (int m = 0; m < DIM; ++m) qhat[m] = 0;
    *delta = 0.0f;
    return;
  }
  float inv = 127.0f / amax;
  for (int m = 0; m < DIM; ++m) {
    float t = qv[m] * inv;
    float r = rintf(t); /* round to nearest, ties to even */
    if (r > QMAX) r = QMAX;
    if (r < -QMAX) r = -QMAX;
    qhat[m] = (int8_t)r;
  }
  *delta = amax / 127.0f;
}

void oracle_quantize_query(int hadamard, const float* q, int64_t n_vec,
                           int8_t* qhat, float* delta, float* q_rot) {
  for (int64_t v = 0; v < n_vec; ++v) {
    float qr[DIM];
    if (hadamard)
      oracle_fwht_query(q + v * DIM, qr);
    else
      memcpy(qr, q + v * DIM, sizeof qr);
    if (q_rot) memcpy(q_rot + v * DIM, qr, sizeof qr);
    quantize_vector(qr, qhat + v * DIM, delta + v);
  }
}

/* ---------------------------------------------------------------------- */
/* Key code (Sec. II-A, II-D): value s * sigma * (1 + j/2^k) 2^-e.           */
/* The code of an element is the grid value nearest to u = fl32(|x|/s) in   */
/* log2 distance, found here by brute force over the whole grid in fp64.    */
/* u below 2^-(E+1/2) (the log-midpoint under the smallest magnitude) is    */
/* flushed to the exact zero; u above the top saturates (nearest anyway).   */

typedef struct {
  int neg, e, j, zero;
} elem_code;

/* log2 of every grid value (1 + j/2^k) 2^-e, index e * 2^k + j. */
static void grid_log2(int k, double* out) {
  int nj = 1 << k;
  for (int e = 0; e <= EXP_MAX; ++e)
    for (int j = 0; j < nj; ++j)
      out[e * nj + j] = log2((1.0 + (double)j / nj) * ldexp(1.0, -e));
}

static elem_code encode_element(float x, float s, int k, const double* glog) {
  elem_code c = {0, ZERO_FIELD, 0, 1};
  if (!(s > 0.0f)) return c;           /* no scale: everything is zero     */
  if (x == 0.0f || isnan(x)) return c; /* exact zero (or undefined input)  */
  float u = fabsf(x) / s;              /* one correctly rounded division   */
  if (!(u > 0.0f)) return c;           /* underflowed ratio                */
  double lu = log2((double)u);
  if (lu < -((double)EXP_MAX + 0.5)) return c;
  int nj = 1 << k;
  int best_e = 0, best_j = nj - 1; /* the top value (saturation)             */
  if (!isinf(lu)) {
    double best = INFINITY;
    for (int e = 0; e <= EXP_MAX; ++e) {
      for (int j = 0; j < nj; ++j) {
        double dist = fabs(lu - glog[e * nj + j]);
        if (dist < best) {
          best = dist;
          best_e = e;
          best_j = j;
        }
      }
    }
  }
  c.neg = x < 0.0f;
  c.e = best_e;
  c.j = best_j;
  c.zero = 0;
  return c;
}

int oracle_encode_keys(int mant_bits, int hadamard, const uint16_t* k_fp16,
                       int64_t n_rows, int scale_mode, float* key_scale,
                       uint8_t* codes_se, uint8_t* codes_m) {
  if (mant_bits < 0 || mant_bits > 4) return -1;
  double glog[(EXP_MAX + 1) * 16];
  grid_log2(mant_bits, glog);
  for (int64_t r = 0; r < n_rows; ++r) {
    float kf[DIM], kr[DIM];
    for (int m = 0; m < DIM; ++m) kf[m] = oracle_half_to_float(k_fp16[r * DIM + m]);
    if (hadamard)
      rotate_key_row(kf, kr);
    else
      memcpy(kr, kf, sizeof kr);
    float s;
    if (scale_mode == 0) {
      s = 0.0f;
      for (int m = 0; m < DIM; ++m)
        if (fabsf(kr[m]) > s) s = fabsf(kr[m]);
      key_scale[r] = s;
    } else {
      s = key_scale[r];
    }
    uint8_t* se = codes_se + r * (DIM / 2);
    memset(se, 0, DIM / 2);
    uint8_t* mp = mant_bits ? codes_m + r * 8 * mant_bits : NULL;
    if (mp) memset(mp, 0, (size_t)8 * mant_bits);
    for (int m = 0; m < DIM; ++m) {
      elem_code c = encode_element(kr[m], s, mant_bits, glog);
      int nib = c.zero ? ZERO_FIELD : ((c.neg << 3) | c.e);
      se[m / 2] |= (uint8_t)(nib << (4 * (m % 2)));
      for (int b = 0; b < mant_bits; ++b)
        if (!c.zero && ((c.j >> b) & 1)) mp[8 * b + m / 8] |= (uint8_t)(1u << (m % 8));
    }
  }
  return 0;
}

/* Decode one element code from the cache layout. */
static void read_code(const uint8_t* se, const uint8_t* mp, int k, int m,
                      int* neg, int* e, int* j) {
  int nib = (se[m / 2] >> (4 * (m % 2))) & 15;
  *neg = (nib >> 3) & 1;
  *e = nib & 7;
  int jj = 0;
  for (int b = 0; b < k; ++b) jj |= ((mp[8 * b + m / 8] >> (m % 8)) & 1) << b;
  *j = jj;
}

/* Exact score accumulator at head-room F (eq. sac, generalised to PoT-Mk at
 * scale 2^-(F+k)): acc = sum_m sigma_m q^_m (2^k + j_m) 2^(F - e_m), over
 * non-zero codes. Computed with integer multiplications by powers of two in
 * int64; returns -2 if a term would need a negative exponent (a right shift,
 * excluded by eq. exact) and -3 if the sum leaves int32. */
static int sac_score(const int8_t* qh, const uint8_t* se, const uint8_t* mp,
                     int k, int F, int32_t* acc_out) {
  int64_t acc = 0;
  for (int m = 0; m < DIM; ++m) {
    int neg, e, j;
    read_code(se, mp, k, m, &neg, &e, &j);
    if (e == ZERO_FIELD) continue;
    int r = F - e;
    if (r < 0) return -2;
    int64_t pow2 = (int64_t)1 << r;
    int64_t term = (int64_t)qh[m] * ((int64_t)(1 << k) + j) * pow2;
    acc += neg ? -term : term;
  }
  if (acc > INT32_MAX || acc < INT32_MIN) return -3;
  *acc_out = (int32_t)acc;
  return 0;
}

/* ---------------------------------------------------------------------- */
/* Softmax over log2-domain scores x (Sec. II-E).                           */
/*  - two-pass reference: M = ceil(max x), w = 2^(x - M) in fp64, O = sum  */
/*    w V / sum w.                                                          */
/*  - online form (tile > 0): per split a running integer M updated per     */
/*    tile, exact 2^(M_old - M_new) rescales, splits merged with exact      */
/*    2^(M_s - M) factors. Used by tests to pin online == two-pass.         */

/* One cache row of values: fp16 (v16), or INT8 codes v8 with the per-token */
/* power-of-two scale 2^-g (Sec. II-E), whose value is v8[d] * 2^-g.        */
typedef struct {
  const uint16_t* v16;
  const int8_t* v8;
  int g;
} value_row;

static double value_at(const value_row* r, int d) {
  if (r->v8) return ldexp((double)r->v8[d], -r->g); /* exact */
  return (double)oracle_half_to_float(r->v16[d]);
}

/* Weight of a key with log2-domain score x under the integer maximum M.     */
/*  pow2 = 0: the softmax weight 2^(x - M) (eq. logsm with exact exp2).     */
/*  pow2 = 1: the power-of-two weight A~ = 2^-k of eq. logsm, k = M - c with  */
/*  c = ceil(x - 1/2), i.e. k = M - x rounded half up. x - 1/2 is formed in   */
/*  fp64, where it is exact for every finite fp32 x (below 2^53 the two       */
/*  operands fit 54 bits; above, x is an even integer and the tie rounds back */
/*  to x, whose ceiling is still x - 1/2 rounded up); in fp32 it is not       */
/*  (x = -0.5 + 2^-25 would round to -1).                                     */
/*  (The paper says "round"; rounding half up makes k - M a function of x    */
/*  alone, so a running maximum that rises by any integer rescales exactly.) */
static double key_weight(float x, int32_t M, int pow2) {
  if (pow2) return ldexp(1.0, (int)ceil((double)x - 0.5) - M);
  return exp2((double)x - (double)M);
}

static void softmax_av(const float* x, const value_row* vrows, int T,
                       int split_len, int tile, int pow2, int32_t* m_final,
                       int32_t* m_split, double* out) {
  float xmax = -INFINITY;
  for (int t = 0; t < T; ++t)
    if (x[t] > xmax) xmax = x[t];
  int32_t M = (int32_t)ceilf(xmax);
  if (m_final) *m_final = M;
  int n_split = (T + split_len - 1) / split_len;
  if (m_split) {
    for (int s = 0; s < n_split; ++s) {
      float sm = -INFINITY;
      for (int t = s * split_len; t < T && t < (s + 1) * split_len; ++t)
        if (x[t] > sm) sm = x[t];
      m_split[s] = (int32_t)ceilf(sm);
    }
  }
  if (!out) return;
  if (tile <= 0) {
    double l = 0.0, o[DIM] = {0};
    for (int t = 0; t < T; ++t) {
      double w = key_weight(x[t], M, pow2);
      l += w;
      for (int d = 0; d < DIM; ++d) o[d] += w * value_at(&vrows[t], d);
    }
    for (int d = 0; d < DIM; ++d) out[d] = o[d] / l;
    return;
  }
  /* online */
  int32_t* Ms = (int32_t*)malloc(sizeof(int32_t) * n_split);
  double* ls = (double*)malloc(sizeof(double) * n_split);
  double* os = (double*)malloc(sizeof(double) * n_split * DIM);
  for (int s = 0; s < n_split; ++s) {
    int32_t Mrun = INT32_MIN;
    double l = 0.0, o[DIM] = {0};
    int t_end = (s + 1) * split_len < T ? (s + 1) * split_len : T;
    for (int t0 = s * split_len; t0 < t_end; t0 += tile) {
      int t1 = t0 + tile < t_end ? t0 + tile : t_end;
      float tm = -INFINITY;
      for (int t = t0; t < t1; ++t)
        if (x[t] > tm) tm = x[t];
      int32_t Mt = (int32_t)ceilf(tm);
      if (Mt > Mrun) {
        if (Mrun != INT32_MIN) {
          double f = ldexp(1.0, Mrun - Mt); /* exact power of two */
          l *= f;
          for (int d = 0; d < DIM; ++d) o[d] *= f;
        }
        Mrun = Mt;
      }
      for (int t = t0; t < t1; ++t) {
        double w = key_weight(x[t], Mrun, pow2);
        l += w;
        for (int d = 0; d < DIM; ++d) o[d] += w * value_at(&vrows[t], d);
      }
    }
    Ms[s] = Mrun;
    ls[s] = l;
    memcpy(os + s * DIM, o, sizeof o);
  }
  int32_t Mg = INT32_MIN;
  for (int s = 0; s < n_split; ++s)
    if (Ms[s] > Mg) Mg = Ms[s];
  double L = 0.0, O[DIM] = {0};
  for (int s = 0; s < n_split; ++s) {
    double f = ldexp(1.0, Ms[s] - Mg);
    L += f * ls[s];
    for (int d = 0; d < DIM; ++d) O[d] += f * os[s * DIM + d];
  }
  for (int d = 0; d < DIM; ++d) out[d] = O[d] / L;
  free(Ms);
  free(ls);
  free(os);
}

/* ---------------------------------------------------------------------- */
/* Decode attention with PoT keys, whole problem.                           */
/*  x_t = fl32(fl32(float(acc_t) * s_t) * c), c = fl32(fl32(Delta *         */
/*  log2e) * 2^-(F+k+3)); 2^-3 = 1/sqrt(64) (eq. attn), log2e moves the     */
/*  softmax to base 2 (eq. logsm).                                          */
/* Optional outputs may be NULL. scores/x are [B][Hq][T], m_split is        */
/* [B][Hq][ceil(T/split_len)], out is [B][Hq][64] in fp64.                  */

static int pot_decode_impl(int mant_bits, int frac_bits, int hadamard,
                           const float* q, const uint8_t* codes_se,
                           const uint8_t* codes_m, const float* key_scale,
                           const uint16_t* v, const int8_t* v8, const int8_t* v_exp,
                           int64_t t_cap, const int32_t* kv_head_of_q,
                           int B, int Hq, int Hkv, int T, int split_len, int tile, int pow2,
                           int8_t* qhat_out, float* delta_out, int32_t* scores_out,
                           float* x_out, int32_t* m_final, int32_t* m_split,
                           double* out) {
  if (T < 1 || T > t_cap || split_len < 1) return -1;
  int k = mant_bits;
  int n_split = (T + split_len - 1) / split_len;
  float* x = (float*)malloc(sizeof(float) * T);
  value_row* vrows = (value_row*)malloc(sizeof(value_row) * T);
  int rc = 0;
  for (int b = 0; b < B && rc == 0; ++b) {
    for (int i = 0; i < Hq && rc == 0; ++i) {
      int h = kv_head_of_q[i];
      int64_t bh = (int64_t)b * Hq + i;
      int8_t qh[DIM];
      float delta;
      oracle_quantize_query(hadamard, q + bh * DIM, 1, qh, &delta, NULL);
      if (qhat_out) memcpy(qhat_out + bh * DIM, qh, DIM);
      if (delta_out) delta_out[bh] = delta;
      float c = ldexpf(delta * LOG2E_F32, -(frac_bits + k + 3));
      for (int t = 0; t < T; ++t) {
        int64_t row = ((int64_t)b * Hkv + h) * t_cap + t;
        int32_t acc;
        rc = sac_score(qh, codes_se + row * (DIM / 2),
                       k ? codes_m + row * 8 * k : NULL, k, frac_bits, &acc);
        if (rc) break;
        if (scores_out) scores_out[bh * T + t] = acc;
        x[t] = ((float)acc * key_scale[row]) * c;
        if (x_out) x_out[bh * T + t] = x[t];
        vrows[t].v16 = v8 ? NULL : v + row * DIM;
        vrows[t].v8 = v8 ? v8 + row * DIM : NULL;
        vrows[t].g = v8 ? v_exp[row] : 0;
      }
      if (rc) break;
      softmax_av(x, vrows, T, split_len, tile, pow2, m_final ? m_final + bh : NULL,
                 m_split ? m_split + bh * n_split : NULL,
                 out ? out + bh * DIM : NULL);
    }
  }
  free(x);
  free(vrows);
  return rc;
}

int oracle_pot_decode(int mant_bits, int frac_bits, int hadamard,
                      const float* q, const uint8_t* codes_se,
                      const uint8_t* codes_m, const float* key_scale,
                      const uint16_t* v, int64_t t_cap, const int32_t* kv_head_of_q,
                      int B, int Hq, int Hkv, int T, int split_len, int tile,
                      int8_t* qhat_out, float* delta_out, int32_t* scores_out,
                      float* x_out, int32_t* m_final, int32_t* m_split,
                      double* out) {
  return pot_decode_impl(mant_bits, frac_bits, hadamard, q, codes_se, codes_m, key_scale, v,
                         NULL, NULL, t_cap, kv_head_of_q, B, Hq, Hkv, T, split_len, tile, 0,
                         qhat_out, delta_out, scores_out, x_out, m_final, m_split, out);
}

/* The same with the values as INT8 codes v8 [rows][64] and per-row exponents */
/* v_exp [rows] (value v8 * 2^-v_exp, Sec. II-E).                            */
int oracle_pot_decode_v8(int mant_bits, int frac_bits, int hadamard,
                         const float* q, const uint8_t* codes_se,
                         const uint8_t* codes_m, const float* key_scale,
                         const int8_t* v8, const int8_t* v_exp, int64_t t_cap,
                         const int32_t* kv_head_of_q, int B, int Hq, int Hkv, int T,
                         int split_len, int tile, int8_t* qhat_out, float* delta_out,
                         int32_t* scores_out, float* x_out, int32_t* m_final,
                         int32_t* m_split, double* out) {
  return pot_decode_impl(mant_bits, frac_bits, hadamard, q, codes_se, codes_m, key_scale, NULL,
                         v8, v_exp, t_cap, kv_head_of_q, B, Hq, Hkv, T, split_len, tile, 0,
                         qhat_out, delta_out, scores_out, x_out, m_final, m_split, out);
}

/* Both products by powers of two (Sec. II-E, eq. logsm and eq. av): the     */
/* same scores, INT8 values v8 * 2^-v_exp, and the power-of-two weights      */
/* A~_t = 2^-k_t: O = sum_t A~_t v_t / sum_t A~_t (the normalisation eq. av   */
/* leaves out), every product A~_t v_t exact, sums in fp64. No k_max cut.     */
int oracle_pot_decode_v8_pow2(int mant_bits, int frac_bits, int hadamard,
                              const float* q, const uint8_t* codes_se,
                              const uint8_t* codes_m, const float* key_scale,
                              const int8_t* v8, const int8_t* v_exp, int64_t t_cap,
                              const int32_t* kv_head_of_q, int B, int Hq, int Hkv, int T,
                              int split_len, int tile, int8_t* qhat_out, float* delta_out,
                              int32_t* scores_out, float* x_out, int32_t* m_final,
                              int32_t* m_split, double* out) {
  return pot_decode_impl(mant_bits, frac_bits, hadamard, q, codes_se, codes_m, key_scale, NULL,
                         v8, v_exp, t_cap, kv_head_of_q, B, Hq, Hkv, T, split_len, tile, 1,
                         qhat_out, delta_out, scores_out, x_out, m_final, m_split, out);
}

/* Attention of one query over given log2-domain scores x[T] and INT8 value  */
/* rows v8[T][64] * 2^-v_exp[t] (test hook for the weight rules): pow2 = 0   */
/* softmax weights, 1 power-of-two weights; tile > 0 runs the online form.   */
int oracle_attend_x(const float* x, const int8_t* v8, const int8_t* v_exp, int T,
                    int split_len, int tile, int pow2, int32_t* m_final, double* out) {
  if (T < 1 || split_len < 1) return -1;
  value_row* vrows = (value_row*)malloc(sizeof(value_row) * T);
  for (int t = 0; t < T; ++t) {
    vrows[t].v16 = NULL;
    vrows[t].v8 = v8 + (int64_t)t * DIM;
    vrows[t].g = v_exp[t];
  }
  softmax_av(x, vrows, T, split_len, tile, pow2, m_final, NULL, out);
  free(vrows);
  return 0;
}

/* ---------------------------------------------------------------------- */
/* INT8 values with a power-of-two per-token scale (Sec. II-E): the paper   */
/* stores V as INT8 codes with a scale 2^-g per token; how g and the codes  */
/* are rounded is not stated. Reading used here: g is the largest integer   */
/* with max_d |v_d| * 2^g <= 127 (g = 0 for an all-zero row) and           */
/* v^_d = round-half-even(v_d * 2^g), so |v^_d| <= 127 and the row maximum  */
/* lands in [64, 127].                                                      */

int oracle_quantize_values(const uint16_t* v_fp16, int64_t n_rows, int8_t* vhat,
                           int8_t* v_exp) {
  for (int64_t r = 0; r < n_rows; ++r) {
    double v[DIM], amax = 0.0;
    for (int d = 0; d < DIM; ++d) {
      v[d] = (double)oracle_half_to_float(v_fp16[r * DIM + d]);
      if (v[d] != v[d] || isinf(v[d])) return -1;
      if (fabs(v[d]) > amax) amax = fabs(v[d]);
    }
    int g = 0;
    if (amax > 0.0) {
      while (ldexp(amax, g) > QMAX) --g;        /* exact: scaling by 2^g */
      while (ldexp(amax, g + 1) <= QMAX) ++g;
    }
    if (g < -128 || g > 127) return -2;
    v_exp[r] = (int8_t)g;
    for (int d = 0; d < DIM; ++d) {
      double c = nearbyint(ldexp(v[d], g)); /* default rounding: half to even */
      if (c > QMAX || c < -QMAX) return -3;
      vhat[r * DIM + d] = (int8_t)c;
    }
  }
  return 0;
}

/* ---------------------------------------------------------------------- */
/* INT8 uniform key comparator: s = fl32(amax/127), k^ = clamp(rne(fl32(K' * */
/* fl32(127/amax)))), score acc = sum q^ k^ (exact int), x = fl32(fl32(      */
/* float(acc) * s) * fl32(fl32(Delta*log2e) * 2^-3)).                        */

int oracle_int8_encode_keys(int hadamard, const uint16_t* k_fp16,
                            int64_t n_rows, float* key_scale, int8_t* codes) {
  for (int64_t r = 0; r < n_rows; ++r) {
    float kf[DIM], kr[DIM];
    for (int m = 0; m < DIM; ++m) kf[m] = oracle_half_to_float(k_fp16[r * DIM + m]);
    if (hadamard)
      rotate_key_row(kf, kr);
    else
      memcpy(kr, kf, sizeof kr);
    quantize_vector(kr, codes + r * DIM, key_scale + r);
  }
  return 0;
}

int oracle_int8_decode(int hadamard, const float* q, const int8_t* codes,
                       const float* key_scale, const uint16_t* v, int64_t t_cap,
                       const int32_t* kv_head_of_q, int B, int Hq, int Hkv,
                       int T, int split_len, int8_t* qhat_out,
                       float* delta_out, int32_t* scores_out, int32_t* m_final,
                       int32_t* m_split, double* out) {
  if (T < 1 || T > t_cap || split_len < 1) return -1;
  int n_split = (T + split_len - 1) / split_len;
  float* x = (float*)malloc(sizeof(float) * T);
  value_row* vrows = (value_row*)malloc(sizeof(value_row) * T);
  for (int b = 0; b < B; ++b) {
    for (int i = 0; i < Hq; ++i) {
      int h = kv_head_of_q[i];
      int64_t bh = (int64_t)b * Hq + i;
      int8_t qh[DIM];
      float delta;
      oracle_quantize_query(hadamard, q + bh * DIM, 1, qh, &delta, NULL);
      if (qhat_out) memcpy(qhat_out + bh * DIM, qh, DIM);
      if (delta_out) delta_out[bh] = delta;
      float c = ldexpf(delta * LOG2E_F32, -3);
      for (int t = 0; t < T; ++t) {
        int64_t row = ((int64_t)b * Hkv + h) * t_cap + t;
        int64_t acc = 0;
        for (int m = 0; m < DIM; ++m) acc += (int64_t)qh[m] * codes[row * DIM + m];
        if (scores_out) scores_out[bh * T + t] = (int32_t)acc;
        x[t] = ((float)acc * key_scale[row]) * c;
        vrows[t].v16 = v + row * DIM;
        vrows[t].v8 = NULL;
        vrows[t].g = 0;
      }
      softmax_av(x, vrows, T, split_len, 0, 0, m_final ? m_final + bh : NULL,
                 m_split ? m_split + bh * n_split : NULL,
                 out ? out + bh * DIM : NULL);
    }
  }
  free(x);
  free(vrows);
  return 0;
}

/* ---------------------------------------------------------------------- */
/* FP16 baseline: q rounded to fp16; S = q16 . K / sqrt(64) and the softmax */
/* and A.V in fp64 (the plain definition of eq. attn on an fp16 cache).     */

int oracle_fp16_decode(const float* q, const uint16_t* k, const uint16_t* v,
                       int64_t t_cap, const int32_t* kv_head_of_q, int B,
                       int Hq, int Hkv, int T, double* out) {
  if (T < 1 || T > t_cap) return -1;
  double* sc = (double*)malloc(sizeof(double) * T);
  for (int b = 0; b < B; ++b) {
    for (int i = 0; i < Hq; ++i) {
      int h = kv_head_of_q[i];
      int64_t bh = (int64_t)b * Hq + i;
      double q16[DIM];
      for (int m = 0; m < DIM; ++m)
        q16[m] = oracle_half_to_float(oracle_float_to_half(q[bh * DIM + m]));
      double smax = -INFINITY;
      for (int t = 0; t < T; ++t) {
        int64_t row = ((int64_t)b * Hkv + h) * t_cap + t;
        double s = 0.0;
        for (int m = 0; m < DIM; ++m) s += q16[m] * oracle_half_to_float(k[row * DIM + m]);
        sc[t] = s / 8.0;
        if (sc[t] > smax) smax = sc[t];
      }
      double l = 0.0, o[DIM] = {0};
      for (int t = 0; t < T; ++t) {
        int64_t row = ((int64_t)b * Hkv + h) * t_cap + t;
        double w = exp(sc[t] - smax);
        l += w;
        for (int d = 0; d < DIM; ++d) o[d] += w * oracle_half_to_float(v[row * DIM + d]);
      }
      for (int d = 0; d < DIM; ++d) out[bh * DIM + d] = o[d] / l;
    }
  }
  free(sc);
  return 0;
}
