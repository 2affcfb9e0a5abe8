/*
 * quake_oracle.c — plain, slow, obviously-correct CPU oracle for QuAKE
 * (arXiv:2412.00408).
 *
 * TEST INFRASTRUCTURE. Only the test suite, the smoke check and the CPU
 * baseline of the benchmark load this library. The HIP product path never
 * includes, links or calls anything here, and nothing here is shared with it.
 *
 * Build (fp contraction OFF, no fast-math, so every fused multiply-add the
 * method prescribes is an explicit fmaf() and nothing else is fused):
 *   gcc -O2 -std=c11 -ffp-contract=off -fno-fast-math -fPIC -shared \
 *       -o liboracle.so quake_oracle.c -lm
 *
 * What each function follows:
 *   qo_quake      Sec. II-B Eq. 2-3, Sec. III-A Eq. 5 (QuAKE), Sec. III-B Eq. 6
 *                 and Algorithm 1 (QuAKE2), with explicit constants c0, c1.
 *                 Every operator takes mode QO_Q2M too: QuAKE2 with the
 *                 coefficients of Eq. 6 that minimise the worst-case relative
 *                 error (the grid-search optimum of Sec. III-B, here solved by
 *                 the Remez exchange; qo_q2m_coefficients).
 *   qo_exp        Sec. III-A: e^(a x + b) with the affine map folded into c0, c1.
 *   qo_softmax    Sec. III-C, Algorithm 2 (SoftMax-QuAKEx).
 *   qo_gelu       Sec. II-C Eq. 4 rewritten as Sec. III-D Eq. 7.
 *   qo_sigmoid    Sec. III-D logistic function (and SiLU = x * logistic).
 *   qo_softmax_causal
 *                 Algorithm 2 on rows whose entries past a causal limit are
 *                 masked: entry (r, j) takes part iff j <= r mod period + shift;
 *                 masked entries are not read and give 0 (as -inf inputs would).
 *   qo_softmax_unfused, qo_gelu_unfused
 *                 the operators of Sec. V-A's fusion study (Table IV) with the
 *                 standard exponential plugged in: softmax computes (v - m) * t
 *                 and then e^s; GELU computes k * x * (1/0.044715 + x^2) and then
 *                 e^-s; EXACT mode is the vanilla operator with exp.
 *   qo_softmax_numerators
 *                 Algorithm 2 without the final division: the exponentials of
 *                 a binary32 row against its max, and the row sum (attention).
 *   qo_gelu_f32in qo_gelu on binary32 inputs with output in any format (the
 *                 epilogue of a matrix product: GELU of the binary32 sums).
 *   qo_exp16      Sec. II-A/II-B in a 16-bit format's own layout: Eq. 3 with
 *                 the l_m and B of binary16 / bfloat16, Algorithm 1 with the
 *                 16-bit masks and the refinement in that format's arithmetic.
 *   qo_round      IEEE-754 round-to-nearest-even from double to binary32,
 *                 binary16 and bfloat16 (the output formats).
 *
 * Readings taken where the paper is silent (each also listed in the design
 * notes): convert_to_int truncates toward zero; x*c0 + c1 is one binary32 fma;
 * (a_m^2 + 2)/3 is fmaf(a_m, a_m, 2) * fl32(1/3) (QO_Q2_DIV keeps the literal
 * division for comparison); l is clamped to [0, 255*2^23] before the
 * conversion (the v_min clamp of Algorithm 2, which as printed mixes units);
 * the Schraudolph bias 0.0436 applies to first-order QuAKE outside softmax
 * only; an all -inf softmax row gives zeros; constants are evaluated in double
 * from their definitions and rounded once to binary32; sums are accumulated in
 * double and the final division is done in double and rounded once.
 */
#include <math.h>
#include <stdint.h>
#include <string.h>

/* ---- mode / dtype codes (same numeric values as the public ABI enums) ---- */
enum { QO_EXACT = 0, QO_Q1 = 1, QO_Q2 = 2, QO_Q2M = 3, QO_Q2_DIV = 4 };
enum { QO_F32 = 0, QO_F16 = 1, QO_BF16 = 2 };

/* ---- IEEE binary32 layout, Sec. II-A Eq. 1: l_e = 8, l_m = 23, B = 127 ---- */
#define LM 23
#define BIAS 127
/* Masks of Algorithm 1: keep mantissa / keep sign+exponent / exponent := B. */
#define MASK_MANT 0x007FFFFFu
#define MASK_SIGN_EXP 0xFF800000u
#define EXP_B 0x3F800000u

static const double LN2 = 0.693147180559945309417232121458176568; /* ln 2 */
static const double TWO_LM = 8388608.0;                            /* 2^23 */

static uint32_t f2u(float f) { uint32_t u; memcpy(&u, &f, 4); return u; }
static float u2f(uint32_t u) { float f; memcpy(&f, &u, 4); return f; }

/* ------------------------------------------------------------------------ */
/* Constants, each from its real-number definition in double, rounded once. */
/* ------------------------------------------------------------------------ */

/* 127 * 2^23: c1 of the plain natural exponential (Sec. III-A). */
static float k127(void) { return (float)(BIAS * TWO_LM); }

/* Upper clamp of l: biased exponent 255, mantissa 0 = bits of +inf. */
static float l_hi(void) { return (float)(255.0 * TWO_LM); }

/* Eq. 5 with p = a/ln2 (natural exp folded into base 2): c0 = 2^23 * p. */
static float c0_of(double a) { return (float)((a / LN2) * TWO_LM); }

/* Eq. 5 with q = b/ln2, plus the Schraudolph bias for first order:
 * c1 = 2^23 * (B - beta + q), beta = 0.0436 (Sec. III-A). */
static float c1_of(double b, int mode) {
  double beta = (mode == QO_Q1) ? 0.0436 : 0.0;
  return (float)(((BIAS - beta) + b / LN2) * TWO_LM);
}

/* fl32(1/3): a0 = 1/3 of the continuity-constrained coefficients, Sec. III-B. */
static float third(void) { return (float)(1.0 / 3.0); }

/*
 * Minimax coefficients of Eq. 6: the quadratic y(a) = a0 a^2 + a1 a + a2 that
 * minimises the worst-case relative error |y(a) 2^(1-a) - 1| over a = a_m in
 * [1, 2] (f = a - 1 in [0, 1)), the problem the paper solves by grid search
 * (Sec. III-B). Solved here by the Remez exchange: the best quadratic's error
 * takes its extreme value E with alternating signs at four points, both ends
 * and the two interior roots of e'(a) = 0. With w(a) = 2^(1-a),
 * e'(a) = w (y'(a) - ln2 y(a)), so the interior extrema are the roots of the
 * quadratic ln2 a0 a^2 + (ln2 a1 - 2 a0) a + (ln2 a2 - a1). Each step solves
 * the 4x4 linear system y(r_i) w(r_i) - (-1)^i E = 1 on the current points
 * r_i and moves the interior points to those roots. Computed once in double
 * when the library loads; each coefficient is then rounded once to binary32.
 */
static double q2m_c[3], q2m_e, q2m_ref[4];
static float q2m_f[3];

/* Gaussian elimination with partial pivoting on a 4x5 augmented matrix. */
static void solve4(double m[4][5], double* out) {
  for (int c = 0; c < 4; ++c) {
    int piv = c;
    for (int r = c + 1; r < 4; ++r)
      if (fabs(m[r][c]) > fabs(m[piv][c])) piv = r;
    for (int k = 0; k < 5; ++k) {
      double t = m[c][k];
      m[c][k] = m[piv][k];
      m[piv][k] = t;
    }
    for (int r = 0; r < 4; ++r) {
      if (r == c) continue;
      double f = m[r][c] / m[c][c];
      for (int k = c; k < 5; ++k) m[r][k] -= f * m[c][k];
    }
  }
  for (int c = 0; c < 4; ++c) out[c] = m[c][4] / m[c][c];
}

static void q2m_remez(void) {
  double r[4] = {1.0, 4.0 / 3.0, 5.0 / 3.0, 2.0};
  double sol[4] = {1.0 / 3.0, 0.0, 2.0 / 3.0, 0.0};
  for (int it = 0; it < 100; ++it) {
    double m[4][5];
    for (int i = 0; i < 4; ++i) {
      double w = exp2(1.0 - r[i]);
      m[i][0] = r[i] * r[i] * w;
      m[i][1] = r[i] * w;
      m[i][2] = w;
      m[i][3] = (i % 2) ? 1.0 : -1.0;   /* -(-1)^i E */
      m[i][4] = 1.0;
    }
    solve4(m, sol);
    /* interior extrema: roots of A a^2 + B a + C */
    double A = LN2 * sol[0], B = LN2 * sol[1] - 2.0 * sol[0], C = LN2 * sol[2] - sol[1];
    double disc = sqrt(B * B - 4.0 * A * C);
    double q = -0.5 * (B + (B >= 0 ? disc : -disc));
    double x1 = q / A, x2 = C / q;
    double lo = x1 < x2 ? x1 : x2, hi = x1 < x2 ? x2 : x1;
    double moved = fabs(lo - r[1]) + fabs(hi - r[2]);
    r[1] = lo;
    r[2] = hi;
    if (moved < 1e-15) break;
  }
  for (int k = 0; k < 3; ++k) {
    q2m_c[k] = sol[k];
    q2m_f[k] = (float)sol[k];
  }
  q2m_e = fabs(sol[3]);
  for (int k = 0; k < 4; ++k) q2m_ref[k] = r[k];
}

__attribute__((constructor)) static void qo_init(void) { q2m_remez(); }

/* 1/0.044715 of Eq. 7. */
static float a_gelu(void) { return (float)(1.0 / 0.044715); }

/* Scale of the logistic argument in Eq. 7: 2 * 0.044715 * sqrt(2/pi). */
static double k_gelu(void) { return 2.0 * 0.044715 * sqrt(2.0 / 3.14159265358979323846264338327950288); }

/* ------------------------------------------------------------------------ */
/* The approximation itself.                                                */
/* ------------------------------------------------------------------------ */

/*
 * QuAKE / QuAKE2 of one binary32 input with explicit c0, c1.
 *   order QO_Q1     : Eq. 2-3 — z = int(l), result = z's bits as a float.
 *   order QO_Q2     : Algorithm 1 — a_m = 1 + {.} from z's mantissa with the
 *                     exponent field set to B; y_m = (a_m^2 + 2)/3 (Eq. 6,
 *                     a0 = 1/3, a1 = 0, a2 = 2/3) as fmaf(a_m, a_m, 2) * fl(1/3);
 *                     result = z's sign+exponent field joined with y_m's mantissa.
 *   order QO_Q2M    : as QO_Q2 with the minimax coefficients of Eq. 6 (above),
 *                     y_m = fmaf(fmaf(a0, a_m, a1), a_m, a2) (Horner, two FMAs);
 *                     y_m stays inside [1, 2), so the same join applies.
 *                     Where a_m = 1 (z's mantissa field is 0: every integer
 *                     exponent, and both ends of the clamp) y_m is taken as 1,
 *                     the value 2^0 itself, so the result is z's bits: exact
 *                     powers of two, 0 for l <= 0 (masked -inf entries) and
 *                     +inf at the top of the clamp, as with the paper's
 *                     coefficients (the optimum's y_m(1) = 1.0017 would join
 *                     to a nonzero denormal at the bottom and NaN at the top).
 *   order QO_Q2_DIV : as QO_Q2 with the literal float expression (a*a + 2) / 3.
 */
static float quake_one(float x, float c0, float c1, int order) {
  float l = fmaf(x, c0, c1);             /* Eq. 5, one rounding */
  if (!(l > 0.0f)) l = 0.0f;             /* clamp below (also -inf, NaN) */
  if (l > l_hi()) l = l_hi();            /* clamp above (+inf, overflow) */
  int32_t z = (int32_t)l;                /* convert_to_int, toward zero */
  if (order == QO_Q1) return u2f((uint32_t)z);   /* int_bits_as_float */

  float am = u2f(((uint32_t)z & MASK_MANT) | EXP_B);
  float ym;
  if (order == QO_Q2_DIV) {
    ym = (am * am + 2.0f) / 3.0f;
  } else if (order == QO_Q2M) {
    ym = fmaf(fmaf(q2m_f[0], am, q2m_f[1]), am, q2m_f[2]);
  } else {
    ym = fmaf(am, am, 2.0f) * third();
  }
  uint32_t yi = ((uint32_t)z & MASK_SIGN_EXP) + f2u(ym) - EXP_B;
  if (order == QO_Q2M && ((uint32_t)z & MASK_MANT) == 0) yi = (uint32_t)z;
  return u2f(yi);
}

/*
 * The exact exponential of the comparison (EXACT) operators: 2^s correctly
 * rounded to binary32, the format the paper computes in (Sec. II-A), so it
 * overflows to +inf like expf once 2^s exceeds the largest binary32 value.
 */
static float exp2_binary32(float s) { return (float)exp2((double)s); }

/* ------------------------------------------------------------------------ */
/* Format conversion (I/O only; the method computes in binary32).           */
/* ------------------------------------------------------------------------ */

/*
 * Round a double to a binary format with p significand bits (implicit bit
 * included) and normal exponents [emin, emax], round-to-nearest-even, with
 * gradual underflow and overflow to infinity. Returns the rounded value as a
 * double (exactly representable in the target format).
 */
static double round_format(double v, int p, int emin, int emax) {
  if (isnan(v) || isinf(v) || v == 0.0) return v;
  double a = fabs(v);
  int e2;
  frexp(a, &e2);                 /* a = f * 2^e2, f in [0.5, 1) */
  int E = e2 - 1;                /* floor(log2 a) */
  if (E < emin) E = emin;        /* subnormal range: fixed quantum */
  double quantum = ldexp(1.0, E - (p - 1));
  double r = nearbyint(a / quantum) * quantum;   /* ties to even */
  double maxfin = ldexp(2.0 - ldexp(1.0, 1 - p), emax);
  if (r > maxfin) r = INFINITY;
  return copysign(r, v);
}

static uint16_t enc_bf16(double v) {
  if (isnan(v)) return (uint16_t)(signbit(v) ? 0xFFC0u : 0x7FC0u);
  double r = round_format(v, 8, -126, 127);     /* exact in binary32 */
  return (uint16_t)(f2u((float)r) >> 16);
}

static uint16_t enc_f16(double v) {
  uint16_t s = signbit(v) ? 0x8000u : 0u;
  if (isnan(v)) return (uint16_t)(s | 0x7E00u);
  double r = fabs(round_format(v, 11, -14, 15));
  if (isinf(r)) return (uint16_t)(s | 0x7C00u);
  if (r == 0.0) return s;
  int e2;
  frexp(r, &e2);
  int E = e2 - 1;
  if (E < -14) return (uint16_t)(s | (uint16_t)ldexp(r, 24));   /* subnormal */
  uint16_t mant = (uint16_t)(ldexp(r, -E) * 1024.0 - 1024.0);
  return (uint16_t)(s | (uint16_t)((E + 15) << 10) | mant);
}

static float dec_bf16(uint16_t h) { return u2f((uint32_t)h << 16); }

static float dec_f16(uint16_t h) {
  int s = (h >> 15) & 1, e = (h >> 10) & 31, m = h & 1023;
  float v;
  if (e == 0) v = ldexpf((float)m, -24);
  else if (e == 31) v = m ? NAN : INFINITY;
  else v = ldexpf((float)(1024 + m), e - 25);
  return s ? -v : v;
}

static float load_el(const void* p, int64_t i, int dt) {
  if (dt == QO_F32) return ((const float*)p)[i];
  if (dt == QO_F16) return dec_f16(((const uint16_t*)p)[i]);
  return dec_bf16(((const uint16_t*)p)[i]);
}

/* Store a value, rounding once from double to the output format. */
static void store_el(void* p, int64_t i, int dt, double v) {
  if (dt == QO_F32) ((float*)p)[i] = (float)v;
  else if (dt == QO_F16) ((uint16_t*)p)[i] = enc_f16(v);
  else ((uint16_t*)p)[i] = enc_bf16(v);
}

static int bad_args(int dt, int mode) {
  if (dt < QO_F32 || dt > QO_BF16) return 2;
  if (mode < QO_EXACT || mode > QO_Q2_DIV) return 3;
  return 0;
}

/* ------------------------------------------------------------------------ */
/* Exported functions.                                                      */
/* ------------------------------------------------------------------------ */

/* Fixed constants, for tests: fills out[0..9]. */
void qo_constants(float* out) {
  out[0] = c0_of(1.0);             /* C0_EXP  = 2^23 log2 e          */
  out[1] = k127();                 /* K127    = 127 * 2^23           */
  out[2] = c1_of(0.0, QO_Q1);      /* C1_Q1   = (127 - 0.0436) 2^23  */
  out[3] = l_hi();                 /* L_HI    = 255 * 2^23           */
  out[4] = a_gelu();               /* A_GELU  = 1/0.044715           */
  out[5] = (float)(-(k_gelu() / LN2) * TWO_LM);   /* C0_GELU         */
  out[6] = third();                /* THIRD                          */
  out[7] = c0_of(-1.0);            /* C0_NEG  = -2^23 log2 e         */
  out[8] = (float)(1.0 / LN2);     /* log2 e (EXACT-mode scale)      */
  out[9] = (float)(-k_gelu() / LN2);   /* EXACT-mode GELU scale      */
}

/* The minimax coefficients of Eq. 6 (double), their worst-case relative
 * error E and the four equioscillation points: out[0..2], out[3], out[4..7]. */
void qo_q2m_coefficients(double* out) {
  for (int k = 0; k < 3; ++k) out[k] = q2m_c[k];
  out[3] = q2m_e;
  for (int k = 0; k < 4; ++k) out[4 + k] = q2m_ref[k];
}

/* c0 of the softmax for temperature t (Algorithm 2): 2^23 t / ln2. */
float qo_softmax_c0(float t, int mode) {
  if (mode == QO_EXACT) return (float)((double)t / LN2);
  return (float)(((double)t / LN2) * TWO_LM);
}

/* Raw QuAKE with explicit constants, binary32 in and out. */
int qo_quake(const float* x, float* y, int64_t n, float c0, float c1, int order) {
  if (order != QO_Q1 && order != QO_Q2 && order != QO_Q2M && order != QO_Q2_DIV) return 3;
  for (int64_t i = 0; i < n; ++i) y[i] = quake_one(x[i], c0, c1, order);
  return 0;
}

/* e^(a x + b), Sec. III-A. */
int qo_exp(const void* x, void* y, int64_t n, int dt, int mode, float a, float b) {
  int err = bad_args(dt, mode);
  if (err) return err;
  if (mode == QO_EXACT) {
    float c0e = (float)((double)a / LN2), c1e = (float)((double)b / LN2);
    for (int64_t i = 0; i < n; ++i) {
      float s = fmaf(load_el(x, i, dt), c0e, c1e);
      store_el(y, i, dt, exp2((double)s));
    }
  } else {
    float c0 = c0_of(a), c1 = c1_of(b, mode);
    for (int64_t i = 0; i < n; ++i)
      store_el(y, i, dt, (double)quake_one(load_el(x, i, dt), c0, c1, mode));
  }
  return 0;
}

/* Logistic function (silu = 0) or SiLU x * logistic(x) (silu != 0). */
int qo_sigmoid(const void* x, void* y, int64_t n, int dt, int mode, int silu) {
  int err = bad_args(dt, mode);
  if (err) return err;
  float c0 = c0_of(-1.0), c1 = c1_of(0.0, mode);
  float c0e = (float)(-1.0 / LN2);
  for (int64_t i = 0; i < n; ++i) {
    float xv = load_el(x, i, dt);
    double e = (mode == QO_EXACT) ? (double)exp2_binary32(fmaf(xv, c0e, 0.0f))
                                  : (double)quake_one(xv, c0, c1, mode);
    double num = silu ? (double)xv : 1.0;
    store_el(y, i, dt, num / (1.0 + e));
  }
  return 0;
}

/* GELU via Eq. 7: x * sigma(k * x * (1/0.044715 + x^2)), k = 2*0.044715*sqrt(2/pi). */
int qo_gelu(const void* x, void* y, int64_t n, int dt, int mode) {
  int err = bad_args(dt, mode);
  if (err) return err;
  float A = a_gelu();
  float c0 = (float)(-(k_gelu() / LN2) * TWO_LM), c1 = c1_of(0.0, mode);
  float c0e = (float)(-k_gelu() / LN2);
  for (int64_t i = 0; i < n; ++i) {
    float xv = load_el(x, i, dt);
    float u = fmaf(xv, xv, A);      /* 1/0.044715 + x^2, one FMA */
    float w = xv * u;
    double e = (mode == QO_EXACT) ? (double)exp2_binary32(fmaf(w, c0e, 0.0f))
                                  : (double)quake_one(w, c0, c1, mode);
    store_el(y, i, dt, (double)xv / (1.0 + e));
  }
  return 0;
}

/*
 * Row softmax of t*x, Algorithm 2. `tmp` is caller scratch of cols doubles.
 * Row r of x starts at element r*ldx, row r of y at r*ldy.
 */
int qo_softmax(const void* x, void* y, int64_t rows, int64_t cols, int64_t ldx,
               int64_t ldy, int dt, int mode, float t, double* tmp) {
  int err = bad_args(dt, mode);
  if (err) return err;
  float c0 = qo_softmax_c0(t, mode);
  for (int64_t r = 0; r < rows; ++r) {
    const int64_t bx = r * ldx, by = r * ldy;
    float m = -INFINITY;
    for (int64_t j = 0; j < cols; ++j) {
      float v = load_el(x, bx + j, dt);
      if (v > m) m = v;
    }
    if (m == -INFINITY) {                       /* fully masked row */
      for (int64_t j = 0; j < cols; ++j) store_el(y, by + j, dt, 0.0);
      continue;
    }
    double sum = 0.0;
    if (mode == QO_EXACT) {
      float c1e = fmaf(-c0, m, 0.0f);
      for (int64_t j = 0; j < cols; ++j) {
        tmp[j] = (double)exp2_binary32(fmaf(load_el(x, bx + j, dt), c0, c1e));
        sum += tmp[j];
      }
    } else {
      float c1 = fmaf(-c0, m, k127());          /* 127*2^23 - c0*m */
      for (int64_t j = 0; j < cols; ++j) {
        tmp[j] = (double)quake_one(load_el(x, bx + j, dt), c0, c1, mode);
        sum += tmp[j];
      }
    }
    for (int64_t j = 0; j < cols; ++j) store_el(y, by + j, dt, tmp[j] / sum);
  }
  return 0;
}

/*
 * Softmax with an implicit causal mask: row r uses only its first
 * L = min(cols, r mod period + shift + 1) entries; the others are treated as
 * -inf without being read (exactly what explicit -inf entries give under
 * Algorithm 2 with the clamp of l), and their outputs are 0.
 */
int qo_softmax_causal(const void* x, void* y, int64_t rows, int64_t cols, int64_t ldx,
                      int64_t ldy, int64_t period, int64_t shift, int dt, int mode, float t,
                      double* tmp) {
  int err = bad_args(dt, mode);
  if (err) return err;
  if (period <= 0) return 1;
  float c0 = qo_softmax_c0(t, mode);
  for (int64_t r = 0; r < rows; ++r) {
    const int64_t bx = r * ldx, by = r * ldy;
    int64_t L = r % period + shift + 1;
    if (L > cols) L = cols;
    if (L < 0) L = 0;
    float m = -INFINITY;
    for (int64_t j = 0; j < L; ++j) {
      float v = load_el(x, bx + j, dt);
      if (v > m) m = v;
    }
    for (int64_t j = L; j < cols; ++j) store_el(y, by + j, dt, 0.0);
    if (m == -INFINITY) {
      for (int64_t j = 0; j < L; ++j) store_el(y, by + j, dt, 0.0);
      continue;
    }
    double sum = 0.0;
    float c1 = (mode == QO_EXACT) ? fmaf(-c0, m, 0.0f) : fmaf(-c0, m, k127());
    for (int64_t j = 0; j < L; ++j) {
      float v = load_el(x, bx + j, dt);
      tmp[j] = (mode == QO_EXACT) ? (double)exp2_binary32(fmaf(v, c0, c1))
                                  : (double)quake_one(v, c0, c1, mode);
      sum += tmp[j];
    }
    for (int64_t j = 0; j < L; ++j) store_el(y, by + j, dt, tmp[j] / sum);
  }
  return 0;
}

/* ------------------------------------------------------------------------ */
/* Unfused ("plug-in") operators of the fusion study (Sec. V-A, Table IV).  */
/* ------------------------------------------------------------------------ */

/* The standard natural exponential of a binary32 argument: QuAKE with
 * c0 = 2^23 log2 e and c1 = (127 - beta) 2^23 (Sec. III-A), or the vanilla
 * exp in binary32 (EXACT: 2^(s * fl(log2 e)), the product rounded to binary32). */
static float std_exp(float s, int mode) {
  if (mode == QO_EXACT) return exp2_binary32(s * (float)(1.0 / LN2));
  return quake_one(s, c0_of(1.0), c1_of(0.0, mode), mode);
}

/* Softmax without folding: s_j = (v_j - m) * t in binary32, then e^s_j. */
int qo_softmax_unfused(const void* x, void* y, int64_t rows, int64_t cols, int64_t ldx,
                       int64_t ldy, int dt, int mode, float t, double* tmp) {
  int err = bad_args(dt, mode);
  if (err) return err;
  for (int64_t r = 0; r < rows; ++r) {
    const int64_t bx = r * ldx, by = r * ldy;
    float m = -INFINITY;
    for (int64_t j = 0; j < cols; ++j) {
      float v = load_el(x, bx + j, dt);
      if (v > m) m = v;
    }
    if (m == -INFINITY) {
      for (int64_t j = 0; j < cols; ++j) store_el(y, by + j, dt, 0.0);
      continue;
    }
    double sum = 0.0;
    for (int64_t j = 0; j < cols; ++j) {
      float d = load_el(x, bx + j, dt) - m;   /* max subtraction */
      float s = d * t;                        /* temperature     */
      tmp[j] = (double)std_exp(s, mode);
      sum += tmp[j];
    }
    for (int64_t j = 0; j < cols; ++j) store_el(y, by + j, dt, tmp[j] / sum);
  }
  return 0;
}

/*
 * Algorithm 2 up to the normalisation, for binary32 score rows (the scores of
 * an attention head): p[r, j] = QuAKEx(s[r, j]) with c1 from the row max (the
 * EXACT mode exponentiates the same base-2 argument), and sums[r] = sum_j p[r, j]
 * in double. -inf entries give 0; an all -inf row gives zeros and sum 0.
 */
int qo_softmax_numerators(const float* s, float* p, double* sums, int64_t rows, int64_t cols,
                          int mode, float t) {
  int err = bad_args(QO_F32, mode);
  if (err) return err;
  float c0 = qo_softmax_c0(t, mode);
  for (int64_t r = 0; r < rows; ++r) {
    const float* sr = s + r * cols;
    float* pr = p + r * cols;
    float m = -INFINITY;
    for (int64_t j = 0; j < cols; ++j)
      if (sr[j] > m) m = sr[j];
    double sum = 0.0;
    if (m == -INFINITY) {
      for (int64_t j = 0; j < cols; ++j) pr[j] = 0.0f;
    } else if (mode == QO_EXACT) {
      float c1e = fmaf(-c0, m, 0.0f);
      for (int64_t j = 0; j < cols; ++j) {
        pr[j] = exp2_binary32(fmaf(sr[j], c0, c1e));
        sum += pr[j];
      }
    } else {
      float c1 = fmaf(-c0, m, k127());
      for (int64_t j = 0; j < cols; ++j) {
        pr[j] = quake_one(sr[j], c0, c1, mode);
        sum += pr[j];
      }
    }
    sums[r] = sum;
  }
  return 0;
}

/* GELU via Eq. 7 of binary32 inputs (e.g. the binary32 accumulators of a
 * matrix product), output rounded once to format dt. */
int qo_gelu_f32in(const float* x, void* y, int64_t n, int dt, int mode) {
  int err = bad_args(dt, mode);
  if (err) return err;
  float A = a_gelu();
  float c0 = (float)(-(k_gelu() / LN2) * TWO_LM), c1 = c1_of(0.0, mode);
  float c0e = (float)(-k_gelu() / LN2);
  for (int64_t i = 0; i < n; ++i) {
    float xv = x[i];
    float u = fmaf(xv, xv, A);
    float w = xv * u;
    double e = (mode == QO_EXACT) ? (double)exp2_binary32(fmaf(w, c0e, 0.0f))
                                  : (double)quake_one(w, c0, c1, mode);
    store_el(y, i, dt, (double)xv / (1.0 + e));
  }
  return 0;
}

/* GELU through Eq. 7 without folding its constants into the exponential:
 * s = k * (x * (1/0.044715 + x^2)), y = x / (1 + e^-s). */
int qo_gelu_unfused(const void* x, void* y, int64_t n, int dt, int mode) {
  int err = bad_args(dt, mode);
  if (err) return err;
  float A = a_gelu();
  float k = (float)k_gelu();
  for (int64_t i = 0; i < n; ++i) {
    float xv = load_el(x, i, dt);
    float u = fmaf(xv, xv, A);
    float w = xv * u;
    float s = w * k;
    double e = (double)std_exp(-s, mode);
    store_el(y, i, dt, (double)xv / (1.0 + e));
  }
  return 0;
}

/* ------------------------------------------------------------------------ */
/* QuAKE built in a 16-bit format's own layout (Sec. II-A, II-B).           */
/* ------------------------------------------------------------------------ */

/*
 * e^(a x + b) for binary16 / bfloat16 inputs and outputs, with Eq. 3 taken in
 * the output format itself: z = (x/ln2 + B) 2^l_m is the 16-bit pattern of
 * the result (binary16: l_e = 5, l_m = 10, B = 15; bfloat16: l_e = 8,
 * l_m = 7, B = 127), no binary32 result and no narrowing.
 *   l = fmaf(x, c0, c1) in binary32 (x widened exactly), c0 = fl32(2^l_m a/ln2),
 *       c1 = fl32(2^l_m (B - beta + b/ln2)), beta = 0.0436 for QuAKE only;
 *   l clamped to [0, (2^l_e - 1) 2^l_m] (the top is the pattern of +inf);
 *   z = (int) l, truncating: the 16-bit result of QuAKE (Eq. 2, 3);
 *   QuAKE2 (Algorithm 1 with the 16-bit masks): a_m = (z & (2^l_m - 1)) |
 *       (B << l_m) in [1, 2); y_m = (a_m^2 + 2) / 3 in the format's own
 *       arithmetic, each operation rounded to nearest even once:
 *         binary16: t = fl16(a_m a_m + 2) (one fused operation), y_m = fl16(t fl16(1/3));
 *         bfloat16: t = a_m a_m + 2 (exact in binary32), y_m = fl_bf16(fl32(t fl32(1/3)))
 *       (bfloat16 arithmetic is binary32 arithmetic rounded to bfloat16);
 *       result = z's sign and exponent fields joined with y_m's mantissa.
 * x and y hold raw 16-bit patterns. Modes QO_Q1, QO_Q2 only.
 */
static uint16_t quake16_one(float x, float c0, float c1, int dt, int order) {
  const int lm = (dt == QO_F16) ? 10 : 7;
  const int bias = (dt == QO_F16) ? 15 : 127;
  const int le = (dt == QO_F16) ? 5 : 8;
  const uint32_t mant = (1u << lm) - 1u;
  const float top = (float)(((1 << le) - 1) * (1 << lm));
  float l = fmaf(x, c0, c1);
  if (!(l > 0.0f)) l = 0.0f;
  if (l > top) l = top;
  const uint32_t z = (uint32_t)(int32_t)l;
  if (order == QO_Q1) return (uint16_t)z;
  const uint32_t am_bits = (z & mant) | ((uint32_t)bias << lm);
  uint32_t ym_bits;
  if (dt == QO_F16) {
    const double am = (double)dec_f16((uint16_t)am_bits);
    const double third16 = (double)dec_f16(enc_f16(1.0 / 3.0));
    const double t = (double)dec_f16(enc_f16(am * am + 2.0));   /* exact in double, rounded once */
    ym_bits = enc_f16(t * third16);                             /* exact in double, rounded once */
  } else {
    const float am = dec_bf16((uint16_t)am_bits);
    const float t = fmaf(am, am, 2.0f);                         /* exact in binary32 */
    const float p = t * (float)(1.0 / 3.0);                     /* binary32 rounding */
    ym_bits = enc_bf16((double)p);
  }
  return (uint16_t)((z & ~mant & 0xFFFFu) | (ym_bits & mant));
}

int qo_exp16(const void* x, void* y, int64_t n, int dt, int mode, float a, float b) {
  if (dt != QO_F16 && dt != QO_BF16) return 2;
  if (mode != QO_Q1 && mode != QO_Q2) return 3;
  const double two_lm = (dt == QO_F16) ? 1024.0 : 128.0;
  const double bias = (dt == QO_F16) ? 15.0 : 127.0;
  const double beta = (mode == QO_Q1) ? 0.0436 : 0.0;
  const float c0 = (float)(((double)a / LN2) * two_lm);
  const float c1 = (float)(((bias - beta) + (double)b / LN2) * two_lm);
  for (int64_t i = 0; i < n; ++i)
    ((uint16_t*)y)[i] = quake16_one(load_el(x, i, dt), c0, c1, dt, mode);
  return 0;
}

/* Rounding of doubles to an output format, exposed for tests. */
int qo_round(const double* v, void* out, int64_t n, int dt) {
  if (dt < QO_F32 || dt > QO_BF16) return 2;
  for (int64_t i = 0; i < n; ++i) store_el(out, i, dt, v[i]);
  return 0;
}

/* Decoding of an input format to binary32, exposed for tests. */
int qo_decode(const void* in, float* out, int64_t n, int dt) {
  if (dt < QO_F32 || dt > QO_BF16) return 2;
  for (int64_t i = 0; i < n; ++i) out[i] = load_el(in, i, dt);
  return 0;
}
