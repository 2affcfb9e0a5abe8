/*
 * Edge-case driver for the CPU oracle (test infrastructure only), built with
 * AddressSanitizer and UndefinedBehaviorSanitizer (float-to-int cast overflow
 * included) by tests/test_oracle_sanitized.py. It runs every exported oracle
 * function over special binary32 values (zeros, denormals, the largest finite
 * values, infinities, NaN), a strided sweep of binary32 bit patterns, every
 * 16-bit pattern of binary16 and bfloat16, softmax rows with masks, extreme
 * temperatures and strides, and causal limits at and beyond the row ends.
 * Besides "no sanitizer report" it checks a few facts that hold for any input:
 * outputs of exp are >= 0 or NaN, softmax rows with a finite maximum sum to 1,
 * masked softmax outputs are exactly 0.
 * Exit status 0 on success; the sanitizers abort on the first report.
 */
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

int qo_quake(const float* x, float* y, int64_t n, float c0, float c1, int order);
int qo_exp(const void* x, void* y, int64_t n, int dt, int mode, float a, float b);
int qo_sigmoid(const void* x, void* y, int64_t n, int dt, int mode, int silu);
int qo_gelu(const void* x, void* y, int64_t n, int dt, int mode);
int qo_gelu_unfused(const void* x, void* y, int64_t n, int dt, int mode);
int qo_softmax(const void* x, void* y, int64_t rows, int64_t cols, int64_t ldx, int64_t ldy,
               int dt, int mode, float t, double* tmp);
int qo_softmax_unfused(const void* x, void* y, int64_t rows, int64_t cols, int64_t ldx,
                       int64_t ldy, int dt, int mode, float t, double* tmp);
int qo_softmax_causal(const void* x, void* y, int64_t rows, int64_t cols, int64_t ldx,
                      int64_t ldy, int64_t period, int64_t shift, int dt, int mode, float t,
                      double* tmp);
int qo_exp16(const void* x, void* y, int64_t n, int dt, int mode, float a, float b);
int qo_round(const double* v, void* out, int64_t n, int dt);
int qo_decode(const void* in, float* out, int64_t n, int dt);
float qo_softmax_c0(float t, int mode);

static int failures = 0;
#define EXPECT(c, ...)                     \
  do {                                     \
    if (!(c)) {                            \
      printf("FAIL: " __VA_ARGS__);        \
      printf("\n");                        \
      failures++;                          \
    }                                      \
  } while (0)

static float u2f(uint32_t u) { float f; memcpy(&f, &u, 4); return f; }

static const uint32_t SPECIAL[] = {
    0x00000000u, 0x80000000u, 0x00000001u, 0x80000001u, 0x007FFFFFu, 0x807FFFFFu,
    0x00800000u, 0x80800000u, 0x3F800000u, 0xBF800000u, 0x42B17218u, 0xC2B17218u,
    0x42B20000u, 0xC2CE0000u, 0x42FE0000u, 0xC2FE0000u, 0x4B000000u, 0xCB000000u,
    0x7F7FFFFFu, 0xFF7FFFFFu, 0x7F800000u, 0xFF800000u, 0x7FC00000u, 0xFFC00000u,
    0x7F800001u, 0x3EAAAAABu, 0x4E7E0000u, 0x4F7F0000u, 0xCF000000u, 0x4F000000u};
#define NSPECIAL (sizeof(SPECIAL) / sizeof(SPECIAL[0]))

/* Values of format dt as raw elements (float or uint16) in buf; returns count. */
static int64_t fill_inputs(void* buf, int dt) {
  if (dt == 0) {
    float* f = (float*)buf;
    int64_t n = 0;
    for (size_t i = 0; i < NSPECIAL; ++i) f[n++] = u2f(SPECIAL[i]);
    for (uint64_t b = 0; b <= 0xFFFFFFFFull; b += 4099u) f[n++] = u2f((uint32_t)b);
    return n;
  }
  uint16_t* h = (uint16_t*)buf;
  for (int64_t i = 0; i < 65536; ++i) h[i] = (uint16_t)i;
  return 65536;
}

static void elementwise(void) {
  const int64_t cap = 1100000;
  void* x = malloc(cap * 4);
  void* y = malloc(cap * 4);
  for (int dt = 0; dt < 3; ++dt) {
    const int64_t n = fill_inputs(x, dt);
    float* dec = (float*)malloc(n * 4);
    float* out = (float*)malloc(n * 4);
    EXPECT(qo_decode(x, dec, n, dt) == 0, "decode dt=%d", dt);
    for (int mode = 0; mode < 5; ++mode) {
      const float ab[][2] = {{1.0f, 0.0f}, {-1.0f, 0.0f}, {0.5f, -3.0f}, {1e30f, 0.0f},
                             {1e-30f, 5.0f}};
      for (size_t k = 0; k < sizeof(ab) / sizeof(ab[0]); ++k) {
        EXPECT(qo_exp(x, y, n, dt, mode, ab[k][0], ab[k][1]) == 0, "exp");
        EXPECT(qo_decode(y, out, n, dt) == 0, "decode");
        for (int64_t i = 0; i < n; ++i)
          EXPECT(isnan(out[i]) || out[i] >= 0.0f, "exp < 0 dt=%d mode=%d i=%lld", dt, mode,
                 (long long)i);
      }
      EXPECT(qo_sigmoid(x, y, n, dt, mode, 0) == 0, "sigmoid");
      EXPECT(qo_decode(y, out, n, dt) == 0, "decode");
      for (int64_t i = 0; i < n; ++i)
        EXPECT(isnan(dec[i]) || (out[i] >= 0.0f && out[i] <= 1.0f), "sigmoid out of [0,1]");
      EXPECT(qo_sigmoid(x, y, n, dt, mode, 1) == 0, "silu");
      EXPECT(qo_gelu(x, y, n, dt, mode) == 0, "gelu");
      EXPECT(qo_gelu_unfused(x, y, n, dt, mode) == 0, "gelu unfused");
      if (dt > 0 && (mode == 1 || mode == 2)) {
        const float ab16[][2] = {{1.0f, 0.0f}, {-1.0f, 0.0f}, {3e4f, 0.0f}, {1e-30f, -7.0f}};
        for (size_t k = 0; k < 4; ++k)
          EXPECT(qo_exp16(x, y, n, dt, mode, ab16[k][0], ab16[k][1]) == 0, "exp16");
      }
      if (mode > 0) {
        float* fy = (float*)y;
        EXPECT(qo_quake(dec, fy, n, 12102203.0f, 1065353216.0f, mode) == 0, "quake");
        EXPECT(qo_quake(dec, fy, n, -1e30f, 3e9f, mode) == 0, "quake extreme constants");
      }
    }
    free(dec);
    free(out);
  }
  /* rounding of doubles beyond every format's range, and of tiny values */
  double v[] = {0.0, -0.0, 1e-320, -1e-320, 5.9e-8, 2.9e-8, 65519.0, 65520.0, 3.4e38, 3.5e38,
                1e300, -1e300, INFINITY, -INFINITY, NAN, 1.0 + 1e-16};
  uint32_t out32[16];
  for (int dt = 0; dt < 3; ++dt) EXPECT(qo_round(v, out32, 16, dt) == 0, "round");
  free(x);
  free(y);
}

static void softmax(void) {
  const int64_t rows = 7, cols = 301, ld = 333;
  float* x = (float*)malloc(sizeof(float) * rows * ld);
  float* y = (float*)malloc(sizeof(float) * rows * ld);
  uint16_t* xh = (uint16_t*)malloc(2 * rows * ld);
  uint16_t* yh = (uint16_t*)malloc(2 * rows * ld);
  double* tmp = (double*)malloc(sizeof(double) * cols);
  uint32_t s = 7u;
  for (int64_t i = 0; i < rows * ld; ++i) {
    s = s * 1664525u + 1013904223u;
    x[i] = ((float)(s >> 8) / 16777216.0f - 0.5f) * 200.0f;
  }
  for (int64_t j = 0; j < cols; ++j) x[1 * ld + j] = -INFINITY;  /* fully masked row */
  for (int64_t j = 0; j < cols; j += 2) x[2 * ld + j] = -INFINITY;
  x[3 * ld + 5] = 3.4e38f;                                        /* huge max */
  x[4 * ld + 0] = -3.4e38f;
  for (int64_t j = 0; j < cols; ++j) x[5 * ld + j] = 1e-40f;      /* denormal row */
  x[6 * ld + 9] = NAN;
  for (int64_t i = 0; i < rows * ld; ++i) xh[i] = (uint16_t)(s = s * 1664525u + 1013904223u) ;
  const float temps[] = {1.4e-45f, 1e-30f, 0.125f, 1.0f, 1e10f, 2.8e31f};
  for (int mode = 0; mode < 5; ++mode) {
    for (size_t k = 0; k < sizeof(temps) / sizeof(temps[0]); ++k) {
      const float t = temps[k];
      if (!isfinite(qo_softmax_c0(t, mode))) continue;
      EXPECT(qo_softmax(x, y, rows, cols, ld, ld, 0, mode, t, tmp) == 0, "softmax");
      for (int64_t r = 0; r < rows; ++r) {
        if (r == 6) continue;  /* NaN row: unspecified */
        float m = -INFINITY;
        for (int64_t j = 0; j < cols; ++j) m = x[r * ld + j] > m ? x[r * ld + j] : m;
        /* Algorithm 2 folds the row maximum into c1 = 127 * 2^23 - c0 * m in
         * binary32; past |t m| of about 1e9 that rounding alone can push every
         * exponent to 0 or +inf, so the row-sum property is checked inside
         * the folded form's range only. */
        if (r != 1 && !((double)t * fabs((double)m) <= 1e8)) continue;
        double sum = 0.0;
        for (int64_t j = 0; j < cols; ++j) sum += y[r * ld + j];
        if (r == 1) EXPECT(sum == 0.0, "masked row");
        else EXPECT(fabs(sum - 1.0) < 1e-4, "row %lld sum %g mode %d t %g", (long long)r, sum,
                    mode, (double)t);
        if (r == 2)
          for (int64_t j = 0; j < cols; j += 2)
            EXPECT(y[2 * ld + j] == 0.0f, "-inf entry mode %d t %g", mode, (double)t);
      }
      EXPECT(qo_softmax_unfused(x, y, rows, cols, ld, ld, 0, mode, t, tmp) == 0, "unfused");
      for (int dt = 1; dt < 3; ++dt) {
        EXPECT(qo_softmax(xh, yh, rows, cols, ld, ld, dt, mode, t, tmp) == 0, "softmax 16");
        EXPECT(qo_softmax_unfused(xh, yh, rows, cols, ld, ld, dt, mode, t, tmp) == 0, "u16");
      }
      const int64_t shifts[] = {-400, -1, 0, 1, 300, 1000000};
      const int64_t periods[] = {1, 3, 301, 1000};
      for (size_t a = 0; a < 6; ++a)
        for (size_t b = 0; b < 4; ++b) {
          EXPECT(qo_softmax_causal(x, y, rows, cols, ld, ld, periods[b], shifts[a], 0, mode, t,
                                   tmp) == 0, "causal");
          for (int64_t r = 0; r < rows; ++r) {
            int64_t L = r % periods[b] + shifts[a] + 1;
            for (int64_t j = L < 0 ? 0 : L; j < cols; ++j)
              EXPECT(y[r * ld + j] == 0.0f, "causal masked output");
          }
        }
    }
  }
  EXPECT(qo_softmax(x, y, 0, cols, ld, ld, 0, 2, 1.0f, tmp) == 0, "zero rows");
  free(x); free(y); free(xh); free(yh); free(tmp);
}

int main(void) {
  elementwise();
  softmax();
  printf("%s (%d failures)\n", failures ? "oracle edges FAILED" : "oracle edges passed", failures);
  return failures ? 1 : 0;
}
