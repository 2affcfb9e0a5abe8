/*
 * quake.h — C ABI of libquake, the MI355X (gfx950) implementation of QuAKE:
 * the IEEE-754 bit-construction approximation of exp with the affine input
 * transform folded into its two constants, the second-order (QuAKE2) mantissa
 * refinement, and the Softmax, GELU and Logistic operators built on it.
 *
 * Paper: S. K. Narayanaswami, G. Srinivasan, B. Ravindran, "QuAKE: Speeding up
 * Model Inference Using Quick and Approximate Kernels for Exponential
 * Non-Linearities", arXiv:2412.00408.
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 * - Pointers x and y are DEVICE pointers (memory the caller allocated on the
 *   current HIP device, e.g. by torch). The library never allocates, frees or
 *   retains them. x and y have the same element type (quake_dtype); all
 *   arithmetic is binary32. In-place (x == y) is allowed; partial overlap is
 *   undefined. Any alignment is accepted. Element-aligned buffers are read
 *   and written as aligned 16-byte vectors: 16-byte-aligned ones directly;
 *   the elementwise operators (below 2^31 elements) and the softmax rows at
 *   the same offset from 16 bytes in x and y through the aligned 16-byte
 *   blocks that hold their bytes, with the elements outside the operand
 *   never written (up to 15 bytes around an operand may be read, never
 *   outside a 16-byte block that holds some of its bytes). Other layouts take
 *   scalar kernels.
 * - `stream` is a hipStream_t passed as an opaque pointer (NULL = the legacy
 *   default stream). Every call is asynchronous and stream-ordered: the status
 *   covers argument validation and the launch itself (hipGetLastError right
 *   after the launch); a fault inside a kernel surfaces at the caller's next
 *   synchronisation.
 * - A size of zero returns QUAKE_OK and launches nothing. Negative sizes, a
 *   NULL pointer with a nonzero size, or a row stride smaller than the row
 *   length return QUAKE_EINVAL before any HIP call. Unknown enum values return
 *   QUAKE_EDTYPE / QUAKE_EMODE. No C++ exception crosses this interface.
 * - Sizes above 2^31 elements are split into several launches by the library.
 * - NaN inputs give unspecified (but finite-time, fault-free) outputs.
 *
 * The three modes (quake_mode):
 *   QUAKE_EXACT  the same fused binary32 argument, exponentiated with the GPU's
 *                hardware base-2 exponential instead of the bit construction.
 *                This is the comparison ("vanilla") kernel.
 *   QUAKE_1      first-order QuAKE, Sec. III-A: l = c0*x + c1 (Eq. 5, one fused
 *                multiply-add), z = convert_to_int(l), result = bits of z read
 *                as a float (Eq. 2, Eq. 3).
 *   QUAKE_2      QuAKE2, Sec. III-B and Algorithm 1: the mantissa of z is
 *                refined with y_m = (a_m^2 + 2)/3 (Eq. 6 with a0 = 1/3, a1 = 0,
 *                a2 = 2/3), evaluated as fmaf(a_m, a_m, 2) * fl(1/3), and joined
 *                to the exponent field of z.
 *   QUAKE_2M     QuAKE2 with the coefficients of Eq. 6 that minimise the
 *                worst-case relative error over [0, 1) (the optimum of the
 *                paper's grid search, Sec. III-B; solved exactly by the Remez
 *                exchange: a0 = 0.33718944, a1 = -0.016742593, a2 = 0.68127793
 *                in binary32, worst case 0.1725 %): y_m = fmaf(fmaf(a0, a_m,
 *                a1), a_m, a2), joined as in QUAKE_2. Where a_m = 1 (integer
 *                exponents, both clamp ends) the result is z's bits, so 0, +inf
 *                and exact powers of two are kept. Half QuAKE2's worst-case
 *                error, not continuous at binade edges, monotone.
 *   Before convert_to_int, l is clamped to [0, 255 * 2^23] (our reading of the
 *   v_min clamp of Algorithm 2, applied to every operator): inputs whose result
 *   underflows give 0 (or a denormal ramp), +inf or overflowing inputs give
 *   +inf, and the float-to-int conversion can never overflow.
 */
#ifndef QUAKE_H
#define QUAKE_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define QUAKE_ABI_VERSION 5

typedef enum {
  QUAKE_F32 = 0,  /* IEEE binary32 */
  QUAKE_F16 = 1,  /* IEEE binary16 */
  QUAKE_BF16 = 2  /* bfloat16 (upper half of binary32) */
} quake_dtype;

typedef enum {
  QUAKE_EXACT = 0,
  QUAKE_1 = 1,
  QUAKE_2 = 2,
  QUAKE_2M = 3
} quake_mode;

typedef enum {
  QUAKE_OK = 0,
  QUAKE_EINVAL = 1,  /* bad pointer / size / stride / scalar argument */
  QUAKE_EDTYPE = 2,  /* unknown quake_dtype */
  QUAKE_EMODE = 3,   /* unknown quake_mode */
  QUAKE_EHIP = 4,    /* a HIP runtime call or kernel launch failed */
  QUAKE_ENOSCRATCH = 5  /* quake_softmax_noalloc: the shape needs more than its fixed scratch */
} quake_status;

/*
 * quake_exp — y[i] = e^(a*x[i] + b), elementwise over n contiguous elements.
 * Sec. III-A, Eq. 5: the affine map is folded into the constants,
 *   c0 = fl32(2^23 * a / ln2),  c1 = fl32(2^23 * (127 - beta + b / ln2)),
 * each evaluated in double and rounded once. beta is the Schraudolph bias
 * 0.0436 in QUAKE_1 (Sec. III-A) and 0 in QUAKE_2 and QUAKE_2M (QuAKE2 is
 * exact at integer powers of two, Sec. III-B). QUAKE_EXACT computes exp2(fmaf(x, fl32(a/ln2),
 * fl32(b/ln2))) with the hardware exp2.
 *   x, y : device buffers of n elements of `dtype`, contiguous.
 *   a, b : finite, with c0 and c1 finite in binary32 (|a|, |b| below about
 *          2.8e31 in QUAKE_1/QUAKE_2, 2.3e38 in QUAKE_EXACT); otherwise
 *          QUAKE_EINVAL.
 * QUAKE_1, QUAKE_2 and QUAKE_2M outputs are bit-exact functions of the input.
 */
quake_status quake_exp(const void* x, void* y, int64_t n, quake_dtype dtype,
                       quake_mode mode, float a, float b, void* stream);

/*
 * quake_softmax — row-wise softmax(t * x) of a row-major matrix,
 * Sec. III-C, Algorithm 2: m = max_j x[r, j]; c0 = fl32(2^23 * t / ln2);
 * c1 = fmaf(-c0, m, 127 * 2^23); y[r, j] = QuAKEx(x[r, j]) / sum_j QuAKEx(x[r, j]).
 * Every exponent of a row is taken against the row's final maximum (QuAKE is
 * not multiplicative, so online rescaling of partial sums would change the
 * result). Sums are accumulated in fp32 within each 16-byte vector, then
 * across vectors, lanes and waves in fp32 (16-bit rows of up to 16384
 * elements held by one wave or one 256-thread workgroup) or double (all
 * other rows), and in double across the workgroups of a split row.
 *   x    : device, rows x cols elements, row r at x + r*ldx (elements).
 *   y    : device, row r at y + r*ldy (elements).
 *   ldx, ldy >= cols. cols >= 1 when rows >= 1.
 *   t    : temperature, finite and > 0, with c0 finite in binary32 (t below
 *          about 2.8e31 in QUAKE_1/QUAKE_2); otherwise QUAKE_EINVAL.
 * Rows may hold -inf (masking); those entries give exactly 0, and a row that
 * is entirely -inf gives a row of zeros. +inf inputs are unspecified.
 * Folding m into c1 (one binary32 rounding of c0*m) shifts every exponent's
 * argument by up to |t*m| * 2^-24 (natural-log units); rows with |t*m| above
 * about 1e9 are outside the folded form's range and may give NaN.
 * Rows whose start is not 16-byte aligned (a length that is not a multiple
 * of 16 bytes, an offset base) but lies at the same offset from a 16-byte
 * boundary in x and y are read as the aligned 16-byte blocks that cover them:
 * up to 15 bytes before and after each row are read (never written, and
 * never outside the 16-byte blocks that hold the row's own first and last
 * bytes); other layouts take a scalar kernel.
 * Rows of more than 16384 elements do not fit one wave's or one 256-thread
 * workgroup's registers. Without a workspace, such a row of up to 129024
 * (binary32) or 131072 (16-bit) elements (a few fewer for a row whose start
 * is not 16-byte aligned) is held by one 512-thread workgroup in its
 * registers and LDS (each element read once); longer rows, and the layouts
 * that take the scalar kernel, are reduced by one workgroup that reads the
 * row three times (max, sum, normalise; the re-reads are served by the
 * caches). quake_softmax_ws computes the same operator for long rows (the
 * partial sums in another order) over several workgroups per row, every
 * element read from HBM once (rows that are not 16-byte aligned: when
 * ceil(cols / 16384) chunks cover the aligned blocks of every row, else the
 * one-workgroup kernels). The library allocates nothing and keeps no
 * state.
 */
quake_status quake_softmax(const void* x, void* y, int64_t rows, int64_t cols,
                           int64_t ldx, int64_t ldy, quake_dtype dtype,
                           quake_mode mode, float t, void* stream);

/*
 * quake_softmax_workspace_size — bytes of device workspace quake_softmax_ws
 * uses for rows x cols (any dtype): 0 when rows fit one workgroup's registers
 * (cols <= 16384) or when cols > 2^22 (such rows take the workspace-free
 * kernel), else 256 + 12 * G * R + 4 * R rounded up to 256, with
 * G = ceil(cols / 16384) chunks per row and R = min(rows, 1024) rows per
 * launch (6656 bytes for 64 x 128256). bytes: host pointer, non-NULL.
 */
quake_status quake_softmax_workspace_size(int64_t rows, int64_t cols, quake_dtype dtype,
                                          int64_t* bytes);

/*
 * quake_softmax_ws — quake_softmax (Algorithm 2, same arguments, same results
 * up to the summation order of the partial sums) where rows longer than one
 * workgroup's registers (16384 < cols <= 2^22, vectorisable layout) are split
 * into G chunks of 16384 elements held by G workgroups. Every exponent of a
 * row needs the row's final max (Algorithm 2; QuAKE is not multiplicative, so
 * partial sums cannot be rescaled), so the chunks exchange their maxima, then
 * their sums, through `workspace`; x is read once from HBM.
 *   workspace       : device memory owned by the caller, 16-byte aligned, of
 *                     at least quake_softmax_workspace_size(rows, cols) bytes
 *                     (else QUAKE_EINVAL), zero-filled before its first use
 *                     (e.g. hipMemset or torch.zeros). Every call returns the
 *                     slots to zero when it completes, so one workspace serves
 *                     any number of stream-ordered calls (and graph replays).
 *                     Calls that may run concurrently (different streams)
 *                     need different workspaces. NULL (with workspace_bytes
 *                     0) gives exactly quake_softmax.
 *   Word 0 of the workspace (uint32) is the exchange's wait limit in ticks of
 *   the GPU's 100 MHz constant clock, 0 meaning the default of 10000 (100 us):
 *   a workgroup that has waited that long for a peer's value computes it from
 *   x itself, with the peer's loads and summation order, so the result is the
 *   same bits; progress never depends on the peers being resident (other
 *   streams may hold any number of CUs); 0xFFFFFFFF means no waiting at all
 *   (every workgroup computes every chunk value of its row from x: the same
 *   bits, about G times the reads). Word 1 (uint32) counts the
 *   workgroups that did so (a diagnostic; the library only increments it).
 *   Bytes 8 .. 255 are reserved and must stay zero.
 * Other arguments, layout, errors and input contract as quake_softmax.
 */
quake_status quake_softmax_ws(const void* x, void* y, int64_t rows, int64_t cols, int64_t ldx,
                              int64_t ldy, quake_dtype dtype, quake_mode mode, float t,
                              void* workspace, int64_t workspace_bytes, void* stream);

/*
 * quake_softmax_noalloc — quake_softmax_ws without a workspace argument, for
 * callers that cannot allocate device memory (code under HIP graph capture,
 * tight serving loops, harnesses that forbid hipMalloc): the exchange uses a
 * fixed 262144-byte device array of the library instead, one per GPU, held
 * until the process ends. No allocation or free happens in this call; the
 * first call on a device looks the array up and clears it with a kernel on
 * `stream`. Same arguments (minus the workspace), same kernels and the same
 * bits as quake_softmax_ws. Shapes whose workspace
 * (quake_softmax_workspace_size) exceeds 262144 bytes return
 * QUAKE_ENOSCRATCH before any HIP call (rows <= 1024 with cols <= 327680, or
 * 64 rows of up to 2^22, fit); shapes needing no workspace run as
 * quake_softmax. Every call on one GPU shares that GPU's array, which every
 * call leaves zeroed: calls that may overlap on one GPU (different streams,
 * host threads) race and must not be issued.
 */
quake_status quake_softmax_noalloc(const void* x, void* y, int64_t rows, int64_t cols, int64_t ldx,
                                   int64_t ldy, quake_dtype dtype, quake_mode mode, float t,
                                   void* stream);

/*
 * quake_gelu — tanh-form GELU (Sec. II-C, Eq. 4) rewritten as
 * x * sigma(2*0.044715*sqrt(2/pi) * x * (1/0.044715 + x^2)) (Sec. III-D, Eq. 7):
 *   u = fmaf(x, x, fl32(1/0.044715)); w = x*u;
 *   e = QuAKEx(w) with c0 = fl32(-2^23 * 2*0.044715*sqrt(2/pi) / ln2),
 *       c1 = 127*2^23 (QUAKE_2) or (127 - 0.0436)*2^23 (QUAKE_1);
 *   y = x / (1 + e).
 * x, y: device buffers of n contiguous elements. GELU(+-inf) is unspecified.
 */
quake_status quake_gelu(const void* x, void* y, int64_t n, quake_dtype dtype,
                        quake_mode mode, void* stream);

/*
 * quake_sigmoid — Logistic sigma(x) = 1 / (1 + e^-x) (Sec. III-D), or, when
 * silu != 0, SiLU x * sigma(x) = x / (1 + e^-x). e^-x is QuAKEx with
 * c0 = fl32(-2^23 / ln2) (Eq. 5 with p = -1) and the c1 of quake_exp.
 * x, y: device buffers of n contiguous elements. +-inf inputs are allowed
 * (sigma(-inf) = 0, sigma(+inf) = 1).
 */
quake_status quake_sigmoid(const void* x, void* y, int64_t n, quake_dtype dtype,
                           quake_mode mode, int silu, void* stream);

/*
 * quake_softmax_causal — quake_softmax with an implicit causal mask, as in
 * attention scores: entry (r, j) takes part iff j <= (r mod period) + shift;
 * masked entries are NOT read and their outputs are exactly 0, which is what
 * quake_softmax gives for -inf entries at those positions (Algorithm 2 with
 * the clamp of l). A row with no live entry gives zeros. For self-attention
 * with rows = batch*heads*seq and cols = seq, use period = seq, shift = 0;
 * for queries aligned to the end of a longer key range, shift = cols - seq.
 *   period       : 1 <= period <= 2^31 - 1; |shift| <= 2^40; otherwise QUAKE_EINVAL.
 *   write_masked : nonzero writes 0 to every masked output; zero leaves
 *                  masked outputs that lie in 16-byte vectors without live
 *                  entries unwritten (for consumers that never read them, such
 *                  as a causal P*V product), so only about half the outputs
 *                  are stored.
 * Other arguments as quake_softmax. Only the live entries are read from HBM.
 */
quake_status quake_softmax_causal(const void* x, void* y, int64_t rows, int64_t cols,
                                  int64_t ldx, int64_t ldy, int64_t period, int64_t shift,
                                  int write_masked, quake_dtype dtype, quake_mode mode, float t,
                                  void* stream);

/*
 * quake_softmax_unfused, quake_gelu_unfused — the same operators in the
 * "plug-in" form of the paper's fusion study (Sec. V-A, Table IV): the
 * affine input transform is not folded into the exponential's constants.
 * Softmax computes s = (x - m) * t in binary32 (m the row max) and then the
 * standard exponential e^s; GELU computes s = k * x * (1/0.044715 + x^2),
 * k = fl32(2*0.044715*sqrt(2/pi)), and then e^-s. The standard exponential is
 * QuAKEx with c0 = fl32(2^23/ln2), c1 = (127 - beta)*2^23 (beta as in
 * quake_exp), or, in QUAKE_EXACT, the hardware exp2 of fl32(s * fl32(1/ln2)) —
 * the vanilla operator. Arguments, layout, errors and input contract are
 * those of quake_softmax / quake_gelu. These exist to measure what the
 * folding saves; results differ from the fused operators only by the
 * binary32 rounding of the exponential's argument.
 */
quake_status quake_softmax_unfused(const void* x, void* y, int64_t rows, int64_t cols,
                                   int64_t ldx, int64_t ldy, quake_dtype dtype,
                                   quake_mode mode, float t, void* stream);
quake_status quake_gelu_unfused(const void* x, void* y, int64_t n, quake_dtype dtype,
                                quake_mode mode, void* stream);

/*
 * quake_exp16 — y[i] = e^(a*x[i] + b) with QuAKE / QuAKE2 built directly in
 * the 16-bit format's own layout (Sec. II-A notes the construction holds for
 * any IEEE-style format; Eq. 3 with that format's l_m and B, Algorithm 1 with
 * its masks): binary16 (l_e = 5, l_m = 10, B = 15) or bfloat16 (l_e = 8,
 * l_m = 7, B = 127). No binary32 result is formed and nothing is narrowed:
 *   l = fmaf(x, c0, c1) in binary32, c0 = fl32(2^l_m a / ln2),
 *   c1 = fl32(2^l_m (B - beta + b / ln2)) (beta as in quake_exp);
 *   l clamped to [0, (2^l_e - 1) 2^l_m]; z = (int) l is the 16-bit result of
 *   QUAKE_1; QUAKE_2 sets z's mantissa to that of y_m = (a_m^2 + 2)/3,
 *   a_m = (z & (2^l_m - 1)) | (B << l_m), evaluated in the format's own
 *   arithmetic: binary16 fl16(fl16(a_m a_m + 2) fl16(1/3)); bfloat16
 *   fl_bf16(fl32((a_m a_m + 2) fl32(1/3))).
 * The mantissa carries l_m bits, so results are coarser than quake_exp's
 * (QUAKE_2 worst case about 0.38 % in binary16, 1 % in bfloat16, over normal
 * results). Outputs are bit-exact functions of the input.
 *   x, y  : device buffers of n contiguous elements of `dtype`.
 *   dtype : QUAKE_F16 or QUAKE_BF16 (else QUAKE_EDTYPE).
 *   mode  : QUAKE_1 or QUAKE_2 (else QUAKE_EMODE).
 *   a, b  : finite, with c0, c1 finite; otherwise QUAKE_EINVAL.
 */
quake_status quake_exp16(const void* x, void* y, int64_t n, quake_dtype dtype, quake_mode mode,
                         float a, float b, void* stream);

/*
 * quake_linear_gelu — y = GELU(x w^T), or y = x w^T when gelu == 0: the
 * up-projection of a transformer MLP with its activation fused. The GELU is
 * Eq. 7 with the exponential of `mode` (Sec. III-D, as quake_gelu), applied
 * to the binary32 accumulators in the epilogue of a matrix-core product; the
 * paper applies QuAKE to standalone operators, this is the same operator
 * fused into its producer.
 *   x : device, m x k 16-bit (dtype), row r at x + r*ldx (elements),
 *       16-byte aligned.
 *   w : device, n x k 16-bit (a linear layer's weight), row r at w + r*ldw,
 *       16-byte aligned.
 *   y : device, m x n 16-bit, row r at y + r*ldy.
 *   k, ldx, ldw: multiples of 8; ldx, ldw >= k; ldy >= n; k <= 2^31 - 257,
 *       m <= 2^31 - 129, n <= 2^31 - 193.
 *   dtype : QUAKE_BF16 or QUAKE_F16 (binary16), the format of x, w and y
 *       (else QUAKE_EDTYPE); mode: any quake_mode.
 * Products are accumulated in binary32 (order unspecified), then the GELU of
 * each accumulator is rounded to the 16-bit format. m == 0 or n == 0 launches nothing;
 * other bad sizes, strides or alignments return QUAKE_EINVAL.
 */
quake_status quake_linear_gelu(const void* x, const void* w, void* y, int64_t m, int64_t n,
                               int64_t k, int64_t ldx, int64_t ldw, int64_t ldy,
                               quake_dtype dtype, quake_mode mode, int gelu, void* stream);

/*
 * quake_attention — o = softmax(t q k^T) v for every head: scaled dot-product
 * attention whose softmax is Algorithm 2 (Sec. III-C) with the exponential of
 * `mode`, fused with both products. Each query's exponentials are taken
 * against the max of its whole score row (no online rescaling), so the
 * probabilities are the ones quake_softmax gives for those scores; they are
 * rounded to the 16-bit format before the second product, and the row sum (of
 * the binary32 exponentials) divides the binary32 result, rounded to the
 * 16-bit format.
 *   q, k : device, [heads, seq, dim] 16-bit (dtype), contiguous, 16-byte aligned.
 *   vt   : device, v transposed: [heads, dim, ldv] 16-bit, element
 *          (h, d, j) = v[h, j, d]; ldv >= seq, 2-byte aligned. Columns
 *          seq .. ldv-1 may hold anything (they do not affect o). With vt
 *          16-byte aligned and ldv a multiple of 8 the rows are read as
 *          16-byte vectors, else element by element.
 *   o    : device, [heads, seq, dim] 16-bit, contiguous, 8-byte aligned; it
 *          must not overlap q, k or vt (other workgroups still read them).
 *   dim == 64 and seq <= 131072. Up to 1024 keys a query's scores stay in
 *   registers (one pass: 32 queries per workgroup of four waves up to 512
 *   keys, eight waves beyond); longer sequences take two passes over the keys
 *   (the scores once for the row max, then again for the exponentials and the
 *   second product), with the same arithmetic as one pass of four waves;
 *   t > 0 finite (1/sqrt(dim) for the usual scaling); causal != 0 lets query
 *   i use keys j <= i only (masked keys are neither loaded nor multiplied).
 *   dtype : QUAKE_BF16 or QUAKE_F16, the format of q, k, vt and o (else
 *   QUAKE_EDTYPE); mode: any quake_mode.
 * Scores are binary32 sums of the exact 16-bit products (order unspecified).
 * heads == 0 or seq == 0 launches nothing; other bad sizes, strides,
 * alignments or t return QUAKE_EINVAL.
 */
quake_status quake_attention(const void* q, const void* k, const void* vt, void* o, int64_t heads,
                             int64_t seq, int64_t dim, int64_t ldv, quake_dtype dtype,
                             quake_mode mode, float t, int causal, void* stream);

/*
 * quake_stream_copy — a measurement aid, not part of the method: copies
 * `bytes` (a multiple of 16, below 2^35) from x to y with plain non-temporal
 * 16-byte loads and stores, in one of the launch shapes the operators use, so
 * that an operator's time can be set against the time this device takes to
 * move the same bytes. shape: 0 resident grid of 8 workgroups per CU, two
 * vectors per lane per step, software-pipelined (the mid-size elementwise
 * kernels' shape); 1 one vector per lane (the large elementwise kernels'
 * shape); 2 resident grid of 4 workgroups per CU, four vectors per lane per
 * step; 3 read only (x is read, y is written only if a 16-byte vector's four
 * words XOR to 0x9E3779B9, which the caller's data should avoid); 4 write
 * only (zeros to y; x unused). x, y: device, 16-byte aligned, not overlapping.
 * Other shapes, sizes or alignments return QUAKE_EINVAL.
 */
quake_status quake_stream_copy(const void* x, void* y, int64_t bytes, int shape, void* stream);

/* Static, human-readable name of a status code (never NULL). */
const char* quake_status_str(quake_status s);

/* Returns QUAKE_ABI_VERSION of the built library. */
int quake_abi_version(void);

#ifdef __cplusplus
}
#endif

#endif /* QUAKE_H */
