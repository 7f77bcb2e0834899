/*
 * hobflops_oracle.h -- scalar CPU reference for HOBFLOPS custom-precision
 * floating-point arithmetic.
 *
 * TEST INFRASTRUCTURE ONLY. This is the oracle that the GPU path is checked
 * against. It shares no code with the GPU library, is not tuned, and is only
 * ever loaded by the tests, the smoke check and the CPU-baseline leg of the
 * benchmark. Nothing in the product path links it.
 *
 * Number format (paper, Sec. 3.3 "Design Flow"): a FloPoCo floating-point word
 * is a 2-bit exception field, a sign bit, a wE-bit exponent and a wF-bit
 * fraction; the significand has an implicit leading one and there are no
 * subnormal numbers. A code is held LSB-first in an integer:
 *     bits [0, wF)            fraction F
 *     bits [wF, wF+wE)        exponent E
 *     bit  wF+wE              sign s
 *     bits [wF+wE+1, wF+wE+3) exception field x (x = 1 means "normal")
 * so NB = 3 + wE + wF bits per value (the paper's NINBITS, Sec. 3.4).
 * Bits of a code above NB are ignored on input and zero on output.
 *
 * Readings of points the paper leaves open (all shared with the GPU path and
 * listed in the design notes): x = 0 zero, 2 infinity, 3 NaN; bias
 * 2^(wE-1)-1; every exponent value E is an ordinary binade; round to nearest,
 * ties to even, after every operation, with an unbounded exponent first and the
 * range check after; overflow -> signed infinity; underflow -> zero with the
 * sign of the exact value; IEEE-754 rules for specials and zero signs; outputs
 * canonical (E = F = 0 for zero and infinity, s = E = F = 0 for NaN).
 *
 * Limits: 2 <= wE <= 8 and 1 <= wF <= 23 for every format argument (so that
 * IEEE binary16, bfloat16 and binary32 are all expressible).
 * Functions return HFO_BAD_FORMAT (all ones) for a format outside the limits.
 */
#ifndef HOBFLOPS_ORACLE_H
#define HOBFLOPS_ORACLE_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define HFO_BAD_FORMAT (~(uint64_t)0)

/* Rounding modes. Round to nearest, ties to even, is the paper's mode for
 * every operation (Sec. 4); round toward zero is its second one, used for the
 * MACs of the type sweep (Sec. 4): the dropped bits of the exact value are
 * discarded. In both modes the exponent range is checked after rounding
 * (overflow gives infinity) and exact cancellation gives +0. Conversion from
 * float32 always rounds to nearest. */
#define HFO_RNE 0
#define HFO_RTZ 1

/* Scalar operations on codes. */
uint64_t hfo_quantize_f32(float f, int wE, int wF);
float    hfo_decode_f32(uint64_t code, int wE, int wF);
uint64_t hfo_mul(uint64_t a, uint64_t b, int wE, int wF_in, int wF_out);
uint64_t hfo_add(uint64_t a, uint64_t b, int wE, int wF);
uint64_t hfo_convert(uint64_t a, int wE, int wF_src, int wF_dst);
uint64_t hfo_relu(uint64_t a, int wE, int wF);
uint64_t hfo_muladd(uint64_t a, uint64_t b, uint64_t c, int wE, int wF_in, int wF_acc);
/* The same with an explicit rounding mode (HFO_RNE or HFO_RTZ; any other
 * value gives HFO_BAD_FORMAT). */
uint64_t hfo_mul_rm(uint64_t a, uint64_t b, int wE, int wF_in, int wF_out, int mode);
uint64_t hfo_add_rm(uint64_t a, uint64_t b, int wE, int wF, int mode);
uint64_t hfo_convert_rm(uint64_t a, int wE, int wF_src, int wF_dst, int mode);
uint64_t hfo_muladd_rm(uint64_t a, uint64_t b, uint64_t c, int wE, int wF_in, int wF_acc, int mode);

/* Element-wise array forms (same semantics, n elements). Return 0, or -1 on a
 * bad format. */
int hfo_quantize_f32_array(const float* src, size_t n, int wE, int wF, uint64_t* dst);
int hfo_decode_f32_array(const uint64_t* src, size_t n, int wE, int wF, float* dst);
int hfo_mul_array(const uint64_t* a, const uint64_t* b, size_t n, int wE, int wF_in,
                  int wF_out, uint64_t* r);
int hfo_add_array(const uint64_t* a, const uint64_t* b, size_t n, int wE, int wF, uint64_t* r);
int hfo_convert_array(const uint64_t* a, size_t n, int wE, int wF_src, int wF_dst, uint64_t* r);
int hfo_relu_array(const uint64_t* a, size_t n, int wE, int wF, uint64_t* r);
int hfo_muladd_array(const uint64_t* a, const uint64_t* b, const uint64_t* c, size_t n, int wE,
                     int wF_in, int wF_acc, uint64_t* r);
int hfo_mul_rm_array(const uint64_t* a, const uint64_t* b, size_t n, int wE, int wF_in,
                     int wF_out, int mode, uint64_t* r);
int hfo_add_rm_array(const uint64_t* a, const uint64_t* b, size_t n, int wE, int wF, int mode,
                     uint64_t* r);
int hfo_convert_rm_array(const uint64_t* a, size_t n, int wE, int wF_src, int wF_dst, int mode,
                         uint64_t* r);
int hfo_muladd_rm_array(const uint64_t* a, const uint64_t* b, const uint64_t* c, size_t n, int wE,
                        int wF_in, int wF_acc, int mode, uint64_t* r);

/* Multi-channel multi-kernel convolution (paper, Sec. 3.4).
 * ifm: codes in in_fmt, NHWC [N][H][W][C]; w: codes in in_fmt, HWIO
 * [KH][KW][C][M]; ofm: codes in out_fmt, [N][OH][OW][M] with
 * OH = (H + 2*pad - KH)/stride + 1 (likewise OW).
 * For every output: acc = +0 in acc_fmt; for ky, then kx, then c:
 *   acc = add(acc, mul(w[ky][kx][c][m], x)), x = +0 for a padding tap;
 * then ofm = convert(act(acc), acc_fmt -> out_fmt); act 0 = none, 1 = ReLU.
 * Every mul, add and the final convert round in mode `round` (HFO_RNE or
 * HFO_RTZ).
 * All formats share wE. nthreads <= 0 means one thread per online CPU.
 * Returns 0, or -1 on bad arguments. */
typedef struct {
  int N, H, W, C, M, KH, KW, stride, pad;
  int wE, wF_in, wF_acc, wF_out, act;
  int round;
} hfo_conv_desc;

int hfo_conv2d(const uint64_t* ifm, const uint64_t* w, uint64_t* ofm, const hfo_conv_desc* d,
               int nthreads);

/* The same convolution evaluated only at npts output points; pts holds
 * (n, oy, ox, m) quadruples, out receives one code per point. */
int hfo_conv2d_points(const uint64_t* ifm, const uint64_t* w, const int64_t* pts, size_t npts,
                      uint64_t* out, const hfo_conv_desc* d, int nthreads);

/* Number of threads hfo_conv2d would use for nthreads <= 0. */
int hfo_default_threads(void);

/* The code, in format (wE, wF), of 1/n for an integer n >= 1, rounded to
 * nearest with ties to even (the scale factor of average pooling). Returns
 * HFO_BAD_FORMAT for a bad format or n = 0. */
uint64_t hfo_recip(uint64_t n, int wE, int wF);

/* Global average pooling, the layer between the last convolution and the
 * fully connected layer of MobileNets that the paper proposes to build in the
 * HOBFLOPS format (Sec. 4, on where the format transformation happens).
 * in: codes in in_fmt, [N][H][W][C]; out: codes in out_fmt, [N][C].
 * For every (n, c): acc = +0 in acc_fmt; for y, then x:
 *   acc = add(acc, widen(in[n][y][x][c]))       (widening to acc_fmt is exact)
 * then out = mul(acc, s) rounded into out_fmt, with s = hfo_recip(H*W) in
 * acc_fmt. The adds and the mul round in mode `round`.
 * All formats share wE; wF_in <= wF_acc. Returns 0, or -1 on bad arguments. */
int hfo_avgpool(const uint64_t* in, uint64_t* out, int N, int H, int W, int C, int wE, int wF_in,
                int wF_acc, int wF_out, int round);

#ifdef __cplusplus
}
#endif
#endif
