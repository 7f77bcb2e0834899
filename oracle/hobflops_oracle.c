/*
 * hobflops_oracle.c -- scalar CPU reference (oracle) for HOBFLOPS custom-precision
 * floating-point arithmetic and the MCMK convolution built from it.
 *
 * TEST INFRASTRUCTURE ONLY: see hobflops_oracle.h. Plain, slow and meant to be
 * checked by eye: every value is decoded to an exact integer significand and a
 * power-of-two exponent, the exact product or sum is formed in a wide integer,
 * and one rounding step turns it into a code.
 *
 * Paper passages followed:
 *   format ............ Sec. 3.3 (FloPoCo word: exception, sign, exponent,
 *                       fraction with implicit one, no subnormals)
 *   MAC widths ........ Table 3 and Sec. 3.4 (multiplier output has wF+1
 *                       fraction bits for the "single" MAC types)
 *   rounding .......... Sec. 4 (round to nearest, ties to even)
 *   IEEE behaviour .... Sec. 3.3 (operators match IEEE-754 on quantized values)
 *   convolution ....... Sec. 3.4 and the convolution figure (multiply, then add
 *                       into the accumulator, optional ReLU, OFM in HOBFLOPS form)
 */
#include "hobflops_oracle.h"

#include <math.h>
#include <pthread.h>
#include <string.h>
#include <unistd.h>

/* ------------------------------------------------------------------------ */
/* Fixed-width unsigned big integer: enough for the exact sum of two values of
 * the widest supported format (exponent span 2^8 plus a 24-bit significand). */

#define NLIMB 12 /* 384 bits */
typedef struct {
  uint32_t w[NLIMB]; /* little-endian 32-bit limbs */
} big;

static void big_set_shl(big* r, uint64_t v, int sh) /* r = v << sh */
{
  memset(r, 0, sizeof *r);
  for (int i = 0; i < 64; i++)
    if ((v >> i) & 1) {
      int k = i + sh;
      r->w[k / 32] |= (uint32_t)1 << (k % 32);
    }
}

static int big_cmp(const big* a, const big* b)
{
  for (int i = NLIMB - 1; i >= 0; i--) {
    if (a->w[i] > b->w[i]) return 1;
    if (a->w[i] < b->w[i]) return -1;
  }
  return 0;
}

static void big_add(big* r, const big* a, const big* b)
{
  uint64_t carry = 0;
  for (int i = 0; i < NLIMB; i++) {
    uint64_t t = (uint64_t)a->w[i] + b->w[i] + carry;
    r->w[i] = (uint32_t)t;
    carry = t >> 32;
  }
}

static void big_sub(big* r, const big* a, const big* b) /* requires a >= b */
{
  int64_t borrow = 0;
  for (int i = 0; i < NLIMB; i++) {
    int64_t t = (int64_t)a->w[i] - b->w[i] - borrow;
    borrow = t < 0;
    r->w[i] = (uint32_t)(t + (borrow ? ((int64_t)1 << 32) : 0));
  }
}

static int big_bit(const big* a, int k)
{
  if (k < 0 || k >= 32 * NLIMB) return 0;
  return (a->w[k / 32] >> (k % 32)) & 1;
}

static int big_bitlen(const big* a) /* index of the highest set bit, plus one */
{
  for (int k = 32 * NLIMB - 1; k >= 0; k--)
    if (big_bit(a, k)) return k + 1;
  return 0;
}

static int big_any_below(const big* a, int k) /* any set bit in positions [0, k) */
{
  for (int i = 0; i < k; i++)
    if (big_bit(a, i)) return 1;
  return 0;
}

static uint64_t big_field(const big* a, int lo, int n) /* bits [lo, lo+n), n <= 63 */
{
  uint64_t v = 0;
  for (int i = 0; i < n; i++) v |= (uint64_t)big_bit(a, lo + i) << i;
  return v;
}

/* ------------------------------------------------------------------------ */
/* Codes. */

enum { EXN_ZERO = 0, EXN_NORMAL = 1, EXN_INF = 2, EXN_NAN = 3 };

typedef struct {
  int wE, wF;
} fmt_t;

typedef struct {
  int exn, s;
  int64_t E;  /* biased exponent field */
  uint64_t F; /* fraction field */
} fields_t;

static int fmt_ok(fmt_t f) { return f.wE >= 2 && f.wE <= 8 && f.wF >= 1 && f.wF <= 23; }
static int mode_ok(int mode) { return mode == HFO_RNE || mode == HFO_RTZ; }
static int64_t bias_of(fmt_t f) { return ((int64_t)1 << (f.wE - 1)) - 1; }

static fields_t decode(uint64_t code, fmt_t f)
{
  fields_t r;
  r.F = code & (((uint64_t)1 << f.wF) - 1);
  r.E = (int64_t)((code >> f.wF) & (((uint64_t)1 << f.wE) - 1));
  r.s = (int)((code >> (f.wF + f.wE)) & 1);
  r.exn = (int)((code >> (f.wF + f.wE + 1)) & 3);
  return r;
}

static uint64_t encode(int exn, int s, uint64_t E, uint64_t F, fmt_t f)
{
  return ((uint64_t)exn << (f.wF + f.wE + 1)) | ((uint64_t)s << (f.wF + f.wE)) | (E << f.wF) | F;
}

static uint64_t make_zero(int s, fmt_t f) { return encode(EXN_ZERO, s, 0, 0, f); }
static uint64_t make_inf(int s, fmt_t f) { return encode(EXN_INF, s, 0, 0, f); }
static uint64_t make_nan(fmt_t f) { return encode(EXN_NAN, 0, 0, 0, f); }

/* Canonical form of a decoded value (fields of non-normal values dropped). */
static uint64_t canonical(fields_t v, fmt_t f)
{
  switch (v.exn) {
    case EXN_ZERO: return make_zero(v.s, f);
    case EXN_INF: return make_inf(v.s, f);
    case EXN_NAN: return make_nan(f);
    default: return encode(EXN_NORMAL, v.s, (uint64_t)v.E, v.F, f);
  }
}

/* Significand (with the implicit one) and power-of-two exponent of a normal
 * value: value = (-1)^s * sig * 2^exp2 exactly. */
static uint64_t sig_of(fields_t v, fmt_t f) { return ((uint64_t)1 << f.wF) + v.F; }
static int64_t exp2_of(fields_t v, fmt_t f) { return v.E - bias_of(f) - f.wF; }

/* ------------------------------------------------------------------------ */
/* Rounding: the correctly rounded code, in format f, of (-1)^s * M * 2^e
 * for an exact integer M > 0, to nearest with ties to even (HFO_RNE) or toward
 * zero (HFO_RTZ: the dropped bits are discarded). The rounding is done with an
 * unbounded exponent; the exponent range is checked afterwards: above the
 * largest binade gives infinity (in both modes), below the smallest gives zero
 * (there are no subnormal numbers). */
static uint64_t round_value(fmt_t f, int s, const big* M, int64_t e, int mode)
{
  int p = big_bitlen(M) - 1; /* M lies in [2^p, 2^(p+1)) */
  int64_t u = p + e;         /* value lies in [2^u, 2^(u+1)) */
  uint64_t sig;              /* wF+1 significant bits, leading one included */
  if (p <= f.wF) {
    sig = big_field(M, 0, p + 1) << (f.wF - p); /* exact, nothing to round */
  } else {
    int k = p - f.wF; /* number of bits dropped */
    sig = big_field(M, k, f.wF + 1);
    int half_bit = big_bit(M, k - 1);        /* first dropped bit */
    int below_half = big_any_below(M, k - 1); /* any later dropped bit */
    int round_up = mode == HFO_RNE && half_bit && (below_half || (sig & 1));
    if (round_up) sig += 1;
    if (sig == ((uint64_t)1 << (f.wF + 1))) { /* carried into a new binade */
      sig >>= 1;
      u += 1;
    }
  }
  int64_t Eb = u + bias_of(f);
  if (Eb > (((int64_t)1 << f.wE) - 1)) return make_inf(s, f);
  if (Eb < 0) return make_zero(s, f);
  return encode(EXN_NORMAL, s, (uint64_t)Eb, sig - ((uint64_t)1 << f.wF), f);
}

/* ------------------------------------------------------------------------ */
/* Operations. */

uint64_t hfo_mul_rm(uint64_t a, uint64_t b, int wE, int wF_in, int wF_out, int mode)
{
  fmt_t fi = {wE, wF_in}, fo = {wE, wF_out};
  if (!fmt_ok(fi) || !fmt_ok(fo) || !mode_ok(mode)) return HFO_BAD_FORMAT;
  fields_t A = decode(a, fi), B = decode(b, fi);
  int s = A.s ^ B.s;
  if (A.exn == EXN_NAN || B.exn == EXN_NAN) return make_nan(fo);
  if ((A.exn == EXN_INF && B.exn == EXN_ZERO) || (A.exn == EXN_ZERO && B.exn == EXN_INF))
    return make_nan(fo);
  if (A.exn == EXN_INF || B.exn == EXN_INF) return make_inf(s, fo);
  if (A.exn == EXN_ZERO || B.exn == EXN_ZERO) return make_zero(s, fo);
  big P;
  big_set_shl(&P, sig_of(A, fi) * sig_of(B, fi), 0); /* exact: at most 48 bits */
  return round_value(fo, s, &P, exp2_of(A, fi) + exp2_of(B, fi), mode);
}

uint64_t hfo_add_rm(uint64_t a, uint64_t b, int wE, int wF, int mode)
{
  fmt_t f = {wE, wF};
  if (!fmt_ok(f) || !mode_ok(mode)) return HFO_BAD_FORMAT;
  fields_t A = decode(a, f), B = decode(b, f);
  if (A.exn == EXN_NAN || B.exn == EXN_NAN) return make_nan(f);
  if (A.exn == EXN_INF && B.exn == EXN_INF) return A.s == B.s ? make_inf(A.s, f) : make_nan(f);
  if (A.exn == EXN_INF) return make_inf(A.s, f);
  if (B.exn == EXN_INF) return make_inf(B.s, f);
  if (A.exn == EXN_ZERO && B.exn == EXN_ZERO) return make_zero(A.s & B.s, f);
  if (A.exn == EXN_ZERO) return canonical(B, f);
  if (B.exn == EXN_ZERO) return canonical(A, f);
  /* Both normal: align both significands to the smaller exponent, exactly. */
  int64_t ea = exp2_of(A, f), eb = exp2_of(B, f);
  int64_t emin = ea < eb ? ea : eb;
  big X, Y, S;
  big_set_shl(&X, sig_of(A, f), (int)(ea - emin));
  big_set_shl(&Y, sig_of(B, f), (int)(eb - emin));
  int s;
  if (A.s == B.s) {
    big_add(&S, &X, &Y);
    s = A.s;
  } else {
    int c = big_cmp(&X, &Y);
    if (c == 0) return make_zero(0, f); /* exact cancellation gives +0, in both modes */
    if (c > 0) {
      big_sub(&S, &X, &Y);
      s = A.s;
    } else {
      big_sub(&S, &Y, &X);
      s = B.s;
    }
  }
  return round_value(f, s, &S, emin, mode);
}

uint64_t hfo_convert_rm(uint64_t a, int wE, int wF_src, int wF_dst, int mode)
{
  fmt_t fs = {wE, wF_src}, fd = {wE, wF_dst};
  if (!fmt_ok(fs) || !fmt_ok(fd) || !mode_ok(mode)) return HFO_BAD_FORMAT;
  fields_t A = decode(a, fs);
  if (A.exn == EXN_NAN) return make_nan(fd);
  if (A.exn == EXN_INF) return make_inf(A.s, fd);
  if (A.exn == EXN_ZERO) return make_zero(A.s, fd);
  big M;
  big_set_shl(&M, sig_of(A, fs), 0);
  return round_value(fd, A.s, &M, exp2_of(A, fs), mode);
}

uint64_t hfo_mul(uint64_t a, uint64_t b, int wE, int wF_in, int wF_out)
{
  return hfo_mul_rm(a, b, wE, wF_in, wF_out, HFO_RNE);
}

uint64_t hfo_add(uint64_t a, uint64_t b, int wE, int wF) { return hfo_add_rm(a, b, wE, wF, HFO_RNE); }

uint64_t hfo_convert(uint64_t a, int wE, int wF_src, int wF_dst)
{
  return hfo_convert_rm(a, wE, wF_src, wF_dst, HFO_RNE);
}

uint64_t hfo_relu(uint64_t a, int wE, int wF)
{
  fmt_t f = {wE, wF};
  if (!fmt_ok(f)) return HFO_BAD_FORMAT;
  fields_t A = decode(a, f);
  if (A.exn == EXN_NAN) return make_nan(f);
  if (A.s) return make_zero(0, f); /* negative normal, -inf and -0 all give +0 */
  return canonical(A, f);
}

uint64_t hfo_muladd_rm(uint64_t a, uint64_t b, uint64_t c, int wE, int wF_in, int wF_acc, int mode)
{
  uint64_t p = hfo_mul_rm(a, b, wE, wF_in, wF_acc, mode);
  uint64_t cw = hfo_convert_rm(c, wE, wF_in, wF_acc, mode); /* widening: exact */
  if (p == HFO_BAD_FORMAT || cw == HFO_BAD_FORMAT) return HFO_BAD_FORMAT;
  return hfo_add_rm(cw, p, wE, wF_acc, mode);
}

uint64_t hfo_muladd(uint64_t a, uint64_t b, uint64_t c, int wE, int wF_in, int wF_acc)
{
  return hfo_muladd_rm(a, b, c, wE, wF_in, wF_acc, HFO_RNE);
}

/* float32 -> code: the exact float32 value (subnormals included) rounded once. */
uint64_t hfo_quantize_f32(float x, int wE, int wF)
{
  fmt_t f = {wE, wF};
  if (!fmt_ok(f)) return HFO_BAD_FORMAT;
  uint32_t bits;
  memcpy(&bits, &x, 4);
  int s = (int)(bits >> 31);
  uint32_t ef = (bits >> 23) & 0xFF, frac = bits & 0x7FFFFF;
  if (ef == 0xFF) return frac ? make_nan(f) : make_inf(s, f);
  if (ef == 0 && frac == 0) return make_zero(s, f);
  uint64_t M = ef ? (frac | 0x800000u) : frac;
  int64_t e = ef ? (int64_t)ef - 150 : -149;
  big Mb;
  big_set_shl(&Mb, M, 0);
  return round_value(f, s, &Mb, e, HFO_RNE);
}

/* code -> float32: exact value formed in double (exact for wF <= 23 and the
 * supported exponent range), then one IEEE round-to-nearest-even conversion. */
float hfo_decode_f32(uint64_t code, int wE, int wF)
{
  fmt_t f = {wE, wF};
  if (!fmt_ok(f)) return NAN;
  fields_t A = decode(code, f);
  if (A.exn == EXN_NAN) {
    uint32_t qnan = 0x7FC00000u;
    float r;
    memcpy(&r, &qnan, 4);
    return r;
  }
  if (A.exn == EXN_INF) return A.s ? -INFINITY : INFINITY;
  if (A.exn == EXN_ZERO) return A.s ? -0.0f : 0.0f;
  double v = ldexp((double)sig_of(A, f), (int)exp2_of(A, f));
  return (float)(A.s ? -v : v);
}

/* ------------------------------------------------------------------------ */
/* Array forms. */

#define FMT_CHECK(we, wf) \
  do {                    \
    fmt_t f_ = {we, wf};  \
    if (!fmt_ok(f_)) return -1; \
  } while (0)

int hfo_quantize_f32_array(const float* src, size_t n, int wE, int wF, uint64_t* dst)
{
  FMT_CHECK(wE, wF);
  for (size_t i = 0; i < n; i++) dst[i] = hfo_quantize_f32(src[i], wE, wF);
  return 0;
}

int hfo_decode_f32_array(const uint64_t* src, size_t n, int wE, int wF, float* dst)
{
  FMT_CHECK(wE, wF);
  for (size_t i = 0; i < n; i++) dst[i] = hfo_decode_f32(src[i], wE, wF);
  return 0;
}

int hfo_mul_array(const uint64_t* a, const uint64_t* b, size_t n, int wE, int wF_in, int wF_out,
                  uint64_t* r)
{
  FMT_CHECK(wE, wF_in);
  FMT_CHECK(wE, wF_out);
  for (size_t i = 0; i < n; i++) r[i] = hfo_mul(a[i], b[i], wE, wF_in, wF_out);
  return 0;
}

int hfo_add_array(const uint64_t* a, const uint64_t* b, size_t n, int wE, int wF, uint64_t* r)
{
  FMT_CHECK(wE, wF);
  for (size_t i = 0; i < n; i++) r[i] = hfo_add(a[i], b[i], wE, wF);
  return 0;
}

int hfo_convert_array(const uint64_t* a, size_t n, int wE, int wF_src, int wF_dst, uint64_t* r)
{
  FMT_CHECK(wE, wF_src);
  FMT_CHECK(wE, wF_dst);
  for (size_t i = 0; i < n; i++) r[i] = hfo_convert(a[i], wE, wF_src, wF_dst);
  return 0;
}

int hfo_relu_array(const uint64_t* a, size_t n, int wE, int wF, uint64_t* r)
{
  FMT_CHECK(wE, wF);
  for (size_t i = 0; i < n; i++) r[i] = hfo_relu(a[i], wE, wF);
  return 0;
}

int hfo_muladd_array(const uint64_t* a, const uint64_t* b, const uint64_t* c, size_t n, int wE,
                     int wF_in, int wF_acc, uint64_t* r)
{
  FMT_CHECK(wE, wF_in);
  FMT_CHECK(wE, wF_acc);
  for (size_t i = 0; i < n; i++) r[i] = hfo_muladd(a[i], b[i], c[i], wE, wF_in, wF_acc);
  return 0;
}

int hfo_mul_rm_array(const uint64_t* a, const uint64_t* b, size_t n, int wE, int wF_in,
                     int wF_out, int mode, uint64_t* r)
{
  FMT_CHECK(wE, wF_in);
  FMT_CHECK(wE, wF_out);
  if (!mode_ok(mode)) return -1;
  for (size_t i = 0; i < n; i++) r[i] = hfo_mul_rm(a[i], b[i], wE, wF_in, wF_out, mode);
  return 0;
}

int hfo_add_rm_array(const uint64_t* a, const uint64_t* b, size_t n, int wE, int wF, int mode,
                     uint64_t* r)
{
  FMT_CHECK(wE, wF);
  if (!mode_ok(mode)) return -1;
  for (size_t i = 0; i < n; i++) r[i] = hfo_add_rm(a[i], b[i], wE, wF, mode);
  return 0;
}

int hfo_convert_rm_array(const uint64_t* a, size_t n, int wE, int wF_src, int wF_dst, int mode,
                         uint64_t* r)
{
  FMT_CHECK(wE, wF_src);
  FMT_CHECK(wE, wF_dst);
  if (!mode_ok(mode)) return -1;
  for (size_t i = 0; i < n; i++) r[i] = hfo_convert_rm(a[i], wE, wF_src, wF_dst, mode);
  return 0;
}

int hfo_muladd_rm_array(const uint64_t* a, const uint64_t* b, const uint64_t* c, size_t n, int wE,
                        int wF_in, int wF_acc, int mode, uint64_t* r)
{
  FMT_CHECK(wE, wF_in);
  FMT_CHECK(wE, wF_acc);
  if (!mode_ok(mode)) return -1;
  for (size_t i = 0; i < n; i++) r[i] = hfo_muladd_rm(a[i], b[i], c[i], wE, wF_in, wF_acc, mode);
  return 0;
}

/* ------------------------------------------------------------------------ */
/* Convolution. */

static int conv_ok(const hfo_conv_desc* d)
{
  if (!d) return 0;
  if (d->N < 1 || d->H < 1 || d->W < 1 || d->C < 1 || d->M < 1 || d->KH < 1 || d->KW < 1)
    return 0;
  if (d->stride < 1 || d->pad < 0) return 0;
  if (d->H + 2 * d->pad < d->KH || d->W + 2 * d->pad < d->KW) return 0;
  if (d->act != 0 && d->act != 1) return 0;
  if (!mode_ok(d->round)) return 0;
  fmt_t a = {d->wE, d->wF_in}, b = {d->wE, d->wF_acc}, c = {d->wE, d->wF_out};
  return fmt_ok(a) && fmt_ok(b) && fmt_ok(c);
}

static int out_h(const hfo_conv_desc* d) { return (d->H + 2 * d->pad - d->KH) / d->stride + 1; }
static int out_w(const hfo_conv_desc* d) { return (d->W + 2 * d->pad - d->KW) / d->stride + 1; }

/* One output of the convolution, accumulated in the fixed order ky, kx, c. */
static uint64_t conv_one(const uint64_t* ifm, const uint64_t* w, const hfo_conv_desc* d, int n,
                         int oy, int ox, int m)
{
  fmt_t fin = {d->wE, d->wF_in}, facc = {d->wE, d->wF_acc};
  uint64_t acc = make_zero(0, facc);
  uint64_t pad_zero = make_zero(0, fin);
  for (int ky = 0; ky < d->KH; ky++)
    for (int kx = 0; kx < d->KW; kx++)
      for (int c = 0; c < d->C; c++) {
        int iy = oy * d->stride + ky - d->pad;
        int ix = ox * d->stride + kx - d->pad;
        uint64_t x = pad_zero;
        if (iy >= 0 && iy < d->H && ix >= 0 && ix < d->W)
          x = ifm[(((size_t)n * d->H + iy) * d->W + ix) * d->C + c];
        uint64_t wv = w[(((size_t)ky * d->KW + kx) * d->C + c) * d->M + m];
        uint64_t p = hfo_mul_rm(wv, x, d->wE, d->wF_in, d->wF_acc, d->round);
        acc = hfo_add_rm(acc, p, d->wE, d->wF_acc, d->round);
      }
  if (d->act == 1) acc = hfo_relu(acc, d->wE, d->wF_acc);
  return hfo_convert_rm(acc, d->wE, d->wF_acc, d->wF_out, d->round);
}

typedef struct {
  const uint64_t* ifm;
  const uint64_t* w;
  uint64_t* out;
  const int64_t* pts; /* NULL for the full convolution */
  size_t count;       /* rows (n, oy) or points */
  const hfo_conv_desc* d;
  int tid, nthreads;
} conv_job;

static void* conv_worker(void* arg)
{
  conv_job* j = (conv_job*)arg;
  const hfo_conv_desc* d = j->d;
  int OH = out_h(d), OW = out_w(d);
  for (size_t r = (size_t)j->tid; r < j->count; r += (size_t)j->nthreads) {
    if (j->pts) {
      const int64_t* p = j->pts + 4 * r;
      j->out[r] = conv_one(j->ifm, j->w, d, (int)p[0], (int)p[1], (int)p[2], (int)p[3]);
    } else {
      int n = (int)(r / (size_t)OH), oy = (int)(r % (size_t)OH);
      for (int ox = 0; ox < OW; ox++)
        for (int m = 0; m < d->M; m++)
          j->out[(((size_t)n * OH + oy) * OW + ox) * d->M + m] =
              conv_one(j->ifm, j->w, d, n, oy, ox, m);
    }
  }
  return NULL;
}

int hfo_default_threads(void)
{
  long n = sysconf(_SC_NPROCESSORS_ONLN);
  return n < 1 ? 1 : (int)n;
}

static int run_conv(const uint64_t* ifm, const uint64_t* w, uint64_t* out, const int64_t* pts,
                    size_t count, const hfo_conv_desc* d, int nthreads)
{
  if (nthreads <= 0) nthreads = hfo_default_threads();
  if (nthreads > 256) nthreads = 256;
  pthread_t th[256];
  conv_job jobs[256];
  for (int t = 0; t < nthreads; t++) {
    conv_job j = {ifm, w, out, pts, count, d, t, nthreads};
    jobs[t] = j;
  }
  if (nthreads == 1) {
    conv_worker(&jobs[0]);
    return 0;
  }
  int started = 0;
  for (int t = 0; t < nthreads; t++) {
    if (pthread_create(&th[t], NULL, conv_worker, &jobs[t]) != 0) break;
    started++;
  }
  for (int t = 0; t < started; t++) pthread_join(th[t], NULL);
  /* Any job whose thread could not start runs here. */
  for (int t = started; t < nthreads; t++) conv_worker(&jobs[t]);
  return 0;
}

int hfo_conv2d(const uint64_t* ifm, const uint64_t* w, uint64_t* ofm, const hfo_conv_desc* d,
               int nthreads)
{
  if (!conv_ok(d) || !ifm || !w || !ofm) return -1;
  return run_conv(ifm, w, ofm, NULL, (size_t)d->N * (size_t)out_h(d), d, nthreads);
}

int hfo_conv2d_points(const uint64_t* ifm, const uint64_t* w, const int64_t* pts, size_t npts,
                      uint64_t* out, const hfo_conv_desc* d, int nthreads)
{
  if (!conv_ok(d) || !ifm || !w || !out || (!pts && npts)) return -1;
  int OH = out_h(d), OW = out_w(d);
  for (size_t i = 0; i < npts; i++) {
    const int64_t* p = pts + 4 * i;
    if (p[0] < 0 || p[0] >= d->N || p[1] < 0 || p[1] >= OH || p[2] < 0 || p[2] >= OW ||
        p[3] < 0 || p[3] >= d->M)
      return -1;
  }
  return run_conv(ifm, w, out, pts, npts, d, nthreads);
}

/* ------------------------------------------------------------------------ */
/* Average pooling. */

uint64_t hfo_recip(uint64_t n, int wE, int wF)
{
  fmt_t f = {wE, wF};
  if (!fmt_ok(f) || n == 0 || n > ((uint64_t)1 << 32)) return HFO_BAD_FORMAT;
  /* 1/n = (q + r/n) * 2^-k with q = floor(2^k / n) of at least wF+3 bits;
   * a sticky bit below q (set when r != 0) keeps the rounding exact */
  int ln = 0;
  while (ln < 64 && (n >> ln) != 0) ln++;
  int k = wF + 3 + ln;
  uint64_t q = ((uint64_t)1 << k) / n, r = ((uint64_t)1 << k) % n;
  big M;
  big_set_shl(&M, (q << 1) | (r != 0), 0);
  return round_value(f, 0, &M, -(int64_t)k - 1, HFO_RNE);
}

int hfo_avgpool(const uint64_t* in, uint64_t* out, int N, int H, int W, int C, int wE, int wF_in,
                int wF_acc, int wF_out, int round)
{
  fmt_t fi = {wE, wF_in}, fa = {wE, wF_acc}, fo = {wE, wF_out};
  if (!in || !out || N < 1 || H < 1 || W < 1 || C < 1 || !fmt_ok(fi) || !fmt_ok(fa) ||
      !fmt_ok(fo) || wF_in > wF_acc || !mode_ok(round))
    return -1;
  uint64_t scale = hfo_recip((uint64_t)H * (uint64_t)W, wE, wF_acc);
  for (int n = 0; n < N; n++) {
    for (int c = 0; c < C; c++) {
      uint64_t acc = make_zero(0, fa);
      for (int y = 0; y < H; y++) {
        for (int x = 0; x < W; x++) {
          uint64_t v = in[(((size_t)n * H + y) * W + x) * C + c];
          acc = hfo_add_rm(acc, hfo_convert_rm(v, wE, wF_in, wF_acc, round), wE, wF_acc, round);
        }
      }
      out[(size_t)n * C + c] = hfo_mul_rm(acc, scale, wE, wF_acc, wF_out, round);
    }
  }
  return 0;
}
