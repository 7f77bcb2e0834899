/*
 * hobflops.h -- C ABI of libhobflops.so: bitsliced custom-precision
 * floating-point (HOBFLOPS) arithmetic and MCMK convolution on MI355X (gfx950).
 *
 * Number format (paper Sec. 3.3): a FloPoCo word of NB = 3 + wE + wF bits,
 * held LSB first in a code: fraction F in bits [0, wF), exponent E in
 * [wF, wF+wE), sign at wF+wE, 2-bit exception field above it (00 zero,
 * 01 normal, 10 infinity, 11 NaN). Exponent bias 2^(wE-1) - 1; no subnormal
 * numbers; every E is an ordinary binade. Every operation rounds to nearest,
 * ties to even (paper Sec. 4), with an unbounded exponent first and the range
 * check after: overflow gives a signed infinity, underflow a zero with the sign
 * of the exact value. NaN, infinity and zero signs follow IEEE-754. Results are
 * canonical: E = F = 0 for zero and infinity, s = E = F = 0 for NaN.
 *
 * Plane layout PL32 (bitslice-parallel layout of paper Sec. 3.2): a tensor of
 * logical shape [rows][len], packed along len, is stored as uint32
 * words[rows][ceil(len/32)][NB]; bit j of words[r][g][b] is bit b of the code
 * of element (r, 32*g + j). Lanes past len hold code 0 (+0).
 *
 * Conventions for every entry point:
 *  - Pointers are device pointers (HBM) owned by the caller; the library
 *    allocates no device memory. Inputs and outputs of one call must not
 *    overlap. Pointers must be 4-byte aligned.
 *  - `stream` is a hipStream_t (NULL = the default stream). Calls enqueue work
 *    on it and return without synchronising.
 *  - Arguments are checked before anything is launched; a rejected call
 *    launches nothing and returns a negative status (see below).
 *  - Supported widths: 2 <= wE <= 8, 1 <= wF <= 23, NB <= 32. The convolution
 *    and element-wise MAC run only for the format combinations and rounding
 *    modes the library was generated for (hobflops_conv2d_supported /
 *    hobflops_muladd_supported); other combinations return
 *    HOBFLOPS_EUNSUPPORTED.
 *  - Apart from two diagnostics of the split convolution kernel's bounded
 *    waits (the give-up count and the wait limit, see hobflops_wait_failures),
 *    the library keeps no state between calls; it is safe to call from
 *    several host threads.
 *
 * Where this interface differs from the plain one the paper's problem
 * statement suggests (format widths, tensor shapes, one accumulation order):
 *  - hobflops_plane_words returns a status and writes the count through a
 *    pointer, so that an overflowing size is an error rather than a value;
 *  - the rounding mode is an argument of hobflops_muladd, hobflops_avgpool and
 *    hobflops_netlist_ops and a field of hobflops_conv_desc, since the paper
 *    measures round-toward-zero as well as nearest-even (Sec. 4); its values
 *    are spelled HOBFLOPS_ROUND_NEAREST_EVEN and HOBFLOPS_ROUND_TOWARD_ZERO;
 *  - hobflops_conv_desc adds `algo` (the kernel shape) and `ofm_kind` (the
 *    unpack fused into the last layer's epilogue, Sec. 3.4);
 *  - hobflops_netlist_ops reports the fused MAC, the multiplier, the
 *    accumulating adder and the element-wise MAC separately;
 *  - hobflops_pack_batch, hobflops_avgpool, hobflops_conv2d_algo and the
 *    *_supported queries are additions.
 */
#ifndef HOBFLOPS_H
#define HOBFLOPS_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct {
  int wE; /* exponent bits */
  int wF; /* fraction bits */
} hobflops_fmt;

enum {
  HOBFLOPS_OK = 0,
  HOBFLOPS_EINVAL = -1,       /* bad size, shape, format or null pointer */
  HOBFLOPS_EUNSUPPORTED = -2, /* valid request, no generated kernel for it */
  HOBFLOPS_EALIGN = -3,       /* a pointer is not 4-byte aligned */
  HOBFLOPS_EHIP = -4          /* the HIP runtime reported an error */
};

enum { HOBFLOPS_SRC_F32 = 0, HOBFLOPS_SRC_CODE_U32 = 1 };
/* Rounding of the multiply-accumulate operations (paper Sec. 4): to nearest
 * with ties to even, or toward zero (the dropped bits of the exact value are
 * discarded). In both modes the exponent range is checked after rounding, so
 * an overflow gives a signed infinity, and an exact cancellation gives +0.
 * hobflops_pack always rounds to nearest even. */
enum { HOBFLOPS_ROUND_NEAREST_EVEN = 0, HOBFLOPS_ROUND_TOWARD_ZERO = 1 };
enum { HOBFLOPS_ORDER_KY_KX_C = 0 };
enum { HOBFLOPS_ACT_NONE = 0, HOBFLOPS_ACT_RELU = 1 };
/* Kernel shape of hobflops_conv2d (results are identical for all four):
 * FUSED runs multiplier and adder on the same wave; SPLIT runs them on
 * separate waves of the same CU (one accumulator/multiplier pair per SIMD) so
 * that a launch with few accumulator chains can still fill the VALU;
 * SPLIT_COMPACT is SPLIT in a form of which two workgroups share a CU (two
 * pairs per SIMD, two products per hand-over). AUTO picks SPLIT when the
 * launch has at most one accumulator wave (64 positions of one 32-kernel
 * tile) per SIMD of the device, SPLIT_COMPACT (else SPLIT) when it has at most
 * two, and FUSED otherwise. */
enum {
  HOBFLOPS_ALGO_AUTO = 0,
  HOBFLOPS_ALGO_FUSED = 1,
  HOBFLOPS_ALGO_SPLIT = 2,
  HOBFLOPS_ALGO_SPLIT_COMPACT = 3
};
/* What hobflops_conv2d writes to ofm: PL32 planes of out_fmt (the next
 * layer's input, the default), or with the unpack fused into the epilogue
 * (the last layer, paper Sec. 3.4), one value per element, row-major
 * [N*OH*OW][M]: float32 as hobflops_unpack writes them, or uint32 codes. */
enum { HOBFLOPS_OFM_PLANES = 0, HOBFLOPS_OFM_F32 = 1, HOBFLOPS_OFM_CODE_U32 = 2 };

/* Number of uint32 words of a PL32 tensor: rows * ceil(len/32) * NB.
 * Returns HOBFLOPS_OK and writes *words, or HOBFLOPS_EINVAL. */
int hobflops_plane_words(int64_t rows, int64_t len, hobflops_fmt f, int64_t* words);

/* Quantise and pack (paper Sec. 3.4 and the convolution figure: data are
 * transformed to the bitslice layout before the first layer).
 * src: rows*len elements, row-major; kind HOBFLOPS_SRC_F32 = float32 values,
 * each rounded to format f (the exact float32 value, subnormals included;
 * NaN -> NaN, +-inf -> +-inf, +-0 -> +-0); kind HOBFLOPS_SRC_CODE_U32 = codes
 * in format f (bits above NB ignored; fields of non-normal codes are kept as
 * given). planes: hobflops_plane_words(rows, len, f) words, fully written. */
int hobflops_pack(const void* src, int kind, int64_t rows, int64_t len, hobflops_fmt f,
                  uint32_t* planes, void* stream);

/* One tensor of hobflops_pack_batch: the arguments of a hobflops_pack call
 * other than the format and the stream. */
typedef struct {
  const void* src;
  int kind;
  int64_t rows;
  int64_t len;
  uint32_t* planes;
} hobflops_pack_job;

/* hobflops_pack of several tensors of one format in few kernel launches: one
 * per 8 jobs (a job of more than 2^30 values counts as several). Before the
 * paper's first layer both the IFM and the kernels are transformed (Sec. 3.4);
 * packed together they take one launch instead of two. jobs: host array of
 * count entries (count >= 0; jobs may be NULL when count is 0), read before
 * the call returns. Every job is checked as hobflops_pack checks its
 * arguments, all before anything is launched, so that an error launches
 * nothing; jobs with no values are skipped. The results are those of one
 * hobflops_pack call per job; a job's planes must not overlap the src or the
 * planes of another job. */
int hobflops_pack_batch(const hobflops_pack_job* jobs, int count, hobflops_fmt f, void* stream);

/* Unpack (paper Sec. 3.4: transformed back to floats after the last layer).
 * planes: PL32 tensor of format f; dst: rows*len elements, row-major; kind
 * HOBFLOPS_SRC_CODE_U32 writes codes (bits above NB zero), HOBFLOPS_SRC_F32
 * writes float32: the exact value rounded to nearest even float32 (exact for
 * wE <= 7), NaN as 0x7FC00000. */
int hobflops_unpack(const uint32_t* planes, int64_t rows, int64_t len, hobflops_fmt f, int kind,
                    void* dst, void* stream);

/* Multi-channel multi-kernel convolution whose every multiply-add is a
 * bitsliced custom-precision multiply followed by an add (paper Sec. 3.4).
 *   ifm: PL32, rows N*H*W (NHWC order), len C, format in_fmt
 *   w:   PL32, rows KH*KW*C (HWIO order, row (ky*KW + kx)*C + c), len M, in_fmt
 *   ofm: PL32, rows N*OH*OW, len M, format out_fmt; OH = (H + 2*pad - KH)/stride + 1
 *        (ofm_kind HOBFLOPS_OFM_PLANES), or N*OH*OW*M float32 values or uint32
 *        codes of out_fmt, row-major (HOBFLOPS_OFM_F32 / _CODE_U32)
 * For each output (n, oy, ox, m): acc = +0 in acc_fmt; for ky, then kx, then c:
 *   acc = add(acc, mul(w[ky][kx][c][m], x)), x the IFM value or +0 for a
 *   padding tap, mul rounding into acc_fmt and add rounding in acc_fmt; then
 *   ofm = convert(act(acc)) into out_fmt (ReLU: NaN stays NaN, negatives and -0
 *   give +0). All formats share wE; acc_fmt.wF >= in_fmt.wF. With
 *   acc_fmt.wF = in_fmt.wF + 1 this is the paper's "single" MAC type, with
 *   2 * in_fmt.wF + 1 its "extended" type, whose products are exact (Table 3).
 *   round: HOBFLOPS_ROUND_* for every mul, add and the final convert; order
 *   must be HOBFLOPS_ORDER_KY_KX_C. algo SPLIT (SPLIT_COMPACT) returns
 *   HOBFLOPS_EUNSUPPORTED for a variant generated without that kernel (its
 *   netlists do not fit the registers); AUTO then picks among the others. */
typedef struct {
  int N, H, W, C, M, KH, KW, stride, pad;
  hobflops_fmt in_fmt, acc_fmt, out_fmt;
  int act, round, order;
  int algo;     /* HOBFLOPS_ALGO_* */
  int ofm_kind; /* HOBFLOPS_OFM_* */
} hobflops_conv_desc;

int hobflops_conv2d(const uint32_t* ifm, const uint32_t* w, uint32_t* ofm,
                    const hobflops_conv_desc* d, void* stream);

/* 1 if hobflops_conv2d has a kernel for d's formats, activation, rounding
 * mode and (for HOBFLOPS_ALGO_SPLIT and _SPLIT_COMPACT) kernel shape, else 0. */
int hobflops_conv2d_supported(const hobflops_conv_desc* d);

/* The kernel shape hobflops_conv2d runs d in (HOBFLOPS_ALGO_FUSED, _SPLIT or
 * _SPLIT_COMPACT): d->algo itself, or for HOBFLOPS_ALGO_AUTO the shape AUTO
 * picks on the current device. Returns that value (>= 1), or a negative
 * status: HOBFLOPS_EINVAL for a bad descriptor, HOBFLOPS_EUNSUPPORTED where
 * hobflops_conv2d_supported is 0, HOBFLOPS_EHIP if AUTO cannot query the
 * device. Launches nothing. */
int hobflops_conv2d_algo(const hobflops_conv_desc* d);

/* Element-wise r = add(widen(c), mul(a, b)) over n elements of flat PL32
 * tensors (rows 1, len n): a, b, c in in_fmt, r in acc_fmt (same wE,
 * acc_fmt.wF >= in_fmt.wF); the product is rounded into acc_fmt, c widened
 * exactly, the sum rounded once more (the paper's MAC: a multiplier then an
 * adder, Sec. 3.3 and Table 3), both in mode round (HOBFLOPS_ROUND_*). */
int hobflops_muladd(const uint32_t* a, const uint32_t* b, const uint32_t* c, uint32_t* r,
                    int64_t n, hobflops_fmt in_fmt, hobflops_fmt acc_fmt, int round,
                    void* stream);

int hobflops_muladd_supported(hobflops_fmt in_fmt, hobflops_fmt acc_fmt, int round);

/* Bitwise VALU instructions per 32-lane word in the generated netlists of a
 * MAC (in_fmt x in_fmt -> acc_fmt, then acc_fmt + acc_fmt, rounding mode
 * round): the convolution's fused multiply-add step, its multiplier and its
 * accumulating adder alone (the split kernel's two wave roles; 0 where that
 * kernel was not generated), and the element-wise kernel's MAC (the paper's
 * gate count, Sec. 4: throughput follows it). Returns HOBFLOPS_OK,
 * HOBFLOPS_EINVAL or HOBFLOPS_EUNSUPPORTED; any output pointer may be NULL. */
int hobflops_netlist_ops(hobflops_fmt in_fmt, hobflops_fmt acc_fmt, int round, int* conv_mac_ops,
                         int* conv_mul_ops, int* conv_accum_ops, int* muladd_ops);

/* Global average pooling on PL32 planes: the pooling layer the paper proposes
 * to build in the packed format, between MobileNets' last convolution and its
 * fully connected layer (Sec. 4, on where the format transformation happens).
 *   in:  [N * H * W][ceil(C/32)][NB_in]  (the planes of an NHWC tensor, as a
 *        convolution writes them; padding channels hold +0)
 *   out: [N][ceil(C/32)][NB_out]          (device memory owned by the caller)
 * For each (n, c): acc = +0 in acc_fmt; for y, then x:
 *   acc = add(acc, widen(in[n][y][x][c]))  (widening to acc_fmt is exact)
 * then out = mul(acc, s) rounded into out_fmt, s the code of 1/(H*W) in
 * acc_fmt rounded to nearest even (+0 if below the format's range). The adds
 * and the multiply round in mode round (HOBFLOPS_ROUND_*). All formats share
 * wE; acc_fmt.wF >= in_fmt.wF. in and out must not overlap.
 * Returns HOBFLOPS_EINVAL (shape, format, null pointer), HOBFLOPS_EALIGN,
 * HOBFLOPS_EUNSUPPORTED (combination not generated) or HOBFLOPS_EHIP. */
int hobflops_avgpool(const uint32_t* in, uint32_t* out, int N, int H, int W, int C,
                     hobflops_fmt in_fmt, hobflops_fmt acc_fmt, hobflops_fmt out_fmt, int round,
                     void* stream);

/* 1 if hobflops_avgpool has a kernel for these formats and rounding mode. */
int hobflops_avgpool_supported(hobflops_fmt in_fmt, hobflops_fmt acc_fmt, hobflops_fmt out_fmt,
                               int round);

/* Bitwise VALU instructions per 32-lane word of the pooling netlists: one
 * accumulating add and the final multiply. Any output pointer may be NULL. */
int hobflops_avgpool_netlist_ops(hobflops_fmt in_fmt, hobflops_fmt acc_fmt, hobflops_fmt out_fmt,
                                 int round, int* accum_ops, int* scale_ops);

/* Diagnostics of the split convolution kernel (HOBFLOPS_ALGO_SPLIT and
 * _SPLIT_COMPACT). Its
 * multiplier and accumulator waves hand products over through counters in
 * LDS; every wait for a counter sleeps at most a bounded number of times
 * (about 64 clocks each), so that a counter that never came would end the
 * wait instead of hanging the GPU. A wait that reaches its bound without the
 * counter is a give-up: that launch's results are invalid, and one give-up is
 * added to a per-device count.
 *
 * hobflops_wait_failures: synchronises the current device, writes its
 * give-up count (since the library was loaded or last reset) to *count, and
 * sets it to zero if reset is nonzero. For tests and monitoring, not for hot
 * loops. Returns HOBFLOPS_OK, HOBFLOPS_EINVAL (count NULL) or HOBFLOPS_EHIP.
 *
 * hobflops_set_wait_limit: the bound, in sleeps, for launches made after the
 * call, process-wide (default 1048576, about 30 ms of sleeping per wait). With
 * 0 a wait gives up when its first look does not find the counter: tests use
 * it to check that give-ups are counted. The kernels still finish normally.
 * hobflops_get_wait_limit returns the current bound. */
int hobflops_wait_failures(uint32_t* count, int reset);
int hobflops_set_wait_limit(uint32_t sleeps);
uint32_t hobflops_get_wait_limit(void);

/* Text for a status code; for HOBFLOPS_EHIP, the last HIP error of this
 * thread. The pointer stays valid until the next call on the same thread. */
const char* hobflops_status_string(int status);

#ifdef __cplusplus
}
#endif
#endif
