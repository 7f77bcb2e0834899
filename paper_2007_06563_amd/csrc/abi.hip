// C ABI of libhobflops.so (declared in include/hobflops.h): argument checks,
// variant dispatch and launches. The only value computed on the host is the
// pooling scale, the code of 1/(H*W) (recip_code); all MAC arithmetic runs in
// the kernels.
#include <hip/hip_runtime.h>
#include <limits.h>
#include <stdint.h>
#include <stdio.h>
#include <string.h>

#include <atomic>
#include <mutex>
#include <vector>

#include "hobflops.h"
#include "pack.hpp"
#include "registry.hpp"

using namespace hobflops;

namespace {

thread_local char g_errbuf[256];

// Give-ups of the split kernel's bounded waits (a diagnostic: each one means
// that launch's results are invalid). One word per device, in this file's
// device code; kernels get its address, taken once per device with that
// device current (the symbol's host-side name is not a device address).
__device__ uint32_t g_wait_fail_word;
constexpr int kMaxDevices = 64;
std::mutex g_wait_mutex;
uint32_t* g_wait_fail_ptr[kMaxDevices];
std::atomic<uint32_t> g_spin_cap{kSpinCap};

// The give-up word of the current device (*ptr), or a HIP error.
hipError_t wait_fail_word(uint32_t** ptr) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(g_wait_mutex);
  if (!g_wait_fail_ptr[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(g_wait_fail_word));
    if (e != hipSuccess) return e;
    g_wait_fail_ptr[dev] = static_cast<uint32_t*>(p);
  }
  *ptr = g_wait_fail_ptr[dev];
  return hipSuccess;
}

int fmt_ok(hobflops_fmt f) {
  return f.wE >= 2 && f.wE <= 8 && f.wF >= 1 && f.wF <= 23 && 3 + f.wE + f.wF <= 32;
}
int aligned(const void* p) { return ((uintptr_t)p & 3u) == 0; }

int hip_status(hipError_t e) {
  if (e == hipSuccess) return HOBFLOPS_OK;
  snprintf(g_errbuf, sizeof g_errbuf, "HIP error %d: %s", (int)e, hipGetErrorString(e));
  return HOBFLOPS_EHIP;
}

const ConvVariant* find_conv(const hobflops_conv_desc* d) {
  for (int i = 0; i < kNumConvVariants; ++i) {
    const ConvVariant& v = kConvVariants[i];
    if (v.wE == d->in_fmt.wE && v.wF_in == d->in_fmt.wF && v.wF_acc == d->acc_fmt.wF &&
        v.wF_out == d->out_fmt.wF && v.act == d->act && v.round == d->round)
      return &v;
  }
  return nullptr;
}

const MuladdVariant* find_muladd(hobflops_fmt in, hobflops_fmt acc, int round) {
  for (int i = 0; i < kNumMuladdVariants; ++i) {
    const MuladdVariant& v = kMuladdVariants[i];
    if (v.wE == in.wE && v.wF_in == in.wF && v.wF_acc == acc.wF && acc.wE == in.wE &&
        v.round == round)
      return &v;
  }
  return nullptr;
}

const PoolVariant* find_pool(hobflops_fmt in, hobflops_fmt acc, hobflops_fmt out, int round) {
  if (acc.wE != in.wE || out.wE != in.wE) return nullptr;
  for (int i = 0; i < kNumPoolVariants; ++i) {
    const PoolVariant& v = kPoolVariants[i];
    if (v.wE == in.wE && v.wF_in == in.wF && v.wF_acc == acc.wF && v.wF_out == out.wF &&
        v.round == round)
      return &v;
  }
  return nullptr;
}

// The code of 1/n (n >= 1) in format f, to nearest with ties to even. With
// 2^(t-1) <= n < 2^t: a power of two is exact; otherwise 1/n = (2^t/n) 2^-t
// with 2^t/n in (1, 2), whose fraction bits are floor(2^(t+wF)/n) - 2^wF,
// rounded by the remainder. Below the smallest normal the code is +0.
uint32_t recip_code(uint64_t n, hobflops_fmt f) {
  int t = 0;
  while (t < 64 && (n >> t) != 0) ++t;
  const int64_t bias = ((int64_t)1 << (f.wE - 1)) - 1;
  int64_t u;
  uint64_t frac;
  if ((n & (n - 1)) == 0) {
    u = -(int64_t)(t - 1);
    frac = 0;
  } else {
    u = -(int64_t)t;
    const uint64_t num = (uint64_t)1 << (t + f.wF);
    uint64_t q = num / n;
    const uint64_t r = num % n;
    if (2 * r > n || (2 * r == n && (q & 1u))) ++q;
    if (q == ((uint64_t)1 << (f.wF + 1))) {  // rounded up into the next binade
      q >>= 1;
      ++u;
    }
    frac = q - ((uint64_t)1 << f.wF);
  }
  const int64_t eb = u + bias;
  if (eb < 0) return 0u;
  return (1u << (f.wF + f.wE + 1)) | ((uint32_t)eb << f.wF) | (uint32_t)frac;
}

int round_ok(int round) {
  return round == HOBFLOPS_ROUND_NEAREST_EVEN || round == HOBFLOPS_ROUND_TOWARD_ZERO;
}

// Shape and format checks shared by conv2d and conv2d_supported.
int conv_check(const hobflops_conv_desc* d) {
  if (!d) return HOBFLOPS_EINVAL;
  if (d->N < 1 || d->H < 1 || d->W < 1 || d->C < 1 || d->M < 1 || d->KH < 1 || d->KW < 1 ||
      d->stride < 1 || d->pad < 0)
    return HOBFLOPS_EINVAL;
  if (d->H + 2 * (int64_t)d->pad < d->KH || d->W + 2 * (int64_t)d->pad < d->KW)
    return HOBFLOPS_EINVAL;
  if (!fmt_ok(d->in_fmt) || !fmt_ok(d->acc_fmt) || !fmt_ok(d->out_fmt)) return HOBFLOPS_EINVAL;
  if (d->acc_fmt.wE != d->in_fmt.wE || d->out_fmt.wE != d->in_fmt.wE) return HOBFLOPS_EINVAL;
  if (d->acc_fmt.wF < d->in_fmt.wF) return HOBFLOPS_EINVAL;
  if (d->act != HOBFLOPS_ACT_NONE && d->act != HOBFLOPS_ACT_RELU) return HOBFLOPS_EINVAL;
  if (!round_ok(d->round) || d->order != HOBFLOPS_ORDER_KY_KX_C) return HOBFLOPS_EINVAL;
  if (d->algo != HOBFLOPS_ALGO_AUTO && d->algo != HOBFLOPS_ALGO_FUSED &&
      d->algo != HOBFLOPS_ALGO_SPLIT && d->algo != HOBFLOPS_ALGO_SPLIT_COMPACT)
    return HOBFLOPS_EINVAL;
  if (d->ofm_kind != HOBFLOPS_OFM_PLANES && d->ofm_kind != HOBFLOPS_OFM_F32 &&
      d->ofm_kind != HOBFLOPS_OFM_CODE_U32)
    return HOBFLOPS_EINVAL;
  const int64_t OH = (d->H + 2 * (int64_t)d->pad - d->KH) / d->stride + 1;
  const int64_t OW = (d->W + 2 * (int64_t)d->pad - d->KW) / d->stride + 1;
  const int64_t P = (int64_t)d->N * OH * OW;
  const int64_t MT = (d->M + 31) / 32;
  // index arithmetic inside the kernel is 32-bit for positions and taps
  if (P > (int64_t)1 << 30 || (int64_t)d->N * d->H * d->W > (int64_t)1 << 30 ||
      (int64_t)d->KH * d->KW * d->C > (int64_t)1 << 24 || MT > 65535)
    return HOBFLOPS_EINVAL;
  return HOBFLOPS_OK;
}

}  // namespace

extern "C" {

int hobflops_plane_words(int64_t rows, int64_t len, hobflops_fmt f, int64_t* words) {
  if (!words || rows < 0 || len < 0 || !fmt_ok(f)) return HOBFLOPS_EINVAL;
  const int64_t G = (len + 31) / 32;
  const int64_t nb = 3 + f.wE + f.wF;
  if (rows > 0 && G > INT64_MAX / nb / rows) return HOBFLOPS_EINVAL;
  *words = rows * G * nb;
  return HOBFLOPS_OK;
}

int hobflops_pack(const void* src, int kind, int64_t rows, int64_t len, hobflops_fmt f,
                  uint32_t* planes, void* stream) {
  const hobflops_pack_job job{src, kind, rows, len, planes};
  return hobflops_pack_batch(&job, 1, f, stream);
}

int hobflops_pack_batch(const hobflops_pack_job* jobs, int count, hobflops_fmt f, void* stream) {
  if (count < 0 || (count > 0 && !jobs) || !fmt_ok(f)) return HOBFLOPS_EINVAL;
  std::vector<PackTensor> t;
  t.reserve(count);
  for (int n = 0; n < count; ++n) {
    const hobflops_pack_job& j = jobs[n];
    if (j.rows < 0 || j.len < 0) return HOBFLOPS_EINVAL;
    if (j.kind != HOBFLOPS_SRC_F32 && j.kind != HOBFLOPS_SRC_CODE_U32) return HOBFLOPS_EINVAL;
    if (j.rows == 0 || j.len == 0) continue;
    if (!j.src || !j.planes) return HOBFLOPS_EINVAL;
    if (!aligned(j.src) || !aligned(j.planes)) return HOBFLOPS_EALIGN;
    if ((j.len + 31) / 32 > INT32_MAX) return HOBFLOPS_EINVAL;
    int64_t words;  // rows * groups * NB must not overflow
    if (hobflops_plane_words(j.rows, j.len, f, &words) != HOBFLOPS_OK) return HOBFLOPS_EINVAL;
    t.push_back(PackTensor{j.src, j.kind, j.rows, j.len, j.planes});
  }
  if (t.empty()) return HOBFLOPS_OK;
  return hip_status(
      launch_pack_batch(t.data(), (int)t.size(), f.wE, f.wF, (hipStream_t)stream));
}

int hobflops_unpack(const uint32_t* planes, int64_t rows, int64_t len, hobflops_fmt f, int kind,
                    void* dst, void* stream) {
  if (rows < 0 || len < 0 || !fmt_ok(f)) return HOBFLOPS_EINVAL;
  if (kind != HOBFLOPS_SRC_F32 && kind != HOBFLOPS_SRC_CODE_U32) return HOBFLOPS_EINVAL;
  if (rows == 0 || len == 0) return HOBFLOPS_OK;
  if (!dst || !planes) return HOBFLOPS_EINVAL;
  if (!aligned(dst) || !aligned(planes)) return HOBFLOPS_EALIGN;
  if ((len + 31) / 32 > INT32_MAX) return HOBFLOPS_EINVAL;
  return hip_status(launch_unpack(planes, rows, len, f.wE, f.wF, kind, dst, (hipStream_t)stream));
}

// The kernel shape a conv runs in: d->algo, or for AUTO the choice below,
// made from the launch's chain waves (one accumulator wave per 64 positions
// and 32-kernel tile). Up to one per SIMD: the split kernel, one wave pair per
// SIMD. Up to two: its compact form, two pairs per SIMD in one round of
// workgroups (or the split kernel in two rounds where the compact form was
// not generated). More: the fused kernel, whose waves fill the SIMDs by
// themselves.
static int resolve_algo(const hobflops_conv_desc* d, const ConvVariant* v, int* algo) {
  *algo = d->algo;
  if (d->algo != HOBFLOPS_ALGO_AUTO) return HOBFLOPS_OK;
  int dev = 0, cus = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e == hipSuccess) e = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev);
  if (e != hipSuccess) return hip_status(e);
  const int64_t OH = (d->H + 2 * (int64_t)d->pad - d->KH) / d->stride + 1;
  const int64_t OW = (d->W + 2 * (int64_t)d->pad - d->KW) / d->stride + 1;
  const int64_t P = (int64_t)d->N * OH * OW;
  const int64_t chain_waves = (P + 63) / 64 * ((d->M + 31) / 32);
  const int64_t simds = 4 * (int64_t)cus;
  if (chain_waves <= simds && v->has_split)
    *algo = HOBFLOPS_ALGO_SPLIT;
  else if (chain_waves <= 2 * simds && v->has_compact)
    *algo = HOBFLOPS_ALGO_SPLIT_COMPACT;
  else if (chain_waves <= 2 * simds && v->has_split)
    *algo = HOBFLOPS_ALGO_SPLIT;
  else
    *algo = HOBFLOPS_ALGO_FUSED;
  return HOBFLOPS_OK;
}

int hobflops_conv2d_algo(const hobflops_conv_desc* d) {
  const int st = conv_check(d);
  if (st != HOBFLOPS_OK) return st;
  const ConvVariant* v = find_conv(d);
  if (!v || (d->algo == HOBFLOPS_ALGO_SPLIT && !v->has_split) ||
      (d->algo == HOBFLOPS_ALGO_SPLIT_COMPACT && !v->has_compact))
    return HOBFLOPS_EUNSUPPORTED;
  int algo = 0;
  const int st2 = resolve_algo(d, v, &algo);
  return st2 != HOBFLOPS_OK ? st2 : algo;
}

int hobflops_conv2d_supported(const hobflops_conv_desc* d) {
  if (conv_check(d) != HOBFLOPS_OK) return 0;
  const ConvVariant* v = find_conv(d);
  return v != nullptr && (d->algo != HOBFLOPS_ALGO_SPLIT || v->has_split) &&
         (d->algo != HOBFLOPS_ALGO_SPLIT_COMPACT || v->has_compact);
}

int hobflops_conv2d(const uint32_t* ifm, const uint32_t* w, uint32_t* ofm,
                    const hobflops_conv_desc* d, void* stream) {
  const int st = conv_check(d);
  if (st != HOBFLOPS_OK) return st;
  if (!ifm || !w || !ofm) return HOBFLOPS_EINVAL;
  if (!aligned(ifm) || !aligned(w) || !aligned(ofm)) return HOBFLOPS_EALIGN;
  const ConvVariant* v = find_conv(d);
  if (!v || (d->algo == HOBFLOPS_ALGO_SPLIT && !v->has_split) ||
      (d->algo == HOBFLOPS_ALGO_SPLIT_COMPACT && !v->has_compact))
    return HOBFLOPS_EUNSUPPORTED;
  ConvParams p;
  p.N = d->N;
  p.H = d->H;
  p.W = d->W;
  p.C = d->C;
  p.M = d->M;
  p.KH = d->KH;
  p.KW = d->KW;
  p.stride = d->stride;
  p.pad = d->pad;
  p.OH = (d->H + 2 * d->pad - d->KH) / d->stride + 1;
  p.OW = (d->W + 2 * d->pad - d->KW) / d->stride + 1;
  p.CG = (d->C + 31) / 32;
  p.MT = (d->M + 31) / 32;
  p.P = p.N * p.OH * p.OW;
  p.ofm_kind = d->ofm_kind;
  p.ofm_vec = ((uintptr_t)ofm & 15u) == 0;
  p.spin_cap = g_spin_cap.load(std::memory_order_relaxed);
  {
    const hipError_t e = wait_fail_word(&p.wait_fail);
    if (e != hipSuccess) return hip_status(e);
  }
  int algo = 0;
  {
    const int st2 = resolve_algo(d, v, &algo);
    if (st2 != HOBFLOPS_OK) return st2;
  }
  const int kalgo = algo == HOBFLOPS_ALGO_SPLIT           ? kAlgoSplit
                    : algo == HOBFLOPS_ALGO_SPLIT_COMPACT ? kAlgoSplitCompact
                                                          : kAlgoFused;
  return hip_status(v->launch(ifm, w, ofm, p, kalgo, (hipStream_t)stream));
}

int hobflops_muladd_supported(hobflops_fmt in_fmt, hobflops_fmt acc_fmt, int round) {
  return fmt_ok(in_fmt) && fmt_ok(acc_fmt) && round_ok(round) &&
         find_muladd(in_fmt, acc_fmt, round) != nullptr;
}

int hobflops_muladd(const uint32_t* a, const uint32_t* b, const uint32_t* c, uint32_t* r,
                    int64_t n, hobflops_fmt in_fmt, hobflops_fmt acc_fmt, int round,
                    void* stream) {
  if (n < 0 || !fmt_ok(in_fmt) || !fmt_ok(acc_fmt) || !round_ok(round)) return HOBFLOPS_EINVAL;
  if (acc_fmt.wE != in_fmt.wE || acc_fmt.wF < in_fmt.wF) return HOBFLOPS_EINVAL;
  const MuladdVariant* v = find_muladd(in_fmt, acc_fmt, round);
  if (!v) return HOBFLOPS_EUNSUPPORTED;
  if (n == 0) return HOBFLOPS_OK;
  if (!a || !b || !c || !r) return HOBFLOPS_EINVAL;
  if (!aligned(a) || !aligned(b) || !aligned(c) || !aligned(r)) return HOBFLOPS_EALIGN;
  return hip_status(v->launch(a, b, c, r, (n + 31) / 32, (hipStream_t)stream));
}

int hobflops_avgpool_supported(hobflops_fmt in_fmt, hobflops_fmt acc_fmt, hobflops_fmt out_fmt,
                               int round) {
  return fmt_ok(in_fmt) && fmt_ok(acc_fmt) && fmt_ok(out_fmt) && round_ok(round) &&
         find_pool(in_fmt, acc_fmt, out_fmt, round) != nullptr;
}

int hobflops_avgpool(const uint32_t* in, uint32_t* out, int N, int H, int W, int C,
                     hobflops_fmt in_fmt, hobflops_fmt acc_fmt, hobflops_fmt out_fmt, int round,
                     void* stream) {
  if (N < 1 || H < 1 || W < 1 || C < 1 || (int64_t)H * W > INT32_MAX) return HOBFLOPS_EINVAL;
  if (!fmt_ok(in_fmt) || !fmt_ok(acc_fmt) || !fmt_ok(out_fmt) || !round_ok(round))
    return HOBFLOPS_EINVAL;
  if (acc_fmt.wE != in_fmt.wE || out_fmt.wE != in_fmt.wE || acc_fmt.wF < in_fmt.wF)
    return HOBFLOPS_EINVAL;
  const PoolVariant* v = find_pool(in_fmt, acc_fmt, out_fmt, round);
  if (!v) return HOBFLOPS_EUNSUPPORTED;
  if (!in || !out) return HOBFLOPS_EINVAL;
  if (!aligned(in) || !aligned(out)) return HOBFLOPS_EALIGN;
  PoolParams p;
  p.N = N;
  p.HW = H * W;
  p.CG = (C + 31) / 32;
  p.scale = recip_code((uint64_t)H * (uint64_t)W, acc_fmt);
  return hip_status(v->launch(in, out, p, (hipStream_t)stream));
}

int hobflops_avgpool_netlist_ops(hobflops_fmt in_fmt, hobflops_fmt acc_fmt, hobflops_fmt out_fmt,
                                 int round, int* accum_ops, int* scale_ops) {
  if (!round_ok(round)) return HOBFLOPS_EINVAL;
  const PoolVariant* v = find_pool(in_fmt, acc_fmt, out_fmt, round);
  if (!v) return HOBFLOPS_EUNSUPPORTED;
  if (accum_ops) *accum_ops = v->accum_ops;
  if (scale_ops) *scale_ops = v->scale_ops;
  return HOBFLOPS_OK;
}

int hobflops_netlist_ops(hobflops_fmt in_fmt, hobflops_fmt acc_fmt, int round,
                         int* conv_mac_ops, int* conv_mul_ops, int* conv_accum_ops,
                         int* muladd_ops) {
  int found = 0;
  if (!round_ok(round)) return HOBFLOPS_EINVAL;
  if (conv_mac_ops) *conv_mac_ops = 0;
  if (conv_mul_ops) *conv_mul_ops = 0;
  if (conv_accum_ops) *conv_accum_ops = 0;
  if (muladd_ops) *muladd_ops = 0;
  for (int i = 0; i < kNumConvVariants; ++i) {
    const ConvVariant& v = kConvVariants[i];
    if (v.wE == in_fmt.wE && v.wF_in == in_fmt.wF && v.wF_acc == acc_fmt.wF &&
        acc_fmt.wE == in_fmt.wE && v.round == round) {
      if (conv_mac_ops) *conv_mac_ops = v.mac_ops;
      if (conv_mul_ops) *conv_mul_ops = v.has_split ? v.mul_ops : 0;
      if (conv_accum_ops) *conv_accum_ops = v.has_split ? v.accum_ops : 0;
      found = 1;
      break;
    }
  }
  const MuladdVariant* m = find_muladd(in_fmt, acc_fmt, round);
  if (m) {
    if (muladd_ops) *muladd_ops = m->ops;
    found = 1;
  }
  return found ? HOBFLOPS_OK : HOBFLOPS_EUNSUPPORTED;
}

int hobflops_wait_failures(uint32_t* count, int reset) {
  if (!count) return HOBFLOPS_EINVAL;
  uint32_t* word = nullptr;
  hipError_t e = wait_fail_word(&word);
  if (e == hipSuccess) e = hipDeviceSynchronize();
  if (e == hipSuccess) e = hipMemcpy(count, word, sizeof(uint32_t), hipMemcpyDeviceToHost);
  if (e == hipSuccess && reset) {
    const uint32_t zero = 0;
    e = hipMemcpy(word, &zero, sizeof(uint32_t), hipMemcpyHostToDevice);
  }
  return hip_status(e);
}

int hobflops_set_wait_limit(uint32_t sleeps) {
  g_spin_cap.store(sleeps, std::memory_order_relaxed);
  return HOBFLOPS_OK;
}

uint32_t hobflops_get_wait_limit(void) { return g_spin_cap.load(std::memory_order_relaxed); }

const char* hobflops_status_string(int status) {
  switch (status) {
    case HOBFLOPS_OK: return "ok";
    case HOBFLOPS_EINVAL: return "invalid argument";
    case HOBFLOPS_EUNSUPPORTED: return "no generated kernel for this format combination";
    case HOBFLOPS_EALIGN: return "pointer not 4-byte aligned";
    case HOBFLOPS_EHIP: return g_errbuf[0] ? g_errbuf : "HIP error";
    default: return "unknown status";
  }
}

}  // extern "C"
