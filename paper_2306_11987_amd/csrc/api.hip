// C ABI of libhqlss: argument validation, workspace carving and the launch sequence of
// HQ-MM (forward) and LSS-MM (backward) on the caller's stream.  See include/hqlss.h.
#include <hip/hip_runtime.h>

#include <atomic>
#include <cmath>
#include <mutex>
#include <vector>

#include "../../include/hqlss.h"
#include "common.h"
#include "launch.h"

using namespace hqlss;

namespace {

constexpr int64_t kPad = 128;  // row padding of gathered operands (GEMM tile / K step)

int64_t rup(int64_t x, int64_t m) { return (x + m - 1) / m * m; }
size_t al(size_t x) { return (x + 255) & ~size_t(255); }

bool a16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15) == 0; }
bool a4(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 3) == 0; }

hqlss_status hip_status(hipError_t e) { return e == hipSuccess ? HQLSS_OK : HQLSS_ERR_HIP; }
#define HQ_TRY(expr)                              \
  do {                                            \
    hipError_t e_ = (expr);                       \
    if (e_ != hipSuccess) return HQLSS_ERR_HIP;   \
  } while (0)

// ---------------------------------------------------------------- shape checks
hqlss_status check_shape(int64_t N, int64_t D, int64_t C) {
  if (N < 1 || D < 64 || C < 64 || D % 64 || C % 64) return HQLSS_ERR_SHAPE;
  if (N > (int64_t(1) << 30) || D > (int64_t(1) << 24) || C > (int64_t(1) << 24)) return HQLSS_ERR_SHAPE;
  return HQLSS_OK;
}
hqlss_status check_block(int log2_block, int64_t D) {
  if (log2_block < 0 || log2_block > 7) return HQLSS_ERR_BLOCK;
  if (D % (int64_t(1) << log2_block)) return HQLSS_ERR_BLOCK;
  return HQLSS_OK;
}
hqlss_status check_dtype(int dt) {
  return (dt == HQLSS_F32 || dt == HQLSS_F16 || dt == HQLSS_BF16) ? HQLSS_OK : HQLSS_ERR_DTYPE;
}
const int64_t kI32 = int64_t(1) << 31;
// forward accumulators: 16 x 16 x 49 x D (both operands widened by 16)
hqlss_status check_fwd_overflow(int64_t D) {
  return 256 * 49 * D < kI32 ? HQLSS_OK : HQLSS_ERR_OVERFLOW;
}
// gradient accumulators: 16 x 126 x 7 x K raw, and b x 126 x 7 x K after the transform;
// K = C for dX, K = kept tokens <= N for dW.  Scores: 196 (49 C)(49 D) 2^16 < 2^64.
hqlss_status check_bwd_overflow(int64_t N, int64_t D, int64_t C, int log2_block) {
  const int64_t b = int64_t(1) << log2_block;
  const int64_t kmax = N > C ? N : C;
  const int64_t f = (b > 16 ? b : 16) * 126 * 7;
  if (f * kmax >= kI32) return HQLSS_ERR_OVERFLOW;
  const long double sc = 196.0L * 49.0L * (long double)C * 49.0L * (long double)D * 65536.0L;
  if (sc >= 18446744073709551615.0L) return HQLSS_ERR_OVERFLOW;
  if (N > 65536) return HQLSS_ERR_SHAPE;  // one-workgroup sampler keeps <= 64 tokens per thread
  return HQLSS_OK;
}

// need_amax: the dynamic mode's maxima (the learned-step-size mode has its steps instead)
hqlss_status check_saved(const hqlss_saved_t* s, bool need_amax = true) {
  if (!s || !s->xq || !s->wq || !s->wqT || !s->x_sumsq) return HQLSS_ERR_NULL;
  if (need_amax && !s->amax) return HQLSS_ERR_NULL;
  if (!a16(s->xq) || !a16(s->wq) || !a16(s->wqT) || !a16(s->x_sumsq) ||
      (need_amax && !a4(s->amax)))
    return HQLSS_ERR_ALIGN;
  return HQLSS_OK;
}
// want_dx / want_dw: which deltas the call reads (the forward writes both)
hqlss_status check_lsq(const hqlss_lsq_t* l, bool want_dx, bool want_dw) {
  if (!l || !l->step || (want_dx && !l->delta_x) || (want_dw && !l->delta_w)) return HQLSS_ERR_NULL;
  if (!a4(l->step) || (want_dx && !a16(l->delta_x)) || (want_dw && !a16(l->delta_w)))
    return HQLSS_ERR_ALIGN;
  return HQLSS_OK;
}
hqlss_status check_plan(const lss_plan_t* p) {
  if (!p || !p->qup || !p->qdn || !p->sumsq_up || !p->sumsq_dn || !p->w_up || !p->w_dn ||
      !p->kept || !p->n_kept || !p->amax_g)
    return HQLSS_ERR_NULL;
  if (!a16(p->qup) || !a16(p->qdn) || !a16(p->sumsq_up) || !a16(p->sumsq_dn) || !a16(p->w_up) ||
      !a16(p->w_dn) || !a16(p->kept) || !a4(p->n_kept) || !a4(p->amax_g))
    return HQLSS_ERR_ALIGN;
  return HQLSS_OK;
}

// ---------------------------------------------------------------- workspace layout
// forward head of the workspace: per-workgroup absmax partials of X and W
constexpr size_t kFwdHead = size_t(2) * kQMaxWg * sizeof(float);
size_t fwd_gemm_partial(int64_t N, int64_t D, int64_t C) {
  return al(gemm_partial_bytes(N, C, gemm_splits(N, C, D, true, true)));
}
size_t dx_gemm_partial(int64_t N, int64_t D, int64_t C) {
  return al(gemm_partial_bytes(N, D, gemm_splits(N, D, C, false, true)));
}
size_t dw_gemm_partial(int64_t N, int64_t D, int64_t C) {
  return al(gemm_partial_bytes(C, D, gemm_splits(C, D, (N + 127) / 128 * 128, false, true)));
}
// The forward product of hq_linear_fwd runs on the FP6 MFMA (the quantizer then also writes
// the codes as FP6 into the workspace) when the product is large enough for the faster
// matrix cores to repay the N D + C D bytes of those extra codes: above 2^38 multiply-adds
// (measured at N = 16384: 4096 x 4096 breaks even, 4096 x 11008 and 8192 x 8192 gain
// 54-65 us per launch).  A per-thread test hook forces either product.
thread_local int g_fwd_fp6_override = 0;  // 1: FP6, -1: int8, 0: by size
bool fwd_uses_fp6(int64_t N, int64_t D, int64_t C) {
  if (g_fwd_fp6_override) return g_fwd_fp6_override > 0;
  return (double)N * (double)D * (double)C > 274877906944.0;  // 2^38
}
size_t fwd6_partial(int64_t N, int64_t D, int64_t C);
// int8 product: the absmax partials and the split-K partials; FP6 product (fp6 = true): also
// the FP6 codes of X and W
size_t fwd_bytes(int64_t N, int64_t D, int64_t C, bool fp6) {
  return fp6 ? kFwdHead + al(N * D) + al(C * D) + fwd6_partial(N, D, C)
             : kFwdHead + fwd_gemm_partial(N, D, C);
}
size_t fwd_bytes(int64_t N, int64_t D, int64_t C) { return fwd_bytes(N, D, C, fwd_uses_fp6(N, D, C)); }
// FP6 route: the forward's INT4 codes (X^, W^, W^^T) staged before their conversion
size_t fwd6_partial(int64_t N, int64_t D, int64_t C) {
  return al(gemm_partial_bytes(N, C, gemm6_splits(N, C, D)));
}
size_t fwd6_bytes(int64_t N, int64_t D, int64_t C) {
  return kFwdHead + al(N * D / 2) + al(C * D / 2) + al(D * C / 2) + fwd6_partial(N, D, C);
}
// FP6 backward: K entries of dW (lower rows, plus each upper row in three weight classes,
// each class padded to 128) and their split-K factor; the fp32 sums stay exact while
// 882 N < 2^24 (every entry's weighted products of one output add to at most 126 x 7 per
// token), else each split holds at most 21376 entries (784 per entry)
int64_t ecap6(int64_t N) { return rup(4 * N + 640, 128); }
int dw6_splits(int64_t N, int64_t D, int64_t C) {
  int sp = gemm6_splits(C, D, ecap6(N));
  if (882 * N >= (int64_t(1) << 24)) {
    const int need = (int)((ecap6(N) + 21375) / 21376);
    if (sp < need) sp = need;
  }
  return sp;
}
size_t dx6_bytes(int64_t N, int64_t D, int64_t C) {
  return al(N * C) + al(rup(N, 256) * C) + al(gemm_partial_bytes(N, D, gemm6_splits(N, D, C)));
}
size_t dw6_bytes(int64_t N, int64_t D, int64_t C) {
  return al(C * ecap6(N)) + al(D * ecap6(N)) + al(gemm_partial_bytes(C, D, dw6_splits(N, D, C)));
}
size_t plan6_bytes(int64_t N) { return al(4 * N) + al(4 * ecap6(N)) + al(64); }
// absmax partials of dY, leverage scores [2][round_up(N, 8)], bit-split partials
int64_t score_pitch(int64_t N) { return rup(N, 8); }
size_t plan_scratch_bytes(int64_t N) {
  return al(sizeof(float) * kQMaxWg) + al(8 * score_pitch(N)) + al(sizeof(uint4) * kQMaxWg);
}
size_t plan_bytes(int64_t N, int64_t C) {
  return al(N * C / 2) * 2 + al(4 * N) * 2 + al(N) * 2 + al(4 * N) + al(4) * 2;
}
// block-size search: per-workgroup maxima (float) and error sums (double) of X and W
constexpr size_t kHsizeMaxBytes = size_t(kQMaxWg) * 8 * sizeof(float);
constexpr size_t kHsizeErrBytes = size_t(kQMaxWg) * 8 * sizeof(double);
size_t hsize_bytes() { return 2 * al(kHsizeMaxBytes) + 2 * al(kHsizeErrBytes); }
size_t dx_bytes(int64_t N, int64_t D, int64_t C) {
  return al(rup(N, kPad) * C) + dx_gemm_partial(N, D, C);
}
size_t dw_bytes(int64_t N, int64_t D, int64_t C) {
  return al(C * rup(N, kPad)) + al(D * rup(N, kPad) / 2) + dw_gemm_partial(N, D, C);
}
// dX and dW together: the two products share the int8 operand A_T
size_t grads_bytes(int64_t N, int64_t D, int64_t C, bool dx, bool dw) {
  if (dx && dw) return dx_bytes(N, D, C) + al(D * rup(N, kPad) / 2) + dw_gemm_partial(N, D, C);
  return (dx ? dx_bytes(N, D, C) : 0) + (dw ? dw_bytes(N, D, C) : 0);
}
// learned-step-size mode: per-workgroup sums of acc * delta of the dX and dW epilogues
int64_t lsq_parts_dx(int64_t N, int64_t D, int64_t C) {
  return gemm_epi_parts(N, D, gemm_splits(N, D, C, false, true));
}
int64_t lsq_parts_dw(int64_t N, int64_t D, int64_t C) {
  return gemm_epi_parts(C, D, gemm_splits(C, D, rup(N, kPad), false, true));
}
size_t lsq_parts_bytes(int64_t N, int64_t D, int64_t C, bool dx, bool dw) {
  return (dx ? al(8 * lsq_parts_dx(N, D, C)) : 0) + (dw ? al(8 * lsq_parts_dw(N, D, C)) : 0);
}

struct Carve {
  char* base;
  size_t off, cap;
  template <class T>
  T* take(size_t bytes) {
    off = al(off);
    T* p = reinterpret_cast<T*>(base + off);
    off += bytes;
    return p;
  }
  bool ok() const { return off <= cap; }
};

void plan_from_ws(Carve& w, int64_t N, int64_t C, lss_plan_t* p) {
  p->qup = w.take<uint8_t>(N * C / 2);
  p->qdn = w.take<uint8_t>(N * C / 2);
  p->sumsq_up = w.take<int32_t>(4 * N);
  p->sumsq_dn = w.take<int32_t>(4 * N);
  p->w_up = w.take<uint8_t>(N);
  p->w_dn = w.take<uint8_t>(N);
  p->kept = w.take<int32_t>(4 * N);
  p->n_kept = w.take<int32_t>(4);
  p->amax_g = w.take<float>(4);
}

// ---------------------------------------------------------------- static scratch
// Device memory of the allocation-free forward (hq_linear_fwd_noalloc): the absmax and
// split-K partials that hq_linear_fwd keeps in its caller's workspace.  Each GPU holds its
// own copy of the array, at its own address, until the process ends.  In host code the
// array's name is only a host-side stand-in: kernels get the device address that
// hipGetSymbolAddress returns for the current device.
static __device__ __align__(256) unsigned char scratch[HQLSS_STATIC_SCRATCH_BYTES];

constexpr int kMaxDevices = 64;
std::atomic<void*> g_scratch_ptr[kMaxDevices];  // device address of `scratch`, per device
std::mutex g_scratch_mu;

// The device address of `scratch` on the current device, looked up once per device (with
// that device current) and cached.
hqlss_status scratch_address(void** out) {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return HQLSS_ERR_HIP;
  void* p = g_scratch_ptr[dev].load(std::memory_order_acquire);
  if (!p) {
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    p = g_scratch_ptr[dev].load(std::memory_order_relaxed);
    if (!p) {
      if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) return HQLSS_ERR_HIP;
      g_scratch_ptr[dev].store(p, std::memory_order_release);
    }
  }
  *out = p;
  return HQLSS_OK;
}

// ---------------------------------------------------------------- timing log
struct TimingLog {
  bool on = false;
  std::vector<hipEvent_t> ev;  // pairs
  std::vector<int> ids;
  size_t used = 0;
  bool overflow = false;
};
// Per calling thread: a benchmark hook, so concurrent callers on other threads neither
// record into nor read another thread's log.
thread_local TimingLog g_log;
constexpr size_t kLogPairs = 4096;

// ---------------------------------------------------------------- the two passes
hqlss_status do_fwd(const void* X, const void* W, void* Y, int64_t N, int64_t D, int64_t C,
                    int dt, int k, const hqlss_saved_t* sv, void* ws, bool fp6, hipStream_t s) {
  uint32_t* amax = reinterpret_cast<uint32_t*>(sv->amax);
  float* px = static_cast<float*>(ws);  // [2][kQMaxWg] absmax partials
  float* pw = px + kQMaxWg;
  QJob jx = make_job(X, N, D), jw = make_job(W, C, D);
  HQ_TRY(launch_fwht_absmax(s, dt, k, jx, px, jw, pw));
  if (fp6 && Y) {  // the codes also as FP6 (workspace), the product on the FP6 MFMA
    Carve w{static_cast<char*>(ws), kFwdHead, fwd_bytes(N, D, C, true)};
    uint8_t* x6 = w.take<uint8_t>(N * D);
    uint8_t* w6 = w.take<uint8_t>(C * D);
    int32_t* part = w.take<int32_t>(fwd6_partial(N, D, C));
    const QOut ox{px, jx.wg, sv->amax, sv->xq, sv->x_sumsq, nullptr, x6};
    const QOut ow{pw, jw.wg, sv->amax + 1, sv->wq, nullptr, sv->wqT, w6};
    HQ_TRY(launch_fwht_quant(s, dt, k, jx, ox, jw, ow));
    GemmArgs g{};
    g.A = x6; g.lda = D;
    g.B = w6; g.ldb = D;
    g.M = N; g.N = C; g.K = D;
    g.out = Y; g.ldo = C;
    g.amax1 = amax; g.amax2 = amax + 1;
    g.denom = (float)(int64_t(1) << k);
    g.log2b = k;
    HQ_TRY(launch_gemm6(s, kEpiFwd, dt, g, gemm6_splits(N, C, D), part));
    return HQLSS_OK;
  }
  const QOut ox{px, jx.wg, sv->amax, sv->xq, sv->x_sumsq};
  const QOut ow{pw, jw.wg, sv->amax + 1, sv->wq, nullptr, sv->wqT};  // W^ and W^^T
  HQ_TRY(launch_fwht_quant(s, dt, k, jx, ox, jw, ow));
  if (Y) {
    GemmArgs g{};
    g.A = sv->xq; g.lda = D / 2;
    g.B = sv->wq; g.ldb = D / 2;
    g.M = N; g.N = C; g.K = D;
    g.out = Y; g.ldo = C;
    g.amax1 = amax; g.amax2 = amax + 1;
    g.denom = (float)(int64_t(1) << k);
    g.log2b = k;
    const int sp = gemm_splits(N, C, D, true, true);
    int32_t* part = reinterpret_cast<int32_t*>(static_cast<char*>(ws) + kFwdHead);
    HQ_TRY(launch_gemm(s, kEpiFwd, dt, true, true, g, sp, part));
  }
  return HQLSS_OK;
}

// FP6 route of the forward: the same maxima and INT4 codes as do_fwd (staged in the
// workspace), converted to the padded FP6 layout of the saved state, then the product on
// the FP6 MFMA.  Y equals do_fwd's bit for bit.
hqlss_status do_fwd_fp6(const void* X, const void* W, void* Y, int64_t N, int64_t D, int64_t C,
                        int dt, int k, const hqlss_saved_t* sv, void* ws, hipStream_t s) {
  uint32_t* amax = reinterpret_cast<uint32_t*>(sv->amax);
  float* px = static_cast<float*>(ws);  // [2][kQMaxWg] absmax partials
  float* pw = px + kQMaxWg;
  Carve w{static_cast<char*>(ws), kFwdHead, fwd6_bytes(N, D, C)};
  uint8_t* xq4 = w.take<uint8_t>(N * D / 2);
  uint8_t* wq4 = w.take<uint8_t>(C * D / 2);
  uint8_t* wqT4 = w.take<uint8_t>(D * C / 2);
  int32_t* part = w.take<int32_t>(fwd6_partial(N, D, C));
  QJob jx = make_job(X, N, D), jw = make_job(W, C, D);
  HQ_TRY(launch_fwht_absmax(s, dt, k, jx, px, jw, pw));
  const QOut ox{px, jx.wg, sv->amax, xq4, sv->x_sumsq, nullptr, sv->xq};
  const QOut ow{pw, jw.wg, sv->amax + 1, wq4, nullptr, wqT4, sv->wq};
  HQ_TRY(launch_fwht_quant(s, dt, k, jx, ox, jw, ow));
  HQ_TRY(launch_int4_to_fp6(s, wqT4, sv->wqT, D, C));
  if (Y) {
    GemmArgs g{};
    g.A = sv->xq; g.lda = D;
    g.B = sv->wq; g.ldb = D;
    g.M = N; g.N = C; g.K = D;
    g.out = Y; g.ldo = C;
    g.amax1 = amax; g.amax2 = amax + 1;
    g.denom = (float)(int64_t(1) << k);
    g.log2b = k;
    HQ_TRY(launch_gemm6(s, kEpiFwd, dt, g, gemm6_splits(N, C, D), part));
  }
  return HQLSS_OK;
}

hqlss_status do_fwd_lsq(const void* X, const void* W, void* Y, int64_t N, int64_t D, int64_t C,
                        int dt, int k, const hqlss_saved_t* sv, const hqlss_lsq_t* l, void* ws,
                        hipStream_t s) {
  QJob jx = make_job(X, N, D), jw = make_job(W, C, D);
  const LsqOut ox{l->step, sv->xq, sv->x_sumsq, l->delta_x};
  const LsqOut ow{l->step + 1, sv->wq, nullptr, l->delta_w, sv->wqT};  // W^ and W^^T
  HQ_TRY(launch_fwht_lsq(s, dt, k, jx, ox, jw, ow));
  GemmArgs g{};
  g.A = sv->xq; g.lda = D / 2;
  g.B = sv->wq; g.ldb = D / 2;
  g.M = N; g.N = C; g.K = D;
  g.out = Y; g.ldo = C;
  g.amax1 = reinterpret_cast<const uint32_t*>(l->step);
  g.amax2 = reinterpret_cast<const uint32_t*>(l->step + 1);
  g.steps_mask = 3;
  g.denom = (float)(int64_t(1) << k);
  g.log2b = k;
  const int sp = gemm_splits(N, C, D, true, true);
  HQ_TRY(launch_gemm(s, kEpiFwd, dt, true, true, g, sp, static_cast<int32_t*>(ws)));
  return HQLSS_OK;
}

// ---------------------------------------------------------------- attention BMM (App. A.1)
hqlss_status check_bmm(int64_t B, int64_t N, int64_t M, int64_t P, int dt, int k) {
  hqlss_status st;
  if ((st = check_shape(N, M, P))) return st;
  if (B < 1 || B > 65535 || B * N > (int64_t(1) << 30) || B * P > (int64_t(1) << 30))
    return HQLSS_ERR_SHAPE;
  if ((st = check_block(k, M))) return st;
  return check_dtype(dt);
}
hqlss_status check_bmm_lsq(const hqlss_bmm_lsq_t* l) {
  if (!l || !l->step_q || !l->step_k || !l->delta_q || !l->delta_k) return HQLSS_ERR_NULL;
  if (!a4(l->step_q) || !a4(l->step_k) || !a16(l->delta_q) || !a16(l->delta_k))
    return HQLSS_ERR_ALIGN;
  return HQLSS_OK;
}

hqlss_status do_bmm_fwd(const void* Q, const void* K, void* T, int64_t B, int64_t N, int64_t M,
                        int64_t P, int dt, int k, const hqlss_saved_t* sv,
                        const hqlss_bmm_lsq_t* l, hipStream_t s) {
  QJob jq = make_job_batched(Q, B, N, M), jk = make_job_batched(K, B, P, M);
  const LsqOut oq{l->step_q, sv->xq, sv->x_sumsq, l->delta_q};
  const LsqOut ok{l->step_k, sv->wq, nullptr, l->delta_k, sv->wqT};  // K^ and K^^T per batch
  HQ_TRY(launch_fwht_lsq(s, dt, k, jq, oq, jk, ok));
  GemmArgs g{};
  g.A = sv->xq; g.lda = M / 2;
  g.B = sv->wq; g.ldb = M / 2;
  g.M = N; g.N = P; g.K = M;
  g.out = T; g.ldo = P;
  g.amax1 = reinterpret_cast<const uint32_t*>(l->step_q);
  g.amax2 = reinterpret_cast<const uint32_t*>(l->step_k);
  g.steps_mask = 3;
  g.denom = (float)(int64_t(1) << k);
  g.log2b = k;
  g.batch = (int)B;
  g.bs_a = N * M / 2;
  g.bs_b = P * M / 2;
  g.bs_out = N * P;
  HQ_TRY(launch_gemm(s, kEpiFwd, dt, true, true, g, 1, nullptr));
  return HQLSS_OK;
}

// batched backward workspace: plan arrays, scratch, GEMM operands and step-gradient
// partials of all batches (every batch is in flight at once)
struct BmmWs {
  int64_t parts;  // absmax / bit-split partials of all batches (upper bound)
  int64_t kp;     // padded kept-token count per batch
  int64_t tiles_dx, tiles_dw;
};
BmmWs bmm_ws_dims(int64_t B, int64_t N, int64_t M, int64_t P) {
  return {B + kBatchWgSlack, rup(N, kPad), gemm_epi_parts(N, M, 1), gemm_epi_parts(P, M, 1)};
}
size_t bmm_bwd_bytes(int64_t B, int64_t N, int64_t M, int64_t P, bool dq, bool dk) {
  const BmmWs d = bmm_ws_dims(B, N, M, P);
  size_t t = 2 * al(B * N * P / 2) + 2 * al(4 * B * N) + 2 * al(B * N) + al(4 * B * N) +
             al(4 * B) * 2;
  t += al(4 * d.parts) + al(4 * B * 2 * score_pitch(N)) + al(16 * d.parts);
  if (dq || dk) t += al(B * d.kp * P);  // A_T, read by both gradient products
  if (dq) t += al(8 * B * d.tiles_dx);
  if (dk) t += al(B * M * d.kp / 2) + al(8 * B * d.tiles_dw);
  return t;
}

hqlss_status do_bmm_bwd(const void* dT, const hqlss_saved_t* sv, const hqlss_bmm_lsq_t* l,
                        void* dQ, void* dK, float* dstep_q, float* dstep_k, int64_t B, int64_t N,
                        int64_t M, int64_t P, int dt, int k, int64_t budget, uint64_t seed,
                        uint64_t offset, Carve& w, hipStream_t s) {
  const BmmWs d = bmm_ws_dims(B, N, M, P);
  const int64_t pitch = score_pitch(N);
  const uint64_t ostride = (uint64_t)((N * P + 7) / 8);  // counter blocks per batch (8 per block)
  uint8_t* qup = w.take<uint8_t>(B * N * P / 2);
  uint8_t* qdn = w.take<uint8_t>(B * N * P / 2);
  int32_t* su = w.take<int32_t>(4 * B * N);
  int32_t* sd = w.take<int32_t>(4 * B * N);
  uint8_t* wu = w.take<uint8_t>(B * N);
  uint8_t* wd = w.take<uint8_t>(B * N);
  int32_t* kept = w.take<int32_t>(4 * B * N);
  int32_t* nk = w.take<int32_t>(4 * B);
  float* ag = w.take<float>(4 * B);
  float* pg = w.take<float>(4 * d.parts);
  uint32_t* scores = w.take<uint32_t>(4 * B * 2 * pitch);
  uint4* bparts = w.take<uint4>(16 * d.parts);
  int8_t* Ag = w.take<int8_t>(B * d.kp * P);
  double* px = dQ ? w.take<double>(8 * B * d.tiles_dx) : nullptr;
  uint8_t* XtT = dK ? w.take<uint8_t>(B * M * d.kp / 2) : nullptr;
  double* pw = dK ? w.take<double>(8 * B * d.tiles_dw) : nullptr;
  if (!w.ok()) return HQLSS_ERR_WORKSPACE;

  // per-batch bit split and sample (App. A.1: every batch as a linear operator)
  QJob jg = make_job_batched(dT, B, N, P), none = make_job(nullptr, 0, P);
  HQ_TRY(launch_fwht_absmax(s, dt, 0, jg, pg, none, nullptr));
  const int nparts = jg.wg;
  const BsOut o{ag, qup, qdn, su, sd, sv->x_sumsq, scores, pitch, bparts, ostride};
  HQ_TRY(launch_bit_split(s, dt, jg, pg, nparts, o, seed, offset));
  HQ_TRY(launch_lss_plan(s, su, scores, pitch, bparts, jg.wg, N, budget, seed, offset, wu, wd,
                         kept, nk, B, ostride));
  HQ_TRY(launch_build_operands(s, dt, qup, qdn, wu, wd, kept, nk, sv->xq, N, P, M, Ag, XtT, dQ,
                               B));
  const uint32_t* agb = reinterpret_cast<const uint32_t*>(ag);
  const float denom = (float)(kBsRatio * (int64_t(1) << k));
  if (dQ) {  // grad Q_b = s_K[b] (I_Q o grad T_b K^_b) H^T on the kept rows
    GemmArgs g{};
    g.A = Ag; g.lda = P;
    g.B = sv->wqT; g.ldb = P / 2;
    g.M = N; g.m_dev = nk; g.N = M; g.K = P;
    g.out_rows = kept;
    g.amax1 = agb; g.amax2 = reinterpret_cast<const uint32_t*>(l->step_k);
    g.steps_mask = 2; g.denom = denom; g.log2b = k;
    g.out = dQ; g.ldo = M;
    g.delta = l->delta_q; g.ds_part = px;
    g.batch = (int)B;
    g.bs_a = d.kp * P; g.bs_b = M * P / 2; g.bs_out = N * M; g.bs_rows = N; g.bs_delta = N * M;
    HQ_TRY(launch_gemm(s, kEpiDxL, dt, false, true, g, 1, nullptr));
  }
  if (dK) {  // grad K_b = s_Q[b] (I_K o grad T_b^T Q^_b) H^T over the kept tokens
    GemmArgs g{};
    g.A = Ag; g.lda = P; g.a_kmajor = 1;
    g.B = XtT; g.ldb = d.kp / 2;
    g.M = P; g.N = M; g.K = d.kp; g.k_dev = nk;
    g.amax1 = agb; g.amax2 = reinterpret_cast<const uint32_t*>(l->step_q);
    g.steps_mask = 2; g.denom = denom; g.log2b = k;
    g.out = dK; g.ldo = M;
    g.delta = l->delta_k; g.ds_part = pw;
    g.batch = (int)B;
    g.bs_a = d.kp * P; g.bs_b = M * d.kp / 2; g.bs_out = P * M; g.bs_delta = P * M;
    HQ_TRY(launch_gemm(s, kEpiDwL, dt, false, true, g, 1, nullptr));
  }
  const bool sq = dQ && dstep_q, sk = dK && dstep_k;
  if (sq || sk) {  // g(s) = 1 / sqrt(Q_P numel) per batch (App. A.3)
    const double gq = 1.0 / std::sqrt(7.0 * (double)N * (double)M);
    const double gk = 1.0 / std::sqrt(7.0 * (double)P * (double)M);
    HQ_TRY(launch_lsq_step_grad(s, px, sq ? d.tiles_dx : 0, pw, sk ? d.tiles_dw : 0, ag,
                                l->step_q, l->step_k, k, gq, gk, sq ? dstep_q : nullptr,
                                sk ? dstep_k : nullptr, B));
  }
  return HQLSS_OK;
}

// do_plan's scratch: the absmax partials, then the scores (lss_grad_plan starts it at the
// workspace's first byte, so the scores sit at plan_scores_offset() there)
size_t plan_scores_offset() { return al(sizeof(float) * kQMaxWg); }

hqlss_status do_plan(const void* dY, const hqlss_saved_t* sv, const lss_plan_t* p, int64_t N,
                     int64_t C, int dt, int64_t budget, uint64_t seed, uint64_t offset,
                     Carve& w, hipStream_t s) {
  float* pg = w.take<float>(sizeof(float) * kQMaxWg);
  const int64_t pitch = score_pitch(N);
  uint32_t* scores = w.take<uint32_t>(8 * pitch);
  uint4* bparts = w.take<uint4>(sizeof(uint4) * kQMaxWg);
  QJob jg = make_job(dY, N, C), none = make_job(nullptr, 0, C);
  HQ_TRY(launch_fwht_absmax(s, dt, 0, jg, pg, none, nullptr));
  const int nparts = jg.wg;  // absmax partials of dY
  const BsOut o{p->amax_g, p->qup, p->qdn, p->sumsq_up, p->sumsq_dn, sv->x_sumsq, scores, pitch,
                bparts};
  HQ_TRY(launch_bit_split(s, dt, jg, pg, nparts, o, seed, offset));
  HQ_TRY(launch_lss_plan(s, p->sumsq_up, scores, pitch, bparts, jg.wg, N, budget, seed, offset,
                         p->w_up, p->w_dn, p->kept, p->n_kept));
  return HQLSS_OK;
}

// lsq (may be null): the learned-step-size mode: masked epilogues, and the step-size
// gradients into dstep (if not null).
hqlss_status do_grads(const lss_plan_t* p, const hqlss_saved_t* sv, void* dX, void* dW,
                      int32_t* acc, int which_acc, int64_t N, int64_t D, int64_t C, int dt,
                      int k, Carve& w, hipStream_t s, const hqlss_lsq_t* lsq = nullptr,
                      float* dstep = nullptr) {
  const uint32_t* amax = lsq ? reinterpret_cast<const uint32_t*>(lsq->step)
                             : reinterpret_cast<const uint32_t*>(sv->amax);
  const int smask = lsq ? 2 : 0;  // operand 2 (s_W or s_X) is a step in the LSQ mode
  const uint32_t* ag = reinterpret_cast<const uint32_t*>(p->amax_g);
  const float denom = (float)(kBsRatio * (int64_t(1) << k));
  const bool want_dx = dX || (acc && which_acc == 1);
  const bool want_dw = dW || (acc && which_acc == 2);
  const int64_t Kp = rup(N, kPad);
  // The dW product reads the dX operand A_T itself, k-major (its kept rows are the K of
  // dW), through transposing LDS reads.
  int8_t* Ag = nullptr;
  int32_t* part_dx = nullptr;
  const int sp_dx = gemm_splits(N, D, C, false, true);
  if (want_dx || want_dw) Ag = w.take<int8_t>(Kp * C);
  if (want_dx) part_dx = w.take<int32_t>(gemm_partial_bytes(N, D, sp_dx));
  uint8_t* XtT = nullptr;
  int32_t* part_dw = nullptr;
  const int sp_dw = gemm_splits(C, D, Kp, false, true);
  if (want_dw) {
    XtT = w.take<uint8_t>(D * Kp / 2);
    part_dw = w.take<int32_t>(gemm_partial_bytes(C, D, sp_dw));
  }
  double* px = (lsq && dX) ? w.take<double>(8 * lsq_parts_dx(N, D, C)) : nullptr;
  double* pw = (lsq && dW) ? w.take<double>(8 * lsq_parts_dw(N, D, C)) : nullptr;
  if (!w.ok()) return HQLSS_ERR_WORKSPACE;
  HQ_TRY(launch_build_operands(s, dt, p->qup, p->qdn, p->w_up, p->w_dn, p->kept, p->n_kept, sv->xq,
                               N, C, D, Ag, XtT, dX));
  if (want_dx) {
    GemmArgs g{};
    g.A = Ag; g.lda = C;
    g.B = sv->wqT; g.ldb = C / 2;
    g.M = N; g.m_dev = p->n_kept; g.N = D; g.K = C;
    g.out_rows = p->kept;
    g.amax1 = ag; g.amax2 = amax + 1; g.denom = denom; g.log2b = k;
    g.steps_mask = smask;
    if (dX) {
      g.out = dX; g.ldo = D;
      if (lsq) { g.delta = lsq->delta_x; g.ds_part = px; }
      HQ_TRY(launch_gemm(s, lsq ? kEpiDxL : kEpiDx, dt, false, true, g, sp_dx, part_dx));
    }
    if (acc && which_acc == 1) {
      g.out = acc; g.ldo = D;
      HQ_TRY(launch_gemm(s, kEpiAcc, dt, false, true, g, sp_dx, part_dx));
    }
  }
  if (want_dw) {
    GemmArgs g{};
    g.A = Ag; g.lda = C; g.a_kmajor = 1;
    g.B = XtT; g.ldb = Kp / 2;
    g.M = C; g.N = D; g.K = Kp; g.k_dev = p->n_kept;
    g.amax1 = ag; g.amax2 = amax; g.denom = denom; g.log2b = k;
    g.steps_mask = smask;
    if (dW) {
      g.out = dW; g.ldo = D;
      if (lsq) { g.delta = lsq->delta_w; g.ds_part = pw; }
      HQ_TRY(launch_gemm(s, lsq ? kEpiDwL : kEpiDw, dt, false, true, g, sp_dw, part_dw));
    }
    if (acc && which_acc == 2) {
      g.out = acc; g.ldo = D;
      HQ_TRY(launch_gemm(s, kEpiAcc, dt, false, true, g, sp_dw, part_dw));
    }
  }
  if (lsq && dstep) {
    // g(s) = 1 / sqrt(Q_P numel) with Q_P = 7 (App. A.3)
    const double gx = 1.0 / std::sqrt(7.0 * (double)N * (double)D);
    const double gw = 1.0 / std::sqrt(7.0 * (double)C * (double)D);
    HQ_TRY(launch_lsq_step_grad(s, px, px ? lsq_parts_dx(N, D, C) : 0, pw,
                                pw ? lsq_parts_dw(N, D, C) : 0, p->amax_g, lsq->step,
                                lsq->step + 1, k, gx, gw, dstep, dstep + 1));
  }
  return HQLSS_OK;
}

// FP6 route of the backward GEMMs: the same plan, operands in the padded FP6 layout ordered
// for the route's exact weights (fp6_plan), products on the FP6 MFMA.  Every accumulator and
// output equals do_grads' bit for bit.
hqlss_status do_grads_fp6(const lss_plan_t* p, const hqlss_saved_t* sv, void* dX, void* dW,
                          int32_t* acc, int which_acc, int64_t N, int64_t D, int64_t C, int dt,
                          int k, Carve& w, hipStream_t s) {
  const uint32_t* amax = reinterpret_cast<const uint32_t*>(sv->amax);
  const uint32_t* ag = reinterpret_cast<const uint32_t*>(p->amax_g);
  const float denom = (float)(kBsRatio * (int64_t(1) << k));
  const bool want_dx = dX || (acc && which_acc == 1);
  const bool want_dw = dW || (acc && which_acc == 2);
  const int64_t ecap = ecap6(N);
  int32_t* order6 = w.take<int32_t>(4 * N);
  int32_t* ent = w.take<int32_t>(4 * ecap);
  int32_t* cnt = w.take<int32_t>(64);  // [0] n_up, [8..12] class bounds
  uint8_t *a_dn = nullptr, *a_up = nullptr, *a_dw = nullptr, *x_dw = nullptr;
  int32_t *part_dx = nullptr, *part_dw = nullptr;
  const int sp_dx = gemm6_splits(N, D, C), sp_dw = dw6_splits(N, D, C);
  if (want_dx) {
    a_dn = w.take<uint8_t>(N * C);
    a_up = w.take<uint8_t>(rup(N, 256) * C);
    part_dx = w.take<int32_t>(gemm_partial_bytes(N, D, sp_dx));
  }
  if (want_dw) {
    a_dw = w.take<uint8_t>(C * ecap);
    x_dw = w.take<uint8_t>(D * ecap);
    part_dw = w.take<int32_t>(gemm_partial_bytes(C, D, sp_dw));
  }
  if (!w.ok()) return HQLSS_ERR_WORKSPACE;
  HQ_TRY(launch_fp6_plan(s, p->w_up, p->w_dn, N, order6, cnt, ent, cnt + 8));
  HQ_TRY(launch_fp6_build(s, dt, p->qup, p->qdn, p->w_up, p->w_dn, order6, p->n_kept, cnt, ent,
                          cnt + 8, sv->xq, N, C, D, ecap, a_dn, a_up, a_dw, x_dw, dX));
  if (want_dx) {
    GemmArgs g{};
    g.A = a_dn; g.lda = C;
    g.B = sv->wqT; g.ldb = C;
    g.M = N; g.m_dev = p->n_kept; g.N = D; g.K = C;
    g.out_rows = order6;
    g.amax1 = ag; g.amax2 = amax + 1; g.denom = denom; g.log2b = k;
    g.f6_kind = 1; g.A2 = a_up; g.m2_dev = cnt; g.w_up = p->w_up; g.w_dn = p->w_dn;
    if (dX) {
      g.out = dX; g.ldo = D;
      HQ_TRY(launch_gemm6(s, kEpiDx, dt, g, sp_dx, part_dx));
    }
    if (acc && which_acc == 1) {
      g.out = acc; g.ldo = D;
      HQ_TRY(launch_gemm6(s, kEpiAcc, dt, g, sp_dx, part_dx));
    }
  }
  if (want_dw) {
    GemmArgs g{};
    g.A = a_dw; g.lda = ecap;
    g.B = x_dw; g.ldb = ecap;
    g.M = C; g.N = D; g.K = ecap; g.k_dev = cnt + 12;
    g.amax1 = ag; g.amax2 = amax; g.denom = denom; g.log2b = k;
    g.f6_kind = 2; g.kcls = cnt + 8;
    if (dW) {
      g.out = dW; g.ldo = D;
      HQ_TRY(launch_gemm6(s, kEpiDw, dt, g, sp_dw, part_dw));
    }
    if (acc && which_acc == 2) {
      g.out = acc; g.ldo = D;
      HQ_TRY(launch_gemm6(s, kEpiAcc, dt, g, sp_dw, part_dw));
    }
  }
  return HQLSS_OK;
}

// the FP6 backward's extra shape limit: the dX sums of 14 / w_dn times the upper pass plus
// the lower pass are half-integers below 735 C, exact in fp32 for C <= 11412
hqlss_status check_bwd6_overflow(int64_t C) {
  return 2 * 735 * C < (int64_t(1) << 24) ? HQLSS_OK : HQLSS_ERR_OVERFLOW;
}

hqlss_status check_bwd_common(const void* dY, const hqlss_saved_t* saved, int64_t N, int64_t D,
                              int64_t C, int dt, int log2_block, int64_t budget,
                              bool need_amax = true) {
  if (!dY) return HQLSS_ERR_NULL;
  hqlss_status st;
  if ((st = check_shape(N, D, C))) return st;
  if ((st = check_block(log2_block, D))) return st;
  if ((st = check_dtype(dt))) return st;
  if ((st = check_saved(saved, need_amax))) return st;
  if (!a16(dY)) return HQLSS_ERR_ALIGN;
  if ((st = check_bwd_overflow(N, D, C, log2_block))) return st;
  if (budget > 2 * N || budget < HQLSS_BUDGET_KEEP_NONZERO) return HQLSS_ERR_ARG;
  return HQLSS_OK;
}

// 0 -> N (Sec. 4.2), HQLSS_BUDGET_KEEP_NONZERO -> 2N (every non-zero row kept), else itself.
int64_t resolve_budget(int64_t budget_rows, int64_t N) {
  if (budget_rows == 0) return N;
  if (budget_rows == HQLSS_BUDGET_KEEP_NONZERO) return 2 * N;
  return budget_rows;
}

}  // namespace

namespace hqlss {

const char* kernel_name(int id) {
  static const char* names[kKCount] = {"fwht_absmax", "fwht_quant", "bit_split", "lss_plan", "build_operands",
                                       "gemm_fwd", "gemm_dx", "gemm_dw", "gemm_acc",
                                       "gemm_reduce", "copy", "hsize_max", "hsize_err",
                                       "hsize_pick", "lsq_quant", "lsq_step_grad", "fp6_convert",
                                       "fp6_plan", "fp6_build"};
  return (id >= 0 && id < kKCount) ? names[id] : "?";
}

void timing_begin(hipStream_t s) {
  if (!g_log.on) return;
  if (g_log.used >= kLogPairs) { g_log.overflow = true; return; }
  (void)hipEventRecord(g_log.ev[2 * g_log.used], s);
}
void timing_end(hipStream_t s, int id) {
  if (!g_log.on || g_log.used >= kLogPairs) return;
  (void)hipEventRecord(g_log.ev[2 * g_log.used + 1], s);
  g_log.ids[g_log.used] = id;
  ++g_log.used;
}

}  // namespace hqlss

extern "C" {

size_t hqlss_workspace_bytes(int which, int64_t N, int64_t D, int64_t C) {
  if (N < 1 || D < 1 || C < 1) return 0;
  switch (which) {
    case HQLSS_WS_FWD: return fwd_bytes(N, D, C);
    case HQLSS_WS_BWD_DX: return plan_bytes(N, C) + plan_scratch_bytes(N) + dx_bytes(N, D, C);
    case HQLSS_WS_BWD_DW: return plan_bytes(N, C) + plan_scratch_bytes(N) + dw_bytes(N, D, C);
    case HQLSS_WS_BWD: return plan_bytes(N, C) + plan_scratch_bytes(N) + grads_bytes(N, D, C, true, true);
    case HQLSS_WS_FROM_PLAN: return grads_bytes(N, D, C, true, true);
    case HQLSS_WS_PLAN: return plan_scratch_bytes(N);
    case HQLSS_WS_HSIZE: return hsize_bytes();
    case HQLSS_WS_FWD_LSQ: return fwd_gemm_partial(N, D, C);
    case HQLSS_WS_FWD_FP6: return fwd6_bytes(N, D, C);
    case HQLSS_WS_BWD_FP6:
      return plan_bytes(N, C) + plan_scratch_bytes(N) + plan6_bytes(N) + dx6_bytes(N, D, C) +
             dw6_bytes(N, D, C);
    case HQLSS_WS_FROM_PLAN_FP6: return plan6_bytes(N) + dx6_bytes(N, D, C) + dw6_bytes(N, D, C);
    case HQLSS_WS_BWD_LSQ:
      return plan_bytes(N, C) + plan_scratch_bytes(N) + grads_bytes(N, D, C, true, true) +
             lsq_parts_bytes(N, D, C, true, true);
  }
  return 0;
}

size_t hqlss_bmm_workspace_bytes(int which, int64_t B, int64_t N, int64_t M, int64_t P) {
  if (B < 1 || N < 1 || M < 1 || P < 1) return 0;
  switch (which) {
    case HQLSS_WS_BMM_FWD: return 0;
    case HQLSS_WS_BMM_BWD: return bmm_bwd_bytes(B, N, M, P, true, true);
  }
  return 0;
}

hqlss_status lss_bmm_bwd_lsq(const void* dT, const hqlss_saved_t* saved,
                             const hqlss_bmm_lsq_t* lsq, void* dQ, void* dK, float* dstep_q,
                             float* dstep_k, int64_t B, int64_t N, int64_t M, int64_t P,
                             hqlss_dtype dt, int log2_block, int64_t budget_rows, uint64_t seed,
                             uint64_t offset, void* ws, size_t ws_bytes, void* stream) {
  if (!dT) return HQLSS_ERR_NULL;
  if (!dQ && !dK) return HQLSS_ERR_NULL;
  hqlss_status st;
  if ((st = check_bmm(B, N, M, P, dt, log2_block))) return st;
  if ((st = check_saved(saved, false))) return st;
  if ((st = check_bmm_lsq(lsq))) return st;
  if (!a16(dT) || (dQ && !a16(dQ)) || (dK && !a16(dK)) || (ws && !a16(ws)) ||
      (dstep_q && !a4(dstep_q)) || (dstep_k && !a4(dstep_k)))
    return HQLSS_ERR_ALIGN;
  if ((st = check_bwd_overflow(N, M, P, log2_block))) return st;
  if (budget_rows > 2 * N || budget_rows < HQLSS_BUDGET_KEEP_NONZERO) return HQLSS_ERR_ARG;
  if (!ws || ws_bytes < bmm_bwd_bytes(B, N, M, P, dQ != nullptr, dK != nullptr))
    return HQLSS_ERR_WORKSPACE;
  Carve w{static_cast<char*>(ws), 0, ws_bytes};
  return do_bmm_bwd(dT, saved, lsq, dQ, dK, dstep_q, dstep_k, B, N, M, P, dt, log2_block,
                    resolve_budget(budget_rows, N), seed, offset, w,
                    static_cast<hipStream_t>(stream));
}

hqlss_status hq_bmm_fwd_lsq(const void* Q, const void* K, void* T, int64_t B, int64_t N,
                            int64_t M, int64_t P, hqlss_dtype dt, int log2_block,
                            const hqlss_saved_t* saved, const hqlss_bmm_lsq_t* lsq, void* ws,
                            size_t ws_bytes, void* stream) {
  (void)ws;
  (void)ws_bytes;
  if (!Q || !K || !T) return HQLSS_ERR_NULL;
  hqlss_status st;
  if ((st = check_bmm(B, N, M, P, dt, log2_block))) return st;
  if ((st = check_saved(saved, false))) return st;
  if ((st = check_bmm_lsq(lsq))) return st;
  if (!a16(Q) || !a16(K) || !a16(T)) return HQLSS_ERR_ALIGN;
  if ((st = check_fwd_overflow(M))) return st;
  return do_bmm_fwd(Q, K, T, B, N, M, P, dt, log2_block, saved, lsq,
                    static_cast<hipStream_t>(stream));
}

uint64_t lss_philox_offset_advance(int64_t N, int64_t C) {
  if (N < 1 || C < 1) return 0;
  return (uint64_t)((N * C + 7) / 8);
}

const char* hqlss_status_string(hqlss_status s) {
  switch (s) {
    case HQLSS_OK: return "ok";
    case HQLSS_ERR_NULL: return "a required pointer is NULL";
    case HQLSS_ERR_SHAPE: return "invalid shape (N >= 1; D, C positive multiples of 64)";
    case HQLSS_ERR_BLOCK: return "invalid Hadamard block (0 <= log2_block <= 7, D % 2^k == 0)";
    case HQLSS_ERR_ALIGN: return "pointer not aligned (16 bytes for arrays, 4 for scalars)";
    case HQLSS_ERR_DTYPE: return "unknown dtype";
    case HQLSS_ERR_WORKSPACE: return "workspace too small";
    case HQLSS_ERR_OVERFLOW: return "shape would overflow an int32 accumulator or int64 score";
    case HQLSS_ERR_HIP: return "HIP launch or runtime error";
    case HQLSS_ERR_ARG: return "invalid argument";
    case HQLSS_ERR_SCRATCH:
      return "shape needs more scratch than the static array (HQLSS_STATIC_SCRATCH_BYTES) holds";
  }
  return "unknown status";
}

hqlss_status hq_linear_fwd(const void* X, const void* W, void* Y, int64_t N, int64_t D, int64_t C,
                           hqlss_dtype dt, int log2_block, const hqlss_saved_t* saved, void* ws,
                           size_t ws_bytes, void* stream) {
  if (!X || !W || !Y) return HQLSS_ERR_NULL;
  hqlss_status st;
  if ((st = check_shape(N, D, C))) return st;
  if ((st = check_block(log2_block, D))) return st;
  if ((st = check_dtype(dt))) return st;
  if ((st = check_saved(saved))) return st;
  if (!a16(X) || !a16(W) || !a16(Y)) return HQLSS_ERR_ALIGN;
  if ((st = check_fwd_overflow(D))) return st;
  const bool fp6 = fwd_uses_fp6(N, D, C);
  if (!ws || ws_bytes < fwd_bytes(N, D, C, fp6)) return HQLSS_ERR_WORKSPACE;
  if (!a16(ws)) return HQLSS_ERR_ALIGN;
  return do_fwd(X, W, Y, N, D, C, dt, log2_block, saved, ws, fp6, static_cast<hipStream_t>(stream));
}

hqlss_status hq_linear_fwd_noalloc(const void* X, const void* W, void* Y, int64_t N, int64_t D,
                                   int64_t C, hqlss_dtype dt, int log2_block,
                                   const hqlss_saved_t* saved, void* stream) {
  if (!X || !W || !Y) return HQLSS_ERR_NULL;
  hqlss_status st;
  if ((st = check_shape(N, D, C))) return st;
  if ((st = check_block(log2_block, D))) return st;
  if ((st = check_dtype(dt))) return st;
  if ((st = check_saved(saved))) return st;
  if (!a16(X) || !a16(W) || !a16(Y)) return HQLSS_ERR_ALIGN;
  if ((st = check_fwd_overflow(D))) return st;
  if (fwd_bytes(N, D, C, false) > HQLSS_STATIC_SCRATCH_BYTES) return HQLSS_ERR_SCRATCH;
  void* ws = nullptr;
  if ((st = scratch_address(&ws))) return st;
  return do_fwd(X, W, Y, N, D, C, dt, log2_block, saved, ws, false, static_cast<hipStream_t>(stream));
}

hqlss_status hq_linear_fwd_fp6(const void* X, const void* W, void* Y, int64_t N, int64_t D, int64_t C,
                               hqlss_dtype dt, int log2_block, const hqlss_saved_t* saved, void* ws,
                               size_t ws_bytes, void* stream) {
  if (!X || !W || !Y) return HQLSS_ERR_NULL;
  hqlss_status st;
  if ((st = check_shape(N, D, C))) return st;
  if ((st = check_block(log2_block, D))) return st;
  if ((st = check_dtype(dt))) return st;
  if ((st = check_saved(saved))) return st;
  if (!a16(X) || !a16(W) || !a16(Y)) return HQLSS_ERR_ALIGN;
  if ((st = check_fwd_overflow(D))) return st;
  if (!ws || ws_bytes < fwd6_bytes(N, D, C)) return HQLSS_ERR_WORKSPACE;
  if (!a16(ws)) return HQLSS_ERR_ALIGN;
  return do_fwd_fp6(X, W, Y, N, D, C, dt, log2_block, saved, ws, static_cast<hipStream_t>(stream));
}

hqlss_status hq_linear_fwd_lsq(const void* X, const void* W, void* Y, int64_t N, int64_t D,
                               int64_t C, hqlss_dtype dt, int log2_block,
                               const hqlss_saved_t* saved, const hqlss_lsq_t* lsq, void* ws,
                               size_t ws_bytes, void* stream) {
  if (!X || !W || !Y) return HQLSS_ERR_NULL;
  hqlss_status st;
  if ((st = check_shape(N, D, C))) return st;
  if ((st = check_block(log2_block, D))) return st;
  if ((st = check_dtype(dt))) return st;
  if ((st = check_saved(saved, false))) return st;
  if ((st = check_lsq(lsq, true, true))) return st;
  if (!a16(X) || !a16(W) || !a16(Y)) return HQLSS_ERR_ALIGN;
  if ((st = check_fwd_overflow(D))) return st;
  const size_t need = fwd_gemm_partial(N, D, C);
  if (need && (!ws || ws_bytes < need)) return HQLSS_ERR_WORKSPACE;
  if (ws && !a16(ws)) return HQLSS_ERR_ALIGN;
  return do_fwd_lsq(X, W, Y, N, D, C, dt, log2_block, saved, lsq, ws,
                    static_cast<hipStream_t>(stream));
}

hqlss_status hq_choose_hadamard_size(const void* X, const void* W, int64_t N, int64_t D,
                                     int64_t C, hqlss_dtype dt, int max_log2_block,
                                     int32_t* log2_block_out, double* mse_out, void* ws,
                                     size_t ws_bytes, void* stream) {
  if (!X || !W || !log2_block_out || !mse_out) return HQLSS_ERR_NULL;
  hqlss_status st;
  if ((st = check_shape(N, D, C))) return st;
  if (max_log2_block < 0 || max_log2_block > 7) return HQLSS_ERR_BLOCK;
  if ((st = check_dtype(dt))) return st;
  if (!a16(X) || !a16(W) || !a4(log2_block_out) ||
      (reinterpret_cast<uintptr_t>(mse_out) & 7) != 0)
    return HQLSS_ERR_ALIGN;
  if (!ws || ws_bytes < hsize_bytes()) return HQLSS_ERR_WORKSPACE;
  if (!a16(ws)) return HQLSS_ERR_ALIGN;
  Carve w{static_cast<char*>(ws), 0, ws_bytes};
  float* mx0 = w.take<float>(kHsizeMaxBytes);
  float* mx1 = w.take<float>(kHsizeMaxBytes);
  double* e0 = w.take<double>(kHsizeErrBytes);
  double* e1 = w.take<double>(kHsizeErrBytes);
  QJob jx = make_job(X, N, D), jw = make_job(W, C, D);
  HQ_TRY(launch_hsize_search(static_cast<hipStream_t>(stream), dt, jx, jw, mx0, mx1, e0, e1,
                             max_log2_block, log2_block_out, mse_out));
  return HQLSS_OK;
}

hqlss_status lss_grad_plan(const void* dY, const hqlss_saved_t* saved, const lss_plan_t* plan,
                           int64_t N, int64_t D, int64_t C, hqlss_dtype dt, int64_t budget_rows,
                           uint64_t seed, uint64_t offset, void* ws, size_t ws_bytes,
                           void* stream) {
  hqlss_status st;
  if ((st = check_bwd_common(dY, saved, N, D, C, dt, 0, budget_rows))) return st;
  if ((st = check_plan(plan))) return st;
  if (!ws || ws_bytes < plan_scratch_bytes(N)) return HQLSS_ERR_WORKSPACE;
  if (!a16(ws)) return HQLSS_ERR_ALIGN;
  const int64_t B = resolve_budget(budget_rows, N);
  Carve w{static_cast<char*>(ws), 0, ws_bytes};
  return do_plan(dY, saved, plan, N, C, dt, B, seed, offset, w, static_cast<hipStream_t>(stream));
}

hqlss_status lss_linear_bwd_from_plan(const lss_plan_t* plan, const hqlss_saved_t* saved,
                                      void* dX, void* dW, int64_t N, int64_t D, int64_t C,
                                      hqlss_dtype dt, int log2_block, void* ws, size_t ws_bytes,
                                      void* stream) {
  if (!dX && !dW) return HQLSS_ERR_NULL;
  hqlss_status st;
  if ((st = check_shape(N, D, C))) return st;
  if ((st = check_block(log2_block, D))) return st;
  if ((st = check_dtype(dt))) return st;
  if ((st = check_saved(saved))) return st;
  if ((st = check_plan(plan))) return st;
  if ((dX && !a16(dX)) || (dW && !a16(dW)) || (ws && !a16(ws))) return HQLSS_ERR_ALIGN;
  if ((st = check_bwd_overflow(N, D, C, log2_block))) return st;
  const size_t need = grads_bytes(N, D, C, dX != nullptr, dW != nullptr);
  if (!ws || ws_bytes < need) return HQLSS_ERR_WORKSPACE;
  Carve w{static_cast<char*>(ws), 0, ws_bytes};
  return do_grads(plan, saved, dX, dW, nullptr, 0, N, D, C, dt, log2_block, w,
                  static_cast<hipStream_t>(stream));
}

static hqlss_status bwd_impl(const void* dY, const hqlss_saved_t* saved, void* dX, void* dW,
                             int64_t N, int64_t D, int64_t C, hqlss_dtype dt, int log2_block,
                             int64_t budget_rows, uint64_t seed, uint64_t offset, void* ws,
                             size_t ws_bytes, void* stream) {
  if (!dX && !dW) return HQLSS_ERR_NULL;
  hqlss_status st;
  if ((st = check_bwd_common(dY, saved, N, D, C, dt, log2_block, budget_rows))) return st;
  if ((dX && !a16(dX)) || (dW && !a16(dW)) || (ws && !a16(ws))) return HQLSS_ERR_ALIGN;
  const size_t need = plan_bytes(N, C) + plan_scratch_bytes(N) + grads_bytes(N, D, C, dX != nullptr, dW != nullptr);
  if (!ws || ws_bytes < need) return HQLSS_ERR_WORKSPACE;
  hipStream_t s = static_cast<hipStream_t>(stream);
  Carve w{static_cast<char*>(ws), 0, ws_bytes};
  lss_plan_t p;
  plan_from_ws(w, N, C, &p);
  const int64_t B = resolve_budget(budget_rows, N);
  if ((st = do_plan(dY, saved, &p, N, C, dt, B, seed, offset, w, s))) return st;
  return do_grads(&p, saved, dX, dW, nullptr, 0, N, D, C, dt, log2_block, w, s);
}

hqlss_status lss_linear_bwd(const void* dY, const hqlss_saved_t* saved, void* dX, void* dW,
                            int64_t N, int64_t D, int64_t C, hqlss_dtype dt, int log2_block,
                            int64_t budget_rows, uint64_t seed, uint64_t offset, void* ws,
                            size_t ws_bytes, void* stream) {
  return bwd_impl(dY, saved, dX, dW, N, D, C, dt, log2_block, budget_rows, seed, offset, ws,
                  ws_bytes, stream);
}

hqlss_status lss_linear_bwd_fp6(const void* dY, const hqlss_saved_t* saved, void* dX, void* dW,
                                int64_t N, int64_t D, int64_t C, hqlss_dtype dt, int log2_block,
                                int64_t budget_rows, uint64_t seed, uint64_t offset, void* ws,
                                size_t ws_bytes, void* stream) {
  if (!dX && !dW) return HQLSS_ERR_NULL;
  hqlss_status st;
  if ((st = check_bwd_common(dY, saved, N, D, C, dt, log2_block, budget_rows))) return st;
  if ((st = check_bwd6_overflow(C))) return st;
  if ((dX && !a16(dX)) || (dW && !a16(dW)) || (ws && !a16(ws))) return HQLSS_ERR_ALIGN;
  const size_t need = plan_bytes(N, C) + plan_scratch_bytes(N) + plan6_bytes(N) +
                      (dX ? dx6_bytes(N, D, C) : 0) + (dW ? dw6_bytes(N, D, C) : 0);
  if (!ws || ws_bytes < need) return HQLSS_ERR_WORKSPACE;
  hipStream_t s = static_cast<hipStream_t>(stream);
  Carve w{static_cast<char*>(ws), 0, ws_bytes};
  lss_plan_t p;
  plan_from_ws(w, N, C, &p);
  const int64_t B = resolve_budget(budget_rows, N);
  if ((st = do_plan(dY, saved, &p, N, C, dt, B, seed, offset, w, s))) return st;
  return do_grads_fp6(&p, saved, dX, dW, nullptr, 0, N, D, C, dt, log2_block, w, s);
}

hqlss_status lss_linear_bwd_dx(const void* dY, const hqlss_saved_t* saved, void* dX, int64_t N,
                               int64_t D, int64_t C, hqlss_dtype dt, int log2_block,
                               int64_t budget_rows, uint64_t seed, uint64_t offset, void* ws,
                               size_t ws_bytes, void* stream) {
  if (!dX) return HQLSS_ERR_NULL;
  return bwd_impl(dY, saved, dX, nullptr, N, D, C, dt, log2_block, budget_rows, seed, offset, ws,
                  ws_bytes, stream);
}

hqlss_status lss_linear_bwd_dw(const void* dY, const hqlss_saved_t* saved, void* dW, int64_t N,
                               int64_t D, int64_t C, hqlss_dtype dt, int log2_block,
                               int64_t budget_rows, uint64_t seed, uint64_t offset, void* ws,
                               size_t ws_bytes, void* stream) {
  if (!dW) return HQLSS_ERR_NULL;
  return bwd_impl(dY, saved, nullptr, dW, N, D, C, dt, log2_block, budget_rows, seed, offset, ws,
                  ws_bytes, stream);
}

hqlss_status lss_linear_bwd_lsq(const void* dY, const hqlss_saved_t* saved,
                                const hqlss_lsq_t* lsq, void* dX, void* dW, float* dstep,
                                int64_t N, int64_t D, int64_t C, hqlss_dtype dt, int log2_block,
                                int64_t budget_rows, uint64_t seed, uint64_t offset, void* ws,
                                size_t ws_bytes, void* stream) {
  if (!dX && !dW) return HQLSS_ERR_NULL;
  hqlss_status st;
  if ((st = check_bwd_common(dY, saved, N, D, C, dt, log2_block, budget_rows, false))) return st;
  if ((st = check_lsq(lsq, dX != nullptr, dW != nullptr))) return st;
  if ((dX && !a16(dX)) || (dW && !a16(dW)) || (ws && !a16(ws)) || (dstep && !a4(dstep)))
    return HQLSS_ERR_ALIGN;
  const size_t need = plan_bytes(N, C) + plan_scratch_bytes(N) + grads_bytes(N, D, C, dX != nullptr, dW != nullptr) +
                      lsq_parts_bytes(N, D, C, dX, dW);
  if (!ws || ws_bytes < need) return HQLSS_ERR_WORKSPACE;
  hipStream_t s = static_cast<hipStream_t>(stream);
  Carve w{static_cast<char*>(ws), 0, ws_bytes};
  lss_plan_t p;
  plan_from_ws(w, N, C, &p);
  const int64_t B = resolve_budget(budget_rows, N);
  if ((st = do_plan(dY, saved, &p, N, C, dt, B, seed, offset, w, s))) return st;
  return do_grads(&p, saved, dX, dW, nullptr, 0, N, D, C, dt, log2_block, w, s, lsq, dstep);
}

hqlss_status hqlss_debug_gemm_acc(int which, const lss_plan_t* plan, const hqlss_saved_t* saved,
                                  int32_t* acc, int64_t N, int64_t D, int64_t C, void* ws,
                                  size_t ws_bytes, void* stream) {
  if (!acc) return HQLSS_ERR_NULL;
  hqlss_status st;
  if ((st = check_shape(N, D, C))) return st;
  if ((st = check_saved(saved))) return st;
  if (!a16(acc)) return HQLSS_ERR_ALIGN;
  hipStream_t s = static_cast<hipStream_t>(stream);
  if (which == 0) {
    if ((st = check_fwd_overflow(D))) return st;
    GemmArgs g{};
    g.A = saved->xq; g.lda = D / 2;
    g.B = saved->wq; g.ldb = D / 2;
    g.M = N; g.N = C; g.K = D;
    g.out = acc; g.ldo = C;
    const int sp = gemm_splits(N, C, D, true, true);
    if (sp > 1 && (!ws || ws_bytes < fwd_bytes(N, D, C, false))) return HQLSS_ERR_WORKSPACE;
    int32_t* part = sp > 1 ? reinterpret_cast<int32_t*>(static_cast<char*>(ws) + kFwdHead)
                           : nullptr;
    return hip_status(launch_gemm(s, kEpiAcc, HQLSS_F32, true, true, g, sp, part));
  }
  if (which == 10) {  // the forward product on the FP6 route (saved codes in the FP6 layout)
    if ((st = check_fwd_overflow(D))) return st;
    GemmArgs g{};
    g.A = saved->xq; g.lda = D;
    g.B = saved->wq; g.ldb = D;
    g.M = N; g.N = C; g.K = D;
    g.out = acc; g.ldo = C;
    const int sp = gemm6_splits(N, C, D);
    if (sp > 1 && (!ws || ws_bytes < kFwdHead + fwd6_partial(N, D, C))) return HQLSS_ERR_WORKSPACE;
    int32_t* part = sp > 1 ? reinterpret_cast<int32_t*>(static_cast<char*>(ws) + kFwdHead)
                           : nullptr;
    return hip_status(launch_gemm6(s, kEpiAcc, HQLSS_F32, g, sp, part));
  }
  if (which == 11 || which == 12) {  // the gradient products on the FP6 route
    if ((st = check_plan(plan))) return st;
    if ((st = check_bwd_overflow(N, D, C, 0))) return st;
    if ((st = check_bwd6_overflow(C))) return st;
    const size_t need = plan6_bytes(N) + (which == 11 ? dx6_bytes(N, D, C) : dw6_bytes(N, D, C));
    if (!ws || ws_bytes < need) return HQLSS_ERR_WORKSPACE;
    if (!a16(ws)) return HQLSS_ERR_ALIGN;
    Carve w{static_cast<char*>(ws), 0, ws_bytes};
    return do_grads_fp6(plan, saved, nullptr, nullptr, acc, which - 10, N, D, C, HQLSS_F32, 0, w, s);
  }
  if (which != 1 && which != 2) return HQLSS_ERR_ARG;
  if ((st = check_plan(plan))) return st;
  if ((st = check_bwd_overflow(N, D, C, 0))) return st;
  const size_t need = which == 1 ? dx_bytes(N, D, C) : dw_bytes(N, D, C);
  if (!ws || ws_bytes < need) return HQLSS_ERR_WORKSPACE;
  if (!a16(ws)) return HQLSS_ERR_ALIGN;
  Carve w{static_cast<char*>(ws), 0, ws_bytes};
  return do_grads(plan, saved, nullptr, nullptr, acc, which, N, D, C, HQLSS_F32, 0, w, s);
}

hqlss_status hqlss_timing_enable(int on) {
  if (on && !g_log.on) {
    if (g_log.ev.empty()) {
      g_log.ev.resize(2 * kLogPairs);
      g_log.ids.resize(kLogPairs);
      for (auto& e : g_log.ev)
        if (hipEventCreate(&e) != hipSuccess) return HQLSS_ERR_HIP;
    }
    g_log.used = 0;
    g_log.overflow = false;
    g_log.on = true;
  } else if (!on) {
    g_log.on = false;
  }
  return HQLSS_OK;
}

int hqlss_timing_read(int* ids, float* ms, int cap) {
  int n = 0;
  for (size_t i = 0; i < g_log.used; ++i) {
    if (hipEventSynchronize(g_log.ev[2 * i + 1]) != hipSuccess) return -1;
    float t = 0.f;
    if (hipEventElapsedTime(&t, g_log.ev[2 * i], g_log.ev[2 * i + 1]) != hipSuccess) return -1;
    if (n < cap) {
      ids[n] = g_log.ids[i];
      ms[n] = t;
      ++n;
    }
  }
  g_log.used = 0;
  return n;
}

const char* hqlss_kernel_name(int id) { return hqlss::kernel_name(id); }

void hqlss_debug_set_gemm_splits(int splits) { hqlss::gemm_set_split_override(splits); }
void hqlss_debug_set_gemm_tile_n(int bn) { hqlss::gemm_set_tile_override(bn); }
void hqlss_debug_set_fwd_fp6(int mode) { g_fwd_fp6_override = mode > 0 ? 1 : mode < 0 ? -1 : 0; }

size_t hqlss_debug_plan_scores_offset(int64_t N, int64_t* pitch) {
  if (N < 1) {
    if (pitch) *pitch = 0;
    return 0;
  }
  if (pitch) *pitch = score_pitch(N);
  return plan_scores_offset();
}

hqlss_status hqlss_debug_copy(const void* src, void* dst, size_t bytes, void* stream) {
  if (!src || !dst) return HQLSS_ERR_NULL;
  if (!a16(src) || !a16(dst)) return HQLSS_ERR_ALIGN;
  if (bytes % 16) return HQLSS_ERR_ARG;
  if (!bytes) return HQLSS_OK;
  return hip_status(launch_copy(static_cast<hipStream_t>(stream), src, dst, (int64_t)bytes));
}

}  // extern "C"
