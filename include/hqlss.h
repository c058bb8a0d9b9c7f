/*
 * hqlss.h -- C ABI of the INT4 quantised linear operator of
 * "Training Transformers with 4-bit Integers" (Xi, Li, Chen, Zhu; arXiv 2306.11987),
 * built for AMD Instinct MI355X (gfx950).
 *
 * One linear layer Y = X W^T, X: N x D activations (N tokens), W: C x D weights
 * (Sec. 3, Eq. 1).
 *
 *   forward   HQ-MM  (Sec. 3.3, Procedure HQ-MM): block-diagonal Hadamard transform of
 *             X and W, per-tensor INT4 quantisation, integer GEMM, dequantisation.
 *   backward  LSS-MM (Sec. 4.2, Procedure LSS-MM; App. A.3): bit splitting of dY into
 *             upper/lower INT4 halves, leverage-score sampling of the 2N stacked rows,
 *             integer GEMMs for dX and dW, dequantisation and the H^T of the STE
 *             gradients (Sec. 4).
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 * Memory      All pointers are DEVICE pointers unless stated.  The caller allocates every
 *             buffer (inputs, outputs, the saved state, the plan, the workspace); the
 *             library allocates and frees nothing and keeps no pointer after returning.
 * Layout      Row-major, contiguous.  X [N][D], W [C][D], Y/dY [N][C], dX [N][D], dW [C][D].
 *             INT4 codes are packed two per byte, even column in the low nibble:
 *             byte = (q[2i+1] << 4) | (q[2i] & 15)  (App. A.6, data pack).
 * Dtypes      X, W, Y, dY, dX, dW all use `dt`.  Codes are in [-7, 7] (Q_N = Q_P = 7,
 *             Sec. 3.1).  Integer GEMMs accumulate exactly in int32; scales and epilogues
 *             are fp32.
 * Hadamard    b = 2^log2_block, 0 <= log2_block <= 7.  The unnormalised +-1 Sylvester
 *             matrix H_u is used (H_u H_u^T = b I, Sec. 3.3); the 2^-k factor is folded
 *             into the dequantisation scales.
 * Scales      Dynamic per-tensor absmax: a = max|v|, s = a / 7, codes
 *             clamp(rint(v * fl(7/a)), -7, 7).  Bit splitting uses s_up = a_g / 7 and
 *             s_dn = s_up / 14.
 * Shapes      N >= 1; D and C multiples of 64; D a multiple of b.  N need not be a
 *             multiple of anything.
 * Streams     All work is enqueued on `stream` (a hipStream_t; 0 = the null stream) and
 *             runs asynchronously; no entry point synchronises the host.  Counts that
 *             the sample produces (the number of kept tokens) stay on the device.
 * Errors      Arguments are validated on the host before anything is launched; a
 *             non-zero hqlss_status is returned and nothing is enqueued.  A failed
 *             launch returns HQLSS_ERR_HIP.  No C++ exception crosses this ABI.
 * Threads     Calls may be issued from several host threads on different streams, with
 *             distinct buffers.  The test hooks and the kernel-timing log below are
 *             per calling thread.
 * RNG         Philox4x32-10 (Salmon et al., SC'11) with key = (lo32(seed), hi32(seed)) and
 *             counter = (lo32(blk), hi32(blk), stream, 0), blk = offset + (i >> 3);
 *             element i uses 16-bit half (i & 1) of output word ((i >> 1) & 3).
 *             Stream 0: stochastic rounding of the lower bit-split half, i = n*C + c.
 *             Stream 1: Bernoulli masks of the lower rows, i = n.
 *             Equal (seed, offset, budget) give bit-identical codes and samples.
 */
#ifndef HQLSS_H
#define HQLSS_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum { HQLSS_F32 = 0, HQLSS_F16 = 1, HQLSS_BF16 = 2 } hqlss_dtype;

typedef enum {
  HQLSS_OK = 0,
  HQLSS_ERR_NULL = 1,      /* a required pointer is NULL                               */
  HQLSS_ERR_SHAPE = 2,     /* N < 1, D or C not a positive multiple of 64               */
  HQLSS_ERR_BLOCK = 3,     /* log2_block outside [0, 7] or D % 2^log2_block != 0         */
  HQLSS_ERR_ALIGN = 4,     /* a pointer is not 16-byte aligned                          */
  HQLSS_ERR_DTYPE = 5,     /* unknown dtype                                             */
  HQLSS_ERR_WORKSPACE = 6, /* ws_bytes smaller than hqlss_workspace_bytes(...)          */
  HQLSS_ERR_OVERFLOW = 7,  /* an int32 accumulator or an int64 score could overflow    */
  HQLSS_ERR_HIP = 8,       /* a HIP launch or runtime call failed                       */
  HQLSS_ERR_ARG = 9,       /* any other invalid argument (e.g. budget, which)           */
  HQLSS_ERR_SCRATCH = 10   /* the shape needs more scratch than the static array holds
                              (allocation-free entry point only)                         */
} hqlss_status;

/* State written by the forward pass and read by the backward pass: the codes X^ and W^,
 * which the backward reuses from the forward rather than recomputing (Sec. 4).
 * Caller-allocated device memory; it must stay alive and unmodified from hq_linear_fwd
 * until the backward calls have run. */
typedef struct {
  uint8_t *xq;      /* [N][D/2]  INT4 codes of X H_u                                  */
  uint8_t *wq;      /* [C][D/2]  INT4 codes of W H_u                                  */
  uint8_t *wqT;     /* [D][C/2]  the same codes, transposed (row d holds column d of W^) */
  int32_t *x_sumsq; /* [N]       sum_d xq[n][d]^2 (feeds the leverage scores)          */
  float *amax;      /* [2]       a_x = max|X H_u|, a_w = max|W H_u|  (s = a / 7)        */
} hqlss_saved_t;

/* The quantised gradient and its sample (Sec. 4.2, Procedure LSS-MM steps 1-4).
 * Caller-allocated device memory, written by lss_grad_plan. */
typedef struct {
  uint8_t *qup;      /* [N][C/2]  upper INT4 codes of dY                               */
  uint8_t *qdn;      /* [N][C/2]  lower INT4 codes of dY (stochastically rounded)      */
  int32_t *sumsq_up; /* [N]       sum_c qup^2                                          */
  int32_t *sumsq_dn; /* [N]       sum_c qdn^2                                          */
  uint8_t *w_up;     /* [N]       weight of the upper row: 1 if kept, else 0            */
  uint8_t *w_dn;     /* [N]       weight m/p of the lower row: 0, 1, 2, 4, 8 or 16      */
  int32_t *kept;     /* [N]       ascending tokens with w_up + w_dn > 0 (first n_kept)   */
  int32_t *n_kept;   /* [1]       |T|, the number of kept tokens                        */
  float *amax_g;     /* [1]       a_g = max|dY|  (s_up = a_g / 7, s_dn = s_up / 14)      */
} lss_plan_t;

/* Learned-step-size (LSQ) mode (Sec. 3.1, Eq. 2; App. A.3): static step sizes given by the
 * caller instead of the per-tensor maxima.  step holds s_X, s_W as device fp32 scalars, the
 * steps of the transformed tensors X H_u and W H_u (unnormalised Hadamard domain, so a code
 * q stands for s q there); each must be finite and at least 2^-126, else the codes are
 * unspecified.  delta_x [N][D] and delta_w [C][D] are fp16 (IEEE binary16 bit patterns)
 * written by hq_linear_fwd_lsq and read by lss_linear_bwd_lsq: delta = q - I r with
 * r = fl(v fl(1/s)) and I = [-7 <= r <= 7], the factor of the step-size gradient; the
 * clip indicator I is recovered from it as |delta| <= 1/2.  Caller-allocated, 16-byte
 * aligned device memory. */
typedef struct {
  const float *step;   /* [2]      s_X, s_W                                                */
  uint16_t *delta_x;   /* [N][D]   fp16 delta_X                                            */
  uint16_t *delta_w;   /* [C][D]   fp16 delta_W                                            */
} hqlss_lsq_t;

/* Attention BMM T = BMM(Q, K^T) with per-batch learned steps (App. A.1): B independent
 * problems with Q_b [N][M], K_b [P][M], T_b [N][P] (in the terms of the linear operator
 * X = Q_b, W = K_b, D = M, C = P).  step_q and step_k hold one step per batch (device fp32,
 * as for hqlss_lsq_t); delta_q [B][N][M] and delta_k [B][P][M] are the forward's fp16
 * deltas.  The saved state of a batched call is the linear operator's per batch, stored
 * batch after batch: xq [B][N][M/2], wq [B][P][M/2], wqT [B][M][P/2], x_sumsq [B][N];
 * amax is not used. */
typedef struct {
  const float *step_q;  /* [B]        */
  const float *step_k;  /* [B]        */
  uint16_t *delta_q;    /* [B][N][M]  */
  uint16_t *delta_k;    /* [B][P][M]  */
} hqlss_bmm_lsq_t;

/* budget_rows value selecting the keep-every-non-zero-row sample (see lss_grad_plan). */
#define HQLSS_BUDGET_KEEP_NONZERO (-1)

/* Workspace sizes (bytes) for the entry points below, which = HQLSS_WS_*. */
enum { HQLSS_WS_FWD = 0, HQLSS_WS_BWD_DX = 1, HQLSS_WS_BWD_DW = 2, HQLSS_WS_BWD = 3,
       HQLSS_WS_FROM_PLAN = 4, HQLSS_WS_PLAN = 5, HQLSS_WS_HSIZE = 6, HQLSS_WS_FWD_LSQ = 7,
       HQLSS_WS_BWD_LSQ = 8, HQLSS_WS_FWD_FP6 = 9, HQLSS_WS_BWD_FP6 = 10,
       HQLSS_WS_FROM_PLAN_FP6 = 11 };
/* Workspace sizes of the batched entry points (B problems of the given shape). */
enum { HQLSS_WS_BMM_FWD = 0, HQLSS_WS_BMM_BWD = 1 };
size_t hqlss_bmm_workspace_bytes(int which, int64_t B, int64_t N, int64_t M, int64_t P);
size_t hqlss_workspace_bytes(int which, int64_t N, int64_t D, int64_t C);

/* HQ-MM forward (Sec. 3.3, Eq. 3; Procedure HQ-MM).
 *   1. v_x = X H_u, v_w = W H_u in fp32 (radix-2 FWHT, strides ascending);
 *   2. a_x = max|v_x|, a_w = max|v_w|; codes clamp(rint(v * fl(7/a)), -7, 7) -> saved;
 *   3. acc = X^ W^^T (int32, exact);
 *   4. Y = fl(alpha * acc), alpha = fl(fl(s_x s_w) / 2^k), cast to dt.
 * X [N][D], W [C][D] inputs; Y [N][C] output; saved: outputs (all fields required);
 * ws: scratch of at least hqlss_workspace_bytes(HQLSS_WS_FWD, ...) bytes.
 * Products of more than 2^38 multiply-adds (N D C) run step 3 on the FP6 MFMA, as
 * hq_linear_fwd_fp6 does (every code is exact in e2m3 and the fp32 sums are exact), with
 * the codes written a second time as FP6 into the workspace; acc, Y and the saved codes are
 * the same bits either way, only the workspace size differs. */
hqlss_status hq_linear_fwd(const void *X, const void *W, void *Y, int64_t N, int64_t D,
                           int64_t C, hqlss_dtype dt, int log2_block,
                           const hqlss_saved_t *saved, void *ws, size_t ws_bytes,
                           void *stream);

/* Allocation-free HQ-MM forward, for callers that cannot allocate device memory: code under
 * HIP graph capture, tight serving loops, harnesses that forbid hipMalloc.  Identical to
 * hq_linear_fwd (same steps, arguments, layouts, results and errors) except that the
 * workspace is not passed: the absmax and split-K partials live in a static device array of
 * HQLSS_STATIC_SCRATCH_BYTES that the library owns, one copy per GPU, held until the
 * process ends.  Nothing is allocated or freed by the call.
 *   - HQLSS_ERR_SCRATCH when hqlss_workspace_bytes(HQLSS_WS_FWD, N, D, C) exceeds
 *     HQLSS_STATIC_SCRATCH_BYTES (only small outputs over a long K split along K and need
 *     more than the absmax partials); use hq_linear_fwd then.
 *   - The array keeps the last call's contents; nothing in it needs to start at zero (every
 *     partial is written before it is read).
 *   - Calls that overlap on one GPU (several streams or threads) race on the array:
 *     serialise them.  The current HIP device must be the device of `stream`. */
#define HQLSS_STATIC_SCRATCH_BYTES ((size_t)8 << 20)
hqlss_status hq_linear_fwd_noalloc(const void *X, const void *W, void *Y, int64_t N, int64_t D,
                                   int64_t C, hqlss_dtype dt, int log2_block,
                                   const hqlss_saved_t *saved, void *stream);

/* FP6 route of HQ-MM (Sec. 3.3, Eq. 3; Procedure HQ-MM), for gfx950's FP6 matrix cores:
 * every INT4 code |q| <= 7 is exact in e2m3 and the fp32 accumulation of their products is
 * exact (integers below 2^24), so the product runs on the FP6 MFMA at twice the int8 rate
 * and Y equals hq_linear_fwd's bit for bit.  Steps, arguments and errors as hq_linear_fwd;
 * only the saved codes differ in layout: saved->xq [N][D], saved->wq [C][D] and saved->wqT
 * [D][C] hold one byte per code, every 32 codes of a row being 24 bytes of e2m3 fields
 * (code i at bits 6i..6i+5 of the little-endian 192-bit group) and 8 zero bytes.
 * e2m3 (OCP Microscaling Formats): sign, 2 exponent bits with bias 1, 3 mantissa bits.
 * ws: at least hqlss_workspace_bytes(HQLSS_WS_FWD_FP6, ...) bytes. */
hqlss_status hq_linear_fwd_fp6(const void *X, const void *W, void *Y, int64_t N, int64_t D,
                               int64_t C, hqlss_dtype dt, int log2_block,
                               const hqlss_saved_t *saved, void *ws, size_t ws_bytes,
                               void *stream);

/* FP6 route of LSS-MM (Sec. 4.2, Procedure LSS-MM, App. A.3), after hq_linear_fwd_fp6 (saved
 * in the FP6 layout): the same bit split, leverage scores and sample as lss_linear_bwd, and
 * dX, dW equal to its outputs bit for bit; the two products run on the FP6 MFMA.  The
 * weighted rows 14 w_up q_up + w_dn q_dn do not fit e2m3, so the route keeps the two code
 * planes apart and applies the weights exactly on the fp32 accumulators: dX rows of tokens
 * with an upper row run a first K pass over the upper codes, scaled by 14 / w_dn before the
 * lower pass and by w_dn after it; dW takes its K entries grouped by weight 2^4 .. 2^0 (an
 * upper row, weight 14 = 8 + 4 + 2, once in each of three classes) and doubles its sums at
 * every class boundary.  Arguments, sampling and errors as lss_linear_bwd, plus
 * HQLSS_ERR_OVERFLOW for C > 11412 (the upper-pass sums must stay exact in fp32).
 * ws: at least hqlss_workspace_bytes(HQLSS_WS_BWD_FP6, ...) bytes. */
hqlss_status lss_linear_bwd_fp6(const void *dY, const hqlss_saved_t *saved, void *dX, void *dW,
                                int64_t N, int64_t D, int64_t C, hqlss_dtype dt, int log2_block,
                                int64_t budget_rows, uint64_t seed, uint64_t offset, void *ws,
                                size_t ws_bytes, void *stream);

/* HQ-MM forward with learned step sizes (Sec. 3.3 Procedure HQ-MM with step 2 done by LSQ,
 * Eq. 2; App. A.3).
 *   1. v_x = X H_u, v_w = W H_u in fp32, as hq_linear_fwd;
 *   2. r = fl(v fl(1/s)), codes clamp(rint(r), -7, 7) -> saved; delta -> lsq (one pass,
 *      no maximum);
 *   3. acc = X^ W^^T (int32, exact);
 *   4. Y = fl(alpha * acc), alpha = fl(fl(s_X s_W) / 2^k), cast to dt.
 * saved: xq, wq, wqT, x_sumsq are written (amax is neither read nor written and may be
 * NULL); lsq: step read, delta_x and delta_w written.  ws: at least
 * hqlss_workspace_bytes(HQLSS_WS_FWD_LSQ, ...) bytes (may be NULL when that is 0). */
hqlss_status hq_linear_fwd_lsq(const void *X, const void *W, void *Y, int64_t N, int64_t D,
                               int64_t C, hqlss_dtype dt, int log2_block,
                               const hqlss_saved_t *saved, const hqlss_lsq_t *lsq, void *ws,
                               size_t ws_bytes, void *stream);

/* Forward of the attention BMM (App. A.1): for every batch b, hq_linear_fwd_lsq with
 * X = Q_b, W = K_b, steps step_q[b], step_k[b]:
 *   codes and deltas of Q_b H_u and K_b H_u (one pass), T_b = fl(alpha_b acc_b) with
 *   alpha_b = fl(fl(step_q[b] step_k[b]) / 2^k), cast to dt.
 * Q [B][N][M], K [B][P][M] inputs; T [B][N][P] output; M and P positive multiples of 64
 * (and M % 2^k == 0), 1 <= B <= 65535, B N and B P at most 2^30.  Every batch runs in the
 * same launches (batch strides, no per-batch host work).  ws: at least
 * hqlss_bmm_workspace_bytes(HQLSS_WS_BMM_FWD, ...) bytes (may be NULL when that is 0). */
hqlss_status hq_bmm_fwd_lsq(const void *Q, const void *K, void *T, int64_t B, int64_t N,
                            int64_t M, int64_t P, hqlss_dtype dt, int log2_block,
                            const hqlss_saved_t *saved, const hqlss_bmm_lsq_t *lsq, void *ws,
                            size_t ws_bytes, void *stream);

/* Backward of the attention BMM (App. A.1): for every batch b, lss_linear_bwd_lsq with
 * dY = dT_b, X = Q_b, W = K_b and the steps of batch b: its own bit split (scale s_up,b),
 * leverage scores c_{b,i} and sample, drawing its random numbers at counter offset
 * offset + b * lss_philox_offset_advance(N, P); then
 *   dQ_b = fl(alpha * FWHT_b(I_Q o acc_dx)), dK_b = fl(alpha * FWHT_b(I_K o acc_dw)),
 *   dstep_q[b], dstep_k[b] as dstep[0], dstep[1] of lss_linear_bwd_lsq (g = 1/sqrt(7 N M)
 *   and 1/sqrt(7 P M)).
 * dT [B][N][P] input; dQ [B][N][M] or NULL, dK [B][P][M] or NULL (at least one);
 * dstep_q, dstep_k: device fp32 [B] or NULL (dstep_q is written only with dQ, dstep_k only
 * with dK).  saved and lsq as written by hq_bmm_fwd_lsq.  budget_rows per batch as for
 * lss_linear_bwd.  Shapes as for hq_bmm_fwd_lsq, and N <= 65536.  ws: at least
 * hqlss_bmm_workspace_bytes(HQLSS_WS_BMM_BWD, ...) bytes (less suffices with dQ or dK NULL). */
hqlss_status lss_bmm_bwd_lsq(const void *dT, const hqlss_saved_t *saved,
                             const hqlss_bmm_lsq_t *lsq, void *dQ, void *dK, float *dstep_q,
                             float *dstep_k, int64_t B, int64_t N, int64_t M, int64_t P,
                             hqlss_dtype dt, int log2_block, int64_t budget_rows, uint64_t seed,
                             uint64_t offset, void *ws, size_t ws_bytes, void *stream);

/* Bit splitting and leverage-score sampling of dY (Sec. 4.2, App. A.2; Procedure LSS-MM
 * steps 1-3, shared by both gradients as in App. A.6).
 *   q_up = rint(dY * fl(7/a_g)); r = that product - q_up; q_dn = SR(fl(14 r)) (stream 0);
 *   scores c_j^2 = w^2 sum q^2 x_sumsq (w = 14 upper, 1 lower), c_j = isqrt(c_j^2 2^16);
 *   p* by the clamp-and-rescale loop of App. A.2 with sum p* = budget (exact integers);
 *   upper rows: kept iff non-zero; lower rows: p~ = 2^-e >= p* (e <= 4, <= 2 if the upper
 *   row is non-zero), m = [u16 < 2^(16-e)] (stream 1), weight m 2^e.
 * budget_rows: 1 .. 2N, or 0 for budget = N (Sec. 4.2: sum p_i = N), or
 * HQLSS_BUDGET_KEEP_NONZERO for budget = 2N, which keeps every non-zero row with weight 1
 * whatever the masks draw: the deterministic rule of the paper's implementation (App. A.6,
 * keep the rows of non-zero norm); dX and dW are then the bit-split product itself.  Any
 * other value is HQLSS_ERR_ARG.  dY [N][C] input; saved is
 * read (x_sumsq); plan: outputs (all fields required); ws: scratch of at least
 * hqlss_workspace_bytes(HQLSS_WS_PLAN, ...) bytes. */
hqlss_status lss_grad_plan(const void *dY, const hqlss_saved_t *saved, const lss_plan_t *plan,
                           int64_t N, int64_t D, int64_t C, hqlss_dtype dt,
                           int64_t budget_rows, uint64_t seed, uint64_t offset, void *ws,
                           size_t ws_bytes, void *stream);

/* LSS-MM gradients from a plan (Sec. 4, Sec. 4.2, App. A.3; Procedure LSS-MM steps 4-6).
 *   A_t = 14 w_up q_up[t] + w_dn q_dn[t] for kept tokens t (|A| <= 126, int8);
 *   dX[t] = fl(alpha_dx * FWHT_b(A_t W^)),           alpha_dx = fl(fl(s_up s_w) / (14 b));
 *   dW    = fl(alpha_dw * FWHT_b(A_T^T X^_T)) rows,  alpha_dw = fl(fl(s_up s_x) / (14 b));
 *   rows of dX of dropped tokens are 0.  FWHT_b is along D, in exact int32.
 * dX [N][D] or NULL, dW [C][D] or NULL (at least one).  saved and plan are inputs. */
hqlss_status lss_linear_bwd_from_plan(const lss_plan_t *plan, const hqlss_saved_t *saved,
                                      void *dX, void *dW, int64_t N, int64_t D, int64_t C,
                                      hqlss_dtype dt, int log2_block, void *ws,
                                      size_t ws_bytes, void *stream);

/* Both gradients from one shared sample: lss_grad_plan into the workspace, then
 * lss_linear_bwd_from_plan.  dX, dW outputs (either may be NULL, not both). */
hqlss_status lss_linear_bwd(const void *dY, const hqlss_saved_t *saved, void *dX, void *dW,
                            int64_t N, int64_t D, int64_t C, hqlss_dtype dt, int log2_block,
                            int64_t budget_rows, uint64_t seed, uint64_t offset, void *ws,
                            size_t ws_bytes, void *stream);

/* Activation gradient alone (Sec. 4.2 "Activation Gradient"; App. A.3).  Same sample as
 * lss_linear_bwd_dw for equal (seed, offset, budget_rows). */
hqlss_status lss_linear_bwd_dx(const void *dY, const hqlss_saved_t *saved, void *dX,
                               int64_t N, int64_t D, int64_t C, hqlss_dtype dt, int log2_block,
                               int64_t budget_rows, uint64_t seed, uint64_t offset, void *ws,
                               size_t ws_bytes, void *stream);

/* Weight gradient alone (Sec. 4.2 "Weight Gradient", Eq. 5). */
hqlss_status lss_linear_bwd_dw(const void *dY, const hqlss_saved_t *saved, void *dW,
                               int64_t N, int64_t D, int64_t C, hqlss_dtype dt, int log2_block,
                               int64_t budget_rows, uint64_t seed, uint64_t offset, void *ws,
                               size_t ws_bytes, void *stream);

/* LSS-MM backward of the learned-step-size forward (Sec. 4, App. A.3): the sample and
 * bit split of lss_linear_bwd, then with the unmasked integer accumulators acc_dx = A_T W^
 * and acc_dw = A_T^T X^_T
 *   dX[t] = fl(alpha_dx * FWHT_b(I_X[t] o acc_dx[t])), dW = fl(alpha_dw * FWHT_b(I_W o acc_dw))
 *   (alpha as in lss_linear_bwd_from_plan with s_X, s_W the steps; I from delta);
 *   dstep[0] = g(s_X) a_dx sum(acc_dx o delta_X[kept]),  a_dx = (s_up / 14) s_W 2^-k,
 *   dstep[1] = g(s_W) a_dw sum(acc_dw o delta_W),         a_dw = (s_up / 14) s_X 2^-k,
 *   g(s_X) = 1 / sqrt(7 N D), g(s_W) = 1 / sqrt(7 C D); the products and the sums are
 *   fp64 (per-workgroup partials added in a fixed order, so results are deterministic),
 *   rounded to fp32 at the end.
 * dX [N][D] or NULL, dW [C][D] or NULL (at least one); dstep: device fp32[2] or NULL (no
 * step-size gradients); dstep[0] is written only with dX, dstep[1] only with dW.  saved:
 * xq, wq, wqT, x_sumsq from hq_linear_fwd_lsq (amax unused); lsq: the same steps and the
 * forward's deltas (delta_x needed with dX, delta_w with dW).  budget_rows, seed and
 * offset as for lss_linear_bwd.  ws: at least hqlss_workspace_bytes(HQLSS_WS_BWD_LSQ, ...)
 * bytes. */
hqlss_status lss_linear_bwd_lsq(const void *dY, const hqlss_saved_t *saved,
                                const hqlss_lsq_t *lsq, void *dX, void *dW, float *dstep,
                                int64_t N, int64_t D, int64_t C, hqlss_dtype dt, int log2_block,
                                int64_t budget_rows, uint64_t seed, uint64_t offset, void *ws,
                                size_t ws_bytes, void *stream);

/* Choice of the Hadamard block size (App. A.5).  For every candidate k (0 <= k <=
 * max_log2_block <= 7, D a multiple of 2^k) the reconstructions V_bar = s int_s(V H) H^T of
 * V = X and V = W, with the forward's codes and steps (fp32 transform, s = fl(a/7), codes
 * rint(v * fl(7/a))), give MSE(V_bar, V) = ||s q - V H_u||^2 / (2^k numel) (Parseval; fp32
 * per-element differences, fp64 sums); the k minimising MSE(X_bar, X) MSE(W_bar, W) is
 * written to *log2_block_out, ties to the smaller k.  X [N][D], W [C][D] inputs (dtype dt,
 * shapes as for hq_linear_fwd); log2_block_out: device int32[1]; mse_out: device
 * double[16], MSE_X(k) at [k] and MSE_W(k) at [8 + k], NaN where k is no candidate (8-byte
 * aligned).  ws: scratch of at least hqlss_workspace_bytes(HQLSS_WS_HSIZE, ...) bytes.
 * Deterministic for a given device.  max_log2_block outside 0..7 is HQLSS_ERR_BLOCK. */
hqlss_status hq_choose_hadamard_size(const void *X, const void *W, int64_t N, int64_t D,
                                     int64_t C, hqlss_dtype dt, int max_log2_block,
                                     int32_t *log2_block_out, double *mse_out, void *ws,
                                     size_t ws_bytes, void *stream);

/* Philox blocks one stream consumes per backward call: advance `offset` by at least this
 * much between calls that must draw independent randomness. */
uint64_t lss_philox_offset_advance(int64_t N, int64_t C);

const char *hqlss_status_string(hqlss_status s);

/* ---- inspection (tests) ------------------------------------------------------------
 * Raw int32 accumulators of the three integer GEMMs, before any scaling or transform:
 *   which 0: acc[N][C]   = X^ W^^T                     (inputs: saved)
 *   which 1: acc[T][D]   = A_T W^  (rows in kept order, T = n_kept rows written)
 *   which 2: acc[C][D]   = A_T^T X^_T
 *   which 10, 11, 12: which 0, 1, 2 on the FP6 route (saved written by hq_linear_fwd_fp6;
 *            11 and 12 need hqlss_workspace_bytes(HQLSS_WS_FROM_PLAN_FP6, ...) bytes)
 * acc is an int32 device buffer of N*C (0, 10), N*D (1, 11) or C*D (2, 12) elements. */
hqlss_status hqlss_debug_gemm_acc(int which, const lss_plan_t *plan, const hqlss_saved_t *saved,
                                  int32_t *acc, int64_t N, int64_t D, int64_t C, void *ws,
                                  size_t ws_bytes, void *stream);

/* Test hook: force the split-K factor of every integer GEMM (0 restores the built-in
 * choice).  Workspace sizes follow the factor in force when they are queried.  The
 * setting is per calling thread: it applies to the calls (and workspace queries) made
 * by the thread that set it, and never to another thread's. */
void hqlss_debug_set_gemm_splits(int splits);

/* Test hook: force the workgroup tile width (128 or 256 output columns) of the forward
 * GEMMs and of the gradient GEMMs whose output is wider than 64 columns, where they are
 * not split along K; any other value restores the built-in choice.  Results do not depend
 * on the width.  Workspace sizes follow the width in force when they are queried.  Per
 * calling thread, as the split hook. */
void hqlss_debug_set_gemm_tile_n(int bn);

/* Test hook: the product of hq_linear_fwd on the FP6 MFMA (mode > 0), on the int8 MFMA
 * (mode < 0), or chosen by size (0, the default).  Results do not depend on it; workspace
 * sizes follow the choice in force when they are queried.  Per calling thread, as the split
 * hook. */
void hqlss_debug_set_fwd_fp6(int mode);

/* Test hook: where lss_grad_plan leaves the integer leverage scores of its sample inside
 * the workspace it was given (Sec. 4.2; see lss_grad_plan for their definition): the
 * scores of the N upper rows start at the returned byte offset, those of the N lower rows
 * `*pitch` uint32 entries later; they stay there until the workspace is reused.  Returns
 * 0 and sets *pitch to 0 for N < 1. */
size_t hqlss_debug_plan_scores_offset(int64_t N, int64_t *pitch);

/* Benchmark hook: a plain device-to-device copy kernel ("copy") of `bytes` bytes (a
 * multiple of 16, both pointers 16-byte aligned, non-overlapping), asynchronous on
 * `stream`.  Its bytes read and written are known exactly, which calibrates hardware
 * traffic counters.  Errors: HQLSS_ERR_NULL, HQLSS_ERR_ALIGN, HQLSS_ERR_ARG (size). */
hqlss_status hqlss_debug_copy(const void *src, void *dst, size_t bytes, void *stream);

/* ---- kernel timing (benchmarks) ------------------------------------------------------
 * When enabled, every kernel the library launches is bracketed by two HIP events
 * recorded on the launch stream.  hqlss_timing_read waits for them, writes up to `cap`
 * (kernel id, milliseconds) pairs and clears the log; hqlss_kernel_name maps ids.  The
 * log is per calling thread: a thread records and reads only its own launches. */
hqlss_status hqlss_timing_enable(int on);
int hqlss_timing_read(int *ids, float *ms, int cap);
const char *hqlss_kernel_name(int id);

#ifdef __cplusplus
}
#endif
#endif /* HQLSS_H */
