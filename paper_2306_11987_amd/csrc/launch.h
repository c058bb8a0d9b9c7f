// Host-side launchers of the HQ-MM / LSS-MM kernels (internal to libhqlss).
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace hqlss {

// Kernel ids for the timing log (kept in sync with kernel_name()).
enum KernelId : int {
  kKAbsmax = 0, kKQuant, kKBitSplit, kKPlan, kKBuild,
  kKGemmFwd, kKGemmDx, kKGemmDw, kKGemmAcc, kKReduce, kKCopy, kKHsizeMax, kKHsizeErr,
  kKHsizePick, kKLsqQuant, kKLsqStepGrad, kKFp6Convert, kKFp6Plan, kKFp6Build, kKCount
};
const char* kernel_name(int id);

// Every launch goes through this hook so that the timing log can bracket it.
void timing_begin(hipStream_t s);
void timing_end(hipStream_t s, int id);

// Plain device copy of `bytes` (a multiple of 16; both pointers 16-byte aligned).
hipError_t launch_copy(hipStream_t s, const void* src, void* dst, int64_t bytes);

// One tensor for the row-group quantisers: rows x cols (cols a multiple of 64), processed
// by `wg` workgroups of 512 threads with 2^log2g lanes per row.  Launchers choose `wg`
// (a grid that is resident at once) and store it back into the job.  A batched job holds
// `batch` such tensors, `bstride` elements apart; `wg` is then per batch, and every
// per-tensor output (codes, row sums, maxima, partials, ...) is one block per batch.
constexpr int kQMaxWg = 1024;  // workgroups (= partial results) of one unbatched job at most
// a batched job has at most kBatchWgSlack + batch workgroups in all (ceil(2 kQMaxWg / B) per batch)
constexpr int kBatchWgSlack = 2 * kQMaxWg;
struct QJob {
  const void* src;
  int64_t rows, cols;
  int log2g;
  int wg;
  int batch;
  int64_t bstride;
};
QJob make_job(const void* src, int64_t rows, int64_t cols);  // rows = 0: an empty job; wg unset
QJob make_job_batched(const void* src, int64_t batch, int64_t rows, int64_t cols);

// Per-workgroup maxima of |block-FWHT(src)| of up to two tensors in one launch:
// part0[0, j0.wg) and part1[0, j1.wg), plain stores (no initialisation needed).
hipError_t launch_fwht_absmax(hipStream_t s, int dt, int log2b, QJob& j0, float* part0,
                              QJob& j1, float* part1);
// Codes of block-FWHT(src) at the maximum of the partials, packed [rows][cols/2]; optional
// per-row sums of squares; the maximum itself is stored to *amax_out.  For the second job
// the same codes can also be written transposed, packed [cols][rows/2] (rows a multiple of
// 16), by extra workgroups of the same launch.
struct QOut {
  const float* part;
  int nparts;
  float* amax_out;
  uint8_t* packed;
  int32_t* row_sumsq;  // may be null
  uint8_t* packed_t;   // may be null; honoured for the second job only
  uint8_t* fp6;        // may be null: the codes again, as FP6 (e2m3) in the padded layout
                       // of fp6.hip (row pitch: cols bytes), row-major
};
hipError_t launch_fwht_quant(hipStream_t s, int dt, int log2b, const QJob& j0, const QOut& o0,
                             const QJob& j1, const QOut& o1);
// Learned-step-size codes of block-FWHT(src) (one pass, no maximum): r = fl(v * fl(1/s)),
// codes clamp(rint(r), -7, 7) packed as above, optional row sums of squares, and
// delta = q - [|r| <= 7] r as fp16 bits [rows][cols].
struct LsqOut {
  const float* step;   // device scalar s > 0 (batched: step[b], one per batch)
  uint8_t* packed;
  int32_t* row_sumsq;  // may be null
  uint16_t* delta;
  uint8_t* packed_t;   // may be null; second job only: codes transposed, as for QOut
};
hipError_t launch_fwht_lsq(hipStream_t s, int dt, int log2b, const QJob& j0, const LsqOut& o0,
                           const QJob& j1, const LsqOut& o1);
// Bit split of dY [N][C] into two packed code planes, their row sums of squares, the
// integer leverage scores scores[t] (upper row) and scores[score_pitch + t] (lower row),
// and per-workgroup {count of non-zero scores, sum lo, sum hi, 0} in parts[0, j.wg).
struct BsOut {
  float* amax_out;
  uint8_t* qup;
  uint8_t* qdn;
  int32_t* sumsq_up;
  int32_t* sumsq_dn;
  const int32_t* x_sumsq;
  uint32_t* scores;
  int64_t score_pitch;
  uint4* parts;
  uint64_t offset_stride;  // batched: Philox counter offset between batches
};
hipError_t launch_bit_split(hipStream_t s, int dt, QJob& j, const float* part, int nparts,
                            const BsOut& o, uint64_t seed, uint64_t offset);
// Hadamard block-size search of X (j0) and W (j1), equal cols (App. A.5): maxima of all
// nested transforms k = 0..7 into mx[wg][8], error sums into err[wg][8] (each buffer
// kQMaxWg * 8 entries), then *k_out and mse_out[16] (MSE_X(k), then MSE_W(k); NaN for k
// not a candidate: k > kmax or cols % 2^k != 0).
hipError_t launch_hsize_search(hipStream_t s, int dt, QJob& j0, QJob& j1, float* mx0, float* mx1,
                               double* err0, double* err1, int kmax, int32_t* k_out,
                               double* mse_out);
// leverage scores, clamp-rescale, masks, compaction (one workgroup per batch; batch b reads
// and writes its own blocks: N rows, 2 score_pitch scores, nparts partials, one n_kept, and
// draws at counter offset + b offset_stride).
hipError_t launch_lss_plan(hipStream_t s, const int32_t* sumsq_up, const uint32_t* scores,
                           int64_t score_pitch, const uint4* parts, int nparts, int64_t N,
                           int64_t budget, uint64_t seed, uint64_t offset, uint8_t* w_up,
                           uint8_t* w_dn, int32_t* kept, int32_t* n_kept, int64_t batch = 1,
                           uint64_t offset_stride = 0);
// GEMM operands of the kept tokens in one pass (any of Ag, XtT, dX may be null):
// Ag [round_up(N,128)][C] weighted rows (int8, K-interleaved; rows < round_up(n_kept,128)
// written) and XtT [D][Kp/2] the gathered X^ rows transposed (packed),
// Kp = round_up(N, 128); rows of dX (dtype dt) of dropped tokens are zeroed.
hipError_t launch_build_operands(hipStream_t s, int dt, const uint8_t* qup, const uint8_t* qdn,
                                 const uint8_t* w_up, const uint8_t* w_dn, const int32_t* kept,
                                 const int32_t* n_kept, const uint8_t* xq, int64_t N, int64_t C,
                                 int64_t D, int8_t* Ag, uint8_t* XtT, void* dX,
                                 int64_t batch = 1);

// Integer GEMM  acc[m][n] = sum_k A[m][k] B[n][k]  (both operands K-contiguous rows).
// kEpiDxL / kEpiDwL: the gradient epilogues of the learned-step-size mode, which mask the
// accumulators by the clip indicator before the transform and sum acc * delta.
enum Epi : int { kEpiFwd = 0, kEpiDx = 1, kEpiDw = 2, kEpiAcc = 3, kEpiPartial = 4, kEpiDxL = 5,
                 kEpiDwL = 6 };
struct GemmArgs {
  const void* A;        // [M][lda] bytes: packed int4 (a_int4) or K-interleaved int8
  const void* B;        // [N][ldb] bytes
  int64_t lda, ldb;     // row pitch in bytes
  int64_t M, N, K;      // K in elements (a multiple of 64); M is an upper bound if m_dev
  const int32_t* m_dev; // if set, M = *m_dev (rows beyond are not computed)
  const int32_t* k_dev; // if set, K = round_up(*k_dev, 128)
  void* out;            // [M][ldo] (or rows out_rows[m]) in `dt`, or int32 for kEpiAcc
  int64_t ldo;
  const int32_t* out_rows;     // kEpiDx: destination row of output row m
  const uint32_t* amax1;       // scale operands of alpha (fp32 bit patterns)
  const uint32_t* amax2;
  float denom;                 // alpha = fl(fl(s1 s2) / denom)
  int log2b;                   // FWHT block of the gradient epilogues
  int steps_mask;              // bit i set: amax(i+1) holds a step s itself (else s = a / 7)
  const uint16_t* delta;       // kEpiDxL / kEpiDwL: fp16 delta, indexed like out (pitch ldo)
  double* ds_part;             // kEpiDxL / kEpiDwL: one sum of acc * delta per workgroup
  // Batched launch (batch > 0): blockIdx.z is the batch b (no split-K), and problem b uses
  // A + b bs_a, B + b bs_b (bytes), out + b bs_out, delta + b bs_delta (elements),
  // out_rows + b bs_rows, one m_dev / k_dev / amax1 / amax2 entry per batch and one block
  // of ds_part entries per batch.
  int batch;
  int64_t bs_a, bs_b, bs_out, bs_rows, bs_delta;
  // FP6 route (launch_gemm6) only.  f6_kind 1: the dX product, whose tiles with rows below
  // *m2_dev run a first K pass over A2 (upper codes, pitch lda) and weight rows by w_up,
  // w_dn of their token out_rows[m]; f6_kind 2: the dW product, whose K entries come in
  // weight classes 2^4 .. 2^0 starting at entries 0, kcls[0..3].
  int f6_kind;
  const void* A2;
  const int32_t* m2_dev;
  const uint8_t* w_up;
  const uint8_t* w_dn;
  const int32_t* kcls;
  // int8 x INT4 kEpiDw / kEpiDwL / kEpiAcc only: A is stored k-major (A[k][m], pitch lda, m positions
  // K-interleaved in groups of 8: the dX operand A_T serves as the dW operand), K whole
  // stages of 128 and M a multiple of 16
  int a_kmajor;
};
// Split-K factor the launcher uses for this shape (1 = no split), and the int32 partial
// buffer it then needs (splits x M x N words).  A non-zero override forces the factor.
int gemm_splits(int64_t M, int64_t N, int64_t K, bool a_int4, bool b_int4);
size_t gemm_partial_bytes(int64_t M, int64_t N, int splits);
void gemm_set_split_override(int splits);
void gemm_set_tile_override(int bn);
hipError_t launch_gemm(hipStream_t s, int epi, int dt, bool a_int4, bool b_int4, const GemmArgs& g,
                       int splits, int32_t* partial);
// Tile widths the launchers choose (forward, gradients), and the split-K reduction with the
// epilogue of `epi` on its own (kEpiAcc, kEpiFwd, kEpiDx, kEpiDw).
int gemm_fwd_bn(int64_t M, int64_t N, int splits, int64_t batch);
int gemm_grad_bn(int64_t M, int64_t N, int splits);
hipError_t launch_gemm_reduce(hipStream_t s, int epi, int dt, const int32_t* P, int S, const GemmArgs& g);
// The same products on the FP6 MFMA: both operands in the padded FP6 layout of
// launch_int4_to_fp6 (lda, ldb = K bytes), results identical to launch_gemm's.
hipError_t launch_gemm6(hipStream_t s, int epi, int dt, const GemmArgs& g, int splits, int32_t* partial);
int gemm6_splits(int64_t M, int64_t N, int64_t K);  // split-K factor of launch_gemm6
int gemm_split_override();                          // the test hook's forced factor (0: none)
// Packed INT4 codes [rows][K/2] (two's complement nibbles, even k in the low nibble) to the
// padded FP6 layout [rows][K]: every 32 codes become 24 bytes of e2m3 fields (field i at
// bits 6i..6i+5, little-endian) followed by 8 zero bytes.  K a multiple of 64.
hipError_t launch_int4_to_fp6(hipStream_t s, const uint8_t* src, uint8_t* dst, int64_t rows, int64_t K);
// Row orders of the FP6 backward from the sample's weights (one workgroup, N <= 65536):
// order6[n_kept] (upper tokens first), *n_up, the dW entries ent[] grouped by weight class
// (capacity 4 N + 640, -1 = padding) and cls[5] = first entries of classes 3, 2, 1, 0 and
// the padded entry count.
hipError_t launch_fp6_plan(hipStream_t s, const uint8_t* w_up, const uint8_t* w_dn, int64_t N,
                           int32_t* order6, int32_t* n_up, int32_t* ent, int32_t* cls);
// FP6 operands of the backward GEMMs (padded FP6 layout):
//   a_dn [N][C]: row i = lower codes of token order6[i] (zero when its w_dn = 0), i < n_kept;
//   a_up [round_up(N, 256)][C]: row i = upper codes of token order6[i] for i < n_up, zero up
//        to the next multiple of 256;
//   a_dw [C][ecap], x_dw [D][ecap]: column e = the codes of entry ent[e] (upper or lower row of
//        its token; X^ row of its token), zero for padding entries; e < cls[4].
// Dropped tokens' rows of dX (dtype dt) are zeroed.  Any output may be null.
hipError_t launch_fp6_build(hipStream_t s, int dt, const uint8_t* qup, const uint8_t* qdn,
                            const uint8_t* w_up, const uint8_t* w_dn, const int32_t* order6,
                            const int32_t* n_kept, const int32_t* n_up, const int32_t* ent,
                            const int32_t* cls, const uint8_t* xq6, int64_t N, int64_t C,
                            int64_t D, int64_t ecap, uint8_t* a_dn, uint8_t* a_up, uint8_t* a_dw,
                            uint8_t* x_dw, void* dX);
// Number of ds_part entries a kEpiDxL / kEpiDwL launch of this shape writes (one per
// workgroup: of the GEMM, or of the reduction after split-K; every entry is written, 0 by
// workgroups without rows).
int64_t gemm_epi_parts(int64_t M, int64_t N, int splits);
// Step-size gradients from the partial sums (one workgroup, fixed order):
// dstep_x = gx * (s_up / 14) s_w 2^-k * sum(px), dstep_w = gw * (s_up / 14) s_x 2^-k *
// sum(pw), s_up = fl(*amax_g / 7), s_x = *step_x, s_w = *step_w; an entry with no partials
// (n = 0) is left unwritten.
// Batched (batch > 1): block b uses px + b nx, pw + b nw and entry b of amax_g, step_x,
// step_w, dstep_x, dstep_w; the linear operator passes step_x = step, step_w = step + 1.
hipError_t launch_lsq_step_grad(hipStream_t s, const double* px, int64_t nx, const double* pw,
                                int64_t nw, const float* amax_g, const float* step_x,
                                const float* step_w, int log2b, double gx, double gw,
                                float* dstep_x, float* dstep_w, int64_t batch = 1);

}  // namespace hqlss
