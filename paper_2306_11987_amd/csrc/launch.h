// Host-side launchers of the HQ-MM / LSS-MM kernels (internal to libhqlss).
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace hqlss {

// Kernel ids for the timing log (kept in sync with kernel_name()).
enum KernelId : int {
  kKZero = 0, kKAbsmax, kKQuant, kKTranspose, kKBitSplit, kKPlan, kKBuildAg, kKBuildDw,
  kKGemmFwd, kKGemmDx, kKGemmDw, kKGemmAcc, kKReduce, kKCopy, kKCount
};
const char* kernel_name(int id);

// Every launch goes through this hook so that the timing log can bracket it.
void timing_begin(hipStream_t s);
void timing_end(hipStream_t s, int id);

// Plain device copy of `bytes` (a multiple of 16; both pointers 16-byte aligned).
hipError_t launch_copy(hipStream_t s, const void* src, void* dst, int64_t bytes);

// Zero up to four u32 buffers (counts in 32-bit words).
hipError_t launch_zero(hipStream_t s, uint32_t* p0, int64_t n0, uint32_t* p1 = nullptr,
                       int64_t n1 = 0, uint32_t* p2 = nullptr, int64_t n2 = 0,
                       uint32_t* p3 = nullptr, int64_t n3 = 0);

// max |rows x cols block-FWHT(src)| -> atomicMax into kSlots zeroed slots (kSlotWords
// words, fp32 bit patterns); consumers reduce the slots.
hipError_t launch_fwht_absmax(hipStream_t s, int dt, int log2b, const void* src, int64_t rows,
                              int64_t cols, uint32_t* slots);
// codes of block-FWHT(src) -> packed [rows][cols/2]; optional per-row sum of squares;
// the reduced maximum is also stored to *amax_out.
hipError_t launch_fwht_quant(hipStream_t s, int dt, int log2b, const void* src, int64_t rows,
                             int64_t cols, const uint32_t* slots, float* amax_out,
                             uint8_t* packed, int32_t* row_sumsq);
// packed [rows][cols/2] -> packed [cols][rows/2] (rows, cols multiples of 64).
hipError_t launch_transpose_packed(hipStream_t s, const uint8_t* src, int64_t rows, int64_t cols,
                                   uint8_t* dst);
// bit split of dY [N][C] into two packed code planes and their row sums of squares.
hipError_t launch_bit_split(hipStream_t s, int dt, const void* g, int64_t N, int64_t C,
                            const uint32_t* slots, float* amax_out, uint8_t* qup, uint8_t* qdn,
                            int32_t* sumsq_up, int32_t* sumsq_dn, uint64_t seed,
                            uint64_t offset);
// leverage scores, clamp-rescale, masks, compaction (one workgroup).
hipError_t launch_lss_plan(hipStream_t s, const int32_t* sumsq_up, const int32_t* sumsq_dn,
                           const int32_t* x_sumsq, int64_t N, int64_t budget, uint64_t seed,
                           uint64_t offset, uint8_t* w_up, uint8_t* w_dn, int32_t* kept,
                           int32_t* n_kept);
// Gathered weighted rows A[i] (int8, K-interleaved) for i < round_up(n_kept, 128).
// Also zeroes the rows of dX (if given, dtype dt) that belong to dropped tokens.
hipError_t launch_build_ag(hipStream_t s, int dt, const uint8_t* qup, const uint8_t* qdn,
                           const uint8_t* w_up, const uint8_t* w_dn, const int32_t* kept,
                           const int32_t* n_kept, int64_t N, int64_t C, int64_t D, int8_t* Ag,
                           void* dX);
// A^T [C][Kp] (int8, K-interleaved) and X^_T^T [D][Kp/2] (packed), Kp = round_up(N, 128).
hipError_t launch_build_dw_operands(hipStream_t s, const uint8_t* qup, const uint8_t* qdn,
                                    const uint8_t* w_up, const uint8_t* w_dn,
                                    const int32_t* kept, const int32_t* n_kept,
                                    const uint8_t* xq, int64_t N, int64_t C, int64_t D,
                                    int8_t* At, uint8_t* XtT);

// Integer GEMM  acc[m][n] = sum_k A[m][k] B[n][k]  (both operands K-contiguous rows).
enum Epi : int { kEpiFwd = 0, kEpiDx = 1, kEpiDw = 2, kEpiAcc = 3, kEpiPartial = 4 };
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
};
// Split-K factor the launcher uses for this shape (1 = no split), and the int32 partial
// buffer it then needs (splits x M x N words).  A non-zero override forces the factor.
int gemm_splits(int64_t M, int64_t N, int64_t K, bool a_int4, bool b_int4);
size_t gemm_partial_bytes(int64_t M, int64_t N, int splits);
void gemm_set_split_override(int splits);
hipError_t launch_gemm(hipStream_t s, int epi, int dt, bool a_int4, bool b_int4, const GemmArgs& g,
                       int splits, int32_t* partial);

}  // namespace hqlss
