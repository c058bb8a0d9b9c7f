// The GEMMs of HQ-MM on the FP6 MFMA of gfx950 (v_mfma_f32_32x32x64_f8f6f4, e2m3 operands).
//
// Every INT4 code |q| <= 7 is exact in e2m3 (1, 2, 3 = 1.5 x 2, 4, 5 = 1.25 x 4, 6, 7 =
// 1.75 x 4), a product of two codes is an integer of at most 49, and the fp32 accumulator
// of a K-long dot product holds integers of at most 49 K < 2^24: exact.  So the FP6 route
// reaches the int8 route's int32 accumulators bit for bit at twice the MFMA rate, with
// operands of one byte per code (the padded layout of fp6.hip) in place of half a byte.
// Kernel and epilogues are the int8 route's (gemm_kernel.h) with the FP6 main loop.
#include "gemm_kernel.h"

namespace hqlss {

namespace {

// FP6 workgroup tiles: 256 x 256, one workgroup of 8 waves per CU, stages of 128 k.
constexpr int kBM6 = 256;

template <int F6K, int EPI, int DT, int LOG2B>
hipError_t run6(hipStream_t s, const GemmArgs& g, int splits, int32_t* partial, int id) {
  if (splits <= 1) return gemm_t<kBM6, true, EPI, DT, LOG2B, kBN, true, F6K>(s, g, 1, id);
  GemmArgs p = g;
  p.out = partial;
  p.ldo = g.N;
  hipError_t e = gemm_t<kBM6, true, kEpiPartial, DT, 0, kBN, true, F6K>(s, p, splits, id);
  if (e != hipSuccess) return e;
  return launch_gemm_reduce(s, EPI, DT, partial, splits, g);
}

// the Hadamard block is a template parameter of the gradient epilogues
template <int F6K, int EPI, int DT>
hipError_t run6_b(hipStream_t s, const GemmArgs& g, int splits, int32_t* partial, int id) {
  switch (g.log2b) {
    case 0: return run6<F6K, EPI, DT, 0>(s, g, splits, partial, id);
    case 1: return run6<F6K, EPI, DT, 1>(s, g, splits, partial, id);
    case 2: return run6<F6K, EPI, DT, 2>(s, g, splits, partial, id);
    case 3: return run6<F6K, EPI, DT, 3>(s, g, splits, partial, id);
    case 4: return run6<F6K, EPI, DT, 4>(s, g, splits, partial, id);
    case 5: return run6<F6K, EPI, DT, 5>(s, g, splits, partial, id);
    case 6: return run6<F6K, EPI, DT, 6>(s, g, splits, partial, id);
    case 7: return run6<F6K, EPI, DT, 7>(s, g, splits, partial, id);
  }
  return hipErrorInvalidValue;
}

template <int F6K, int EPI>
hipError_t run6_dt(hipStream_t s, int dt, const GemmArgs& g, int splits, int32_t* partial, int id) {
  switch (dt) {
    case kF32: return run6_b<F6K, EPI, kF32>(s, g, splits, partial, id);
    case kF16: return run6_b<F6K, EPI, kF16>(s, g, splits, partial, id);
    case kBF16: return run6_b<F6K, EPI, kBF16>(s, g, splits, partial, id);
  }
  return hipErrorInvalidValue;
}

}  // namespace

int gemm6_splits(int64_t M, int64_t N, int64_t K) {
  const int forced = gemm_split_override();
  if (forced) return forced;
  const int64_t slots = 256;  // one workgroup per CU
  const int64_t tiles = ((M + kBM6 - 1) / kBM6) * ((N + kBN - 1) / kBN);
  const int64_t stages = (K + 127) / 128;
  if (2 * tiles >= slots || stages < 16) return 1;
  int64_t sp = slots / tiles;          // all splits resident at once
  const int64_t smax = stages / 8;     // keep >= 8 stages per split
  if (sp > smax) sp = smax;
  return (int)(sp < 1 ? 1 : sp);
}

hipError_t launch_gemm6(hipStream_t s, int epi, int dt, const GemmArgs& g, int splits, int32_t* partial) {
  if (g.f6_kind == kF6Dx) {
    if (epi == kEpiAcc) return run6<kF6Dx, kEpiAcc, kF32, 0>(s, g, splits, partial, kKGemmAcc);
    if (epi == kEpiDx) return run6_dt<kF6Dx, kEpiDx>(s, dt, g, splits, partial, kKGemmDx);
    return hipErrorInvalidValue;
  }
  if (g.f6_kind == kF6Dw) {
    if (epi == kEpiAcc) return run6<kF6Dw, kEpiAcc, kF32, 0>(s, g, splits, partial, kKGemmAcc);
    if (epi == kEpiDw) return run6_dt<kF6Dw, kEpiDw>(s, dt, g, splits, partial, kKGemmDw);
    return hipErrorInvalidValue;
  }
  if (epi == kEpiAcc) return run6<0, kEpiAcc, kF32, 0>(s, g, splits, partial, kKGemmAcc);
  if (epi == kEpiFwd) {
    switch (dt) {
      case kF32: return run6<0, kEpiFwd, kF32, 0>(s, g, splits, partial, kKGemmFwd);
      case kF16: return run6<0, kEpiFwd, kF16, 0>(s, g, splits, partial, kKGemmFwd);
      case kBF16: return run6<0, kEpiFwd, kBF16, 0>(s, g, splits, partial, kKGemmFwd);
    }
  }
  return hipErrorInvalidValue;
}

}  // namespace hqlss
