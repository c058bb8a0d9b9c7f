// Integer GEMMs of HQ-MM and LSS-MM on gfx950 int8 MFMA, with fused epilogues.
//
//   forward  acc = X^ W^^T               (Sec. 3.3, Procedure HQ-MM step 3), then
//            Y = alpha acc                (step 4, dequantise by s_X s_W / 2^k)
//   dX       acc = A_T W^                 (Sec. 4.2, Eq. 6 on the kept rows), then
//            dX[t] = alpha FWHT_b(acc[t]) (the H^T of the STE gradient, Sec. 4)
//   dW       acc = A_T^T X^_T             (Sec. 4.2, Eq. 5 on the kept rows), then
//            dW = alpha FWHT_b(acc)
//
// All three are "NT" products acc[m][n] = sum_k A[m][k] B[n][k] with K-contiguous rows,
// except the A operand of dW: that is A_T itself, stored k-major as the dX product reads
// it, and transposed on its way out of LDS by ds_read_b64_tr_b8 (see gemm_kernel.h).
// CDNA4 has no INT4 matrix instruction, so INT4 codes run on the int8 MFMA
// (v_mfma_i32_32x32x32_i8, int32 accumulation).  INT4 operands stay packed in HBM and in
// LDS and are widened right after the LDS read with two masks per 32-bit word:
// (w << 4) & 0xF0F0F0F0 places the even nibbles, w & 0xF0F0F0F0 the odd ones, in the high
// half of each byte, i.e. 16 x the signed code.  Inside every group of 8 k the register
// order becomes 0,2,4,6,1,3,5,7; int8 operands are stored in that order by their producer,
// and as the reduction over k is order-free the product is exact.  The factor 16 per INT4
// operand is a power of two, removed by an arithmetic shift (or folded into the scale).
//
// Tiling.  Workgroup tile BM x 256 (BM = 128: 4 waves, two workgroups per CU, so every
// SIMD holds two waves and one wave's LDS reads, INT4 widening and epilogue overlap the
// other's MFMAs).  The forward (INT4 x INT4) uses wave tiles of 64 x 128; the gradient
// GEMMs (int8 x INT4) use 128 x 64, as only their n-side operand is widened, or 64 x 128
// for Hadamard blocks of 64 and 128; outputs at most 64 columns wide (attention head
// dimensions) use 64-wide workgroup tiles.  128 int32 accumulators per lane.  The MFMA
// "A" operand carries the n rows and the "B" operand the m rows, so that a lane's
// accumulators run along n: lane l, MFMA tile (i, j), register r holds m = 32 i + (l % 32)
// and n = 16 j + r + (WN / 2) (l / 32) of the wave tile.  This is arranged by the order in
// which the B rows are placed in LDS.  Each lane then owns 16 consecutive n per (i, j),
// and the gradient epilogue's Hadamard transform along n runs in registers, pairing lanes
// l and l ^ 32 for the widest stride.
//
// Main loop.  K advances in stages of 128; operands move from HBM/L2 straight into LDS
// with 16-byte LDS-DMA loads (no register staging), NBUF stages deep, so each stage's
// loads are in flight while the previous one or two are multiplied.  Rows sit in LDS
// without padding, their 16-byte chunks XOR-swizzled by row so that the fragment reads
// (32 rows x one chunk per instruction) hit distinct banks.  A stage boundary is one
// wait on this wave's own loads plus one barrier.
// Epilogue: results are staged through LDS in row chunks so that each store instruction
// writes contiguous 16-byte pieces of whole output rows.  The learned-step gradient
// epilogues first sum acc * delta (fp64) and zero the clipped accumulators (App. A.3).
// Grid z is either the split-K index (int32 partial tiles, summed by reduce_epilogue) or
// the batch of a batched launch (per-batch operand and output strides).  Workgroups take
// tiles in an XCD-aware order over the tiles with rows below the device-side row count.
#include "gemm_kernel.h"

namespace hqlss {

namespace {

template <int DT, int MODE>
__global__ __launch_bounds__(256) void reduce_epilogue_kernel(const int32_t* __restrict__ P, int S,
                                                              GemmArgs g) {
  const int lane = threadIdx.x & 63;
  int64_t M = g.M;
  if (g.m_dev) {
    const int64_t md = *g.m_dev;
    M = md < M ? md : M;
  }
  const uint32_t chunks = (uint32_t)((g.N + 511) / 512);
  const uint32_t items = (uint32_t)M * chunks;
  const uint32_t nw = gridDim.x * 4;
  constexpr bool LSQ = (MODE == kEpiDxL || MODE == kEpiDwL);
  constexpr bool GRAD = (MODE == kEpiDx || MODE == kEpiDw || LSQ);
  constexpr bool ROWMAP = (MODE == kEpiDx || MODE == kEpiDxL);
  float alpha = 0.f;
  if constexpr (MODE != kEpiAcc) alpha = scale_of(g);
  double lsq_sum = 0.0;
  const int b = 1 << g.log2b;
  const int64_t plane = g.M * g.ldo;
  for (uint32_t it = blockIdx.x * 4 + (threadIdx.x >> 6); it < items; it += nw) {
    const int64_t m = it / chunks;
    const int64_t n = (int64_t)(it - (uint32_t)m * chunks) * 512 + lane * 8;
    const bool live = n < g.N;
    int v[8] = {0, 0, 0, 0, 0, 0, 0, 0};
    if (live) {
      for (int z = 0; z < S; ++z) {
        const int32_t* p = P + z * plane + m * g.ldo + n;
        const uint4 u0 = ld_stream<HQ_NT_R_LD>(p), u1 = ld_stream<HQ_NT_R_LD>(p + 4);
        const int4 x0 = make_int4((int)u0.x, (int)u0.y, (int)u0.z, (int)u0.w);
        const int4 x1 = make_int4((int)u1.x, (int)u1.y, (int)u1.z, (int)u1.w);
        v[0] += x0.x; v[1] += x0.y; v[2] += x0.z; v[3] += x0.w;
        v[4] += x1.x; v[5] += x1.y; v[6] += x1.z; v[7] += x1.w;
      }
      if constexpr (LSQ) {  // as in the GEMM epilogue: sum acc * delta, then the mask
        const int64_t drow = ROWMAP ? (int64_t)g.out_rows[m] : m;
        const uint4 d = ld_stream<true>(g.delta + drow * g.ldo + n);
        const uint32_t dw[4] = {d.x, d.y, d.z, d.w};
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          const uint32_t h = (dw[e >> 1] >> (16 * (e & 1))) & 0xFFFFu;
          lsq_sum += (double)v[e] * f16_bits_to_double(h);
          v[e] = inside_of(h) ? v[e] : 0;
        }
      }
    }
    if constexpr (GRAD) {
      if (b > 1) {
#pragma unroll
        for (int e = 0; e < 8; e += 2) { const int a = v[e], c = v[e + 1]; v[e] = a + c; v[e + 1] = a - c; }
      }
      if (b > 2) {
#pragma unroll
        for (int e = 0; e < 8; ++e)
          if ((e & 2) == 0) { const int a = v[e], c = v[e + 2]; v[e] = a + c; v[e + 2] = a - c; }
      }
      if (b > 4) {
#pragma unroll
        for (int e = 0; e < 4; ++e) { const int a = v[e], c = v[e + 4]; v[e] = a + c; v[e + 4] = a - c; }
      }
      for (int mk = 1; mk < b / 8; mk <<= 1) {
        const bool upper = (lane & mk) != 0;
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          const int p = __shfl_xor(v[e], mk);
          v[e] = upper ? (p - v[e]) : (v[e] + p);
        }
      }
    }
    if (!live) continue;
    if constexpr (MODE == kEpiAcc) {
      int32_t* p = static_cast<int32_t*>(g.out) + m * g.ldo + n;
      st_stream<HQ_NT_G_ST>(p, make_uint4((uint32_t)v[0], (uint32_t)v[1], (uint32_t)v[2], (uint32_t)v[3]));
      st_stream<HQ_NT_G_ST>(p + 4, make_uint4((uint32_t)v[4], (uint32_t)v[5], (uint32_t)v[6], (uint32_t)v[7]));
    } else {
      const int64_t orow = ROWMAP ? (int64_t)g.out_rows[m] : m;
      float f[8];
#pragma unroll
      for (int e = 0; e < 8; ++e) f[e] = alpha * (float)v[e];
      store8_stream<DT, HQ_NT_G_ST>(static_cast<char*>(g.out) + (orow * g.ldo + n) * Elem<DT>::bytes, f);
    }
  }
  if constexpr (LSQ) {
    __shared__ double red[4];
    const double t = block_sum_f64<256>(lsq_sum, red);
    if (threadIdx.x == 0) g.ds_part[blockIdx.x] = t;
  }
}

// Step-size gradients (App. A.3): ds = g(s) alpha sum(acc * delta) in fp64 over the
// per-workgroup partials, summed by one workgroup in a fixed order (deterministic).
__global__ __launch_bounds__(256) void lsq_step_grad_kernel(const double* __restrict__ px, int64_t nx,
                                                            const double* __restrict__ pw, int64_t nw,
                                                            const float* __restrict__ amax_g,
                                                            const float* __restrict__ step_x,
                                                            const float* __restrict__ step_w, int log2b,
                                                            double gx, double gw,
                                                            float* __restrict__ dstep_x,
                                                            float* __restrict__ dstep_w) {
  __shared__ double red[4];
  {  // block b: batch b of a batched call
    const int64_t bt = blockIdx.x;
    px += bt * nx;
    pw += bt * nw;
    amax_g += bt;
    step_x += bt;
    step_w += bt;
    dstep_x += bt;
    dstep_w += bt;
  }
  double sx = 0.0, sw = 0.0;
  for (int64_t i = threadIdx.x; i < nx; i += 256) sx += px[i];
  for (int64_t i = threadIdx.x; i < nw; i += 256) sw += pw[i];
  sx = block_sum_f64<256>(sx, red);
  __syncthreads();
  sw = block_sum_f64<256>(sw, red);
  if (threadIdx.x == 0) {
    const double s_dn = (double)step_of(__float_as_uint(*amax_g)) / (double)kBsRatio;
    const double pk = 1.0 / (double)(1 << log2b);
    if (nx > 0) *dstep_x = (float)(gx * (s_dn * (double)*step_w * pk) * sx);
    if (nw > 0) *dstep_w = (float)(gw * (s_dn * (double)*step_x * pk) * sw);
  }
}

// wave tile width: int8 x INT4 GEMMs widen only the n-side operand, so their waves take
// 128 m x 64 n (half the widening per MFMA) unless the Hadamard block spans 64 or 128
// columns (the in-register transform then needs no lane exchange)
int64_t reduce_grid(int64_t M, int64_t N) {
  const int64_t items = M * ((N + 511) / 512);
  int64_t wg = (items + 3) / 4;
  if (wg > 2048) wg = 2048;
  return wg < 1 ? 1 : wg;
}

// Test hooks, per calling thread (a forced width or split-K factor set by one thread
// never reaches another thread's calls): 128 or 256 forces that width (0: the rules below).
thread_local int g_bn_override = 0;

// Workgroup tile width of a gradient GEMM: 64 for outputs at most 64 wide; 128 when the
// 256-wide tiles would fill at most three quarters of one round of two workgroups per CU
// (most CUs would then hold a single workgroup, whose MFMA issue is about half as dense);
// else 256.
int grad_bn(int64_t M, int64_t N, int splits) {
  if (splits > 1) return kBN;
  if (N <= kNarrowBN) return kNarrowBN;
  if (g_bn_override) return g_bn_override;
  const int64_t bm = tile_m<false>();
  const int64_t t256 = ((M + bm - 1) / bm) * ((N + kBN - 1) / kBN);
  return 4 * t256 <= 3 * 512 ? kMidBN : kBN;  // 512 = two workgroups on each of 256 CUs
}

// Tile width of a forward (INT4 x INT4) GEMM by the same rule, the tiles of all batches
// counted; its 128-wide tiles use 64 x 64 wave tiles.
int fwd_bn(int64_t M, int64_t N, int splits, int64_t batch) {
  if (splits > 1) return kBN;
  if (g_bn_override) return g_bn_override;
  const int64_t bm = tile_m<true>();
  const int64_t t256 = ((M + bm - 1) / bm) * ((N + kBN - 1) / kBN) * (batch > 0 ? batch : 1);
  return 4 * t256 <= 3 * 512 ? kMidBN : kBN;
}

// the Hadamard block is a template parameter of the gradient epilogues
template <int BM, bool A4, int EPI, int DT, bool TRA = false>
hipError_t gemm_b(hipStream_t s, const GemmArgs& g, int splits, int id) {
  if constexpr (EPI == kEpiDx || EPI == kEpiDw || EPI == kEpiDxL || EPI == kEpiDwL) {
    const int bn = grad_bn(g.M, g.N, splits);
    if (bn == kMidBN) {
      switch (g.log2b) {
        case 0: return gemm_t<BM, A4, EPI, DT, 0, kMidBN, false, 0, TRA>(s, g, splits, id);
        case 1: return gemm_t<BM, A4, EPI, DT, 1, kMidBN, false, 0, TRA>(s, g, splits, id);
        case 2: return gemm_t<BM, A4, EPI, DT, 2, kMidBN, false, 0, TRA>(s, g, splits, id);
        case 3: return gemm_t<BM, A4, EPI, DT, 3, kMidBN, false, 0, TRA>(s, g, splits, id);
        case 4: return gemm_t<BM, A4, EPI, DT, 4, kMidBN, false, 0, TRA>(s, g, splits, id);
        case 5: return gemm_t<BM, A4, EPI, DT, 5, kMidBN, false, 0, TRA>(s, g, splits, id);
        case 6: return gemm_t<BM, A4, EPI, DT, 6, kMidBN, false, 0, TRA>(s, g, splits, id);
        case 7: return gemm_t<BM, A4, EPI, DT, 7, kMidBN, false, 0, TRA>(s, g, splits, id);
      }
      return hipErrorInvalidValue;
    }
    if (bn == kNarrowBN) {  // narrow output: blocks of at most 64 columns
      switch (g.log2b) {
        case 0: return gemm_t<BM, A4, EPI, DT, 0, kNarrowBN, false, 0, TRA>(s, g, splits, id);
        case 1: return gemm_t<BM, A4, EPI, DT, 1, kNarrowBN, false, 0, TRA>(s, g, splits, id);
        case 2: return gemm_t<BM, A4, EPI, DT, 2, kNarrowBN, false, 0, TRA>(s, g, splits, id);
        case 3: return gemm_t<BM, A4, EPI, DT, 3, kNarrowBN, false, 0, TRA>(s, g, splits, id);
        case 4: return gemm_t<BM, A4, EPI, DT, 4, kNarrowBN, false, 0, TRA>(s, g, splits, id);
        case 5: return gemm_t<BM, A4, EPI, DT, 5, kNarrowBN, false, 0, TRA>(s, g, splits, id);
        case 6: return gemm_t<BM, A4, EPI, DT, 6, kNarrowBN, false, 0, TRA>(s, g, splits, id);
      }
      return hipErrorInvalidValue;
    }
    switch (g.log2b) {
      case 0: return gemm_t<BM, A4, EPI, DT, 0, kBN, false, 0, TRA>(s, g, splits, id);
      case 1: return gemm_t<BM, A4, EPI, DT, 1, kBN, false, 0, TRA>(s, g, splits, id);
      case 2: return gemm_t<BM, A4, EPI, DT, 2, kBN, false, 0, TRA>(s, g, splits, id);
      case 3: return gemm_t<BM, A4, EPI, DT, 3, kBN, false, 0, TRA>(s, g, splits, id);
      case 4: return gemm_t<BM, A4, EPI, DT, 4, kBN, false, 0, TRA>(s, g, splits, id);
      case 5: return gemm_t<BM, A4, EPI, DT, 5, kBN, false, 0, TRA>(s, g, splits, id);
      case 6: return gemm_t<BM, A4, EPI, DT, 6, kBN, false, 0, TRA>(s, g, splits, id);
      case 7: return gemm_t<BM, A4, EPI, DT, 7, kBN, false, 0, TRA>(s, g, splits, id);
    }
    return hipErrorInvalidValue;
  } else {
    if (fwd_bn(g.M, g.N, splits, g.batch) == kMidBN) return gemm_t<BM, A4, EPI, DT, 0, kMidBN, false, 0, TRA>(s, g, splits, id);
    return gemm_t<BM, A4, EPI, DT, 0, kBN, false, 0, TRA>(s, g, splits, id);
  }
}

template <int DT, int MODE>
hipError_t reduce_t(hipStream_t s, const int32_t* P, int S, const GemmArgs& g) {
  const int64_t wg = reduce_grid(g.M, g.N);
  timing_begin(s);
  reduce_epilogue_kernel<DT, MODE><<<(int)wg, 256, 0, s>>>(P, S, g);
  timing_end(s, kKReduce);
  return hipGetLastError();
}

// TRA: A stored k-major (GemmArgs::a_kmajor)
template <bool A4, int EPI, int DT, bool TRA = false>
hipError_t run(hipStream_t s, const GemmArgs& g, int splits, int32_t* partial, int id) {
  constexpr int BM = tile_m<A4>();
  if (splits <= 1) return gemm_b<BM, A4, EPI, DT, TRA>(s, g, 1, id);
  GemmArgs p = g;
  p.out = partial;
  p.ldo = g.N;
  hipError_t e = split_mid(A4, g.N) ? gemm_t<BM, A4, kEpiPartial, DT, 0, kMidBN, false, 0, TRA>(s, p, splits, id)
                                     : gemm_t<BM, A4, kEpiPartial, DT, 0, kBN, false, 0, TRA>(s, p, splits, id);
  if (e != hipSuccess) return e;
  return reduce_t<DT, EPI>(s, partial, splits, g);
}

template <bool A4, int EPI, bool TRA = false>
hipError_t run_dt(hipStream_t s, int dt, const GemmArgs& g, int splits, int32_t* partial, int id) {
  switch (dt) {
    case kF32: return run<A4, EPI, kF32, TRA>(s, g, splits, partial, id);
    case kF16: return run<A4, EPI, kF16, TRA>(s, g, splits, partial, id);
    case kBF16: return run<A4, EPI, kBF16, TRA>(s, g, splits, partial, id);
  }
  return hipErrorInvalidValue;
}

}  // namespace

int gemm_fwd_bn(int64_t M, int64_t N, int splits, int64_t batch) { return fwd_bn(M, N, splits, batch); }
int gemm_grad_bn(int64_t M, int64_t N, int splits) { return grad_bn(M, N, splits); }

hipError_t launch_gemm_reduce(hipStream_t s, int epi, int dt, const int32_t* P, int S, const GemmArgs& g) {
  switch (epi) {
    case kEpiAcc: return reduce_t<kF32, kEpiAcc>(s, P, S, g);
    case kEpiFwd:
      switch (dt) {
        case kF32: return reduce_t<kF32, kEpiFwd>(s, P, S, g);
        case kF16: return reduce_t<kF16, kEpiFwd>(s, P, S, g);
        case kBF16: return reduce_t<kBF16, kEpiFwd>(s, P, S, g);
      }
      break;
    case kEpiDx:
      switch (dt) {
        case kF32: return reduce_t<kF32, kEpiDx>(s, P, S, g);
        case kF16: return reduce_t<kF16, kEpiDx>(s, P, S, g);
        case kBF16: return reduce_t<kBF16, kEpiDx>(s, P, S, g);
      }
      break;
    case kEpiDw:
      switch (dt) {
        case kF32: return reduce_t<kF32, kEpiDw>(s, P, S, g);
        case kF16: return reduce_t<kF16, kEpiDw>(s, P, S, g);
        case kBF16: return reduce_t<kBF16, kEpiDw>(s, P, S, g);
      }
      break;
  }
  return hipErrorInvalidValue;
}

static thread_local int g_split_override = 0;
void gemm_set_split_override(int splits) { g_split_override = splits < 0 ? 0 : splits; }
int gemm_split_override() { return g_split_override; }
void gemm_set_tile_override(int bn) { g_bn_override = (bn == kMidBN || bn == kBN) ? bn : 0; }

int gemm_splits(int64_t M, int64_t N, int64_t K, bool a_int4, bool b_int4) {
  (void)b_int4;
  if (g_split_override) return g_split_override;
  const int64_t bm = a_int4 ? tile_m<true>() : tile_m<false>();
  const int64_t slots = bm == 128 ? 512 : 256;  // workgroups in flight
  const int64_t bn = split_mid(a_int4, N) ? kMidBN : kBN;
  const int64_t tiles = ((M + bm - 1) / bm) * ((N + bn - 1) / bn);
  const int64_t stages = (K + kKS - 1) / kKS;
  if (2 * tiles >= slots || stages < 16) return 1;
  int64_t s = slots / tiles;        // all splits resident at once (no second round)
  const int64_t smax = stages / 8;  // keep >= 8 stages per split
  if (s > smax) s = smax;
  return (int)(s < 1 ? 1 : s);
}

size_t gemm_partial_bytes(int64_t M, int64_t N, int splits) {
  return splits > 1 ? (size_t)splits * M * N * 4 : 0;
}

hipError_t launch_gemm(hipStream_t s, int epi, int dt, bool a_int4, bool b_int4, const GemmArgs& g,
                       int splits, int32_t* partial) {
  if (!b_int4) return hipErrorInvalidValue;
  if (a_int4) {
    if (epi == kEpiFwd) return run_dt<true, kEpiFwd>(s, dt, g, splits, partial, kKGemmFwd);
    if (epi == kEpiAcc) return run<true, kEpiAcc, kF32>(s, g, splits, partial, kKGemmAcc);
  } else if (g.a_kmajor) {
    if (epi == kEpiDw) return run_dt<false, kEpiDw, true>(s, dt, g, splits, partial, kKGemmDw);
    if (epi == kEpiDwL) return run_dt<false, kEpiDwL, true>(s, dt, g, splits, partial, kKGemmDw);
    if (epi == kEpiAcc) return run<false, kEpiAcc, kF32, true>(s, g, splits, partial, kKGemmAcc);
  } else {
    if (epi == kEpiDx) return run_dt<false, kEpiDx>(s, dt, g, splits, partial, kKGemmDx);
    if (epi == kEpiDw) return run_dt<false, kEpiDw>(s, dt, g, splits, partial, kKGemmDw);
    if (epi == kEpiDxL) return run_dt<false, kEpiDxL>(s, dt, g, splits, partial, kKGemmDx);
    if (epi == kEpiDwL) return run_dt<false, kEpiDwL>(s, dt, g, splits, partial, kKGemmDw);
    if (epi == kEpiAcc) return run<false, kEpiAcc, kF32>(s, g, splits, partial, kKGemmAcc);
  }
  return hipErrorInvalidValue;
}

int64_t gemm_epi_parts(int64_t M, int64_t N, int splits) {
  if (splits <= 1) {
    const int64_t bm = tile_m<false>();
    const int64_t bn = grad_bn(M, N, splits);  // as gemm_b chooses
    return ((N + bn - 1) / bn) * ((M + bm - 1) / bm);
  }
  return reduce_grid(M, N);
}

hipError_t launch_lsq_step_grad(hipStream_t s, const double* px, int64_t nx, const double* pw,
                                int64_t nw, const float* amax_g, const float* step_x,
                                const float* step_w, int log2b, double gx, double gw,
                                float* dstep_x, float* dstep_w, int64_t batch) {
  timing_begin(s);
  lsq_step_grad_kernel<<<(unsigned)batch, 256, 0, s>>>(px, nx, pw, nw, amax_g, step_x, step_w, log2b,
                                                       gx, gw, dstep_x, dstep_w);
  timing_end(s, kKLsqStepGrad);
  return hipGetLastError();
}

}  // namespace hqlss
