// Integer GEMMs of HQ-MM and LSS-MM on gfx950 int8 MFMA, with fused epilogues.
//
//   forward  acc = X^ W^^T               (Sec. 3.3, Procedure HQ-MM step 3), then
//            Y = alpha acc                (step 4, dequantise by s_X s_W / 2^k)
//   dX       acc = A_T W^                 (Sec. 4.2, Eq. 6 on the kept rows), then
//            dX[t] = alpha FWHT_b(acc[t]) (the H^T of the STE gradient, Sec. 4)
//   dW       acc = A_T^T X^_T             (Sec. 4.2, Eq. 5 on the kept rows), then
//            dW = alpha FWHT_b(acc)
//
// CDNA4 has no INT4 matrix instruction, so INT4 codes run on the int8 MFMA
// (v_mfma_i32_32x32x32_i8, int32 accumulation).  Both operands are K-contiguous rows.
// INT4 operands stay packed in HBM and in LDS (half the bytes of int8) and are widened
// after the LDS read with two masks per 32-bit word: (w << 4) & 0xF0F0F0F0 puts the even
// nibbles, w & 0xF0F0F0F0 the odd ones, into the high half of each byte, i.e. 16 x the
// signed code.  The k order inside each group of 8 becomes 0,2,4,6,1,3,5,7; int8 operands
// are stored in that same order by their producer, and since the reduction over k is
// order-free the product is exact.  The factor 16 per INT4 operand is an exact power of
// two, removed by an arithmetic shift before any use.
//
// Tiling: 128 x 128 output tile per 256-thread workgroup (2 x 2 waves of 64 x 64, i.e.
// 2 x 2 MFMA 32x32 tiles per wave), K step 128, LDS double buffer with one barrier per
// step; operand rows are padded (16 bytes int8, 8 bytes packed) so that the 32 rows of a
// fragment read fall on distinct LDS banks.
#include "common.h"
#include "launch.h"

namespace hqlss {

namespace {

typedef int v4i __attribute__((ext_vector_type(4)));
typedef int v16i __attribute__((ext_vector_type(16)));

constexpr int BM = 128, BN = 128, BK = 128, kThreads = 256;

template <bool INT4> struct Op {
  static constexpr int row = INT4 ? BK / 2 : BK;       // bytes per row per K step
  static constexpr int pitch = INT4 ? BK / 2 + 8 : BK + 16;
  static constexpr int chunks = row / 16;              // 16-byte chunks per row
};

// One 16-byte MFMA fragment (16 k values of one row) from LDS at k offset kk.
template <bool INT4>
__device__ __forceinline__ v4i read_frag(const uint8_t* base, int row, int kk) {
  if constexpr (INT4) {
    const uint2 w = *reinterpret_cast<const uint2*>(base + row * Op<true>::pitch + kk / 2);
    v4i r;
    r[0] = (int)((w.x << 4) & 0xF0F0F0F0u);
    r[1] = (int)(w.x & 0xF0F0F0F0u);
    r[2] = (int)((w.y << 4) & 0xF0F0F0F0u);
    r[3] = (int)(w.y & 0xF0F0F0F0u);
    return r;
  } else {
    const uint4 w = *reinterpret_cast<const uint4*>(base + row * Op<false>::pitch + kk);
    v4i r;
    r[0] = (int)w.x; r[1] = (int)w.y; r[2] = (int)w.z; r[3] = (int)w.w;
    return r;
  }
}

__device__ __forceinline__ void fwht8_int(int v[8], int b, int lane) {
  if (b > 1) {
#pragma unroll
    for (int j = 0; j < 8; j += 2) { const int a = v[j], c = v[j + 1]; v[j] = a + c; v[j + 1] = a - c; }
  }
  if (b > 2) {
#pragma unroll
    for (int j = 0; j < 8; ++j)
      if ((j & 2) == 0) { const int a = v[j], c = v[j + 2]; v[j] = a + c; v[j + 2] = a - c; }
  }
  if (b > 4) {
#pragma unroll
    for (int j = 0; j < 4; ++j) { const int a = v[j], c = v[j + 4]; v[j] = a + c; v[j + 4] = a - c; }
  }
  for (int m = 1; m < b / 8; m <<= 1) {  // strides 8..64 across the 16 lanes of a row
    const bool upper = (lane & m) != 0;
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const int p = __shfl_xor(v[j], m);
      v[j] = upper ? (p - v[j]) : (v[j] + p);
    }
  }
}

template <bool A4, bool B4, int EPI, int DT>
__global__ __launch_bounds__(kThreads, 2) void gemm_kernel(GemmArgs g) {
  using OA = Op<A4>;
  using OB = Op<B4>;
  constexpr int A_BUF = BM * OA::pitch, B_BUF = BN * OB::pitch;
  constexpr int STAGE = A_BUF + B_BUF;
  constexpr int E_PITCH = BN + 4;  // int32 epilogue tile pitch
  constexpr bool FWHT_EPI = (EPI == kEpiDx || EPI == kEpiDw);
  constexpr int LDS_OPS = 2 * STAGE;
  constexpr int LDS_EPI = FWHT_EPI ? BM * E_PITCH * 4 : 0;
  constexpr int LDS = LDS_OPS > LDS_EPI ? LDS_OPS : LDS_EPI;
  constexpr int SHIFT = (A4 ? 4 : 0) + (B4 ? 4 : 0);
  constexpr int A_CH = BM * OA::chunks / kThreads;  // 16-byte loads per thread per stage
  constexpr int B_CH = BN * OB::chunks / kThreads;
  __shared__ __attribute__((aligned(16))) uint8_t smem[LDS];

  const int tid = threadIdx.x, lane = tid & 63, wid = tid >> 6;
  const int wm = wid >> 1, wn = wid & 1;
  const int64_t m0 = (int64_t)blockIdx.y * BM, n0 = (int64_t)blockIdx.x * BN;
  int64_t M = g.M;
  if (g.m_dev) {
    const int64_t md = *g.m_dev;
    M = md < M ? md : M;
  }
  if (m0 >= M) return;  // whole workgroup: uniform exit before any barrier
  int64_t K = g.K;
  if (g.k_dev) K = ((int64_t)*g.k_dev + BK - 1) / BK * BK;
  const int64_t Ka = A4 ? K / 2 : K, Kb = B4 ? K / 2 : K;  // row extent in bytes
  const int nk = (int)((K + BK - 1) / BK);
  const uint8_t* __restrict__ gA = static_cast<const uint8_t*>(g.A);
  const uint8_t* __restrict__ gB = static_cast<const uint8_t*>(g.B);

  uint4 ra[A_CH], rb[B_CH];
  auto gload = [&](int kt) {
#pragma unroll
    for (int c = 0; c < A_CH; ++c) {
      const int idx = tid + c * kThreads, r = idx / OA::chunks, cc = idx % OA::chunks;
      const int64_t gm = m0 + r, kb = (int64_t)kt * OA::row + cc * 16;
      ra[c] = (gm < M && kb < Ka) ? *reinterpret_cast<const uint4*>(gA + gm * g.lda + kb)
                                  : make_uint4(0u, 0u, 0u, 0u);
    }
#pragma unroll
    for (int c = 0; c < B_CH; ++c) {
      const int idx = tid + c * kThreads, r = idx / OB::chunks, cc = idx % OB::chunks;
      const int64_t gn = n0 + r, kb = (int64_t)kt * OB::row + cc * 16;
      rb[c] = (gn < g.N && kb < Kb) ? *reinterpret_cast<const uint4*>(gB + gn * g.ldb + kb)
                                    : make_uint4(0u, 0u, 0u, 0u);
    }
  };
  auto sstore = [&](int buf) {
    uint8_t* sa = smem + buf * STAGE;
    uint8_t* sb = sa + A_BUF;
#pragma unroll
    for (int c = 0; c < A_CH; ++c) {
      const int idx = tid + c * kThreads, r = idx / OA::chunks, cc = idx % OA::chunks;
      *reinterpret_cast<uint4*>(sa + r * OA::pitch + cc * 16) = ra[c];
    }
#pragma unroll
    for (int c = 0; c < B_CH; ++c) {
      const int idx = tid + c * kThreads, r = idx / OB::chunks, cc = idx % OB::chunks;
      *reinterpret_cast<uint4*>(sb + r * OB::pitch + cc * 16) = rb[c];
    }
  };

  v16i acc[2][2];
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0;

  const int frow = lane & 31, fk = (lane >> 5) * 16;
  if (nk > 0) {
    gload(0);
    sstore(0);
    __syncthreads();
  }
  for (int kt = 0; kt < nk; ++kt) {
    const int cur = kt & 1;
    if (kt + 1 < nk) gload(kt + 1);
    const uint8_t* sa = smem + cur * STAGE;
    const uint8_t* sb = sa + A_BUF;
#pragma unroll
    for (int s = 0; s < BK / 32; ++s) {
      v4i af[2], bf[2];
#pragma unroll
      for (int i = 0; i < 2; ++i) af[i] = read_frag<A4>(sa, wm * 64 + i * 32 + frow, s * 32 + fk);
#pragma unroll
      for (int j = 0; j < 2; ++j) bf[j] = read_frag<B4>(sb, wn * 64 + j * 32 + frow, s * 32 + fk);
#pragma unroll
      for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_i32_32x32x32_i8(af[i], bf[j], acc[i][j], 0, 0, 0);
    }
    if (kt + 1 < nk) sstore(cur ^ 1);
    __syncthreads();
  }

  // accumulator (i, j, r) <-> tile row wm*64 + i*32 + 8*(r/4) + 4*(lane/32) + r%4,
  //                           tile col wn*64 + j*32 + lane%32
  const int rq = 4 * (lane >> 5), cl = lane & 31;
  if constexpr (EPI == kEpiAcc || EPI == kEpiFwd) {
    float alpha = 0.f;
    if constexpr (EPI == kEpiFwd) alpha = alpha_of(*g.amax1, *g.amax2, g.denom);
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
      for (int j = 0; j < 2; ++j)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int64_t gm = m0 + wm * 64 + i * 32 + 8 * (r >> 2) + rq + (r & 3);
          const int64_t gn = n0 + wn * 64 + j * 32 + cl;
          if (gm < M && gn < g.N) {
            const int v = acc[i][j][r] >> SHIFT;
            if constexpr (EPI == kEpiAcc) static_cast<int32_t*>(g.out)[gm * g.ldo + gn] = v;
            else store1<DT>(g.out, gm * g.ldo + gn, alpha * (float)v);
          }
        }
  } else {
    int* E = reinterpret_cast<int*>(smem);
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
      for (int j = 0; j < 2; ++j)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int row = wm * 64 + i * 32 + 8 * (r >> 2) + rq + (r & 3);
          const int col = wn * 64 + j * 32 + cl;
          E[row * E_PITCH + col] = acc[i][j][r] >> SHIFT;
        }
    __syncthreads();
    const float alpha = alpha_of(*g.amax1, *g.amax2, g.denom);
    const int b = 1 << g.log2b;
    const int cg = tid & 15, rs = tid >> 4;
#pragma unroll 1
    for (int pass = 0; pass < BM / 16; ++pass) {
      const int row = pass * 16 + rs;
      int v[8];
      const int4 x0 = *reinterpret_cast<const int4*>(E + row * E_PITCH + cg * 8);
      const int4 x1 = *reinterpret_cast<const int4*>(E + row * E_PITCH + cg * 8 + 4);
      v[0] = x0.x; v[1] = x0.y; v[2] = x0.z; v[3] = x0.w;
      v[4] = x1.x; v[5] = x1.y; v[6] = x1.z; v[7] = x1.w;
      fwht8_int(v, b, lane);
      const int64_t gm = m0 + row, gn = n0 + cg * 8;
      if (gm < M && gn < g.N) {
        const int64_t orow = (EPI == kEpiDx) ? (int64_t)g.out_rows[gm] : gm;
        float f[8];
#pragma unroll
        for (int j = 0; j < 8; ++j) f[j] = alpha * (float)v[j];
        store_vec<DT, 8>(static_cast<char*>(g.out) + (orow * g.ldo + gn) * Elem<DT>::bytes, f);
      }
    }
  }
}

template <bool A4, bool B4, int EPI, int DT>
hipError_t gemm_t(hipStream_t s, const GemmArgs& g, int id) {
  dim3 grid((unsigned)((g.N + BN - 1) / BN), (unsigned)((g.M + BM - 1) / BM));
  timing_begin(s);
  gemm_kernel<A4, B4, EPI, DT><<<grid, kThreads, 0, s>>>(g);
  timing_end(s, id);
  return hipGetLastError();
}

template <bool A4, bool B4, int EPI>
hipError_t gemm_dt(hipStream_t s, int dt, const GemmArgs& g, int id) {
  switch (dt) {
    case kF32: return gemm_t<A4, B4, EPI, kF32>(s, g, id);
    case kF16: return gemm_t<A4, B4, EPI, kF16>(s, g, id);
    case kBF16: return gemm_t<A4, B4, EPI, kBF16>(s, g, id);
  }
  return hipErrorInvalidValue;
}

}  // namespace

hipError_t launch_gemm(hipStream_t s, int epi, int dt, bool a_int4, bool b_int4,
                       const GemmArgs& g) {
  if (a_int4 && b_int4) {
    if (epi == kEpiFwd) return gemm_dt<true, true, kEpiFwd>(s, dt, g, kKGemmFwd);
    if (epi == kEpiAcc) return gemm_t<true, true, kEpiAcc, kF32>(s, g, kKGemmAcc);
  } else if (!a_int4 && b_int4) {
    if (epi == kEpiDx) return gemm_dt<false, true, kEpiDx>(s, dt, g, kKGemmDx);
    if (epi == kEpiDw) return gemm_dt<false, true, kEpiDw>(s, dt, g, kKGemmDw);
    if (epi == kEpiAcc) return gemm_t<false, true, kEpiAcc, kF32>(s, g, kKGemmAcc);
  }
  return hipErrorInvalidValue;
}

}  // namespace hqlss
