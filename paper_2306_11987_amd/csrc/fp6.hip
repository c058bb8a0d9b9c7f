// FP6 (e2m3) operands of the FP6 MFMA route (gemm6.hip).
//
// Padded FP6 layout of a row of K codes (K a multiple of 64): K bytes, every 32 codes one
// 32-byte group holding 24 bytes of e2m3 fields (code i of the group at bits 6i..6i+5 of the
// group read as a little-endian 192-bit string) and 8 zero bytes.  A lane of the MFMA reads
// one such group as its 32 k of one row; the zero bytes keep every group on a 32-byte
// boundary, so the GEMM's 16-byte LDS-DMA loads and swizzled LDS reads are those of the
// INT4 layout at twice the bytes.
//
// e2m3: sign, 2 exponent bits (bias 1), 3 mantissa bits; the integers 1..7 are
// 1.0 x 2^0, 1.0 x 2^1, 1.5 x 2^1, 1.0 x 2^2, 1.25 x 2^2, 1.5 x 2^2, 1.75 x 2^2.
#include "common.h"
#include "launch.h"

namespace hqlss {

namespace {

// e2m3 magnitude byte of |q| = 0..7
constexpr uint64_t kE2m3Mag = 0x1E1C1A1814100800ull;

__device__ __forceinline__ uint32_t e2m3_of_nibble(uint32_t n) {  // two's complement nibble
  const uint32_t neg = n >> 3;
  const uint32_t a = neg ? 16u - n : n;  // |q| (q = -8 does not occur)
  return (uint32_t)((kE2m3Mag >> (8 * a)) & 0xFFu) | (neg << 5);
}

// 16 bytes of packed INT4 (32 codes, even k in the low nibble) -> one 32-byte FP6 group
__device__ __forceinline__ void fp6_group(const uint4& in, uint4& lo, uint4& hi) {
  const uint32_t w[4] = {in.x, in.y, in.z, in.w};
  uint32_t o[8] = {0, 0, 0, 0, 0, 0, 0, 0};
#pragma unroll
  for (int i = 0; i < 32; ++i) {
    const uint32_t f = e2m3_of_nibble((w[i >> 3] >> (4 * (i & 7))) & 15u);
    const int bit = 6 * i, d = bit >> 5, sh = bit & 31;
    o[d] |= f << sh;
    if (sh > 26) o[d + 1] |= f >> (32 - sh);
  }
  lo = make_uint4(o[0], o[1], o[2], o[3]);
  hi = make_uint4(o[4], o[5], 0u, 0u);
}

__global__ __launch_bounds__(256) void int4_to_fp6_kernel(const uint8_t* __restrict__ src,
                                                          uint8_t* __restrict__ dst, int64_t rows,
                                                          int64_t K) {
  const int64_t groups = K / 32, items = rows * groups;
  for (int64_t it = (int64_t)blockIdx.x * 256 + threadIdx.x; it < items; it += (int64_t)gridDim.x * 256) {
    const int64_t r = it / groups, g = it - r * groups;
    const uint4 in = ld_stream<true>(src + r * (K / 2) + g * 16);
    uint4 lo, hi;
    fp6_group(in, lo, hi);
    uint8_t* p = dst + r * K + g * 32;
    *reinterpret_cast<uint4*>(p) = lo;
    *reinterpret_cast<uint4*>(p + 16) = hi;
  }
}

// e2m3 field of an integer code |q| <= 7
__device__ __forceinline__ uint32_t e2m3_of_int(int q) {
  const uint32_t a = (uint32_t)(q < 0 ? -q : q);
  return (uint32_t)((kE2m3Mag >> (8 * a)) & 0xFFu) | (q < 0 ? 0x20u : 0u);
}
// the integer of an e2m3 field that holds one (|v| = (8 + m) >> (4 - e), 0 for e = 0)
__device__ __forceinline__ int int_of_e2m3(uint32_t f) {
  const uint32_t e = (f >> 3) & 3u, m = f & 7u;
  const int a = e ? (int)((8u + m) >> (4u - e)) : 0;
  return (f & 0x20u) ? -a : a;
}

// 32 integer codes -> one 32-byte FP6 group (24 bytes of fields, 8 zero bytes)
__device__ __forceinline__ void fp6_pack32(const int* q, uint4& lo, uint4& hi) {
  uint32_t o[6] = {0, 0, 0, 0, 0, 0};
#pragma unroll
  for (int i = 0; i < 32; ++i) {
    const uint32_t f = e2m3_of_int(q[i]);
    const int bit = 6 * i, d = bit >> 5, sh = bit & 31;
    o[d] |= f << sh;
    if (sh > 26) o[d + 1] |= f >> (32 - sh);
  }
  lo = make_uint4(o[0], o[1], o[2], o[3]);
  hi = make_uint4(o[4], o[5], 0u, 0u);
}

// dX operands: one thread per (row, 32-code group); blockIdx.y 0: lower rows, 1: upper rows
template <int DT>
__global__ __launch_bounds__(256) void fp6_build_rows_kernel(
    const uint8_t* __restrict__ qup, const uint8_t* __restrict__ qdn, const uint8_t* __restrict__ w_dn,
    const int32_t* __restrict__ order6, const int32_t* __restrict__ n_kept,
    const int32_t* __restrict__ n_up, int64_t C, uint8_t* __restrict__ a_dn, uint8_t* __restrict__ a_up) {
  const bool upper = blockIdx.y == 1;
  uint8_t* out = upper ? a_up : a_dn;
  if (!out) return;
  const int64_t nu = *n_up;
  const int64_t rows = upper ? (nu + 255) / 256 * 256 : (int64_t)*n_kept;
  const int64_t groups = C / 32, items = rows * groups;
  for (int64_t it = (int64_t)blockIdx.x * 256 + threadIdx.x; it < items; it += (int64_t)gridDim.x * 256) {
    const int64_t r = it / groups, g = it - r * groups;
    uint4 in = make_uint4(0u, 0u, 0u, 0u);
    if (!upper || r < nu) {
      const int64_t t = order6[r];
      if (upper || w_dn[t]) in = ld_stream<true>((upper ? qup : qdn) + t * (C / 2) + g * 16);
    }
    int q[32];
#pragma unroll
    for (int i = 0; i < 32; ++i) {
      const uint32_t n = ((i < 8 ? in.x : i < 16 ? in.y : i < 24 ? in.z : in.w) >> (4 * (i & 7))) & 15u;
      q[i] = (int)n - (n >= 8 ? 16 : 0);
    }
    uint4 lo, hi;
    fp6_pack32(q, lo, hi);
    uint8_t* p = out + r * C + g * 32;
    *reinterpret_cast<uint4*>(p) = lo;
    *reinterpret_cast<uint4*>(p + 16) = hi;
  }
}

// dW operands, transposed through an LDS tile of 128 entries x 128 columns: blockIdx.x is
// the entry block, blockIdx.y the column block (C / 128 blocks of a_dw, then D / 128 of
// x_dw; a last partial block of 64 columns is allowed).  The last y block zeroes the dX
// rows of dropped tokens instead.
template <int DT>
__global__ __launch_bounds__(256) void fp6_build_cols_kernel(
    const uint8_t* __restrict__ qup, const uint8_t* __restrict__ qdn, const uint8_t* __restrict__ w_up,
    const uint8_t* __restrict__ w_dn, const int32_t* __restrict__ ent, const int32_t* __restrict__ cls,
    const uint8_t* __restrict__ xq6, int64_t N, int64_t C, int64_t D, int64_t ecap,
    uint8_t* __restrict__ a_dw, uint8_t* __restrict__ x_dw, void* __restrict__ dX) {
  __shared__ int8_t tile[128][128 + 4];
  const int tid = threadIdx.x;
  const int64_t cb = (C + 127) / 128, db = (D + 127) / 128;
  if ((int64_t)blockIdx.y == cb + db) {  // zero the dX rows of dropped tokens
    if (!dX) return;
    const int64_t bytes = D * Elem<DT>::bytes;
    const int64_t t0 = (int64_t)blockIdx.x * 128, t1 = t0 + 128 < N ? t0 + 128 : N;
    for (int64_t t = t0 + (tid >> 6); t < t1; t += 4) {
      if (w_up[t] + w_dn[t]) continue;
      char* row = static_cast<char*>(dX) + t * bytes;
      for (int64_t o = (tid & 63) * 16; o < bytes; o += 64 * 16)
        st_stream<HQ_NT_B_ST>(row + o, make_uint4(0u, 0u, 0u, 0u));
    }
    return;
  }
  const bool isA = (int64_t)blockIdx.y < cb;
  uint8_t* out = isA ? a_dw : x_dw;
  if (!out) return;
  const int64_t e0 = (int64_t)blockIdx.x * 128;
  if (e0 >= (int64_t)cls[4]) return;
  const int64_t col0 = isA ? (int64_t)blockIdx.y * 128 : ((int64_t)blockIdx.y - cb) * 128;
  const int64_t ncol = isA ? C : D;
  // 128 entries x 8 chunks of 16 columns, four per thread
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    const int item = tid + 256 * k, r = item >> 3, qc = (item & 7) * 16;
    int v[16];
#pragma unroll
    for (int j = 0; j < 16; ++j) v[j] = 0;
    const int id = ent[e0 + r];
    if (id >= 0 && col0 + qc < ncol) {
      const int64_t t = id >> 1;
      if (isA) {
        const uint2 w = ld_stream2<HQ_NT_B_LD>(((id & 1) ? qup : qdn) + t * (C / 2) + (col0 + qc) / 2);
#pragma unroll
        for (int j = 0; j < 16; ++j) {
          const uint32_t n = ((j < 8 ? w.x : w.y) >> (4 * (j & 7))) & 15u;
          v[j] = (int)n - (n >= 8 ? 16 : 0);
        }
      } else {  // 16 codes = 12 bytes: half (col / 16) & 1 of the 32-code group col / 32
        const int64_t col = col0 + qc;
        const uint8_t* p = xq6 + t * D + (col / 32) * 32 + ((col / 16) & 1) * 12;
        const uint32_t d0 = *reinterpret_cast<const uint32_t*>(p);
        const uint32_t d1 = *reinterpret_cast<const uint32_t*>(p + 4);
        const uint32_t d2 = *reinterpret_cast<const uint32_t*>(p + 8);
        const uint64_t lo = (uint64_t)d0 | ((uint64_t)d1 << 32);
#pragma unroll
        for (int j = 0; j < 16; ++j) {
          const int bit = 6 * j;
          uint32_t f;
          if (bit + 6 <= 64) f = (uint32_t)(lo >> bit) & 63u;
          else if (bit >= 64) f = (d2 >> (bit - 64)) & 63u;
          else f = ((uint32_t)(lo >> bit) | (d2 << (64 - bit))) & 63u;
          v[j] = int_of_e2m3(f);
        }
      }
    }
#pragma unroll
    for (int j = 0; j < 16; ++j) tile[r][qc + j] = (int8_t)v[j];
  }
  __syncthreads();
  // 128 columns x 4 groups of 32 entries, two per thread
#pragma unroll
  for (int k = 0; k < 2; ++k) {
    const int item = tid + 256 * k, c = item >> 2, gg = item & 3;
    if (col0 + c >= ncol) continue;
    int q[32];
#pragma unroll
    for (int i = 0; i < 32; ++i) q[i] = tile[32 * gg + i][c];
    uint4 lo, hi;
    fp6_pack32(q, lo, hi);
    uint8_t* p = out + (col0 + c) * ecap + e0 + 32 * gg;
    *reinterpret_cast<uint4*>(p) = lo;
    *reinterpret_cast<uint4*>(p + 16) = hi;
  }
}

}  // namespace

hipError_t launch_int4_to_fp6(hipStream_t s, const uint8_t* src, uint8_t* dst, int64_t rows, int64_t K) {
  const int64_t items = rows * (K / 32);
  if (items <= 0) return hipSuccess;
  int64_t wg = (items + 255) / 256;
  if (wg > 4096) wg = 4096;
  timing_begin(s);
  int4_to_fp6_kernel<<<(unsigned)wg, 256, 0, s>>>(src, dst, rows, K);
  timing_end(s, kKFp6Convert);
  return hipGetLastError();
}

hipError_t launch_fp6_build(hipStream_t s, int dt, const uint8_t* qup, const uint8_t* qdn,
                            const uint8_t* w_up, const uint8_t* w_dn, const int32_t* order6,
                            const int32_t* n_kept, const int32_t* n_up, const int32_t* ent,
                            const int32_t* cls, const uint8_t* xq6, int64_t N, int64_t C,
                            int64_t D, int64_t ecap, uint8_t* a_dn, uint8_t* a_up, uint8_t* a_dw,
                            uint8_t* x_dw, void* dX) {
  timing_begin(s);
  if (a_dn || a_up) {
    int64_t wg = ((N + 255) / 256 * 256) * (C / 32) / 256;
    if (wg > 4096) wg = 4096;
    if (wg < 1) wg = 1;
    const dim3 grid((unsigned)wg, 2u);
    switch (dt) {
      case kF32: fp6_build_rows_kernel<kF32><<<grid, 256, 0, s>>>(qup, qdn, w_dn, order6, n_kept, n_up, C, a_dn, a_up); break;
      case kF16: fp6_build_rows_kernel<kF16><<<grid, 256, 0, s>>>(qup, qdn, w_dn, order6, n_kept, n_up, C, a_dn, a_up); break;
      case kBF16: fp6_build_rows_kernel<kBF16><<<grid, 256, 0, s>>>(qup, qdn, w_dn, order6, n_kept, n_up, C, a_dn, a_up); break;
      default: return hipErrorInvalidValue;
    }
  }
  {
    const int64_t eb = (ecap + 127) / 128, cb = (C + 127) / 128, db = (D + 127) / 128;
    const int64_t xb = eb > (N + 127) / 128 ? eb : (N + 127) / 128;  // dX zeroing covers N tokens
    const dim3 grid((unsigned)xb, (unsigned)(cb + db + 1));
    switch (dt) {
      case kF32: fp6_build_cols_kernel<kF32><<<grid, 256, 0, s>>>(qup, qdn, w_up, w_dn, ent, cls, xq6, N, C, D, ecap, a_dw, x_dw, dX); break;
      case kF16: fp6_build_cols_kernel<kF16><<<grid, 256, 0, s>>>(qup, qdn, w_up, w_dn, ent, cls, xq6, N, C, D, ecap, a_dw, x_dw, dX); break;
      case kBF16: fp6_build_cols_kernel<kBF16><<<grid, 256, 0, s>>>(qup, qdn, w_up, w_dn, ent, cls, xq6, N, C, D, ecap, a_dw, x_dw, dX); break;
      default: return hipErrorInvalidValue;
    }
  }
  timing_end(s, kKFp6Build);
  return hipGetLastError();
}

}  // namespace hqlss
