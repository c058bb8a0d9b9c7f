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

}  // namespace hqlss
