// Quantisers of HQ-MM and LSS-MM (gfx950).
//
//  * fwht_absmax / fwht_quant: the Hadamard quantiser HQ (Sec. 3.3): block-diagonal
//    unnormalised Hadamard transform of each row (radix-2 butterflies, strides ascending,
//    fp32), then per-tensor absmax and INT4 codes clamp(rint(v * fl(7/a)), -7, 7)
//    (Sec. 3.1, Eq. 2), packed two per byte (App. A.6) with per-row sums of squares
//    (the ||X_i|| factor of the leverage score, Sec. 4.2).
//  * bit_split: bit splitting of the output gradient (Sec. 4.2, Eq. 4): upper codes by
//    round-to-nearest at s_up = a/7, lower codes by stochastic rounding of 14 x the exact
//    residual (s_dn = s_up / 14), Philox stream 0.
//
// Work decomposition: a wave owns one (row, 512-column chunk) item at a time; each lane
// holds 8 consecutive elements (one 16- or 32-byte load).  A Hadamard block of
// b = 2^k <= 128 columns then lives in b/8 consecutive lanes, so strides 1..4 run in
// registers and strides 8..64 across lanes.  Per-row results reduce inside the wave and
// land with one integer atomic per (row, chunk); per-tensor maxima with one atomic per
// workgroup into one of 64 slots.  All loads are 16-byte vectors, coalesced along the row.
#include "common.h"
#include "launch.h"

namespace hqlss {

namespace {

constexpr int kChunk = 512;  // columns per wave item (64 lanes x 8)
constexpr int kThreads = 256;

// Per-tensor maxima land in kSlots words, one 128-byte line apart, so that the
// workgroups' atomics spread over many L2 channels; a consumer wave reduces them
// (one slot per lane).
__device__ __forceinline__ float read_slots(const uint32_t* __restrict__ slots) {
  return wave_max(__uint_as_float(slots[(threadIdx.x & 63) * kSlotStride]));
}

template <int LOG2B>
__device__ __forceinline__ void fwht8(float v[8], int lane) {
  constexpr int b = 1 << LOG2B;
#pragma unroll
  for (int h = 1; h < 8 && h < b; h <<= 1) {
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      if ((j & h) == 0) {
        const float a = v[j], c = v[j + h];
        v[j] = a + c;
        v[j + h] = a - c;
      }
    }
  }
#pragma unroll
  for (int h = 8; h < b; h <<= 1) {
    const int m = h >> 3;
    const bool upper = (lane & m) != 0;
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const float p = __shfl_xor(v[j], m);
      v[j] = upper ? (p - v[j]) : (v[j] + p);  // (a+c, a-c) with a the lower lane
    }
  }
}

__device__ __forceinline__ int code_of(float v, float inv) {
  float q = rintf(v * inv);
  q = fminf(fmaxf(q, -7.0f), 7.0f);
  return (int)q;
}

__device__ __forceinline__ uint32_t pack8(const int q[8]) {
  uint32_t w = 0;
#pragma unroll
  for (int j = 0; j < 8; ++j) w |= (uint32_t)(q[j] & 15) << (4 * j);
  return w;
}

// Plain 16-byte copy: the reference kernel against which hardware traffic counters are
// calibrated (its bytes read and written are known exactly).
__global__ __launch_bounds__(kThreads) void copy_kernel(const uint4* __restrict__ src,
                                                        uint4* __restrict__ dst, int64_t n) {
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += stride)
    dst[i] = src[i];
}

__global__ __launch_bounds__(kThreads) void zero_kernel(uint32_t* p0, int64_t n0, uint32_t* p1,
                                                        int64_t n1, uint32_t* p2, int64_t n2,
                                                        uint32_t* p3, int64_t n3) {
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  const int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  for (int64_t i = t; i < n0; i += stride) p0[i] = 0;
  for (int64_t i = t; i < n1; i += stride) p1[i] = 0;
  for (int64_t i = t; i < n2; i += stride) p2[i] = 0;
  for (int64_t i = t; i < n3; i += stride) p3[i] = 0;
}

template <int DT, int LOG2B>
__global__ __launch_bounds__(kThreads) void fwht_absmax_kernel(const void* __restrict__ src,
                                                               int64_t rows, int64_t cols,
                                                               uint32_t* __restrict__ slots) {
  __shared__ float wmax[kThreads / kWave];
  const int lane = threadIdx.x & 63;
  const uint32_t chunks = (uint32_t)((cols + kChunk - 1) / kChunk);
  const uint32_t items = (uint32_t)rows * chunks;
  const uint32_t nwaves = gridDim.x * (kThreads / kWave);
  float m = 0.f;
  for (uint32_t it = blockIdx.x * (kThreads / kWave) + (threadIdx.x >> 6); it < items; it += nwaves) {
    const uint32_t row = it / chunks;
    const int64_t col = (int64_t)(it - row * chunks) * kChunk + lane * 8;
    float v[8];
    if (col < cols) {
      load8<DT>(static_cast<const char*>(src) + ((int64_t)row * cols + col) * Elem<DT>::bytes, v);
    } else {
#pragma unroll
      for (int j = 0; j < 8; ++j) v[j] = 0.f;
    }
    fwht8<LOG2B>(v, lane);
#pragma unroll
    for (int j = 0; j < 8; ++j) m = fmaxf(m, fabsf(v[j]));
  }
  m = wave_max(m);
  if (lane == 0) wmax[threadIdx.x >> 6] = m;
  __syncthreads();
  if (threadIdx.x == 0) {
    m = fmaxf(fmaxf(wmax[0], wmax[1]), fmaxf(wmax[2], wmax[3]));
    // one atomic per workgroup, spread over kSlots cache lines; |v| >= 0: uint order
    if (m > 0.f) atomicMax(slots + (blockIdx.x % kSlots) * kSlotStride, __float_as_uint(m));
  }
}

template <int DT, int LOG2B>
__global__ __launch_bounds__(kThreads) void fwht_quant_kernel(
    const void* __restrict__ src, int64_t rows, int64_t cols, const uint32_t* __restrict__ slots,
    float* __restrict__ amax_out, uint8_t* __restrict__ packed, int32_t* __restrict__ row_sumsq) {
  const int lane = threadIdx.x & 63;
  const uint32_t chunks = (uint32_t)((cols + kChunk - 1) / kChunk);
  const uint32_t items = (uint32_t)rows * chunks;
  const uint32_t nwaves = gridDim.x * (kThreads / kWave);
  const float a = read_slots(slots);
  if (blockIdx.x == 0 && threadIdx.x == 0) *amax_out = a;
  const float inv = a > 0.f ? 7.0f / a : 0.f;
  for (uint32_t it = blockIdx.x * (kThreads / kWave) + (threadIdx.x >> 6); it < items; it += nwaves) {
    const uint32_t row = it / chunks;
    const int64_t col = (int64_t)(it - row * chunks) * kChunk + lane * 8;
    const bool live = col < cols;
    float v[8];
    if (live) {
      load8<DT>(static_cast<const char*>(src) + ((int64_t)row * cols + col) * Elem<DT>::bytes, v);
    } else {
#pragma unroll
      for (int j = 0; j < 8; ++j) v[j] = 0.f;
    }
    fwht8<LOG2B>(v, lane);
    int q[8];
    int ss = 0;
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      q[j] = code_of(v[j], inv);
      ss += q[j] * q[j];
    }
    if (live) *reinterpret_cast<uint32_t*>(packed + (int64_t)row * (cols / 2) + col / 2) = pack8(q);
    if (row_sumsq) {
      ss = wave_sum(ss);
      if (lane == 0 && ss) atomicAdd(row_sumsq + row, ss);
    }
  }
}

__device__ __forceinline__ int sext4(uint32_t n) { return (int)(n ^ 8u) - 8; }

__global__ __launch_bounds__(kThreads) void transpose_packed_kernel(const uint8_t* __restrict__ src,
                                                                    int64_t rows, int64_t cols,
                                                                    uint8_t* __restrict__ dst) {
  __shared__ int8_t t[64][65];  // codes [row_local][col_local]
  const int64_t r0 = (int64_t)blockIdx.y * 64, c0 = (int64_t)blockIdx.x * 64;
  const int tid = threadIdx.x;
  const int r = tid >> 2, q = (tid & 3) * 8;  // 64 rows x 4 groups of 8 bytes
  {
    const uint2 w = *reinterpret_cast<const uint2*>(src + (r0 + r) * (cols / 2) + c0 / 2 + q);
    const uint32_t ww[2] = {w.x, w.y};
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const uint32_t byte = (ww[j >> 2] >> (8 * (j & 3))) & 0xFFu;
      t[r][2 * (q + j)] = (int8_t)sext4(byte & 15u);
      t[r][2 * (q + j) + 1] = (int8_t)sext4(byte >> 4);
    }
  }
  __syncthreads();
  {
    uint32_t ww[2] = {0u, 0u};
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const int c = 2 * (q + j);
      const uint32_t byte = ((uint32_t)t[c][r] & 15u) | (((uint32_t)t[c + 1][r] & 15u) << 4);
      ww[j >> 2] |= byte << (8 * (j & 3));
    }
    *reinterpret_cast<uint2*>(dst + (c0 + r) * (rows / 2) + r0 / 2 + q) = make_uint2(ww[0], ww[1]);
  }
}

template <int DT>
__global__ __launch_bounds__(kThreads) void bit_split_kernel(
    const void* __restrict__ g, int64_t N, int64_t C, const uint32_t* __restrict__ slots,
    float* __restrict__ amax_out, uint8_t* __restrict__ qup, uint8_t* __restrict__ qdn,
    int32_t* __restrict__ sumsq_up, int32_t* __restrict__ sumsq_dn, uint64_t seed,
    uint64_t offset) {
  const int lane = threadIdx.x & 63;
  const uint32_t chunks = (uint32_t)((C + kChunk - 1) / kChunk);
  const uint32_t items = (uint32_t)N * chunks;
  const uint32_t nwaves = gridDim.x * (kThreads / kWave);
  const float a = read_slots(slots);
  if (blockIdx.x == 0 && threadIdx.x == 0) *amax_out = a;
  const float inv = a > 0.f ? 7.0f / a : 0.f;
  for (uint32_t it = blockIdx.x * (kThreads / kWave) + (threadIdx.x >> 6); it < items; it += nwaves) {
    const int64_t row = it / chunks;
    const int64_t col = (int64_t)(it - (uint32_t)row * chunks) * kChunk + lane * 8;
    const bool live = col < C;
    float v[8];
    if (live) {
      load8<DT>(static_cast<const char*>(g) + (row * C + col) * Elem<DT>::bytes, v);
    } else {
#pragma unroll
      for (int j = 0; j < 8; ++j) v[j] = 0.f;
    }
    const U4 rnd = philox_block(seed, offset, 0u, (uint64_t)(row * C + col));
    int qu[8], qd[8];
    int su = 0, sd = 0;
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const float x = v[j] * inv;
      const float up = rintf(x);          // |x| <= 7 (1 + 2^-23): |up| <= 7
      const float w = 14.0f * (x - up);   // residual exact; |w| <= 7
      const float fl = floorf(w);
      const float thr = (w - fl) * 65536.0f;
      const int dn = (int)fl + (((float)u16_of(rnd, j) < thr) ? 1 : 0);
      qu[j] = (int)up;
      qd[j] = dn;
      su += qu[j] * qu[j];
      sd += dn * dn;
    }
    if (live) {
      const int64_t o = row * (C / 2) + col / 2;
      *reinterpret_cast<uint32_t*>(qup + o) = pack8(qu);
      *reinterpret_cast<uint32_t*>(qdn + o) = pack8(qd);
    }
    su = wave_sum(su);
    sd = wave_sum(sd);
    if (lane == 0) {
      if (su) atomicAdd(sumsq_up + row, su);
      if (sd) atomicAdd(sumsq_dn + row, sd);
    }
  }
}

// Enough waves to fill the chip several times over; every wave loops over items.
int grid_for(int64_t items) {
  int64_t wg = (items + (kThreads / kWave) - 1) / (kThreads / kWave);
  if (wg > 2048) wg = 2048;
  if (wg < 1) wg = 1;
  return (int)wg;
}

template <int DT, int LOG2B>
hipError_t absmax_t(hipStream_t s, const void* src, int64_t rows, int64_t cols, uint32_t* slots) {
  const int64_t items = rows * ((cols + kChunk - 1) / kChunk);
  timing_begin(s);
  fwht_absmax_kernel<DT, LOG2B><<<grid_for(items), kThreads, 0, s>>>(src, rows, cols, slots);
  timing_end(s, kKAbsmax);
  return hipGetLastError();
}

template <int DT, int LOG2B>
hipError_t quant_t(hipStream_t s, const void* src, int64_t rows, int64_t cols,
                   const uint32_t* slots, float* amax_out, uint8_t* packed, int32_t* row_sumsq) {
  const int64_t items = rows * ((cols + kChunk - 1) / kChunk);
  timing_begin(s);
  fwht_quant_kernel<DT, LOG2B>
      <<<grid_for(items), kThreads, 0, s>>>(src, rows, cols, slots, amax_out, packed, row_sumsq);
  timing_end(s, kKQuant);
  return hipGetLastError();
}

template <template <int, int> class F, int DT, typename... Args>
hipError_t dispatch_block(int log2b, Args... args) {
  switch (log2b) {
    case 0: return F<DT, 0>::run(args...);
    case 1: return F<DT, 1>::run(args...);
    case 2: return F<DT, 2>::run(args...);
    case 3: return F<DT, 3>::run(args...);
    case 4: return F<DT, 4>::run(args...);
    case 5: return F<DT, 5>::run(args...);
    case 6: return F<DT, 6>::run(args...);
    case 7: return F<DT, 7>::run(args...);
  }
  return hipErrorInvalidValue;
}

template <int DT, int LOG2B> struct AbsmaxF {
  static hipError_t run(hipStream_t s, const void* src, int64_t r, int64_t c, uint32_t* a) {
    return absmax_t<DT, LOG2B>(s, src, r, c, a);
  }
};
template <int DT, int LOG2B> struct QuantF {
  static hipError_t run(hipStream_t s, const void* src, int64_t r, int64_t c, const uint32_t* a,
                        float* ao, uint8_t* p, int32_t* ss) {
    return quant_t<DT, LOG2B>(s, src, r, c, a, ao, p, ss);
  }
};

}  // namespace

hipError_t launch_zero(hipStream_t s, uint32_t* p0, int64_t n0, uint32_t* p1, int64_t n1,
                       uint32_t* p2, int64_t n2, uint32_t* p3, int64_t n3) {
  int64_t n = n0 > n1 ? n0 : n1;
  n = n > n2 ? n : n2;
  n = n > n3 ? n : n3;
  int64_t wg = (n + kThreads - 1) / kThreads;
  if (wg > 1024) wg = 1024;
  if (wg < 1) wg = 1;
  timing_begin(s);
  zero_kernel<<<(int)wg, kThreads, 0, s>>>(p0, n0, p1, n1, p2, n2, p3, n3);
  timing_end(s, kKZero);
  return hipGetLastError();
}

hipError_t launch_copy(hipStream_t s, const void* src, void* dst, int64_t bytes) {
  const int64_t n = bytes / 16;
  int64_t wg = (n + kThreads - 1) / kThreads;
  if (wg > 4096) wg = 4096;
  if (wg < 1) wg = 1;
  timing_begin(s);
  copy_kernel<<<(int)wg, kThreads, 0, s>>>(static_cast<const uint4*>(src), static_cast<uint4*>(dst), n);
  timing_end(s, kKCopy);
  return hipGetLastError();
}

hipError_t launch_fwht_absmax(hipStream_t s, int dt, int log2b, const void* src, int64_t rows,
                              int64_t cols, uint32_t* amax_bits) {
  switch (dt) {
    case kF32: return dispatch_block<AbsmaxF, kF32>(log2b, s, src, rows, cols, amax_bits);
    case kF16: return dispatch_block<AbsmaxF, kF16>(log2b, s, src, rows, cols, amax_bits);
    case kBF16: return dispatch_block<AbsmaxF, kBF16>(log2b, s, src, rows, cols, amax_bits);
  }
  return hipErrorInvalidValue;
}

hipError_t launch_fwht_quant(hipStream_t s, int dt, int log2b, const void* src, int64_t rows,
                             int64_t cols, const uint32_t* slots, float* amax_out, uint8_t* packed,
                             int32_t* row_sumsq) {
  switch (dt) {
    case kF32:
      return dispatch_block<QuantF, kF32>(log2b, s, src, rows, cols, slots, amax_out, packed, row_sumsq);
    case kF16:
      return dispatch_block<QuantF, kF16>(log2b, s, src, rows, cols, slots, amax_out, packed, row_sumsq);
    case kBF16:
      return dispatch_block<QuantF, kBF16>(log2b, s, src, rows, cols, slots, amax_out, packed, row_sumsq);
  }
  return hipErrorInvalidValue;
}

hipError_t launch_transpose_packed(hipStream_t s, const uint8_t* src, int64_t rows, int64_t cols,
                                   uint8_t* dst) {
  dim3 grid((unsigned)(cols / 64), (unsigned)(rows / 64));
  timing_begin(s);
  transpose_packed_kernel<<<grid, kThreads, 0, s>>>(src, rows, cols, dst);
  timing_end(s, kKTranspose);
  return hipGetLastError();
}

hipError_t launch_bit_split(hipStream_t s, int dt, const void* g, int64_t N, int64_t C,
                            const uint32_t* slots, float* amax_out, uint8_t* qup, uint8_t* qdn,
                            int32_t* sumsq_up, int32_t* sumsq_dn, uint64_t seed,
                            uint64_t offset) {
  const int64_t items = N * ((C + kChunk - 1) / kChunk);
  const int grid = grid_for(items);
  timing_begin(s);
  switch (dt) {
    case kF32:
      bit_split_kernel<kF32><<<grid, kThreads, 0, s>>>(g, N, C, slots, amax_out, qup, qdn, sumsq_up,
                                                      sumsq_dn, seed, offset);
      break;
    case kF16:
      bit_split_kernel<kF16><<<grid, kThreads, 0, s>>>(g, N, C, slots, amax_out, qup, qdn, sumsq_up,
                                                      sumsq_dn, seed, offset);
      break;
    case kBF16:
      bit_split_kernel<kBF16><<<grid, kThreads, 0, s>>>(g, N, C, slots, amax_out, qup, qdn, sumsq_up,
                                                       sumsq_dn, seed, offset);
      break;
    default:
      return hipErrorInvalidValue;
  }
  timing_end(s, kKBitSplit);
  return hipGetLastError();
}

}  // namespace hqlss
