// Device helpers shared by the HQ-MM / LSS-MM kernels (gfx950, wave64).
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace hqlss {

constexpr int kWave = 64;
constexpr int kQmax = 7;      // Q_N = Q_P = 7 (Sec. 3.1)
constexpr int kBsRatio = 14;  // s_up / s_dn of the bit split

enum Dt : int { kF32 = 0, kF16 = 1, kBF16 = 2 };

// ---------------------------------------------------------------- dtype conversion
// fp16 and bf16 widen to fp32 exactly (subnormals included); fp32 -> fp16/bf16 rounds
// to nearest-even.
template <int DT> struct Elem;
template <> struct Elem<kF32> { static constexpr int bytes = 4; };
template <> struct Elem<kF16> { static constexpr int bytes = 2; };
template <> struct Elem<kBF16> { static constexpr int bytes = 2; };

__device__ __forceinline__ float h2f(uint32_t h) {
  return (float)__builtin_bit_cast(_Float16, (uint16_t)h);
}
__device__ __forceinline__ float bf2f(uint32_t h) { return __uint_as_float(h << 16); }
__device__ __forceinline__ uint32_t f2h(float f) {
  return (uint32_t)__builtin_bit_cast(uint16_t, (_Float16)f);
}
// Two values rounded to nearest-even and packed (the first in the low half), by the
// packed conversions of gfx950 (v_cvt_pk_f16_f32 / v_cvt_pk_bf16_f32).
typedef float f32x2 __attribute__((ext_vector_type(2)));
typedef _Float16 f16x2 __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
template <int DT>
__device__ __forceinline__ uint32_t pack2(float a, float b) {
  const f32x2 x = {a, b};
  if constexpr (DT == kF16) return __builtin_bit_cast(uint32_t, __builtin_convertvector(x, f16x2));
  else return __builtin_bit_cast(uint32_t, __builtin_convertvector(x, bf16x2));
}
__device__ __forceinline__ uint32_t f2bf(float f) {
  uint32_t u = __float_as_uint(f);
  u += 0x7FFFu + ((u >> 16) & 1u);  // inputs are finite
  return u >> 16;
}

// ---------------------------------------------------------------- streaming access
// Loads and stores of data that is touched once per kernel (inputs streamed through a
// quantiser, outputs written for a later kernel) carry the non-temporal hint: they do not
// allocate in the caches, so they neither evict operands other kernels reuse nor wait for
// the write-back of dirty lines a previous kernel left behind.
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
template <bool NT = true>
__device__ __forceinline__ uint4 ld_stream(const void* p) {
  if constexpr (NT) {
    const u32x4 v = __builtin_nontemporal_load(static_cast<const u32x4*>(p));
    return make_uint4(v[0], v[1], v[2], v[3]);
  } else {
    return *static_cast<const uint4*>(p);
  }
}
template <bool NT = true>
__device__ __forceinline__ uint2 ld_stream2(const void* p) {
  if constexpr (NT) {
    const u32x2 v = __builtin_nontemporal_load(static_cast<const u32x2*>(p));
    return make_uint2(v[0], v[1]);
  } else {
    return *static_cast<const uint2*>(p);
  }
}
template <bool NT = true>
__device__ __forceinline__ void st_stream(void* p, uint4 v) {
  if constexpr (NT) {
    const u32x4 w = {v.x, v.y, v.z, v.w};
    __builtin_nontemporal_store(w, static_cast<u32x4*>(p));
  } else {
    *static_cast<uint4*>(p) = v;
  }
}
template <bool NT = true>
__device__ __forceinline__ void st_stream2(void* p, uint2 v) {
  if constexpr (NT) {
    const u32x2 w = {v.x, v.y};
    __builtin_nontemporal_store(w, static_cast<u32x2*>(p));
  } else {
    *static_cast<uint2*>(p) = v;
  }
}
// Cache policy per access site (1 = streaming, 0 = cached).  The maximum pass reads
// cached: the quantizer or bit split that reads the same tensor next then finds part of
// it in the 256 MB MALL.
#ifndef HQ_NT_ABS_LD
#define HQ_NT_ABS_LD 0
#endif
#ifndef HQ_NT_Q_LD
#define HQ_NT_Q_LD 1
#endif
#ifndef HQ_NT_Q_ST
#define HQ_NT_Q_ST 0
#endif
#ifndef HQ_NT_BS_LD
#define HQ_NT_BS_LD 1
#endif
#ifndef HQ_NT_BS_ST
#define HQ_NT_BS_ST 0
#endif
#ifndef HQ_NT_B_LD
#define HQ_NT_B_LD 0
#endif
#ifndef HQ_NT_B_ST
#define HQ_NT_B_ST 0
#endif
#ifndef HQ_NT_G_ST
#define HQ_NT_G_ST 1
#endif
#ifndef HQ_NT_R_LD
#define HQ_NT_R_LD 0
#endif
#ifndef HQ_NT_P_ST
#define HQ_NT_P_ST 0
#endif

// Load 8 consecutive elements starting at p (16-byte aligned for fp16/bf16,
// 32-byte aligned for fp32; streaming) and widen them to fp32.
template <int DT, bool NT = true>
__device__ __forceinline__ void load8(const void* p, float v[8]) {
  if constexpr (DT == kF32) {
    const uint4 a = ld_stream<NT>(p), b = ld_stream<NT>(static_cast<const char*>(p) + 16);
    v[0] = __uint_as_float(a.x); v[1] = __uint_as_float(a.y); v[2] = __uint_as_float(a.z); v[3] = __uint_as_float(a.w);
    v[4] = __uint_as_float(b.x); v[5] = __uint_as_float(b.y); v[6] = __uint_as_float(b.z); v[7] = __uint_as_float(b.w);
  } else {
    uint4 a = ld_stream<NT>(p);
    uint32_t w[4] = {a.x, a.y, a.z, a.w};
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      if constexpr (DT == kF16) {
        v[2 * j] = h2f(w[j] & 0xFFFFu);
        v[2 * j + 1] = h2f(w[j] >> 16);
      } else {
        v[2 * j] = bf2f(w[j] & 0xFFFFu);
        v[2 * j + 1] = bf2f(w[j] >> 16);
      }
    }
  }
}

// Store n (multiple of 4) fp32 values, converting to the element type.
template <int DT, int NV>
__device__ __forceinline__ void store_vec(void* p, const float* v) {
  if constexpr (DT == kF32) {
#pragma unroll
    for (int j = 0; j < NV; j += 4)
      reinterpret_cast<float4*>(p)[j / 4] = make_float4(v[j], v[j + 1], v[j + 2], v[j + 3]);
  } else {
    uint32_t w[NV / 2];
#pragma unroll
    for (int j = 0; j < NV / 2; ++j) {
      w[j] = pack2<DT>(v[2 * j], v[2 * j + 1]);
    }
    if constexpr (NV == 8) {
      *reinterpret_cast<uint4*>(p) = make_uint4(w[0], w[1], w[2], w[3]);
    } else {
#pragma unroll
      for (int j = 0; j < NV / 2; j += 2)
        reinterpret_cast<uint2*>(p)[j / 2] = make_uint2(w[j], w[j + 1]);
    }
  }
}

// store_vec to global memory with the streaming hint (NV = 8).
template <int DT, bool NT = true>
__device__ __forceinline__ void store8_stream(void* p, const float* v) {
  if constexpr (DT == kF32) {
    st_stream<NT>(p, make_uint4(__float_as_uint(v[0]), __float_as_uint(v[1]), __float_as_uint(v[2]), __float_as_uint(v[3])));
    st_stream<NT>(static_cast<char*>(p) + 16,
              make_uint4(__float_as_uint(v[4]), __float_as_uint(v[5]), __float_as_uint(v[6]), __float_as_uint(v[7])));
  } else {
    uint32_t w[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      w[j] = pack2<DT>(v[2 * j], v[2 * j + 1]);
    }
    st_stream<NT>(p, make_uint4(w[0], w[1], w[2], w[3]));
  }
}

template <int DT>
__device__ __forceinline__ void store1(void* p, int64_t idx, float v) {
  if constexpr (DT == kF32) reinterpret_cast<float*>(p)[idx] = v;
  else if constexpr (DT == kF16) reinterpret_cast<uint16_t*>(p)[idx] = (uint16_t)f2h(v);
  else reinterpret_cast<uint16_t*>(p)[idx] = (uint16_t)f2bf(v);
}

// ---------------------------------------------------------------- Philox4x32-10
// Salmon, Moraes, Dror, Shaw, "Parallel Random Numbers: As Easy as 1, 2, 3" (SC'11):
// per round, words 0 and 2 are multiplied by two odd constants into 64-bit products
// (hi, lo) and the state becomes (hi1 ^ w1 ^ k0, lo1, hi0 ^ w3 ^ k1, lo0); the key
// advances by a Weyl sequence between rounds.
struct U4 { uint32_t x, y, z, w; };

__device__ __forceinline__ U4 philox4x32_10(uint32_t c0, uint32_t c1, uint32_t c2, uint32_t c3,
                                            uint32_t k0, uint32_t k1) {
#pragma unroll
  for (int r = 0; r < 10; ++r) {
    if (r) { k0 += 0x9E3779B9u; k1 += 0xBB67AE85u; }
    const uint64_t p0 = (uint64_t)0xD2511F53u * c0;  // one 32 x 32 -> 64 multiply each
    const uint64_t p1 = (uint64_t)0xCD9E8D57u * c2;
    // three-input exclusive or in one v_bitop3_b32 (truth table 0x96)
    const uint32_t n0 = __builtin_amdgcn_bitop3_b32((uint32_t)(p1 >> 32), c1, k0, 0x96);
    const uint32_t n2 = __builtin_amdgcn_bitop3_b32((uint32_t)(p0 >> 32), c3, k1, 0x96);
    c0 = n0; c1 = (uint32_t)p1; c2 = n2; c3 = (uint32_t)p0;
  }
  return U4{c0, c1, c2, c3};
}

// The eight 16-bit uniforms of the Philox block holding elements i0..i0+7 (i0 % 8 == 0).
__device__ __forceinline__ U4 philox_block(uint64_t seed, uint64_t offset, uint32_t stream,
                                           uint64_t i0) {
  const uint64_t blk = offset + (i0 >> 3);
  return philox4x32_10((uint32_t)blk, (uint32_t)(blk >> 32), stream, 0u, (uint32_t)seed,
                       (uint32_t)(seed >> 32));
}
__device__ __forceinline__ uint32_t u16_of(const U4& b, int j) {  // element j of a block
  const uint32_t w = (j >> 1) == 0 ? b.x : (j >> 1) == 1 ? b.y : (j >> 1) == 2 ? b.z : b.w;
  return (j & 1) ? (w >> 16) : (w & 0xFFFFu);
}

// ---------------------------------------------------------------- wave reductions
__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o));
  return v;
}
__device__ __forceinline__ int wave_sum(int v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o);
  return v;
}
__device__ __forceinline__ uint64_t wave_sum_u64(uint64_t v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    uint32_t lo = __shfl_xor((uint32_t)v, o), hi = __shfl_xor((uint32_t)(v >> 32), o);
    v += ((uint64_t)hi << 32) | lo;
  }
  return v;
}

// floor(sqrt(x)) for any 64-bit x: an estimate from the hardware double square root (one
// instruction, not correctly rounded; the estimate is within a step or two of the root),
// clamped to the 32-bit range and corrected in exact integers (no product overflows), so
// the result is exact whatever the estimate's error.
__device__ __forceinline__ uint32_t isqrt64(uint64_t x) {
  uint64_t r = (uint64_t)__builtin_amdgcn_sqrt((double)x);
  if (r > 0xFFFFFFFFull) r = 0xFFFFFFFFull;
  while (r * r > x) --r;
  while (r < 0xFFFFFFFFull && (r + 1) * (r + 1) <= x) ++r;
  return (uint32_t)r;
}

// ---------------------------------------------------------------- scales
// s = fl(a / 7); alpha = fl(fl(s1 * s2) / denom) with denom = 2^k (forward) or 14 * 2^k
// (gradients, s_dn = s_up / 14).  a = 0 gives alpha = 0 (every code is 0 then).
__device__ __forceinline__ float step_of(uint32_t amax_bits) {
  return __uint_as_float(amax_bits) / 7.0f;
}
__device__ __forceinline__ float alpha_of(uint32_t a1, uint32_t a2, float denom) {
  const float p = step_of(a1) * step_of(a2);
  return p / denom;
}

}  // namespace hqlss
