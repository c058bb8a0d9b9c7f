// Quantisers of HQ-MM and LSS-MM (gfx950).
//
//  * fwht_absmax / fwht_quant: the Hadamard quantiser HQ (Sec. 3.3): block-diagonal
//    unnormalised Hadamard transform of each row (radix-2 butterflies, strides ascending,
//    fp32), then per-tensor absmax and INT4 codes clamp(rint(v * fl(7/a)), -7, 7)
//    (Sec. 3.1, Eq. 2), packed two per byte (App. A.6) with per-row sums of squares
//    (the ||X_i|| factor of the leverage score, Sec. 4.2).  One launch serves X and W:
//    X by rows, W by tiles, each tile workgroup writing its codes row-major and also
//    transposed through LDS (the K-contiguous operand of the dX GEMM), so W is read once.
//    On request the codes of X and W are also written as FP6 (e2m3, the padded layout of
//    fp6.hip) for a product on the FP6 MFMA, through the hardware conversion.
//  * fwht_lsq: the same transform quantised at a caller-given (learned) step in one pass,
//    with the fp16 deltas q - I r that the learned-step backward needs (Eq. 2, App. A.3);
//    the second tensor by tiles as above.
//  * bit_split: bit splitting of the output gradient (Sec. 4.2, Eq. 4): upper codes by
//    round-to-nearest at s_up = a/7, lower codes by stochastic rounding of 14 x the exact
//    residual (s_dn = s_up / 14), Philox stream 0.  It also forms the integer leverage
//    scores of both stacked rows of every token and per-workgroup totals of them, which
//    is all the sampler needs.  At a row's end the group reduces the two row sums (one
//    packed reduction for rows of at most 640 columns) and two of its lanes form the two
//    scores, each with one integer square root.
//
// Work decomposition: a row belongs to a group of G lanes (G = the largest power of two
// <= 64 dividing cols/16), so a wave holds 64/G rows and every per-row result (sum of
// squares, scores) is one plain store: no atomics, nothing to pre-zero.  Each lane loads
// 16 consecutive elements per step and keeps two steps in flight.  A Hadamard block
// of b = 2^k <= 128 columns lives in b/16 consecutive lanes of one group (b/16 <= G for
// every admitted shape), so strides 1..8 run in registers and strides 16..64 are lane
// exchanges folded into the butterfly add (DPP) or a swizzle.  Per-tensor maxima leave
// each workgroup as one plain store of a partial; consumers reduce the partials.
// A batched job (the attention BMM) holds many equal tensors; its workgroups are split
// evenly over the batches and every per-tensor output is one block per batch.
//
// These kernels are bound by vector-ALU issue as much as by HBM, so the per-element work
// is kept to a handful of instructions: codes come from the magic-number form of
// round-half-even (x + 1.5 * 2^23 leaves rint(x) in the low mantissa bits, exact for
// |x| < 2^22), packing uses byte permutes, and the sums of squares of the codes are dot
// products of the packed INT4 words with themselves.
#include "common.h"
#include "launch.h"

#include <mutex>
#include <unordered_map>

namespace hqlss {

namespace {

constexpr int kQThreads = 512;
constexpr int kQWaves = kQThreads / kWave;
constexpr int kVE = 16;  // elements per lane per step
constexpr float kRne = 12582912.0f;  // 1.5 * 2^23

template <int DT, bool NT>
__device__ __forceinline__ void load16(const char* p, float v[16]) {
  load8<DT, NT>(p, v);
  load8<DT, NT>(p + 8 * Elem<DT>::bytes, v + 8);
}

// Value of lane (lane ^ M), M in {1, 2, 4}, added to x: DPP quad permutations (folded into
// the add) or a ds_swizzle swap of 4-lane groups.
template <int M>
__device__ __forceinline__ float add_xor_lane(float v, float x) {
  const int i = __float_as_int(v);
  if constexpr (M == 1) return __int_as_float(__builtin_amdgcn_update_dpp(0, i, 0xB1, 0xF, 0xF, true)) + x;
  else if constexpr (M == 2) return __int_as_float(__builtin_amdgcn_update_dpp(0, i, 0x4E, 0xF, 0xF, true)) + x;
  else return __int_as_float(__builtin_amdgcn_ds_swizzle(i, (4 << 10) | 0x1F)) + x;
}

// In-place unnormalised FWHT of blocks of 2^LOG2B consecutive elements; the lane holds 16
// consecutive elements, the lanes of one block are consecutive.  Pairs (a, c) at stride h
// become (a + c, a - c), strides ascending.  Across lanes the lower lane adds its
// partner's value and the upper lane adds its own negated value to the partner's (a - c
// = a + (-c) exactly), so both take one DPP add.
template <int LOG2B>
__device__ __forceinline__ void fwht16(float v[16], int lane) {
  constexpr int b = 1 << LOG2B;
#pragma unroll
  for (int h = 1; h < 16 && h < b; h <<= 1) {
#pragma unroll
    for (int j = 0; j < 16; ++j) {
      if ((j & h) == 0) {
        const float a = v[j], c = v[j + h];
        v[j] = a + c;
        v[j + h] = a - c;
      }
    }
  }
#define HQLSS_XSTAGE(M)                                                       \
  if constexpr (16 * (M) < b) {                                               \
    const uint32_t sgn = (lane & (M)) ? 0x80000000u : 0u;                     \
    _Pragma("unroll") for (int j = 0; j < 16; ++j) {                          \
      const float own = __uint_as_float(__float_as_uint(v[j]) ^ sgn);         \
      v[j] = add_xor_lane<M>(v[j], own);                                      \
    }                                                                         \
  }
  HQLSS_XSTAGE(1)
  HQLSS_XSTAGE(2)
  HQLSS_XSTAGE(4)
#undef HQLSS_XSTAGE
}

// Bits of fl(x + 1.5 * 2^23): rint(x) (half-to-even) sits in the low mantissa bits.
__device__ __forceinline__ uint32_t rne_bits(float x) { return __float_as_uint(x + kRne); }

// 16 consecutive codes (as rne_bits) -> their 12 bytes of FP6 (e2m3) fields, field i at bits
// 6i..6i+5: half of a 32-code group of the padded FP6 layout.  The hardware conversion of
// two 16-float operands interleaves them (field 2k from the first, 2k + 1 from the second),
// so even and odd codes go in separately; the upper 16 fields come out zero.  Exact: the
// codes are integers |q| <= 7, all e2m3 values, and the scale is 1.  The instruction is
// issued through inline assembly with an early-clobber result: the compiler builtin let
// the result registers overlap the source registers, and the instruction then read some
// sources after writing over them (wrong fields at one fixed position of the chunk).
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef int i32x6 __attribute__((ext_vector_type(6)));
__device__ __forceinline__ uint3 fp6_half16(const uint32_t y[16]) {
  f32x16 ev, od;
#pragma unroll
  for (int k = 0; k < 8; ++k) {
    ev[k] = __uint_as_float(y[2 * k]) - kRne;
    od[k] = __uint_as_float(y[2 * k + 1]) - kRne;
    ev[8 + k] = 0.f;
    od[8 + k] = 0.f;
  }
  i32x6 w;
  asm volatile("v_cvt_scalef32_2xpk16_fp6_f32 %0, %1, %2, 1.0" : "=&v"(w) : "v"(ev), "v"(od));
  return make_uint3((uint32_t)w[0], (uint32_t)w[1], (uint32_t)w[2]);
}

// The 16 bytes lane pair (2g, 2g + 1) stores of 32-code group g of a row in the padded FP6
// layout: the even chunk's fields fill bytes 0..11, the odd one's bytes 12..23, then 8 zero
// bytes.  The even lane takes bytes 0..15 (the first word of its partner's fields comes
// over), the odd lane bytes 16..31, so both store one aligned 16-byte piece.  Lanes 2g and
// 2g + 1 must hold chunks 2g and 2g + 1 and both be active.
__device__ __forceinline__ uint4 fp6_chunk16(const uint32_t y[16], bool odd) {
  const uint3 f = fp6_half16(y);
  const uint32_t partner = (uint32_t)__shfl_xor((int)f.x, 1);
  return odd ? make_uint4(f.y, f.z, 0u, 0u) : make_uint4(f.x, f.y, f.z, partner);
}
__device__ __forceinline__ void store_fp6_chunk(uint8_t* row6, int64_t c, const uint4& v) {
  *reinterpret_cast<uint4*>(row6 + (c >> 1) * 32 + (c & 1) * 16) = v;
}

// Pack 8 codes given as rne_bits (low nibbles) into one word, element j at bits 4j.
__device__ __forceinline__ uint32_t pack8_bits(const uint32_t y[8]) {
  uint32_t b[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) b[i] = (y[2 * i + 1] << 4) | (y[2 * i] & 15u);  // valid low byte
  const uint32_t lo = __builtin_amdgcn_perm(b[1], b[0], 0x0C0C0400u);  // [b0, b1, 0, 0]
  const uint32_t hi = __builtin_amdgcn_perm(b[3], b[2], 0x0C0C0400u);  // [b2, b3, 0, 0]
  return __builtin_amdgcn_perm(hi, lo, 0x05040100u);                  // [b0, b1, b2, b3]
}

// Sum of squares of the eight signed nibbles of a packed word, accumulated into acc.
__device__ __forceinline__ int sumsq8(uint32_t w, int acc) {
  return __builtin_amdgcn_sdot8((int)w, (int)w, acc, false);
}

// Sum over the G lanes of a row group (G a power of two; every lane of the group active).
__device__ __forceinline__ int group_sum(int v, int G) {
  for (int o = G >> 1; o > 0; o >>= 1) v += __shfl_xor(v, o);
  return v;
}

// Row-group geometry of one job (one tensor).  The wave walks a uniform sequence of steps
// (row k of its groups, 16-column chunk it), kept several steps ahead in loads whatever
// the row boundaries; group rows past the end re-read the last row and store nothing.
struct Geo {
  int lane, sub, grp, G, rpw, iters;
  int64_t first_row, row_step, rows, steps;
  __device__ Geo(const QJob& j, int wg) {
    lane = threadIdx.x & 63;
    G = 1 << j.log2g;
    sub = lane & (G - 1);
    grp = lane >> j.log2g;
    rpw = 64 >> j.log2g;
    iters = (int)((j.cols / kVE) >> j.log2g);
    const int64_t wave_row0 = ((int64_t)wg * kQWaves + (threadIdx.x >> 6)) * rpw;
    first_row = wave_row0 + grp;
    row_step = (int64_t)j.wg * kQWaves * rpw;
    rows = j.rows;
    steps = wave_row0 < rows ? (rows - wave_row0 + row_step - 1) / row_step * iters : 0;
  }
  // row of step (k, it) for this lane's group, clamped into the tensor
  __device__ int64_t row_of(int64_t k) const {
    const int64_t r = first_row + k * row_step;
    return r < rows ? r : rows - 1;
  }
  __device__ bool valid(int64_t k) const { return first_row + k * row_step < rows; }
};

// max over the first n partial maxima (every thread of the workgroup gets it).
__device__ __forceinline__ float reduce_parts(const float* __restrict__ part, int n) {
  __shared__ float red[kQWaves];
  float m = 0.f;
  for (int i = threadIdx.x; i < n; i += kQThreads) m = fmaxf(m, part[i]);
  m = wave_max(m);
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = m;
  __syncthreads();
  m = red[0];
#pragma unroll
  for (int i = 1; i < kQWaves; ++i) m = fmaxf(m, red[i]);
  return m;
}

// Position of this workgroup in a launch over two (possibly batched) jobs: which job, the
// batch b inside it, and the workgroup index within that batch.
struct QPos {
  bool second;
  int b, wg;
};
__device__ __forceinline__ QPos qpos(const QJob& j0, const QJob& j1) {
  const int n0 = j0.wg * j0.batch;
  const bool second = (int)blockIdx.x >= n0;
  const int idx = second ? (int)blockIdx.x - n0 : (int)blockIdx.x;
  const int per = second ? j1.wg : j0.wg;
  return {second, idx / per, idx % per};
}

// Plain 16-byte copy: the reference kernel against which hardware traffic counters are
// calibrated (its bytes read and written are known exactly).
__global__ __launch_bounds__(256) void copy_kernel(const uint4* __restrict__ src,
                                                   uint4* __restrict__ dst, int64_t n) {
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += stride)
    dst[i] = src[i];
}

// Workgroups [0, j0.wg) serve job 0 and [j0.wg, j0.wg + j1.wg) job 1; each writes the
// maximum |FWHT| of its rows to part[its index within the job].
template <int DT, int LOG2B>
__global__ __launch_bounds__(kQThreads) void fwht_absmax_kernel(QJob j0, QJob j1,
                                                                float* __restrict__ part0,
                                                                float* __restrict__ part1) {
  // steps in flight: 2 measured faster than 4 (fewer registers, more waves per SIMD;
  // -5 % per FFN step's maximum passes, -9 % on the 4096..11008-wide sweep) and than 8
  constexpr int U = 2;
  __shared__ float red[kQWaves];
  const QPos q = qpos(j0, j1);
  const QJob& j = q.second ? j1 : j0;
  const int wg = q.wg;
  const Geo g(j, wg);
  constexpr int EB = Elem<DT>::bytes;
  float m = 0.f;
  const char* base = static_cast<const char*>(j.src) + ((int64_t)q.b * j.bstride + (int64_t)g.sub * kVE) * EB;
  int64_t k = 0;
  int it = 0;
  for (int64_t s0 = 0; s0 < g.steps; s0 += U) {
    float v[U][kVE];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      if (s0 + u < g.steps) {
        load16<DT, HQ_NT_ABS_LD>(base + (g.row_of(k) * j.cols + (int64_t)it * g.G * kVE) * EB, v[u]);
        if (++it == g.iters) { it = 0; ++k; }
      }
    }
#pragma unroll
    for (int u = 0; u < U; ++u) {
      if (s0 + u < g.steps) {  // duplicated rows leave the maximum unchanged
        fwht16<LOG2B>(v[u], g.lane);
#pragma unroll
        for (int e = 0; e < kVE; e += 2) m = fmaxf(m, fmaxf(fabsf(v[u][e]), fabsf(v[u][e + 1])));
      }
    }
  }
  m = wave_max(m);
  if (g.lane == 0) red[threadIdx.x >> 6] = m;
  __syncthreads();
  if (threadIdx.x == 0) {
#pragma unroll
    for (int i = 1; i < kQWaves; ++i) m = fmaxf(m, red[i]);
    m = fmaxf(m, red[0]);
    (q.second ? part1 : part0)[q.b * j.wg + wg] = m;
  }
}

// One tile of the second job (W), quantised by one workgroup: TW columns (whole Hadamard
// blocks) x R rows, 16 elements per lane as in the row kernels, so the transform and the
// rounding are the same operations on the same values.  The workgroup writes the tile's
// codes both ways: row-major from registers (as the row kernels do, with the fp16 deltas
// of the learned-step mode) and transposed through LDS (thread (d, q) packs rows
// 16 q .. 16 q + 15 of column d).  The tiles thus read W once and replace the row
// workgroups of that job.  Rows past the end are loaded from the last row and not stored.
template <int LOG2B> struct TileT {
  static constexpr int TW = (1 << LOG2B) > 64 ? 128 : 64;
  static constexpr int LPR = TW / kVE;         // lanes per row
  static constexpr int R = kQThreads / LPR;    // rows per tile
  __host__ __device__ static int64_t tiles(int64_t rows, int64_t cols) { return (rows + R - 1) / R * (cols / TW); }
};

// LSQ selects the learned-step quantiser: code clamp(rint(v inv), -7, 7) (the clamp first)
// and delta as in fwht_lsq_kernel; else the code rint(v inv) of fwht_quant_kernel.
template <int DT, int LOG2B, bool LSQ>
__device__ void quant_tile(const void* src, int64_t rows, int64_t cols, float inv, int t,
                           uint8_t* __restrict__ packed, uint16_t* __restrict__ delta,
                           uint8_t* __restrict__ packed_t, uint8_t* __restrict__ fp6 = nullptr) {
  using T = TileT<LOG2B>;
  constexpr int TW = T::TW, LPR = T::LPR, R = T::R, PITCH = TW + 4;
  __shared__ uint8_t tile[R * PITCH];
  constexpr int EB = Elem<DT>::bytes;
  const int64_t ntc = cols / TW;
  const int64_t r0 = (int64_t)(t / ntc) * R, c0 = (int64_t)(t % ntc) * TW;
  const int tid = threadIdx.x, rr = tid / LPR, sub = tid % LPR;
  {
    const bool ok = r0 + rr < rows;
    const int64_t r = ok ? r0 + rr : rows - 1;
    float v[kVE];
    load16<DT, HQ_NT_Q_LD>(static_cast<const char*>(src) + (r * cols + c0 + sub * kVE) * EB, v);
    fwht16<LOG2B>(v, tid & 63);
    uint32_t y[kVE], dh[kVE / 2];
#pragma unroll
    for (int e = 0; e < kVE; e += 2) {
      uint32_t h[2];
#pragma unroll
      for (int u = 0; u < 2; ++u) {
        const float x = v[e + u] * inv;
        if constexpr (LSQ) {
          const float rc = __builtin_amdgcn_fmed3f(x, -7.0f, 7.0f);
          const float m = rc + kRne;
          y[e + u] = __float_as_uint(m);
          const float q = m - kRne;
          const float d = (rc == x) ? q - x : q;
          h[u] = (uint32_t)__builtin_bit_cast(uint16_t, (_Float16)d);
        } else {
          y[e + u] = rne_bits(x);
          h[u] = 0u;
        }
      }
      dh[e / 2] = h[0] | (h[1] << 16);
    }
    const int64_t c = (c0 + sub * kVE) / kVE;  // 16-column chunk of the row
    const uint4 f6 = fp6 ? fp6_chunk16(y, (c & 1) != 0) : make_uint4(0u, 0u, 0u, 0u);  // all lanes
    if (ok) {
      st_stream2<HQ_NT_Q_ST>(reinterpret_cast<uint2*>(packed + r * (cols / 2)) + c,
                             make_uint2(pack8_bits(y), pack8_bits(y + 8)));
      if (fp6) store_fp6_chunk(fp6 + r * cols, c, f6);
      if constexpr (LSQ) {
        uint4* dp = reinterpret_cast<uint4*>(delta + r * cols) + 2 * c;
        st_stream<HQ_NT_Q_ST>(dp, make_uint4(dh[0], dh[1], dh[2], dh[3]));
        st_stream<HQ_NT_Q_ST>(dp + 1, make_uint4(dh[4], dh[5], dh[6], dh[7]));
      }
    }
    uint32_t* row = reinterpret_cast<uint32_t*>(tile + rr * PITCH + sub * kVE);
#pragma unroll
    for (int w = 0; w < 4; ++w)
      row[w] = (y[4 * w] & 15u) | ((y[4 * w + 1] & 15u) << 8) | ((y[4 * w + 2] & 15u) << 16) |
               ((y[4 * w + 3] & 15u) << 24);
  }
  __syncthreads();
  const int d = tid / (R / 16), q = tid % (R / 16);
  if (r0 + 16 * q < rows) {
    uint32_t w2[2] = {0u, 0u};
#pragma unroll
    for (int i = 0; i < 16; ++i) w2[i >> 3] |= (uint32_t)tile[(16 * q + i) * PITCH + d] << (4 * (i & 7));
    *reinterpret_cast<uint2*>(packed_t + (c0 + d) * (rows / 2) + r0 / 2 + 8 * q) = make_uint2(w2[0], w2[1]);
  }
}

// Codes of FWHT(rows) at the reduced maximum a; the first workgroup of each job also
// stores a.  When o1.packed_t is set, job 1 has no row workgroups (j1.wg = 0): workgroups
// past job 0's quantise it by tiles (quant_tile), writing its codes and their transpose.
// Row sums of squares are plain stores by the group's first lane.  The clamp to +-7 of the
// definition never engages here: |v| <= a gives |v * fl(7/a)| <= 7 (1 + 2^-24), which
// rounds to at most 7.
template <int DT, int LOG2B>
__global__ __launch_bounds__(kQThreads) void fwht_quant_kernel(QJob j0, QJob j1, QOut o0, QOut o1) {
  constexpr int U = 2;  // steps in flight (2 measured faster than 4, as for the maximum)
  if ((int)blockIdx.x >= j0.wg + j1.wg) {  // uniform per workgroup
    const float a = reduce_parts(o1.part, o1.nparts);
    const int t = (int)blockIdx.x - j0.wg - j1.wg;
    if (t == 0 && threadIdx.x == 0) *o1.amax_out = a;
    quant_tile<DT, LOG2B, false>(j1.src, j1.rows, j1.cols, a > 0.f ? 7.0f / a : 0.f, t, o1.packed,
                                 nullptr, o1.packed_t, o1.fp6);
    return;
  }
  const bool second = (int)blockIdx.x >= j0.wg;
  const QJob& j = second ? j1 : j0;
  const QOut& o = second ? o1 : o0;
  const int wg = second ? (int)blockIdx.x - j0.wg : (int)blockIdx.x;
  const float a = reduce_parts(o.part, o.nparts);
  if (wg == 0 && threadIdx.x == 0) *o.amax_out = a;
  const float inv = a > 0.f ? 7.0f / a : 0.f;
  const Geo g(j, wg);
  constexpr int EB = Elem<DT>::bytes;
  const char* base = static_cast<const char*>(j.src) + (int64_t)g.sub * kVE * EB;
  int64_t k = 0, kp = 0;  // load and process positions
  int it = 0, ip = 0;
  int ss = 0;
  for (int64_t s0 = 0; s0 < g.steps; s0 += U) {
    float v[U][kVE];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      if (s0 + u < g.steps) {
        load16<DT, HQ_NT_Q_LD>(base + (g.row_of(k) * j.cols + (int64_t)it * g.G * kVE) * EB, v[u]);
        if (++it == g.iters) { it = 0; ++k; }
      }
    }
#pragma unroll
    for (int u = 0; u < U; ++u) {
      if (s0 + u < g.steps) {
        fwht16<LOG2B>(v[u], g.lane);
        uint32_t y[kVE];
#pragma unroll
        for (int e = 0; e < kVE; ++e) y[e] = rne_bits(v[u][e] * inv);
        const uint32_t w0 = pack8_bits(y), w1 = pack8_bits(y + 8);
        ss = sumsq8(w1, sumsq8(w0, ss));
        const bool ok = g.valid(kp);
        const int64_t r = g.row_of(kp);
        if (ok) st_stream2<HQ_NT_Q_ST>(reinterpret_cast<uint2*>(o.packed + r * (j.cols / 2)) + (int64_t)ip * g.G + g.sub, make_uint2(w0, w1));
        if (o.fp6) {  // the pair exchange runs in every lane, the store only in valid rows
          const int64_t c = (int64_t)ip * g.G + g.sub;
          const uint4 f6 = fp6_chunk16(y, (c & 1) != 0);
          if (ok) store_fp6_chunk(o.fp6 + r * j.cols, c, f6);
        }
        if (++ip == g.iters) {  // end of the group's row
          if (o.row_sumsq) {
            ss = group_sum(ss, g.G);
            if (ok && g.sub == 0) o.row_sumsq[r] = ss;
          }
          ss = 0;
          ip = 0;
          ++kp;
        }
      }
    }
  }
}

// Learned-step-size codes (Eq. 2 at a caller-given step, after the transform of Sec. 3.3):
// r = fl(v * fl(1/s)), q = clamp(rint(r), -7, 7) and delta = q - [-7 <= r <= 7] r, the
// term that the step-size gradient weights (App. A.3).  One pass: no maximum is needed.
// The clamp comes first (med3), so the magic-number rounding only sees |x| <= 7, and
// rint(clamp(r)) = clamp(rint(r)) as the bounds are integers.  q - r is exact in fp32 (q
// and r lie within a factor of two of each other, or q = 0), then rounded to fp16 (to
// nearest even); |delta| <= 1/2 holds exactly for the entries inside the range and
// |delta| > 1/2 for the clipped ones, so the gradient kernels recover the clip indicator
// from delta alone.
template <int DT, int LOG2B>
__global__ __launch_bounds__(kQThreads) void fwht_lsq_kernel(QJob j0, QJob j1, LsqOut o0, LsqOut o1) {
  // one step in flight: 70-73 registers instead of 96, three workgroups per CU instead of
  // two (the BMM's quantiser 31.3 -> 28.9 us; the FFN's unchanged)
  constexpr int U = 1;
  {  // o1.packed_t set: job 1 by tiles (j1.wg = 0), one tile per workgroup past job 0's
    const int nrow = j0.wg * j0.batch + j1.wg * j1.batch;
    if ((int)blockIdx.x >= nrow) {  // uniform per workgroup
      const int nt = (int)TileT<LOG2B>::tiles(j1.rows, j1.cols);
      const int tt = (int)blockIdx.x - nrow, b = tt / nt;
      const int64_t rc = j1.rows * j1.cols;  // elements of one batch
      quant_tile<DT, LOG2B, true>(static_cast<const char*>(j1.src) + (int64_t)b * j1.bstride * Elem<DT>::bytes,
                                  j1.rows, j1.cols, 1.0f / o1.step[b], tt % nt, o1.packed + b * (rc / 2),
                                  o1.delta + b * rc, o1.packed_t + b * (rc / 2));
      return;
    }
  }
  const QPos qp = qpos(j0, j1);
  const QJob& j = qp.second ? j1 : j0;
  const LsqOut& o = qp.second ? o1 : o0;
  const int wg = qp.wg;
  const float inv = 1.0f / o.step[qp.b];
  const Geo g(j, wg);
  constexpr int EB = Elem<DT>::bytes;
  const char* base = static_cast<const char*>(j.src) + ((int64_t)qp.b * j.bstride + (int64_t)g.sub * kVE) * EB;
  // this batch's outputs
  uint8_t* const packed = o.packed + (int64_t)qp.b * j.rows * (j.cols / 2);
  uint16_t* const delta = o.delta + (int64_t)qp.b * j.rows * j.cols;
  int32_t* const row_sumsq = o.row_sumsq ? o.row_sumsq + (int64_t)qp.b * j.rows : nullptr;
  int64_t k = 0, kp = 0;
  int it = 0, ip = 0;
  int ss = 0;
  for (int64_t s0 = 0; s0 < g.steps; s0 += U) {
    float v[U][kVE];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      if (s0 + u < g.steps) {
        load16<DT, HQ_NT_Q_LD>(base + (g.row_of(k) * j.cols + (int64_t)it * g.G * kVE) * EB, v[u]);
        if (++it == g.iters) { it = 0; ++k; }
      }
    }
#pragma unroll
    for (int u = 0; u < U; ++u) {
      if (s0 + u < g.steps) {
        fwht16<LOG2B>(v[u], g.lane);
        uint32_t y[kVE], dh[kVE / 2];
#pragma unroll
        for (int e = 0; e < kVE; e += 2) {
          uint32_t h[2];
#pragma unroll
          for (int t = 0; t < 2; ++t) {
            const float r = v[u][e + t] * inv;
            const float rc = __builtin_amdgcn_fmed3f(r, -7.0f, 7.0f);
            const float m = rc + kRne;
            y[e + t] = __float_as_uint(m);
            const float q = m - kRne;
            const float d = (rc == r) ? q - r : q;
            h[t] = (uint32_t)__builtin_bit_cast(uint16_t, (_Float16)d);
          }
          dh[e / 2] = h[0] | (h[1] << 16);
        }
        const uint32_t w0 = pack8_bits(y), w1 = pack8_bits(y + 8);
        ss = sumsq8(w1, sumsq8(w0, ss));
        const bool ok = g.valid(kp);
        const int64_t r = g.row_of(kp);
        if (ok) {
          const int64_t c = (int64_t)ip * g.G + g.sub;  // 16-column chunk
          st_stream2<HQ_NT_Q_ST>(reinterpret_cast<uint2*>(packed + r * (j.cols / 2)) + c, make_uint2(w0, w1));
          uint4* dp = reinterpret_cast<uint4*>(delta + r * j.cols) + 2 * c;
          st_stream<HQ_NT_Q_ST>(dp, make_uint4(dh[0], dh[1], dh[2], dh[3]));
          st_stream<HQ_NT_Q_ST>(dp + 1, make_uint4(dh[4], dh[5], dh[6], dh[7]));
        }
        if (++ip == g.iters) {
          if (row_sumsq) {
            ss = group_sum(ss, g.G);
            if (ok && g.sub == 0) row_sumsq[r] = ss;
          }
          ss = 0;
          ip = 0;
          ++kp;
        }
      }
    }
  }
}

// Bit split of dY [N][C] (no transform: the gradient is split as it is, Sec. 4.2) and the
// integer leverage scores of the two stacked rows of every token:
//   c_up = isqrt(14^2 sum q_up^2 * x_sumsq * 2^16),  c_dn = isqrt(sum q_dn^2 * x_sumsq * 2^16)
// (the common factor s_dn s_x dropped).  Each workgroup stores the count of non-zero scores
// and their sum (u64) of its rows as one partial.
template <int DT>
__global__ __launch_bounds__(kQThreads) void bit_split_kernel(QJob j, const float* __restrict__ part,
                                                              int nparts, BsOut o, uint64_t seed,
                                                              uint64_t offset) {
  // one 16-element step per loop pass: the Philox state and the two code planes already
  // hold many registers, and one step (more waves per SIMD) measured 9 % faster than two
  constexpr int U = 1;
  __shared__ uint64_t red_s[kQWaves];
  __shared__ uint32_t red_n[kQWaves];
  // batch b of a batched job: its own maximum, outputs and Philox counter range
  const int b = (int)blockIdx.x / j.wg, wg = (int)blockIdx.x % j.wg;
  const float a = reduce_parts(part + (int64_t)b * nparts, nparts);
  if (wg == 0 && threadIdx.x == 0) o.amax_out[b] = a;
  const float inv = a > 0.f ? 7.0f / a : 0.f;
  // -0.0f, from an argument so that the fma below is not folded into a multiply
  const float nzero = __uint_as_float(0x80000000u | (uint32_t)((uint64_t)j.cols >> 63));
  const Geo g(j, wg);
  const int64_t C = j.cols;
  constexpr int EB = Elem<DT>::bytes;
  uint32_t nnz = 0;
  uint64_t ssum = 0;
  const char* base = static_cast<const char*>(j.src) + ((int64_t)b * j.bstride + (int64_t)g.sub * kVE) * EB;
  offset += (uint64_t)b * o.offset_stride;
  const int64_t rb = (int64_t)b * j.rows;  // first row of this batch in the row-indexed outputs
  uint8_t* const qup = o.qup + rb * (C / 2);
  uint8_t* const qdn = o.qdn + rb * (C / 2);
  uint32_t* const scores = o.scores + (int64_t)b * 2 * o.score_pitch;
  // a row's sums of squared codes are at most 49 C (codes within +-7); below 2^15 both fit
  // one int in 16-bit halves without reaching its sign bit
  const bool packed_sums = 49 * C < 32768;
  int64_t k = 0, kp = 0;
  int it = 0, ip = 0;
  int su = 0, sd = 0;
  for (int64_t s0 = 0; s0 < g.steps; s0 += U) {
    float v[U][kVE];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      if (s0 + u < g.steps) {
        load16<DT, HQ_NT_BS_LD>(base + (g.row_of(k) * C + (int64_t)it * g.G * kVE) * EB, v[u]);
        if (++it == g.iters) { it = 0; ++k; }
      }
    }
#pragma unroll
    for (int u = 0; u < U; ++u) {
      if (s0 + u < g.steps) {
        const bool ok = g.valid(kp);
        const int64_t r = g.row_of(kp);
        const int64_t col = ((int64_t)ip * g.G + g.sub) * kVE;
        uint32_t yu[kVE], yd[kVE];
#pragma unroll
        for (int h = 0; h < 2; ++h) {
          const U4 rnd = philox_block(seed, offset, 0u, (uint64_t)(r * C + col + 8 * h));
#pragma unroll
          for (int e = 0; e < 8; ++e) {
            // fl(v inv): one rounding, so the fma with a -0 addend equals the product
            // (an fp16 operand widens inside the instruction)
            const float x = __builtin_fmaf(v[u][8 * h + e], inv, nzero);
            const uint32_t bu = rne_bits(x);                  // |x| <= 7 (1 + 2^-23)
            // -14 rint(x) exactly from the bits 1.5 * 2^23 + rint(x); then
            // fl(14 x - 14 rint(x)) = fl(14 (x - rint(x))), the residual being exact
            const float m14 = __builtin_fmaf(__uint_as_float(bu), -14.0f, 14.0f * kRne);
            const float w = __builtin_fmaf(x, 14.0f, m14);   // |w| <= 7
            const float fl = floorf(w);
            const float thr = (w - fl) * 65536.0f;
            const uint32_t bd = __float_as_uint(fl + kRne);   // floor(w) in the low bits
            yu[8 * h + e] = bu;
            yd[8 * h + e] = bd + (((float)u16_of(rnd, e) < thr) ? 1u : 0u);
          }
        }
        const uint32_t u0 = pack8_bits(yu), u1 = pack8_bits(yu + 8);
        const uint32_t d0 = pack8_bits(yd), d1 = pack8_bits(yd + 8);
        su = sumsq8(u1, sumsq8(u0, su));
        sd = sumsq8(d1, sumsq8(d0, sd));
        if (ok) {
          const int64_t o8 = r * (C / 16) + (int64_t)ip * g.G + g.sub;  // uint2 index
          st_stream2<HQ_NT_BS_ST>(reinterpret_cast<uint2*>(qup) + o8, make_uint2(u0, u1));
          st_stream2<HQ_NT_BS_ST>(reinterpret_cast<uint2*>(qdn) + o8, make_uint2(d0, d1));
        }
        if (++ip == g.iters) {  // end of the group's row
          if (packed_sums) {  // one reduction of the two halves
            const int p = group_sum(su | (sd << 16), g.G);
            su = p & 0xFFFF;
            sd = (int)((uint32_t)p >> 16);
          } else {
            su = group_sum(su, g.G);
            sd = group_sum(sd, g.G);
          }
          // the group's lane 0 forms the upper row's score and lane 1 the lower row's
          // (G >= 4), so a wave runs one square root per row end, not two in sequence
          if (ok && g.sub < 2) {
            const uint64_t sx = (uint32_t)o.x_sumsq[rb + r];
            const bool upper = g.sub == 0;
            const uint64_t k2 = upper ? (uint64_t)(kBsRatio * kBsRatio) * (uint32_t)su : (uint64_t)(uint32_t)sd;
            const uint32_t c = isqrt64((k2 * sx) << 16);
            if (upper) {
              o.sumsq_up[rb + r] = su;
              o.sumsq_dn[rb + r] = sd;
            }
            scores[(upper ? 0 : o.score_pitch) + r] = c;
            nnz += c > 0;
            ssum += c;
          }
          su = sd = 0;
          ip = 0;
          ++kp;
        }
      }
    }
  }
  nnz = (uint32_t)wave_sum((int)nnz);
  ssum = wave_sum_u64(ssum);
  if (g.lane == 0) {
    red_n[threadIdx.x >> 6] = nnz;
    red_s[threadIdx.x >> 6] = ssum;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    uint32_t n = 0;
    uint64_t t = 0;
#pragma unroll
    for (int i = 0; i < kQWaves; ++i) {
      n += red_n[i];
      t += red_s[i];
    }
    o.parts[(int64_t)b * j.wg + wg] = make_uint4(n, (uint32_t)t, (uint32_t)(t >> 32), 0u);
  }
}

// ---------------------------------------------------------------- block-size search
// Choice of the Hadamard block 2^k (App. A.5): k minimising MSE(X_bar, X) MSE(W_bar, W),
// V_bar = s int_s(V H) H^T.  The transform with strides ascending is nested: after the
// stages of strides 1 .. 2^(k-1) every 2^k block holds its own FWHT, so one pass over the
// data yields the transforms of all k = 0..7 in turn.  The error is taken in the transform
// domain, ||V_bar - V||^2 = ||s q - V H_u||^2 / 2^k (H_u / 2^(k/2) is orthogonal), so it
// needs no inverse transform.  For D not a multiple of 128 the deepest stages mix blocks
// that are no candidates; their values are computed and never used.
constexpr int kLevels = 8;  // k = 0 .. 7
static_assert(kQWaves == kLevels, "pass 2 reduces one level per wave");

// One butterfly stage at stride H (in-lane for H < 16, else across lanes H / 16 apart).
template <int H>
__device__ __forceinline__ void fwht_stage(float v[16], int lane) {
  if constexpr (H < 16) {
#pragma unroll
    for (int j = 0; j < 16; ++j) {
      if ((j & H) == 0) {
        const float a = v[j], c = v[j + H];
        v[j] = a + c;
        v[j + H] = a - c;
      }
    }
  } else {
    constexpr int M = H / 16;
    const uint32_t sgn = (lane & M) ? 0x80000000u : 0u;
#pragma unroll
    for (int j = 0; j < 16; ++j) {
      const float own = __uint_as_float(__float_as_uint(v[j]) ^ sgn);
      v[j] = add_xor_lane<M>(v[j], own);
    }
  }
}

// Calls f(level, v) for level 0 (the input) and after each of the 7 stages.
template <class F>
__device__ __forceinline__ void fwht_nested(float v[16], int lane, F&& f) {
  f(0, v);
  fwht_stage<1>(v, lane);  f(1, v);
  fwht_stage<2>(v, lane);  f(2, v);
  fwht_stage<4>(v, lane);  f(3, v);
  fwht_stage<8>(v, lane);  f(4, v);
  fwht_stage<16>(v, lane); f(5, v);
  fwht_stage<32>(v, lane); f(6, v);
  fwht_stage<64>(v, lane); f(7, v);
}

// Pass 1: per-workgroup maxima of |FWHT_k(rows)| for every k, part[wg * 8 + k].
template <int DT>
__global__ __launch_bounds__(kQThreads) void hsize_max_kernel(QJob j0, QJob j1,
                                                              float* __restrict__ part0,
                                                              float* __restrict__ part1) {
  constexpr int U = 2;
  __shared__ float red[kQWaves][kLevels];
  const bool second = (int)blockIdx.x >= j0.wg;
  const QJob& j = second ? j1 : j0;
  const int wg = second ? (int)blockIdx.x - j0.wg : (int)blockIdx.x;
  const Geo g(j, wg);
  constexpr int EB = Elem<DT>::bytes;
  float m[kLevels];
#pragma unroll
  for (int l = 0; l < kLevels; ++l) m[l] = 0.f;
  const char* base = static_cast<const char*>(j.src) + (int64_t)g.sub * kVE * EB;
  int64_t k = 0;
  int it = 0;
  for (int64_t s0 = 0; s0 < g.steps; s0 += U) {
    float v[U][kVE];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      if (s0 + u < g.steps) {
        load16<DT, HQ_NT_ABS_LD>(base + (g.row_of(k) * j.cols + (int64_t)it * g.G * kVE) * EB, v[u]);
        if (++it == g.iters) { it = 0; ++k; }
      }
    }
#pragma unroll
    for (int u = 0; u < U; ++u) {
      if (s0 + u < g.steps) {  // duplicated rows leave the maxima unchanged
        fwht_nested(v[u], g.lane, [&](int l, const float* x) {
#pragma unroll
          for (int e = 0; e < kVE; e += 2) m[l] = fmaxf(m[l], fmaxf(fabsf(x[e]), fabsf(x[e + 1])));
        });
      }
    }
  }
#pragma unroll
  for (int l = 0; l < kLevels; ++l) {
    const float w = wave_max(m[l]);
    if (g.lane == 0) red[threadIdx.x >> 6][l] = w;
  }
  __syncthreads();
  if (threadIdx.x < kLevels) {
    float r = red[0][threadIdx.x];
#pragma unroll
    for (int i = 1; i < kQWaves; ++i) r = fmaxf(r, red[i][threadIdx.x]);
    (second ? part1 : part0)[wg * kLevels + threadIdx.x] = r;
  }
}

// Pass 2: per-workgroup sums over valid rows of (s_k q - v)^2 for every k, with
// s_k = fl(a_k / 7) and q = rint(v fl(7 / a_k)) the forward quantiser's codes (no clamp
// needed, as there).  Each 16-element chunk is summed in fp32 (one fused multiply-add
// per element on the correctly rounded difference), chunks in fp64; err[wg * 8 + k].
template <int DT>
__global__ __launch_bounds__(kQThreads) void hsize_err_kernel(QJob j0, QJob j1,
                                                              const float* __restrict__ mx0, int n0,
                                                              const float* __restrict__ mx1, int n1,
                                                              double* __restrict__ err0,
                                                              double* __restrict__ err1) {
  constexpr int U = 2;
  __shared__ float amax[kLevels];
  __shared__ double red[kQWaves][kLevels];
  const bool second = (int)blockIdx.x >= j0.wg;
  const QJob& j = second ? j1 : j0;
  const int wg = second ? (int)blockIdx.x - j0.wg : (int)blockIdx.x;
  {  // a_k = max over the pass-1 partials of this tensor: 64 lanes per level
    const float* mx = second ? mx1 : mx0;
    const int n = second ? n1 : n0;
    const int l = threadIdx.x >> 6, lane = threadIdx.x & 63;  // 8 waves = 8 levels
    float r = 0.f;
    for (int i = lane; i < n; i += 64) r = fmaxf(r, mx[i * kLevels + l]);
    r = wave_max(r);
    if (lane == 0) amax[l] = r;
    __syncthreads();
  }
  float inv[kLevels], st[kLevels];
#pragma unroll
  for (int l = 0; l < kLevels; ++l) {
    const float a = amax[l];
    inv[l] = a > 0.f ? 7.0f / a : 0.f;
    st[l] = a / 7.0f;
  }
  const Geo g(j, wg);
  constexpr int EB = Elem<DT>::bytes;
  double acc[kLevels];
#pragma unroll
  for (int l = 0; l < kLevels; ++l) acc[l] = 0.0;
  const char* base = static_cast<const char*>(j.src) + (int64_t)g.sub * kVE * EB;
  int64_t k = 0, kp = 0;
  int it = 0, ip = 0;
  for (int64_t s0 = 0; s0 < g.steps; s0 += U) {
    float v[U][kVE];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      if (s0 + u < g.steps) {
        load16<DT, HQ_NT_ABS_LD>(base + (g.row_of(k) * j.cols + (int64_t)it * g.G * kVE) * EB, v[u]);
        if (++it == g.iters) { it = 0; ++k; }
      }
    }
#pragma unroll
    for (int u = 0; u < U; ++u) {
      if (s0 + u < g.steps) {
        const bool ok = g.valid(kp);
        fwht_nested(v[u], g.lane, [&](int l, const float* x) {
          float e2 = 0.f;
#pragma unroll
          for (int e = 0; e < kVE; ++e) {
            const float q = __builtin_rintf(x[e] * inv[l]);
            const float d = __builtin_fmaf(st[l], q, -x[e]);
            e2 = __builtin_fmaf(d, d, e2);
          }
          acc[l] += ok ? (double)e2 : 0.0;
        });
        if (++ip == g.iters) { ip = 0; ++kp; }
      }
    }
  }
#pragma unroll
  for (int l = 0; l < kLevels; ++l) {
    double w = acc[l];
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) w += __shfl_xor(w, o);
    if (g.lane == 0) red[threadIdx.x >> 6][l] = w;
  }
  __syncthreads();
  if (threadIdx.x < kLevels) {
    double r = red[0][threadIdx.x];
#pragma unroll
    for (int i = 1; i < kQWaves; ++i) r += red[i][threadIdx.x];
    (second ? err1 : err0)[wg * kLevels + threadIdx.x] = r;
  }
}

// Pass 3 (one workgroup of 256): MSE_k = sum / (2^k numel) per tensor, the candidates
// k <= kmax with cols % 2^k == 0, and the argmin of MSE_X MSE_W (ties to the smaller k).
// mse_out[k] = MSE_X(k), mse_out[8 + k] = MSE_W(k), NaN for k not a candidate.
__global__ __launch_bounds__(256) void hsize_pick_kernel(const double* __restrict__ err0, int n0,
                                                         const double* __restrict__ err1, int n1,
                                                         double numel0, double numel1, int64_t cols,
                                                         int kmax, int32_t* __restrict__ k_out,
                                                         double* __restrict__ mse_out) {
  __shared__ double red[2][32][kLevels];
  const int l = threadIdx.x & 7, slot = threadIdx.x >> 3;  // 32 slots per level
  double a = 0.0, b = 0.0;
  for (int i = slot; i < n0; i += 32) a += err0[i * kLevels + l];
  for (int i = slot; i < n1; i += 32) b += err1[i * kLevels + l];
  red[0][slot][l] = a;
  red[1][slot][l] = b;
  __syncthreads();
  if (threadIdx.x == 0) {
    int best = 0;
    double best_obj = 0.0;
    bool any = false;
    for (int k = 0; k < kLevels; ++k) {
      double sx = 0.0, sw = 0.0;
      for (int i = 0; i < 32; ++i) {
        sx += red[0][i][k];
        sw += red[1][i][k];
      }
      const double scale = (double)(1 << k);
      const double mx = numel0 > 0 ? sx / (scale * numel0) : 0.0;
      const double mw = numel1 > 0 ? sw / (scale * numel1) : 0.0;
      const bool cand = k <= kmax && cols % (int64_t(1) << k) == 0;
      const double nan = __longlong_as_double(0x7FF8000000000000LL);
      mse_out[k] = cand ? mx : nan;
      mse_out[kLevels + k] = cand ? mw : nan;
      if (cand) {
        const double obj = mx * mw;
        if (!any || obj < best_obj) {
          best = k;
          best_obj = obj;
          any = true;
        }
      }
    }
    *k_out = best;
  }
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

// Workgroups of kernel f that fit on the device at once (cached per kernel).
int resident_wgs(const void* f) {
  static std::mutex mu;
  static std::unordered_map<const void*, int> cache;
  std::lock_guard<std::mutex> lock(mu);
  auto it = cache.find(f);
  if (it != cache.end()) return it->second;
  int dev = 0, cus = 0, per = 0;
  if (hipGetDevice(&dev) != hipSuccess ||
      hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
      hipOccupancyMaxActiveBlocksPerMultiprocessor(&per, f, kQThreads, 0) != hipSuccess)
    return 256;
  int n = (per > 0 ? per : 1) * (cus > 0 ? cus : 1);
  if (n > kQMaxWg) n = kQMaxWg;
  cache.emplace(f, n);
  return n;
}

int64_t wgs_needed(const QJob& j) {
  if (j.rows <= 0) return 0;
  const int64_t per = (int64_t)(64 >> j.log2g) * kQWaves;
  return (j.rows + per - 1) / per;
}

// Share one resident grid between two jobs: all they need if it fits, else in proportion
// to their sizes (each at least one workgroup).
void fit_grid(QJob& a, QJob& b, int cap) {
  const int64_t na = wgs_needed(a), nb = wgs_needed(b);  // per batch
  if (na * a.batch + nb * b.batch <= cap) {
    a.wg = (int)na;
    b.wg = (int)nb;
    return;
  }
  if (a.batch > 1 || b.batch > 1) {
    // batched: about two resident rounds shared by size, then per batch (many small
    // batches would otherwise get one workgroup each and leave the CUs half occupied);
    // at most kBatchWgSlack + batch workgroups per job in all (the partials bound)
    const double sa = (double)a.rows * a.cols * a.batch, sb = (double)b.rows * b.cols * b.batch;
    const int64_t c2 = 2 * (int64_t)cap;
    const int64_t ca = nb ? (int64_t)(c2 * sa / (sa + sb)) : c2, cb = c2 - ca;
    auto per = [](int64_t c, int64_t n, int64_t batch) {
      int64_t w = (c + batch - 1) / batch;
      if (w > n) w = n;
      return (int)(w < 1 ? 1 : w);
    };
    a.wg = na ? per(ca, na, a.batch) : 0;
    b.wg = nb ? per(cb, nb, b.batch) : 0;
    return;
  }
  const double ba = (double)a.rows * a.cols, bb = (double)b.rows * b.cols;
  int64_t wb = nb ? (int64_t)(cap * bb / (ba + bb) + 0.5) : 0;
  if (nb && wb < 1) wb = 1;
  if (wb > nb) wb = nb;
  int64_t wa = cap - wb;
  if (na && wa < 1) wa = 1;
  if (wa > na) wa = na;
  a.wg = (int)wa;
  b.wg = (int)wb;
}

template <int DT, int LOG2B> struct AbsmaxF {
  static hipError_t run(hipStream_t s, QJob& j0, QJob& j1, float* p0, float* p1) {
    const void* f = reinterpret_cast<const void*>(&fwht_absmax_kernel<DT, LOG2B>);
    fit_grid(j0, j1, resident_wgs(f));
    timing_begin(s);
    fwht_absmax_kernel<DT, LOG2B><<<j0.wg * j0.batch + j1.wg * j1.batch, kQThreads, 0, s>>>(j0, j1, p0, p1);
    timing_end(s, kKAbsmax);
    return hipGetLastError();
  }
};
template <int DT, int LOG2B> struct QuantF {
  static hipError_t run(hipStream_t s, QJob j0, QJob j1, QOut o0, QOut o1) {
    const void* f = reinterpret_cast<const void*>(&fwht_quant_kernel<DT, LOG2B>);
    int64_t nt = 0;
    if (o1.packed_t) {  // job 1 by tiles only
      QJob none = make_job(nullptr, 0, j1.cols);
      fit_grid(j0, none, resident_wgs(f));
      j1.wg = 0;
      nt = TileT<LOG2B>::tiles(j1.rows, j1.cols);
    } else {
      fit_grid(j0, j1, resident_wgs(f));
    }
    timing_begin(s);
    fwht_quant_kernel<DT, LOG2B><<<(unsigned)(j0.wg + j1.wg + nt), kQThreads, 0, s>>>(j0, j1, o0, o1);
    timing_end(s, kKQuant);
    return hipGetLastError();
  }
};

template <int DT, int LOG2B> struct LsqF {
  static hipError_t run(hipStream_t s, QJob j0, QJob j1, LsqOut o0, LsqOut o1) {
    const void* f = reinterpret_cast<const void*>(&fwht_lsq_kernel<DT, LOG2B>);
    int64_t nt = 0;
    if (o1.packed_t) {  // job 1 by tiles only
      QJob none = make_job(nullptr, 0, j1.cols);
      fit_grid(j0, none, resident_wgs(f));
      j1.wg = 0;
      nt = TileT<LOG2B>::tiles(j1.rows, j1.cols) * j1.batch;
    } else {
      fit_grid(j0, j1, resident_wgs(f));
    }
    timing_begin(s);
    fwht_lsq_kernel<DT, LOG2B><<<(unsigned)(j0.wg * j0.batch + j1.wg * j1.batch + nt), kQThreads, 0, s>>>(
        j0, j1, o0, o1);
    timing_end(s, kKLsqQuant);
    return hipGetLastError();
  }
};

int log2_group(int64_t cols) {
  const int64_t v = cols / kVE;
  int l = 0;
  while (l < 6 && v % (int64_t(2) << l) == 0) ++l;
  return l;
}

}  // namespace

QJob make_job(const void* src, int64_t rows, int64_t cols) {
  QJob j{src, rows > 0 ? rows : 0, cols, log2_group(cols), 0, 1, (rows > 0 ? rows : 0) * cols};
  return j;
}

QJob make_job_batched(const void* src, int64_t batch, int64_t rows, int64_t cols) {
  QJob j = make_job(src, rows, cols);
  j.batch = (int)batch;
  return j;
}

hipError_t launch_copy(hipStream_t s, const void* src, void* dst, int64_t bytes) {
  const int64_t n = bytes / 16;
  int64_t wg = (n + 255) / 256;
  if (wg > 4096) wg = 4096;
  if (wg < 1) wg = 1;
  timing_begin(s);
  copy_kernel<<<(int)wg, 256, 0, s>>>(static_cast<const uint4*>(src), static_cast<uint4*>(dst), n);
  timing_end(s, kKCopy);
  return hipGetLastError();
}

hipError_t launch_fwht_absmax(hipStream_t s, int dt, int log2b, QJob& j0, float* part0,
                              QJob& j1, float* part1) {
  switch (dt) {
    case kF32: return dispatch_block<AbsmaxF, kF32, hipStream_t, QJob&, QJob&, float*, float*>(log2b, s, j0, j1, part0, part1);
    case kF16: return dispatch_block<AbsmaxF, kF16, hipStream_t, QJob&, QJob&, float*, float*>(log2b, s, j0, j1, part0, part1);
    case kBF16: return dispatch_block<AbsmaxF, kBF16, hipStream_t, QJob&, QJob&, float*, float*>(log2b, s, j0, j1, part0, part1);
  }
  return hipErrorInvalidValue;
}

hipError_t launch_fwht_quant(hipStream_t s, int dt, int log2b, const QJob& j0, const QOut& o0,
                             const QJob& j1, const QOut& o1) {
  switch (dt) {
    case kF32: return dispatch_block<QuantF, kF32>(log2b, s, j0, j1, o0, o1);
    case kF16: return dispatch_block<QuantF, kF16>(log2b, s, j0, j1, o0, o1);
    case kBF16: return dispatch_block<QuantF, kBF16>(log2b, s, j0, j1, o0, o1);
  }
  return hipErrorInvalidValue;
}

hipError_t launch_fwht_lsq(hipStream_t s, int dt, int log2b, const QJob& j0, const LsqOut& o0,
                           const QJob& j1, const LsqOut& o1) {
  switch (dt) {
    case kF32: return dispatch_block<LsqF, kF32>(log2b, s, j0, j1, o0, o1);
    case kF16: return dispatch_block<LsqF, kF16>(log2b, s, j0, j1, o0, o1);
    case kBF16: return dispatch_block<LsqF, kBF16>(log2b, s, j0, j1, o0, o1);
  }
  return hipErrorInvalidValue;
}

hipError_t launch_bit_split(hipStream_t s, int dt, QJob& j, const float* part, int nparts,
                            const BsOut& o, uint64_t seed, uint64_t offset) {
  const void* f = dt == kF32 ? reinterpret_cast<const void*>(&bit_split_kernel<kF32>)
                  : dt == kF16 ? reinterpret_cast<const void*>(&bit_split_kernel<kF16>)
                               : reinterpret_cast<const void*>(&bit_split_kernel<kBF16>);
  QJob none = make_job(nullptr, 0, j.cols);
  fit_grid(j, none, resident_wgs(f));
  timing_begin(s);
  switch (dt) {
    case kF32:
      bit_split_kernel<kF32><<<j.wg * j.batch, kQThreads, 0, s>>>(j, part, nparts, o, seed, offset);
      break;
    case kF16:
      bit_split_kernel<kF16><<<j.wg * j.batch, kQThreads, 0, s>>>(j, part, nparts, o, seed, offset);
      break;
    case kBF16:
      bit_split_kernel<kBF16><<<j.wg * j.batch, kQThreads, 0, s>>>(j, part, nparts, o, seed, offset);
      break;
    default:
      return hipErrorInvalidValue;
  }
  timing_end(s, kKBitSplit);
  return hipGetLastError();
}


hipError_t launch_hsize_search(hipStream_t s, int dt, QJob& j0, QJob& j1, float* mx0, float* mx1,
                               double* err0, double* err1, int kmax, int32_t* k_out,
                               double* mse_out) {
  const void* fm = dt == kF32 ? reinterpret_cast<const void*>(&hsize_max_kernel<kF32>)
                   : dt == kF16 ? reinterpret_cast<const void*>(&hsize_max_kernel<kF16>)
                                : reinterpret_cast<const void*>(&hsize_max_kernel<kBF16>);
  const void* fe = dt == kF32 ? reinterpret_cast<const void*>(&hsize_err_kernel<kF32>)
                   : dt == kF16 ? reinterpret_cast<const void*>(&hsize_err_kernel<kF16>)
                                : reinterpret_cast<const void*>(&hsize_err_kernel<kBF16>);
  if (dt != kF32 && dt != kF16 && dt != kBF16) return hipErrorInvalidValue;
  QJob a0 = j0, a1 = j1;
  fit_grid(a0, a1, resident_wgs(fm));
  timing_begin(s);
  if (dt == kF32) hsize_max_kernel<kF32><<<a0.wg + a1.wg, kQThreads, 0, s>>>(a0, a1, mx0, mx1);
  else if (dt == kF16) hsize_max_kernel<kF16><<<a0.wg + a1.wg, kQThreads, 0, s>>>(a0, a1, mx0, mx1);
  else hsize_max_kernel<kBF16><<<a0.wg + a1.wg, kQThreads, 0, s>>>(a0, a1, mx0, mx1);
  timing_end(s, kKHsizeMax);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  QJob b0 = j0, b1 = j1;
  fit_grid(b0, b1, resident_wgs(fe));
  timing_begin(s);
  if (dt == kF32)
    hsize_err_kernel<kF32><<<b0.wg + b1.wg, kQThreads, 0, s>>>(b0, b1, mx0, a0.wg, mx1, a1.wg, err0, err1);
  else if (dt == kF16)
    hsize_err_kernel<kF16><<<b0.wg + b1.wg, kQThreads, 0, s>>>(b0, b1, mx0, a0.wg, mx1, a1.wg, err0, err1);
  else
    hsize_err_kernel<kBF16><<<b0.wg + b1.wg, kQThreads, 0, s>>>(b0, b1, mx0, a0.wg, mx1, a1.wg, err0, err1);
  timing_end(s, kKHsizeErr);
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  timing_begin(s);
  hsize_pick_kernel<<<1, 256, 0, s>>>(err0, b0.wg, err1, b1.wg, (double)j0.rows * (double)j0.cols,
                                      (double)j1.rows * (double)j1.cols, j0.cols, kmax, k_out,
                                      mse_out);
  timing_end(s, kKHsizePick);
  j0.wg = b0.wg;
  j1.wg = b1.wg;
  return hipGetLastError();
}

}  // namespace hqlss
