// Leverage-score sampling of the bit-split gradient rows and the GEMM operands it
// selects (gfx950).
//
// lss_plan (one workgroup of 1024 threads, each owning a contiguous run of tokens):
//   1. integer leverage scores of the 2N stacked rows (Sec. 4.2): with the common factor
//      s_dn s_x dropped, c^2 = w^2 * sum q^2 * x_sumsq (w = 14 for the upper row of a token,
//      1 for the lower one) and c = isqrt(c^2 * 2^16), exact;
//   2. inclusion probabilities by the clamp-and-rescale loop of App. A.2 with sum p = B, in
//      exact integers: clamp every row with (B - k) c >= S, then rescale the rest; repeat
//      until nothing new is clamped.  If no more than B rows have c > 0, every such row has
//      p = 1 (the "keep rows with norm > 0" rule the paper's implementation uses, App. A.6);
//   3. upper rows are kept iff non-zero; a lower row with p* < 1 gets p~ = 2^-e >= p*, the
//      smallest power of two (e <= 4, e <= 2 if the token's upper row is non-zero), and is
//      kept iff u16 < 2^(16-e) (Philox stream 1), weight m/p~ = 2^e;
//   4. kept tokens (w_up + w_dn > 0) are compacted in ascending order by a block-wide
//      prefix scan (wave scans with shuffles, then one LDS pass over wave totals).
//
// build_ag / build_dw_operands materialise, for the kept tokens only, the weighted integer
// rows A_t = 14 w_up q_up[t] + w_dn q_dn[t] (|A| <= 126, one int8 operand that carries the
// bit split and the 1/p factors together) and the gathered X^ rows, in the K-contiguous
// layouts the MFMA GEMM reads.  int8 operands use the "K-interleaved" byte order of the
// GEMM: inside every group of 8 consecutive k the bytes hold k = 0,2,4,6,1,3,5,7, the
// order in which a packed INT4 word unpacks for free.
#include "common.h"
#include "launch.h"

namespace hqlss {

namespace {

constexpr int kPlanThreads = 1024;
constexpr int kPlanWaves = kPlanThreads / kWave;

__device__ __forceinline__ uint32_t isqrt64(uint64_t x) {
  uint64_t r = (uint64_t)sqrt((double)x);
  while (r * r > x) --r;
  while ((r + 1) * (r + 1) <= x) ++r;
  return (uint32_t)r;
}

__device__ __forceinline__ uint64_t block_sum_u64(uint64_t v, uint64_t* red) {
  v = wave_sum_u64(v);
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = v;
  __syncthreads();
  uint64_t t = 0;
#pragma unroll
  for (int i = 0; i < kPlanWaves; ++i) t += red[i];
  __syncthreads();
  return t;
}

template <int TPT>
__global__ __launch_bounds__(kPlanThreads) void lss_plan_kernel(
    const int32_t* __restrict__ sumsq_up, const int32_t* __restrict__ sumsq_dn,
    const int32_t* __restrict__ x_sumsq, int N, int64_t B, uint64_t seed, uint64_t offset,
    uint8_t* __restrict__ w_up, uint8_t* __restrict__ w_dn, int32_t* __restrict__ kept,
    int32_t* __restrict__ n_kept) {
  __shared__ uint64_t red[kPlanWaves];
  __shared__ int wtot[kPlanWaves];
  const int tid = threadIdx.x, lane = tid & 63, wid = tid >> 6;
  const int t0 = tid * TPT;

  uint32_t cu[TPT], cd[TPT];
  uint64_t upmask = 0;  // bit j: the token's upper row is non-zero
  int nnz = 0;
#pragma unroll
  for (int j = 0; j < TPT; ++j) {
    const int t = t0 + j;
    cu[j] = cd[j] = 0;
    if (t < N) {
      const uint64_t su = (uint32_t)sumsq_up[t], sd = (uint32_t)sumsq_dn[t];
      const uint64_t sx = (uint32_t)x_sumsq[t];
      cu[j] = isqrt64(((uint64_t)(kBsRatio * kBsRatio) * su * sx) << 16);
      cd[j] = isqrt64((sd * sx) << 16);
      if (su) upmask |= 1ull << j;
    }
    nnz += (cu[j] > 0) + (cd[j] > 0);
  }
  const bool all_nonzero_kept = (int64_t)block_sum_u64((uint64_t)nnz, red) <= B;

  uint64_t clamp_u = 0, clamp_d = 0;
  int64_t R = 0;
  uint64_t S = 0;
  if (!all_nonzero_kept) {
    uint64_t loc = 0;
#pragma unroll
    for (int j = 0; j < TPT; ++j) loc += (uint64_t)cu[j] + cd[j];
    S = block_sum_u64(loc, red);
    int64_t k = 0;
    for (;;) {  // App. A.2: clamp p >= 1, rescale the rest, repeat (uniform across the block)
      R = B - k;
      uint64_t cnt = 0, sum = 0;
#pragma unroll
      for (int j = 0; j < TPT; ++j) {
        if (cu[j] && !((clamp_u >> j) & 1) && (uint64_t)R * cu[j] >= S) {
          clamp_u |= 1ull << j; ++cnt; sum += cu[j];
        }
        if (cd[j] && !((clamp_d >> j) & 1) && (uint64_t)R * cd[j] >= S) {
          clamp_d |= 1ull << j; ++cnt; sum += cd[j];
        }
      }
      const uint64_t ncl = block_sum_u64(cnt, red);
      if (ncl == 0) break;
      k += (int64_t)ncl;
      S -= block_sum_u64(sum, red);
    }
    R = B - k;
  }

  // weights and keep flags
  uint64_t keepmask = 0;
  int nkeep = 0;
  U4 rnd{0, 0, 0, 0};
#pragma unroll
  for (int j = 0; j < TPT; ++j) {
    const int t = t0 + j;
    if (t >= N) continue;
    if (j == 0 || (t & 7) == 0) rnd = philox_block(seed, offset, 1u, (uint64_t)(t & ~7));
    const uint32_t wu = (upmask >> j) & 1;
    uint32_t wd = 0;
    if (cd[j]) {
      if (all_nonzero_kept || ((clamp_d >> j) & 1)) {
        wd = 1;
      } else {
        const int cap = wu ? 2 : 4;
        const uint64_t rc = (uint64_t)R * cd[j];
        int e = 0;
        while (e < cap && (rc << (e + 1)) <= S) ++e;
        const uint32_t u = u16_of(rnd, t & 7);
        wd = (u < (1u << (16 - e))) ? (1u << e) : 0u;
      }
    }
    w_up[t] = (uint8_t)wu;
    w_dn[t] = (uint8_t)wd;
    if (wu + wd) { keepmask |= 1ull << j; ++nkeep; }
  }

  // block-wide exclusive scan of the per-thread keep counts
  int x = nkeep;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const int y = __shfl_up(x, o);
    if (lane >= o) x += y;
  }
  if (lane == 63) wtot[wid] = x;
  __syncthreads();
  int base = 0, total = 0;
#pragma unroll
  for (int i = 0; i < kPlanWaves; ++i) {
    base += (i < wid) ? wtot[i] : 0;
    total += wtot[i];
  }
  int pos = base + x - nkeep;
#pragma unroll
  for (int j = 0; j < TPT; ++j)
    if ((keepmask >> j) & 1) kept[pos++] = t0 + j;
  if (tid == 0) *n_kept = total;
}

__device__ __forceinline__ int sext4(uint32_t n) { return (int)(n ^ 8u) - 8; }

// 8 weighted values (k = 0..7) -> K-interleaved bytes: low word k = 0,2,4,6; high 1,3,5,7.
__device__ __forceinline__ uint2 interleave8(const int a[8]) {
  uint32_t lo = 0, hi = 0;
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    lo |= ((uint32_t)a[2 * j] & 0xFFu) << (8 * j);
    hi |= ((uint32_t)a[2 * j + 1] & 0xFFu) << (8 * j);
  }
  return make_uint2(lo, hi);
}

__device__ __forceinline__ void weighted8(uint32_t up, uint32_t dn, int wu, int wd, int a[8]) {
#pragma unroll
  for (int j = 0; j < 8; ++j)
    a[j] = kBsRatio * wu * sext4((up >> (4 * j)) & 15u) + wd * sext4((dn >> (4 * j)) & 15u);
}

template <int DT>
__global__ __launch_bounds__(256) void build_ag_kernel(
    const uint8_t* __restrict__ qup, const uint8_t* __restrict__ qdn,
    const uint8_t* __restrict__ w_up, const uint8_t* __restrict__ w_dn,
    const int32_t* __restrict__ kept, const int32_t* __restrict__ n_kept, int64_t N, int64_t C,
    int64_t D, int8_t* __restrict__ Ag, void* __restrict__ dX) {
  const int lane = threadIdx.x & 63;
  const int64_t nk = *n_kept;
  const int64_t rows = (nk + 127) / 128 * 128;  // GEMM row tiles read zeros past n_kept
  const int64_t nwaves = (int64_t)gridDim.x * 4;
  const int64_t last = rows > N ? rows : N;
  for (int64_t i = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6); i < last; i += nwaves) {
    if (i < rows) {
      const bool live = i < nk;
      const int64_t t = live ? kept[i] : 0;
      const int wu = live ? w_up[t] : 0, wd = live ? w_dn[t] : 0;
      for (int64_t c = lane * 8; c < C; c += 512) {
        uint2 o = make_uint2(0u, 0u);
        if (live) {
          const uint32_t up = *reinterpret_cast<const uint32_t*>(qup + t * (C / 2) + c / 2);
          const uint32_t dn = *reinterpret_cast<const uint32_t*>(qdn + t * (C / 2) + c / 2);
          int a[8];
          weighted8(up, dn, wu, wd, a);
          o = interleave8(a);
        }
        *reinterpret_cast<uint2*>(Ag + i * C + c) = o;
      }
    }
    // rows of dX that belong to dropped tokens are exactly zero
    if (dX && i < N && (w_up[i] + w_dn[i]) == 0) {
      const int64_t bytes = D * Elem<DT>::bytes;
      char* row = static_cast<char*>(dX) + i * bytes;
      for (int64_t o = lane * 16; o < bytes; o += 64 * 16)
        *reinterpret_cast<uint4*>(row + o) = make_uint4(0u, 0u, 0u, 0u);
    }
  }
}

__global__ __launch_bounds__(256) void build_dw_operands_kernel(
    const uint8_t* __restrict__ qup, const uint8_t* __restrict__ qdn,
    const uint8_t* __restrict__ w_up, const uint8_t* __restrict__ w_dn,
    const int32_t* __restrict__ kept, const int32_t* __restrict__ n_kept,
    const uint8_t* __restrict__ xq, int64_t N, int64_t C, int64_t D, int8_t* __restrict__ At,
    uint8_t* __restrict__ XtT) {
  __shared__ int8_t tile[64][65];  // [kept index][column]
  const int64_t nk = *n_kept;
  const int64_t kp = (nk + 127) / 128 * 128;
  const int64_t i0 = (int64_t)blockIdx.x * 64;
  if (i0 >= kp) return;
  const int64_t pitch = (N + 127) / 128 * 128;  // K pitch of At (bytes) and 2x of XtT
  const bool isA = (int64_t)blockIdx.y < C / 64;
  const int64_t col0 = isA ? (int64_t)blockIdx.y * 64 : ((int64_t)blockIdx.y - C / 64) * 64;
  const int tid = threadIdx.x;
  {
    const int r = tid >> 2, q = (tid & 3) * 16;  // 64 kept rows x 4 x 16 columns
    const int64_t i = i0 + r;
    int v[16];
#pragma unroll
    for (int j = 0; j < 16; ++j) v[j] = 0;
    if (i < nk) {
      const int64_t t = kept[i];
      if (isA) {
        const int wu = w_up[t], wd = w_dn[t];
        const uint2 up = *reinterpret_cast<const uint2*>(qup + t * (C / 2) + (col0 + q) / 2);
        const uint2 dn = *reinterpret_cast<const uint2*>(qdn + t * (C / 2) + (col0 + q) / 2);
        weighted8(up.x, dn.x, wu, wd, v);
        weighted8(up.y, dn.y, wu, wd, v + 8);
      } else {
        const uint2 x = *reinterpret_cast<const uint2*>(xq + t * (D / 2) + (col0 + q) / 2);
#pragma unroll
        for (int j = 0; j < 8; ++j) {
          v[j] = sext4((x.x >> (4 * j)) & 15u);
          v[8 + j] = sext4((x.y >> (4 * j)) & 15u);
        }
      }
    }
#pragma unroll
    for (int j = 0; j < 16; ++j) tile[r][q + j] = (int8_t)v[j];
  }
  __syncthreads();
  {
    const int c = tid >> 2, q = (tid & 3) * 16;  // 64 columns x 4 x 16 kept indices
    if (isA) {
      int a[16];
#pragma unroll
      for (int j = 0; j < 16; ++j) a[j] = tile[q + j][c];
      const uint2 lo = interleave8(a), hi = interleave8(a + 8);
      *reinterpret_cast<uint4*>(At + (col0 + c) * pitch + i0 + q) = make_uint4(lo.x, lo.y, hi.x, hi.y);
    } else {
      uint32_t w0 = 0, w1 = 0;
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        const uint32_t byte = ((uint32_t)tile[q + 2 * j][c] & 15u) |
                              (((uint32_t)tile[q + 2 * j + 1][c] & 15u) << 4);
        if (j < 4) w0 |= byte << (8 * j);
        else w1 |= byte << (8 * (j - 4));
      }
      *reinterpret_cast<uint2*>(XtT + (col0 + c) * (pitch / 2) + (i0 + q) / 2) = make_uint2(w0, w1);
    }
  }
}

template <int TPT>
hipError_t plan_t(hipStream_t s, const int32_t* su, const int32_t* sd, const int32_t* sx, int64_t N,
                  int64_t B, uint64_t seed, uint64_t offset, uint8_t* wu, uint8_t* wd,
                  int32_t* kept, int32_t* nk) {
  timing_begin(s);
  lss_plan_kernel<TPT><<<1, kPlanThreads, 0, s>>>(su, sd, sx, (int)N, B, seed, offset, wu, wd,
                                                   kept, nk);
  timing_end(s, kKPlan);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_lss_plan(hipStream_t s, const int32_t* sumsq_up, const int32_t* sumsq_dn,
                           const int32_t* x_sumsq, int64_t N, int64_t budget, uint64_t seed,
                           uint64_t offset, uint8_t* w_up, uint8_t* w_dn, int32_t* kept,
                           int32_t* n_kept) {
  const int64_t tpt = (N + kPlanThreads - 1) / kPlanThreads;
#define HQLSS_PLAN(T) \
  if (tpt <= T) return plan_t<T>(s, sumsq_up, sumsq_dn, x_sumsq, N, budget, seed, offset, w_up, w_dn, kept, n_kept)
  HQLSS_PLAN(1);
  HQLSS_PLAN(2);
  HQLSS_PLAN(4);
  HQLSS_PLAN(8);
  HQLSS_PLAN(16);
  HQLSS_PLAN(32);
  HQLSS_PLAN(64);
#undef HQLSS_PLAN
  return hipErrorInvalidValue;
}

hipError_t launch_build_ag(hipStream_t s, int dt, const uint8_t* qup, const uint8_t* qdn,
                           const uint8_t* w_up, const uint8_t* w_dn, const int32_t* kept,
                           const int32_t* n_kept, int64_t N, int64_t C, int64_t D, int8_t* Ag,
                           void* dX) {
  int64_t wg = (N + 3) / 4;
  if (wg > 4096) wg = 4096;
  timing_begin(s);
  switch (dt) {
    case kF32:
      build_ag_kernel<kF32><<<(int)wg, 256, 0, s>>>(qup, qdn, w_up, w_dn, kept, n_kept, N, C, D, Ag, dX);
      break;
    case kF16:
      build_ag_kernel<kF16><<<(int)wg, 256, 0, s>>>(qup, qdn, w_up, w_dn, kept, n_kept, N, C, D, Ag, dX);
      break;
    case kBF16:
      build_ag_kernel<kBF16><<<(int)wg, 256, 0, s>>>(qup, qdn, w_up, w_dn, kept, n_kept, N, C, D, Ag, dX);
      break;
    default:
      return hipErrorInvalidValue;
  }
  timing_end(s, kKBuildAg);
  return hipGetLastError();
}

hipError_t launch_build_dw_operands(hipStream_t s, const uint8_t* qup, const uint8_t* qdn,
                                    const uint8_t* w_up, const uint8_t* w_dn,
                                    const int32_t* kept, const int32_t* n_kept,
                                    const uint8_t* xq, int64_t N, int64_t C, int64_t D,
                                    int8_t* At, uint8_t* XtT) {
  const int64_t pitch = (N + 127) / 128 * 128;
  dim3 grid((unsigned)(pitch / 64), (unsigned)(C / 64 + D / 64));
  timing_begin(s);
  build_dw_operands_kernel<<<grid, 256, 0, s>>>(qup, qdn, w_up, w_dn, kept, n_kept, xq, N, C, D,
                                                At, XtT);
  timing_end(s, kKBuildDw);
  return hipGetLastError();
}

}  // namespace hqlss
