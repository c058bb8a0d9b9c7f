// Leverage-score sampling of the bit-split gradient rows and the GEMM operands it
// selects (gfx950).
//
// lss_plan (one workgroup per problem: 1024 threads, 256 for N <= 4096).  Its inputs are
// the integer leverage scores of the 2N stacked rows, formed by the bit-split kernel
// (Sec. 4.2: with the common factor
// s_dn s_x dropped, c^2 = w^2 sum q^2 x_sumsq, w = 14 for the upper row of a token and 1
// for the lower one, c = isqrt(c^2 2^16)), and that kernel's per-workgroup totals:
//   1. inclusion probabilities by the clamp-and-rescale loop of App. A.2 with sum p = B,
//      in exact integers.  Thresholds S/R only fall from one round to the next, so the
//      rows clamped after a round are exactly {c > 0 : R c >= S} for that round's (R, S):
//      a round needs that set's count and sum, and no per-row state (the 1024-thread
//      build takes them from scores binned once, the 256-thread one from a pass over
//      the scores).  If no more
//      than B rows have c > 0, every such row has p = 1 (the "keep rows with norm > 0"
//      rule of the paper's implementation, App. A.6);
//   2. upper rows are kept iff non-zero; a lower row with p* < 1 gets p~ = 2^-e >= p*, the
//      smallest power of two (e <= 4, e <= 2 if the token's upper row is non-zero), and is
//      kept iff u16 < 2^(16-e) (Philox stream 1), weight m/p~ = 2^e;
//   3. kept tokens (w_up + w_dn > 0) are compacted in ascending order: each thread owns 8
//      consecutive tokens per round of 8192 (vector loads and stores, one Philox block),
//      and a block-wide scan of the per-thread counts places them.
//
// build_operands materialises, for the kept tokens only, the weighted integer
// rows A_t = 14 w_up q_up[t] + w_dn q_dn[t] (|A| <= 126, one int8 operand that carries the
// bit split and the 1/p factors together; the dX GEMM reads it K-contiguous, the dW GEMM
// k-major through transposing LDS reads) and the gathered X^ rows, transposed to the
// K-contiguous layout the dW GEMM reads.  The int8 operand uses the "K-interleaved" byte
// order of the GEMM: inside every group of 8 consecutive k the bytes hold
// k = 0,2,4,6,1,3,5,7, the order in which a packed INT4 word unpacks for free.
#include "common.h"
#include "launch.h"

namespace hqlss {

namespace {

// Workgroup sizes of the sampler: 1024 threads, or 256 for short sequences (N <= 4096),
// where four samplers then share a CU (a batched call runs one per batch).  The result
// does not depend on the size: counters are per 8 tokens and every sum is exact.
constexpr int kPlanThreads = 1024;
constexpr int kPlanThreadsSmall = 256;

constexpr int kPlanRegs = 32;  // scores per thread kept in registers (2N <= 32 x threads)

// Sum of a 32-bit value over the wave (every lane gets it): DPP adds inside each row of
// 16 lanes (swap neighbours, swap pairs, mirror halves, mirror the row), then the four row
// sums read as scalars.  Needs every lane of the wave active.
__device__ __forceinline__ uint32_t wave_sum_u32_dpp(uint32_t v) {
  v += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0xB1, 0xF, 0xF, true);   // quad_perm 1,0,3,2
  v += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x4E, 0xF, 0xF, true);   // quad_perm 2,3,0,1
  v += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x141, 0xF, 0xF, true);  // row_half_mirror
  v += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x140, 0xF, 0xF, true);  // row_mirror
  return (uint32_t)__builtin_amdgcn_readlane((int)v, 0) + (uint32_t)__builtin_amdgcn_readlane((int)v, 16) +
         (uint32_t)__builtin_amdgcn_readlane((int)v, 32) + (uint32_t)__builtin_amdgcn_readlane((int)v, 48);
}

// 64-bit wave sum as three 21-bit limbs (64 limbs of at most 22 bits stay below 2^28, so
// each limb sum is exact in 32 bits), recombined modulo 2^64.
__device__ __forceinline__ uint64_t wave_sum_u64_dpp(uint64_t v) {
  constexpr uint64_t kM21 = (1ull << 21) - 1;
  const uint32_t s0 = wave_sum_u32_dpp((uint32_t)(v & kM21));
  const uint32_t s1 = wave_sum_u32_dpp((uint32_t)((v >> 21) & kM21));
  const uint32_t s2 = wave_sum_u32_dpp((uint32_t)(v >> 42));
  return (uint64_t)s0 + ((uint64_t)s1 << 21) + ((uint64_t)s2 << 42);
}

// Two block-wide sums with one barrier.  red holds 2 WAVES words; callers alternate
// between two such buffers, so that a buffer is written again only after the barrier
// that follows every read of it.
template <int WAVES>
__device__ __forceinline__ void block_sum2_u64(uint64_t& a, uint64_t& b, uint64_t* red) {
  a = wave_sum_u64_dpp(a);
  b = wave_sum_u64_dpp(b);
  if ((threadIdx.x & 63) == 0) {
    red[threadIdx.x >> 6] = a;
    red[WAVES + (threadIdx.x >> 6)] = b;
  }
  __syncthreads();
  a = 0;
  b = 0;
#pragma unroll
  for (int i = 0; i < WAVES; ++i) {
    a += red[i];
    b += red[WAVES + i];
  }
}

// Score bins of the 1024-thread sampler's clamp-and-rescale rounds: 32 per octave (the
// position of the leading one, then the next five bits), so the bin never decreases with
// the score: a score in a bin above the threshold's bin is at least the threshold, one in
// a bin below it is smaller, and only the threshold's own bin needs comparisons.
constexpr int kHistBins = 1024;
__device__ __forceinline__ int score_bin(uint32_t c) {  // c > 0
  const int e = 31 - __builtin_clz(c);
  const uint32_t m = e >= 5 ? (c >> (e - 5)) : (c << (5 - e));
  return e * 32 + (int)(m & 31u);
}

// 8 consecutive words from p + t0 (n8 of them valid, the rest 0).
__device__ __forceinline__ void load8u(const uint32_t* p, int t0, int n8, uint32_t v[8]) {
  if (n8 == 8) {
    const uint4 a = *reinterpret_cast<const uint4*>(p + t0), b = *reinterpret_cast<const uint4*>(p + t0 + 4);
    v[0] = a.x; v[1] = a.y; v[2] = a.z; v[3] = a.w;
    v[4] = b.x; v[5] = b.y; v[6] = b.z; v[7] = b.w;
  } else {
#pragma unroll
    for (int j = 0; j < 8; ++j) v[j] = j < n8 ? p[t0 + j] : 0u;
  }
}

template <int kPlanThreads>
__global__ __launch_bounds__(kPlanThreads) void lss_plan_kernel(
    const int32_t* __restrict__ sumsq_up, const uint32_t* __restrict__ scores, int64_t pitch,
    const uint4* __restrict__ parts, int nparts, int N, int64_t B, uint64_t seed,
    uint64_t offset, uint8_t* __restrict__ w_up, uint8_t* __restrict__ w_dn,
    int32_t* __restrict__ kept, int32_t* __restrict__ n_kept, uint64_t offset_stride) {
  constexpr int kPlanWaves = kPlanThreads / kWave;
  __shared__ uint64_t red[4 * kPlanWaves];  // two buffers of block_sum2_u64
  __shared__ int wtot[kPlanWaves];
  // the 1024-thread sampler runs its rounds on binned scores (below): per-bin counts (then
  // the end of each bin's bucket), first slots and sums (then the sums of the bins above),
  // and the non-zero scores bucketed by bin, highest bin first (128 KB of LDS)
  constexpr bool kHist = kPlanThreads == 1024;
  constexpr int kHistCap = kHist ? kPlanRegs * kPlanThreads : 1;
  static_assert(!kHist || kHistBins == kPlanThreads, "one bin per thread in the scan");
  __shared__ uint32_t h_end[kHist ? kHistBins : 1];
  __shared__ uint32_t h_off[kHist ? kHistBins : 1];
  __shared__ uint64_t h_sum[kHist ? kHistBins : 1];
  __shared__ uint32_t h_score[kHistCap];
  __shared__ uint64_t h_rs[2];
  const int tid = threadIdx.x, lane = tid & 63, wid = tid >> 6;
  {  // workgroup b samples batch b of a batched call (its own inputs, outputs and counters)
    const int64_t bt = blockIdx.x;
    sumsq_up += bt * N;
    scores += bt * 2 * pitch;
    parts += bt * nparts;
    w_up += bt * N;
    w_dn += bt * N;
    kept += bt * N;
    n_kept += bt;
    offset += (uint64_t)bt * offset_stride;
  }

  // totals of the bit-split workgroups: non-zero rows and the score sum
  uint64_t nz = 0, st = 0;
  for (int i = tid; i < nparts; i += kPlanThreads) {
    const uint4 p = parts[i];
    nz += p.x;
    st += ((uint64_t)p.z << 32) | p.y;
  }
  block_sum2_u64<kPlanWaves>(nz, st, red);  // buffer 0; the rounds start on buffer 1
  const uint64_t S_all = st;
  const bool all_nonzero_kept = (int64_t)nz <= B;

  // App. A.2 clamp-and-rescale (uniform across the block); each round is one pass over
  // the scores, held in registers when they fit
  uint64_t S = S_all;
  int64_t R = B;
  if (!all_nonzero_kept) {
    const int64_t n2 = 2 * (int64_t)N;
    const bool in_regs = n2 <= (int64_t)kPlanRegs * kPlanThreads;
    uint32_t cs[kPlanRegs];
#pragma unroll
    for (int j = 0; j < kPlanRegs; ++j) {
      const int64_t i = tid + (int64_t)j * kPlanThreads;
      cs[j] = (in_regs && i < n2) ? scores[i < N ? i : pitch + (i - N)] : 0u;
    }
    if (kHist && in_regs) {
      // The same rounds on binned scores.  One pass builds each bin's count and sum, a
      // scan from the top bin down gives the count and sum of all bins above each bin,
      // and a second pass places the scores in per-bin buckets.  A round then takes the
      // bins above its threshold's bin from the scan and compares only the threshold's
      // own bin, in one wave: the rounds' counts and sums, and so their sequence, are
      // those of the full passes.
      for (int b = tid; b < kHistBins; b += kPlanThreads) {
        h_end[b] = 0;
        h_sum[b] = 0;
      }
      __syncthreads();
#pragma unroll
      for (int j = 0; j < kPlanRegs; ++j)
        if (cs[j]) {
          const int b = score_bin(cs[j]);
          atomicAdd(&h_end[b], 1u);
          atomicAdd(reinterpret_cast<unsigned long long*>(&h_sum[b]), (unsigned long long)cs[j]);
        }
      __syncthreads();
      const int hb = kHistBins - 1 - tid;  // thread t scans bin 1023 - t
      const uint32_t c0 = h_end[hb];
      const uint64_t s0 = h_sum[hb];
      uint32_t ci = c0;
      uint64_t si = s0;
#pragma unroll
      for (int o = 1; o < 64; o <<= 1) {
        const uint32_t cy = __shfl_up(ci, o);
        const uint32_t lo = __shfl_up((uint32_t)si, o), hi = __shfl_up((uint32_t)(si >> 32), o);
        if (lane >= o) {
          ci += cy;
          si += ((uint64_t)hi << 32) | lo;
        }
      }
      // red: its last reads (the totals above) came before the barriers since
      if (lane == 63) {
        red[wid] = ci;
        red[kPlanWaves + wid] = si;
      }
      __syncthreads();
      uint32_t cpre = 0;
      uint64_t spre = 0;
#pragma unroll
      for (int i = 0; i < kPlanWaves; ++i)
        if (i < wid) {
          cpre += (uint32_t)red[i];
          spre += red[kPlanWaves + i];
        }
      const uint32_t above = cpre + ci - c0;  // scores in the bins above hb
      h_off[hb] = above;
      h_end[hb] = above;  // the bucket's fill cursor, then its end
      h_sum[hb] = spre + si - s0;
      __syncthreads();
#pragma unroll
      for (int j = 0; j < kPlanRegs; ++j)
        if (cs[j]) h_score[atomicAdd(&h_end[score_bin(cs[j])], 1u)] = cs[j];
      __syncthreads();
      if (wid == 0) {  // the rounds, in one wave (uniform)
        int64_t k = 0, Rr = B;
        uint64_t Sr = S_all;
        // the count grows every round that does not stop, so at most 2N + 1 rounds run;
        // the bound only makes that certain
        for (int64_t round = 0; round <= n2; ++round) {
          Rr = B - k;
          const uint64_t T = Sr == 0 ? 1 : Rr <= 0 ? ~uint64_t(0) : (Sr + (uint64_t)Rr - 1) / (uint64_t)Rr;
          uint64_t cnt = 0, sum = 0;
          if (T <= 0xFFFFFFFFull) {  // else no score reaches it
            const uint32_t T32 = (uint32_t)T;
            const int b = score_bin(T32);
            const uint32_t end = h_end[b];
            uint32_t n = 0;
            uint64_t sm = 0;
            for (uint32_t i = h_off[b] + lane; i < end; i += 64) {
              const uint32_t c = h_score[i];
              if (c >= T32) {
                ++n;
                sm += c;
              }
            }
            cnt = (uint64_t)h_off[b] + wave_sum_u32_dpp(n);
            sum = h_sum[b] + wave_sum_u64_dpp(sm);
          }
          if ((int64_t)cnt == k) break;  // nothing newly clamped
          k = (int64_t)cnt;
          Sr = S_all - sum;
        }
        if (lane == 0) {
          h_rs[0] = (uint64_t)Rr;
          h_rs[1] = Sr;
        }
      }
      __syncthreads();
      R = (int64_t)h_rs[0];
      S = h_rs[1];
    } else {  // full passes (256-thread sampler, or 2N beyond the register-held scores)
      int64_t k = 0;
      int par = 1;
      for (;;) {
        R = B - k;
        // R c >= S  <=>  c >= ceil(S / R) for integers and R > 0: one division per round
        // instead of a 64-bit product per score.  S = 0 admits every non-zero score (as
        // R c >= 0 does); R = 0 with S > 0 admits none.
        const uint64_t T = S == 0 ? 1 : R <= 0 ? ~uint64_t(0) : (S + (uint64_t)R - 1) / (uint64_t)R;
        // T >= 1, so c >= T implies c > 0; a threshold past the 32-bit scores admits none
        const uint32_t T32 = (uint32_t)T;
        uint32_t n = 0;
        uint64_t sum = 0;
        if (T > 0xFFFFFFFFull) {  // uniform
        } else if (in_regs) {
#pragma unroll
          for (int j = 0; j < kPlanRegs; ++j) {
            const uint32_t c = cs[j];
            const bool in = c >= T32;
            n += in;
            sum += in ? c : 0u;
          }
        } else {  // eight loads in flight per thread
          for (int64_t i0 = tid; i0 < n2; i0 += 8 * (int64_t)kPlanThreads) {
            uint32_t c8[8];
#pragma unroll
            for (int u = 0; u < 8; ++u) {
              const int64_t i = i0 + (int64_t)u * kPlanThreads;
              c8[u] = i < n2 ? scores[i < N ? i : pitch + (i - N)] : 0u;
            }
#pragma unroll
            for (int u = 0; u < 8; ++u) {
              const bool in = c8[u] >= T32;
              n += in;
              sum += in ? c8[u] : 0u;
            }
          }
        }
        uint64_t cnt = n;
        block_sum2_u64<kPlanWaves>(cnt, sum, red + 2 * kPlanWaves * par);
        par ^= 1;
        if ((int64_t)cnt == k) break;  // nothing newly clamped
        k = (int64_t)cnt;
        S = S_all - sum;
      }
    }
  }

  // weights, masks and compaction of one round: 8 consecutive tokens per thread
  int base = 0;
  const uint32_t* cdn = scores + pitch;
  const uint32_t* sup = reinterpret_cast<const uint32_t*>(sumsq_up);
  auto round = [&](int t0, int n8, const uint32_t su[8], const uint32_t cd[8]) {
    // Bernoulli draws only when some row has p < 1 (uniform over the workgroup)
    const U4 rnd = all_nonzero_kept ? U4{0u, 0u, 0u, 0u}
                                    : philox_block(seed, offset, 1u, (uint64_t)(t0 > 0 ? t0 : 0));
    uint32_t wu8[2] = {0u, 0u}, wd8[2] = {0u, 0u};
    uint32_t keepmask = 0;
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const uint32_t wu = su[j] ? 1u : 0u;
      uint32_t wd = 0;
      if (cd[j]) {
        const uint64_t rc = (uint64_t)R * cd[j];
        if (all_nonzero_kept || rc >= S) {
          wd = 1;
        } else {
          // e = min(cap, largest e with rc 2^e <= S), here 0 < rc < S: from the bit lengths
          // of rc and S and one comparison
          const int cap = wu ? 2 : 4;
          int e = cap;
          if (rc != 0) {
            const int e0 = __builtin_clzll(rc) - __builtin_clzll(S);
            const int m = (rc << e0) <= S ? e0 : e0 - 1;
            e = m < cap ? m : cap;
          }
          wd = (u16_of(rnd, j) < (1u << (16 - e))) ? (1u << e) : 0u;
        }
      }
      if (j >= n8) wd = 0;
      wu8[j >> 2] |= wu << (8 * (j & 3));
      wd8[j >> 2] |= wd << (8 * (j & 3));
      if (wu + wd) keepmask |= 1u << j;
    }
    if (n8 == 8) {
      *reinterpret_cast<uint2*>(w_up + t0) = make_uint2(wu8[0], wu8[1]);
      *reinterpret_cast<uint2*>(w_dn + t0) = make_uint2(wd8[0], wd8[1]);
    } else {
      for (int j = 0; j < n8; ++j) {
        w_up[t0 + j] = (uint8_t)(wu8[j >> 2] >> (8 * (j & 3)));
        w_dn[t0 + j] = (uint8_t)(wd8[j >> 2] >> (8 * (j & 3)));
      }
    }
    // block-wide exclusive scan of the per-thread keep counts
    const int nkeep = __builtin_popcount(keepmask);
    int x = nkeep;
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
      const int y = __shfl_up(x, o);
      if (lane >= o) x += y;
    }
    if (lane == 63) wtot[wid] = x;
    __syncthreads();
    int pre = 0, total = 0;
#pragma unroll
    for (int i = 0; i < kPlanWaves; ++i) {
      pre += (i < wid) ? wtot[i] : 0;
      total += wtot[i];
    }
    __syncthreads();
    int pos = base + pre + x - nkeep;
#pragma unroll
    for (int j = 0; j < 8; ++j)
      if ((keepmask >> j) & 1) kept[pos++] = t0 + j;
    base += total;
  };
  if (N <= 2 * 8 * kPlanThreads) {
    // both rounds' inputs in one round trip to memory
    uint32_t su[2][8], cd[2][8];
    int t0[2], n8[2];
#pragma unroll
    for (int r = 0; r < 2; ++r) {
      t0[r] = r * 8 * kPlanThreads + 8 * tid;
      n8[r] = t0[r] < N ? (N - t0[r] < 8 ? N - t0[r] : 8) : 0;
      load8u(sup, t0[r], n8[r], su[r]);
      load8u(cdn, t0[r], n8[r], cd[r]);
    }
    round(t0[0], n8[0], su[0], cd[0]);
    if (N > 8 * kPlanThreads) round(t0[1], n8[1], su[1], cd[1]);
  } else {
    for (int r0 = 0; r0 < N; r0 += 8 * kPlanThreads) {
      const int t = r0 + 8 * tid;
      const int n = t < N ? (N - t < 8 ? N - t : 8) : 0;
      uint32_t su[8], cd[8];
      load8u(sup, t, n, su);
      load8u(cdn, t, n, cd);
      round(t, n, su, cd);
    }
  }
  if (tid == 0) *n_kept = base;
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

// One pass over the kept tokens builds every GEMM operand the sample selects: workgroup
// (x, y) takes kept indices [128 x, 128 x + 128) and one block of up to 128 columns (the
// last block of C or D may hold 64).  Blocks of the C columns read q_up, q_dn and the
// weights, form A_t and write it row-major into Ag (the operand of both gradient GEMMs);
// blocks of the D columns gather X^ rows and write them, through an LDS transpose,
// column-major into XtT.  Every row piece written is 128 bytes (64 for XtT), two full
// cache lines.  The last block row zeroes the rows of dX that belong to dropped tokens.
// Rows of Ag and columns of XtT between n_kept and the next multiple of 128 are written as
// zeros (the GEMMs read whole K steps).
constexpr int kBK = 128;  // kept indices per workgroup
constexpr int kBC = 128;  // columns per workgroup
template <int DT>
__global__ __launch_bounds__(256) void build_operands_kernel(
    const uint8_t* __restrict__ qup, const uint8_t* __restrict__ qdn,
    const uint8_t* __restrict__ w_up, const uint8_t* __restrict__ w_dn,
    const int32_t* __restrict__ kept, const int32_t* __restrict__ n_kept,
    const uint8_t* __restrict__ xq, int64_t N, int64_t C, int64_t D, int8_t* __restrict__ Ag,
    uint8_t* __restrict__ XtT, void* __restrict__ dX) {
  __shared__ __attribute__((aligned(16))) int8_t tile[kBK][kBC + 4];  // [kept index][column]
  const int tid = threadIdx.x;
  const int64_t cb = (C + kBC - 1) / kBC, db = (D + kBC - 1) / kBC;
  {  // grid z: batch b of a batched call, every operand one block per batch
    const int64_t bt = blockIdx.z, kpad = (N + 127) / 128 * 128;
    qup += bt * N * (C / 2);
    qdn += bt * N * (C / 2);
    w_up += bt * N;
    w_dn += bt * N;
    kept += bt * N;
    n_kept += bt;
    xq += bt * N * (D / 2);
    if (Ag) Ag += bt * kpad * C;
    if (XtT) XtT += bt * D * (kpad / 2);
    if (dX) dX = static_cast<char*>(dX) + bt * N * D * Elem<DT>::bytes;
  }
  if ((int64_t)blockIdx.y == cb + db) {  // zero the dX rows of dropped tokens
    if (!dX) return;
    const int64_t bytes = D * Elem<DT>::bytes;
    const int64_t t0 = (int64_t)blockIdx.x * kBK, t1 = t0 + kBK < N ? t0 + kBK : N;
    for (int64_t t = t0 + (tid >> 6); t < t1; t += 4) {
      if (w_up[t] + w_dn[t]) continue;
      char* row = static_cast<char*>(dX) + t * bytes;
      for (int64_t o = (tid & 63) * 16; o < bytes; o += 64 * 16)
        st_stream<HQ_NT_B_ST>(row + o, make_uint4(0u, 0u, 0u, 0u));
    }
    return;
  }
  const int64_t nk = *n_kept;
  const int64_t kp = (nk + 127) / 128 * 128;
  const int64_t i0 = (int64_t)blockIdx.x * kBK;
  if (i0 >= kp) return;
  const int64_t pitch = (N + 127) / 128 * 128;  // K pitch of XtT (in codes)
  const bool isA = (int64_t)blockIdx.y < cb;
  if (isA ? !Ag : !XtT) return;
  const int64_t col0 = isA ? (int64_t)blockIdx.y * kBC : ((int64_t)blockIdx.y - cb) * kBC;
  const int64_t ncol = isA ? C : D;
  // 128 kept rows x 4 chunks of 32 columns, two per thread: 16-byte loads of the code rows
  if (isA) {  // uniform: A_t is written row-major straight from registers
#pragma unroll
    for (int k = 0; k < 2; ++k) {
      const int item = tid + 256 * k, r = item >> 2, q = (item & 3) * 32;
      const int64_t i = i0 + r;
      if (col0 + q >= ncol) continue;  // the last block of a 64-multiple width
      int v[32];
#pragma unroll
      for (int j = 0; j < 32; ++j) v[j] = 0;
      if (i < nk) {  // rows past the kept count are the zero padding up to 128
        const int64_t t = kept[i];
        const int wu = w_up[t], wd = w_dn[t];
        const uint4 up = ld_stream<HQ_NT_B_LD>(qup + t * (C / 2) + (col0 + q) / 2);
        const uint4 dn = ld_stream<HQ_NT_B_LD>(qdn + t * (C / 2) + (col0 + q) / 2);
        weighted8(up.x, dn.x, wu, wd, v);
        weighted8(up.y, dn.y, wu, wd, v + 8);
        weighted8(up.z, dn.z, wu, wd, v + 16);
        weighted8(up.w, dn.w, wu, wd, v + 24);
      }
      const uint2 a0 = interleave8(v), a1 = interleave8(v + 8), a2 = interleave8(v + 16),
                  a3 = interleave8(v + 24);
      st_stream<HQ_NT_B_ST>(Ag + i * C + col0 + q, make_uint4(a0.x, a0.y, a1.x, a1.y));
      st_stream<HQ_NT_B_ST>(Ag + i * C + col0 + q + 16, make_uint4(a2.x, a2.y, a3.x, a3.y));
    }
    return;
  }
#pragma unroll
  for (int k = 0; k < 2; ++k) {
    const int item = tid + 256 * k, r = item >> 2, q = (item & 3) * 32;
    const int64_t i = i0 + r;
    uint4 x = make_uint4(0u, 0u, 0u, 0u);
    if (i < nk && col0 + q < ncol) x = ld_stream<HQ_NT_B_LD>(xq + kept[i] * (D / 2) + (col0 + q) / 2);
    // word w of row r sits at word w ^ ((r / 16) % 8) of the row: the transpose below reads
    // one column of 8 row blocks at once, which would otherwise fall on 4 banks
    uint32_t* tp = reinterpret_cast<uint32_t*>(&tile[r][0]);  // 4-byte aligned: pitch 132
    const int sw = (r >> 4) & 7;
    const uint32_t xw[4] = {x.x, x.y, x.z, x.w};
#pragma unroll
    for (int w = 0; w < 8; ++w) {  // bytes 4 w .. 4 w + 3 of the chunk: one code each
      const uint32_t c4 = xw[w >> 1] >> (16 * (w & 1));
      uint32_t b = 0;
#pragma unroll
      for (int j = 0; j < 4; ++j) b |= ((uint32_t)sext4((c4 >> (4 * j)) & 15u) & 0xFFu) << (8 * j);
      tp[(q / 4 + w) ^ sw] = b;
    }
  }
  __syncthreads();
  // 128 columns x 8 chunks of 16 kept indices, four per thread
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    const int item = tid + 256 * k, c = item >> 3, q = (item & 7) * 16;
    if (col0 + c >= ncol) continue;
    const int cs = (((c >> 2) ^ ((q >> 4) & 7)) << 2) | (c & 3);  // column c's byte in rows q..q+15
    uint32_t w0 = 0, w1 = 0;
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const uint32_t byte = ((uint32_t)tile[q + 2 * j][cs] & 15u) |
                            (((uint32_t)tile[q + 2 * j + 1][cs] & 15u) << 4);
      if (j < 4) w0 |= byte << (8 * j);
      else w1 |= byte << (8 * (j - 4));
    }
    st_stream2<HQ_NT_B_ST>(XtT + (col0 + c) * (pitch / 2) + (i0 + q) / 2, make_uint2(w0, w1));
  }
}

// Orders of the kept rows for the FP6 MFMA route (gemm6.hip), one workgroup per problem.
// Categories of a token t: upper (w_up = 1), kept lower-only (w_up = 0, w_dn > 0), and the
// lower weight class e = log2 w_dn (0..4).
//   order6: the kept tokens, upper tokens first, each part ascending (the dX row order:
//           tiles holding upper tokens run a second K pass over the upper codes);
//   ent:    the dW K entries (2 t + 1: the upper row of t, 2 t: its lower row) grouped by
//           weight, classes 2^4 .. 2^0, each class padded with -1 to a multiple of 128 (one
//           GEMM stage).  The upper weight 14 = 8 + 4 + 2 puts each upper row into classes
//           3, 2 and 1 (after that class's lower rows);
//   cls:    the first entries of classes 3, 2, 1, 0 and the padded total.
// Each thread owns a contiguous range of tokens, so a block-wide exclusive scan of the
// per-thread counts places every token in ascending order within its category.
constexpr int kCat = 7;  // upper, lower-only, lower classes 0..4
__global__ __launch_bounds__(1024) void fp6_plan_kernel(
    const uint8_t* __restrict__ w_up, const uint8_t* __restrict__ w_dn, int N,
    int32_t* __restrict__ order6, int32_t* __restrict__ n_up_out, int32_t* __restrict__ ent,
    int32_t* __restrict__ cls) {
  __shared__ int s_cnt[kCat][1024];
  __shared__ int s_tot[kCat];
  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
  const int per = (N + 1023) / 1024;
  const int t0 = tid * per, t1 = min(N, t0 + per);
  int c[kCat];
#pragma unroll
  for (int k = 0; k < kCat; ++k) c[k] = 0;
  for (int t = t0; t < t1; ++t) {
    const int up = w_up[t], dn = w_dn[t];
    if (up) ++c[0];
    else if (dn) ++c[1];
    if (dn) ++c[2 + (31 - __clz(dn))];
  }
#pragma unroll
  for (int k = 0; k < kCat; ++k) s_cnt[k][tid] = c[k];
  __syncthreads();
  if (wv < kCat) {  // wave k: exclusive scan of category k over the 1024 threads
    int v[16], sum = 0;
#pragma unroll
    for (int i = 0; i < 16; ++i) { v[i] = s_cnt[wv][16 * lane + i]; sum += v[i]; }
    int incl = sum;
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
      const int y = __shfl_up(incl, o);
      if (lane >= o) incl += y;
    }
    int run = incl - sum;
#pragma unroll
    for (int i = 0; i < 16; ++i) { s_cnt[wv][16 * lane + i] = run; run += v[i]; }
    if (lane == 63) s_tot[wv] = incl;
  }
  __syncthreads();
  const int n_up = s_tot[0], n_d0 = s_tot[2], n_d1 = s_tot[3], n_d2 = s_tot[4], n_d3 = s_tot[5],
            n_d4 = s_tot[6];
  auto r128 = [](int x) { return (x + 127) & ~127; };
  const int b3 = r128(n_d4), b2 = b3 + r128(n_d3 + n_up), b1 = b2 + r128(n_d2 + n_up),
            b0 = b1 + r128(n_d1 + n_up), ke = b0 + r128(n_d0);
  const int base[5] = {b0, b1, b2, b3, 0};  // first entry of lower class e
  int p_up = s_cnt[0][tid], p_rest = n_up + s_cnt[1][tid];
  int p_d[5];
#pragma unroll
  for (int e = 0; e < 5; ++e) p_d[e] = base[e] + s_cnt[2 + e][tid];
  for (int t = t0; t < t1; ++t) {
    const int up = w_up[t], dn = w_dn[t];
    if (up) {
      order6[p_up] = t;
      ent[b3 + n_d3 + p_up] = 2 * t + 1;
      ent[b2 + n_d2 + p_up] = 2 * t + 1;
      ent[b1 + n_d1 + p_up] = 2 * t + 1;
      ++p_up;
    } else if (dn) {
      order6[p_rest++] = t;
    }
    if (dn) {
      const int e = 31 - __clz(dn);
      ent[p_d[e]++] = 2 * t;
    }
  }
  // padding of every class to its 128-entry boundary
  const int pad_lo[5] = {n_d4, b3 + n_d3 + n_up, b2 + n_d2 + n_up, b1 + n_d1 + n_up, b0 + n_d0};
  const int pad_hi[5] = {b3, b2, b1, b0, ke};
#pragma unroll
  for (int q = 0; q < 5; ++q)
    for (int i = pad_lo[q] + tid; i < pad_hi[q]; i += 1024) ent[i] = -1;
  if (tid == 0) {
    *n_up_out = n_up;
    cls[0] = b3; cls[1] = b2; cls[2] = b1; cls[3] = b0; cls[4] = ke;
  }
}

}  // namespace

hipError_t launch_lss_plan(hipStream_t s, const int32_t* sumsq_up, const uint32_t* scores,
                           int64_t score_pitch, const uint4* parts, int nparts, int64_t N,
                           int64_t budget, uint64_t seed, uint64_t offset, uint8_t* w_up,
                           uint8_t* w_dn, int32_t* kept, int32_t* n_kept, int64_t batch,
                           uint64_t offset_stride) {
  timing_begin(s);
  if (N <= 16 * kPlanThreadsSmall)
    lss_plan_kernel<kPlanThreadsSmall><<<(unsigned)batch, kPlanThreadsSmall, 0, s>>>(
        sumsq_up, scores, score_pitch, parts, nparts, (int)N, budget, seed, offset, w_up, w_dn,
        kept, n_kept, offset_stride);
  else
    lss_plan_kernel<kPlanThreads><<<(unsigned)batch, kPlanThreads, 0, s>>>(
        sumsq_up, scores, score_pitch, parts, nparts, (int)N, budget, seed, offset, w_up, w_dn,
        kept, n_kept, offset_stride);
  timing_end(s, kKPlan);
  return hipGetLastError();
}

hipError_t launch_build_operands(hipStream_t s, int dt, const uint8_t* qup, const uint8_t* qdn,
                                 const uint8_t* w_up, const uint8_t* w_dn, const int32_t* kept,
                                 const int32_t* n_kept, const uint8_t* xq, int64_t N, int64_t C,
                                 int64_t D, int8_t* Ag, uint8_t* XtT, void* dX, int64_t batch) {
  const int64_t pitch = (N + 127) / 128 * 128;
  dim3 grid((unsigned)(pitch / kBK), (unsigned)((C + kBC - 1) / kBC + (D + kBC - 1) / kBC + 1),
            (unsigned)batch);
  timing_begin(s);
  switch (dt) {
    case kF32:
      build_operands_kernel<kF32><<<grid, 256, 0, s>>>(qup, qdn, w_up, w_dn, kept, n_kept, xq, N, C, D, Ag, XtT, dX);
      break;
    case kF16:
      build_operands_kernel<kF16><<<grid, 256, 0, s>>>(qup, qdn, w_up, w_dn, kept, n_kept, xq, N, C, D, Ag, XtT, dX);
      break;
    case kBF16:
      build_operands_kernel<kBF16><<<grid, 256, 0, s>>>(qup, qdn, w_up, w_dn, kept, n_kept, xq, N, C, D, Ag, XtT, dX);
      break;
    default:
      return hipErrorInvalidValue;
  }
  timing_end(s, kKBuild);
  return hipGetLastError();
}

hipError_t launch_fp6_plan(hipStream_t s, const uint8_t* w_up, const uint8_t* w_dn, int64_t N,
                           int32_t* order6, int32_t* n_up, int32_t* ent, int32_t* cls) {
  timing_begin(s);
  fp6_plan_kernel<<<1, 1024, 0, s>>>(w_up, w_dn, (int)N, order6, n_up, ent, cls);
  timing_end(s, kKFp6Plan);
  return hipGetLastError();
}

}  // namespace hqlss
