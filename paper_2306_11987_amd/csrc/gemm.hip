// Integer GEMMs of HQ-MM and LSS-MM on gfx950 int8 MFMA, with fused epilogues.
//
//   forward  acc = X^ W^^T               (Sec. 3.3, Procedure HQ-MM step 3), then
//            Y = alpha acc                (step 4, dequantise by s_X s_W / 2^k)
//   dX       acc = A_T W^                 (Sec. 4.2, Eq. 6 on the kept rows), then
//            dX[t] = alpha FWHT_b(acc[t]) (the H^T of the STE gradient, Sec. 4)
//   dW       acc = A_T^T X^_T             (Sec. 4.2, Eq. 5 on the kept rows), then
//            dW = alpha FWHT_b(acc)
//
// All three are "NT" products acc[m][n] = sum_k A[m][k] B[n][k] with K-contiguous rows.
// CDNA4 has no INT4 matrix instruction, so INT4 codes run on the int8 MFMA
// (v_mfma_i32_32x32x32_i8, int32 accumulation).  INT4 operands stay packed in HBM and in
// LDS and are widened after the LDS read with two masks per 32-bit word:
// (w << 4) & 0xF0F0F0F0 places the even nibbles, w & 0xF0F0F0F0 the odd ones, in the high
// half of each byte, i.e. 16 x the signed code.  Inside every group of 8 k the register
// order becomes 0,2,4,6,1,3,5,7; int8 operands are stored in that order by their producer,
// and as the reduction over k is order-free the product is exact.  The factor 16 per INT4
// operand is a power of two, removed by an arithmetic shift.
//
// Tiling: a BM x 256 tile per 256-thread workgroup, 2 x 2 waves.  INT4 x INT4 (forward) uses
// BM = 256, one workgroup per CU, wave tiles of 128 x 128 (4 x 4 MFMA 32 x 32 tiles,
// accumulators in AGPRs), keeping fragment reads and INT4 widening at 0.5 per MFMA.  The
// int8 x INT4 gradient GEMMs use BM = 128 with two workgroups per CU, so that one
// workgroup's stage boundaries and epilogue overlap the other's MFMAs.  The MFMA "A" operand carries the n rows and the "B"
// operand the m rows, so that a lane's accumulators run along n: lane l, MFMA tile (i, j),
// register r holds m = 32 i + (l % 32) and n = 16 j + r + (BN/4) (l / 32) of the wave tile.
// This is arranged by storing the B rows in LDS in that permuted slot order.  Each lane then
// owns 16 consecutive n per (i, j) (32-byte stores), and the gradient epilogue's Hadamard
// transform along n runs in registers except for the single stride n = BN/4, which pairs
// lanes l and l ^ 32.
//
// Main loop: K in stages of 256 (both operands INT4) or 128, register prefetch of stage s+1
// while stage s computes from LDS, two LDS buffers, one barrier per stage.  All fragments of
// a stage are read from LDS right after the barrier (one latency exposure per stage) and
// widened just before their MFMAs; every operand row sits at a 144-byte pitch, at which the
// fragment reads are free of bank conflicts.
// Epilogue: results are staged through LDS in row chunks so that each store instruction
// writes contiguous 16-byte pieces of whole output rows.  Split-K (gridDim.z > 1) writes
// int32 partial tiles the same way, and reduce_epilogue sums them.
#include "common.h"
#include "launch.h"

namespace hqlss {

namespace {

typedef int v4i __attribute__((ext_vector_type(4)));
typedef int v16i __attribute__((ext_vector_type(16)));

constexpr int kThreads = 256;
constexpr int kBN = 256;  // workgroup tile width (n)
// tile height: 256 (one workgroup per CU) for INT4 x INT4, 128 (two per CU) for int8 x INT4
template <bool A4> constexpr int tile_m() { return A4 ? 256 : 128; }

template <int BM, int BN, bool A4, bool B4>
struct Cfg {
  static constexpr int KS = (A4 && B4) ? 256 : 128;  // K elements per stage
  static constexpr int A_ROW = A4 ? KS / 2 : KS;     // bytes per row per stage (128 or 64)
  static constexpr int B_ROW = B4 ? KS / 2 : KS;
  // 144-byte row pitch: the fragment reads (rows lane % 32, 16-byte column lane / 32) are
  // free of LDS bank conflicts at this pitch (measured); 64-byte rows use it too.
  // 128-row tiles run two workgroups per CU: their 64-byte INT4 rows take an 80-byte pitch
  // (a few bank conflicts) so that two double-buffered stages fit in 80 KB.
  static constexpr int A_PITCH = (BM == 128 && A_ROW == 64) ? 80 : 144;
  static constexpr int B_PITCH = (BM == 128 && B_ROW == 64) ? 80 : 144;
  static constexpr int OCC = BM == 128 ? 2 : 1;  // workgroups per CU
  static constexpr int A_BUF = BM * A_PITCH, B_BUF = BN * B_PITCH;
  static constexpr int STAGE = A_BUF + B_BUF;
  static constexpr int WM = BM / 2, WN = BN / 2;  // wave tile
  static constexpr int TI = WM / 32, TJ = WN / 32;
  static constexpr int A_CPR = A_ROW / 16, B_CPR = B_ROW / 16;  // 16-byte chunks per row
  static constexpr int A_CH = BM * A_CPR / kThreads, B_CH = BN * B_CPR / kThreads;
  static constexpr int PAIRS = KS / 64;  // MFMA k-substep pairs per stage
  static constexpr int SHIFT = (A4 ? 4 : 0) + (B4 ? 4 : 0);
};

// LDS slot of B-tile row n_t (see the file comment): wave half wn, then within the wave
// n_local = 16 j + r + (WN/2) h  ->  slot 32 j + 8 (r / 4) + 4 h + r % 4.
template <int WN>
__device__ __forceinline__ int b_slot(int n_t) {
  const int wn = n_t / WN, nl = n_t % WN;
  const int h = nl / (WN / 2), rem = nl % (WN / 2);
  const int j = rem >> 4, r = rem & 15;
  return wn * WN + 32 * j + 8 * (r >> 2) + 4 * h + (r & 3);
}

// Raw bytes of the two MFMA fragments (k substeps 2q and 2q+1 of a pair) of one 32-row
// operand tile: INT4 16 packed bytes (32 k), int8 32 bytes.  Row `row`, lane half g.
template <bool INT4> struct Raw { uint4 w[INT4 ? 1 : 2]; };

template <bool INT4, int PITCH>
__device__ __forceinline__ Raw<INT4> read_raw(const uint8_t* buf, int row, int pair, int g) {
  Raw<INT4> r;
  if constexpr (INT4) {
    r.w[0] = *reinterpret_cast<const uint4*>(buf + row * PITCH + pair * 32 + g * 16);
  } else {
    const uint8_t* p = buf + row * PITCH + pair * 64 + g * 32;
    r.w[0] = *reinterpret_cast<const uint4*>(p);
    r.w[1] = *reinterpret_cast<const uint4*>(p + 16);
  }
  return r;
}

// Fragment of k substep `half` (0 or 1) of a raw pair; INT4 is widened to 16 x the code.
template <bool INT4>
__device__ __forceinline__ v4i frag_of(const Raw<INT4>& r, int half) {
  v4i f;
  if constexpr (INT4) {
    const uint32_t a = half ? r.w[0].z : r.w[0].x, b = half ? r.w[0].w : r.w[0].y;
    f[0] = (int)((a << 4) & 0xF0F0F0F0u);
    f[1] = (int)(a & 0xF0F0F0F0u);
    f[2] = (int)((b << 4) & 0xF0F0F0F0u);
    f[3] = (int)(b & 0xF0F0F0F0u);
  } else {
    const uint4 w = r.w[half];
    f[0] = (int)w.x; f[1] = (int)w.y; f[2] = (int)w.z; f[3] = (int)w.w;
  }
  return f;
}

// In-register Hadamard transform of one lane's n values of one m row:
// v[j * 16 + r] is n = 16 j + r + (WN/2) h.  Strides 1..8 within r, 16.. within j, and
// stride WN/2 across the lane halves.
template <int TJ>
__device__ __forceinline__ void fwht_lane(int* v, int b, int lane) {
  constexpr int NV = TJ * 16;
#pragma unroll
  for (int h = 1; h < NV; h <<= 1) {
    if (h < b) {
#pragma unroll
      for (int e = 0; e < NV; ++e)
        if ((e & h) == 0) {
          const int a = v[e], c = v[e + h];
          v[e] = a + c;
          v[e + h] = a - c;
        }
    }
  }
  if (b > NV) {  // stride WN/2: partner lane l ^ 32
    const bool upper = (lane & 32) != 0;
#pragma unroll
    for (int e = 0; e < NV; ++e) {
      const int p = __shfl_xor(v[e], 32);
      v[e] = upper ? (p - v[e]) : (v[e] + p);
    }
  }
}

template <int DT>
__device__ __forceinline__ void store16(void* out, int64_t idx, const float* f) {
  char* p = static_cast<char*>(out) + idx * Elem<DT>::bytes;
  if constexpr (DT == kF32) {
    store_vec<DT, 8>(p, f);
    store_vec<DT, 8>(p + 32, f + 8);
  } else {
    store_vec<DT, 8>(p, f);
    store_vec<DT, 8>(p + 16, f + 8);
  }
}

// XCD-aware tile order: workgroups are dispatched round-robin over the 8 XCDs by linear id,
// so the linear id is remapped such that each XCD walks a contiguous run of tiles, n
// fastest: consecutive tiles on one XCD share their A rows in that XCD's L2.
__device__ __forceinline__ void tile_of(int& tm, int& tn) {
  const int tiles_n = gridDim.x, T = gridDim.x * gridDim.y;
  const int L = blockIdx.x + blockIdx.y * gridDim.x;
  int Lp = L;
  if (gridDim.z == 1 && T >= 16) {
    const int x = L % 8, loc = L / 8, q = T / 8, r = T % 8;
    Lp = (x < r) ? x * (q + 1) + loc : r * (q + 1) + (x - r) * q + loc;
  }
  tm = Lp / tiles_n;
  tn = Lp % tiles_n;
}

template <int BM, int BN, bool A4, bool B4, int EPI, int DT>
__global__ __launch_bounds__(kThreads, (BM == 128 ? 2 : 1)) void gemm_kernel(GemmArgs g) {
  using C_ = Cfg<BM, BN, A4, B4>;
  constexpr int TI = C_::TI, TJ = C_::TJ;
  // epilogue staging: rows of BN output elements of ES bytes, written back row-contiguous
  constexpr bool RAW = (EPI == kEpiAcc || EPI == kEpiPartial);
  constexpr int ES = (RAW || DT == kF32) ? 4 : 2;
  constexpr int E_PITCH = BN * ES + 16;
  constexpr int E_ROWS = (2 * C_::STAGE) / E_PITCH >= C_::WM ? C_::WM : C_::WM / 2;
  constexpr int LDS = (2 * C_::STAGE > E_ROWS * E_PITCH) ? 2 * C_::STAGE : E_ROWS * E_PITCH;
  __shared__ __attribute__((aligned(16))) uint8_t smem[LDS];

  const int tid = threadIdx.x, lane = tid & 63, wid = tid >> 6;
  const int wm = wid >> 1, wn = wid & 1;
  int tm, tn;
  tile_of(tm, tn);
  const int64_t m0 = (int64_t)tm * BM, n0 = (int64_t)tn * BN;
  int64_t M = g.M;
  if (g.m_dev) {
    const int64_t md = *g.m_dev;
    M = md < M ? md : M;
  }
  if (m0 >= M) return;  // whole workgroup: uniform exit before any barrier
  int64_t K = g.K;
  if (g.k_dev) K = ((int64_t)*g.k_dev + 127) / 128 * 128;
  // split-K range of this workgroup (whole stages)
  const int nst_all = (int)((K + C_::KS - 1) / C_::KS);
  const int per = (nst_all + (int)gridDim.z - 1) / (int)gridDim.z;
  const int st0 = (int)blockIdx.z * per;
  const int nst = max(0, min(nst_all, st0 + per) - st0);
  const int64_t Ka = A4 ? K / 2 : K, Kb = B4 ? K / 2 : K;  // row extents in bytes
  const uint8_t* __restrict__ gA = static_cast<const uint8_t*>(g.A);
  const uint8_t* __restrict__ gB = static_cast<const uint8_t*>(g.B);

  uint4 ra[C_::A_CH], rb[C_::B_CH];
  auto gload = [&](int st) {
    const int64_t kbA = (int64_t)(st0 + st) * C_::A_ROW, kbB = (int64_t)(st0 + st) * C_::B_ROW;
    // out-of-range pieces load a valid address (row 0, k 0) and are zeroed: no branches
#pragma unroll
    for (int c = 0; c < C_::A_CH; ++c) {
      const int idx = tid + c * kThreads, r = idx / C_::A_CPR, cc = idx % C_::A_CPR;
      const int64_t gm = m0 + r, kb = kbA + cc * 16;
      const bool in = gm < M && kb < Ka;
      uint4 v = *reinterpret_cast<const uint4*>(gA + (in ? gm * g.lda + kb : 0));
      if (!in) v = make_uint4(0u, 0u, 0u, 0u);
      ra[c] = v;
    }
#pragma unroll
    for (int c = 0; c < C_::B_CH; ++c) {
      const int idx = tid + c * kThreads, r = idx / C_::B_CPR, cc = idx % C_::B_CPR;
      const int64_t gn = n0 + r, kb = kbB + cc * 16;
      const bool in = gn < g.N && kb < Kb;
      uint4 v = *reinterpret_cast<const uint4*>(gB + (in ? gn * g.ldb + kb : 0));
      if (!in) v = make_uint4(0u, 0u, 0u, 0u);
      rb[c] = v;
    }
  };
  auto sstore = [&](int buf) {
    uint8_t* sa = smem + buf * C_::STAGE;
    uint8_t* sb = sa + C_::A_BUF;
#pragma unroll
    for (int c = 0; c < C_::A_CH; ++c) {
      const int idx = tid + c * kThreads, r = idx / C_::A_CPR, cc = idx % C_::A_CPR;
      *reinterpret_cast<uint4*>(sa + r * C_::A_PITCH + cc * 16) = ra[c];
    }
#pragma unroll
    for (int c = 0; c < C_::B_CH; ++c) {
      const int idx = tid + c * kThreads, r = idx / C_::B_CPR, cc = idx % C_::B_CPR;
      *reinterpret_cast<uint4*>(sb + b_slot<C_::WN>(r) * C_::B_PITCH + cc * 16) = rb[c];
    }
  };

  v16i acc[TI][TJ];
#pragma unroll
  for (int i = 0; i < TI; ++i)
#pragma unroll
    for (int j = 0; j < TJ; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0;

  const int frow = lane & 31, fg = lane >> 5;
  if (nst > 0) {
    gload(0);
    sstore(0);
    __syncthreads();
  }
  for (int st = 0; st < nst; ++st) {
    const int cur = st & 1;
    if (st + 1 < nst) gload(st + 1);
    const uint8_t* sa = smem + cur * C_::STAGE;
    const uint8_t* sb = sa + C_::A_BUF;
    // Software pipeline over the stage's 32-k steps t (two steps per raw pair p = t / 2):
    // the MFMAs of step t run interleaved with the widening of step t+1's fragments and
    // with the LDS reads of pair p+2, issued two steps before their first use.
    constexpr int STEPS = 2 * C_::PAIRS;
    Raw<B4> rbn[2][TJ];
    Raw<A4> ram[2][TI];
    v4i fb[2][TJ], fa[2][TI];
#pragma unroll
    for (int p = 0; p < 2 && p < C_::PAIRS; ++p) {
#pragma unroll
      for (int j = 0; j < TJ; ++j) rbn[p][j] = read_raw<B4, C_::B_PITCH>(sb, wn * C_::WN + 32 * j + frow, p, fg);
#pragma unroll
      for (int i = 0; i < TI; ++i) ram[p][i] = read_raw<A4, C_::A_PITCH>(sa, wm * C_::WM + 32 * i + frow, p, fg);
    }
#pragma unroll
    for (int j = 0; j < TJ; ++j) fb[0][j] = frag_of<B4>(rbn[0][j], 0);
#pragma unroll
    for (int i = 0; i < TI; ++i) fa[0][i] = frag_of<A4>(ram[0][i], 0);
#pragma unroll
    for (int t = 0; t < STEPS; ++t) {
      const int p = t >> 1, h = t & 1, c = t & 1, n = c ^ 1;
      if (t + 1 < STEPS) {
        const int p1 = (t + 1) >> 1, h1 = (t + 1) & 1;
#pragma unroll
        for (int j = 0; j < TJ; ++j) fb[n][j] = frag_of<B4>(rbn[p1 & 1][j], h1);
#pragma unroll
        for (int i = 0; i < TI; ++i) fa[n][i] = frag_of<A4>(ram[p1 & 1][i], h1);
      }
      if (h == 1 && p + 2 < C_::PAIRS) {  // raw[p & 1] is fully widened now
#pragma unroll
        for (int j = 0; j < TJ; ++j)
          rbn[p & 1][j] = read_raw<B4, C_::B_PITCH>(sb, wn * C_::WN + 32 * j + frow, p + 2, fg);
#pragma unroll
        for (int i = 0; i < TI; ++i)
          ram[p & 1][i] = read_raw<A4, C_::A_PITCH>(sa, wm * C_::WM + 32 * i + frow, p + 2, fg);
      }
#pragma unroll
      for (int i = 0; i < TI; ++i)
#pragma unroll
        for (int j = 0; j < TJ; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_i32_32x32x32_i8(fb[c][j], fa[c][i], acc[i][j], 0, 0, 0);
      // interleave: each MFMA followed by a few VALU (widening) and at most one LDS read
#pragma unroll
      for (int q = 0; q < TI * TJ; ++q) {
        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);  // 1 MFMA
        __builtin_amdgcn_sched_group_barrier(0x002, 3, 0);  // up to 3 VALU
        __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);  // up to 1 DS read
      }
    }
    if (st + 1 < nst) sstore(cur ^ 1);
    __syncthreads();
  }

  // ---------------------------------------------------------------- epilogue
  // values of (i, j): row m = wm*WM + 32 i + (lane % 32), columns n = wn*WN + 16 j +
  // (WN/2)(lane / 32) + r.  They go through LDS so that every store writes whole rows.
  const int ml = lane & 31;
  const int nh = (C_::WN / 2) * (lane >> 5);
  float alpha = 0.f;
  if constexpr (EPI == kEpiFwd) {
    // fl(alpha 2^-SHIFT * fl(acc)) == fl(alpha * fl(acc >> SHIFT)): both scalings are exact
    alpha = alpha_of(*g.amax1, *g.amax2, g.denom) * (1.0f / (float)(1 << C_::SHIFT));
  } else if constexpr (EPI == kEpiDx || EPI == kEpiDw) {
    alpha = alpha_of(*g.amax1, *g.amax2, g.denom);
  }
  if constexpr (EPI == kEpiDx || EPI == kEpiDw) {
    const int b = 1 << g.log2b;
#pragma unroll
    for (int i = 0; i < TI; ++i) {
      int v[TJ * 16];
#pragma unroll
      for (int j = 0; j < TJ; ++j)
#pragma unroll
        for (int r = 0; r < 16; ++r) v[16 * j + r] = acc[i][j][r] >> C_::SHIFT;
      fwht_lane<TJ>(v, b, lane);  // every lane takes part (shuffles)
#pragma unroll
      for (int j = 0; j < TJ; ++j)
#pragma unroll
        for (int r = 0; r < 16; ++r) acc[i][j][r] = v[16 * j + r];
    }
  }
  constexpr int PIECES = BN * ES / 16;  // 16-byte pieces per output row
  char* const out = static_cast<char*>(g.out);
  const int64_t out_plane = (EPI == kEpiPartial) ? (int64_t)blockIdx.z * g.M * g.ldo : 0;
#pragma unroll
  for (int chunk = 0; chunk < BM / E_ROWS; ++chunk) {
    const int r_lo = chunk * E_ROWS;
#pragma unroll
    for (int i = 0; i < TI; ++i) {
      const int row = wm * C_::WM + 32 * i + ml - r_lo;
      if (row < 0 || row >= E_ROWS) continue;
      uint8_t* e = smem + row * E_PITCH;
#pragma unroll
      for (int j = 0; j < TJ; ++j) {
        const int n = wn * C_::WN + 16 * j + nh;
        if constexpr (ES == 4) {
          uint4* p = reinterpret_cast<uint4*>(e + n * 4);
#pragma unroll
          for (int q = 0; q < 4; ++q) {
            uint32_t w[4];
#pragma unroll
            for (int t = 0; t < 4; ++t) {
              const int a = acc[i][j][4 * q + t];
              if constexpr (RAW) w[t] = (uint32_t)(EPI == kEpiPartial || EPI == kEpiAcc ? (a >> C_::SHIFT) : a);
              else w[t] = __float_as_uint(alpha * (float)a);
            }
            p[q] = make_uint4(w[0], w[1], w[2], w[3]);
          }
        } else {
          float f[16];
#pragma unroll
          for (int r = 0; r < 16; ++r) f[r] = alpha * (float)acc[i][j][r];
          store_vec<DT, 8>(e + n * 2, f);
          store_vec<DT, 8>(e + n * 2 + 16, f + 8);
        }
      }
    }
    __syncthreads();
    for (int idx = tid; idx < E_ROWS * PIECES; idx += kThreads) {
      const int r = idx / PIECES, pc = idx % PIECES;
      const int64_t gm = m0 + r_lo + r;
      const int64_t gn = n0 + (int64_t)pc * (16 / ES);
      if (gm < M && gn < g.N) {
        const int64_t orow = (EPI == kEpiDx) ? (int64_t)g.out_rows[gm] : gm;
        *reinterpret_cast<uint4*>(out + (out_plane + orow * g.ldo + gn) * ES) =
            *reinterpret_cast<const uint4*>(smem + r * E_PITCH + pc * 16);
      }
    }
    __syncthreads();
  }
}

// Sum of split-K partials [S][M][N] (int32), then the epilogue of `mode` (kEpiFwd: scale;
// kEpiDx / kEpiDw: Hadamard transform along n, then scale; kEpiAcc: raw int32 copy).
// One wave per (row, 512-column chunk); a lane holds 8 consecutive n.
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
  float alpha = 0.f;
  if constexpr (MODE != kEpiAcc) alpha = alpha_of(*g.amax1, *g.amax2, g.denom);
  const int b = 1 << g.log2b;
  const int64_t plane = g.M * g.ldo;
  for (uint32_t it = blockIdx.x * 4 + (threadIdx.x >> 6); it < items; it += nw) {
    const int64_t m = it / chunks;
    const int64_t n = (int64_t)(it - (uint32_t)m * chunks) * 512 + lane * 8;
    const bool live = n < g.N;
    int v[8] = {0, 0, 0, 0, 0, 0, 0, 0};
    if (live) {
      for (int z = 0; z < S; ++z) {
        const int4* p = reinterpret_cast<const int4*>(P + z * plane + m * g.ldo + n);
        const int4 x0 = p[0], x1 = p[1];
        v[0] += x0.x; v[1] += x0.y; v[2] += x0.z; v[3] += x0.w;
        v[4] += x1.x; v[5] += x1.y; v[6] += x1.z; v[7] += x1.w;
      }
    }
    if constexpr (MODE == kEpiDx || MODE == kEpiDw) {
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
      int4* p = reinterpret_cast<int4*>(static_cast<int32_t*>(g.out) + m * g.ldo + n);
      p[0] = make_int4(v[0], v[1], v[2], v[3]);
      p[1] = make_int4(v[4], v[5], v[6], v[7]);
    } else {
      const int64_t orow = (MODE == kEpiDx) ? (int64_t)g.out_rows[m] : m;
      float f[8];
#pragma unroll
      for (int e = 0; e < 8; ++e) f[e] = alpha * (float)v[e];
      store_vec<DT, 8>(static_cast<char*>(g.out) + (orow * g.ldo + n) * Elem<DT>::bytes, f);
    }
  }
}

template <int BM, int BN, bool A4, bool B4, int EPI, int DT>
hipError_t gemm_t(hipStream_t s, const GemmArgs& g, int splits, int id) {
  dim3 grid((unsigned)((g.N + BN - 1) / BN), (unsigned)((g.M + BM - 1) / BM), (unsigned)splits);
  timing_begin(s);
  gemm_kernel<BM, BN, A4, B4, EPI, DT><<<grid, kThreads, 0, s>>>(g);
  timing_end(s, id);
  return hipGetLastError();
}

template <int DT, int MODE>
hipError_t reduce_t(hipStream_t s, const int32_t* P, int S, const GemmArgs& g) {
  const int64_t items = g.M * ((g.N + 511) / 512);
  int64_t wg = (items + 3) / 4;
  if (wg > 2048) wg = 2048;
  if (wg < 1) wg = 1;
  timing_begin(s);
  reduce_epilogue_kernel<DT, MODE><<<(int)wg, 256, 0, s>>>(P, S, g);
  timing_end(s, kKReduce);
  return hipGetLastError();
}

template <int EPI, int DT>
hipError_t reduce_dt(hipStream_t s, const int32_t* P, int S, const GemmArgs& g) {
  return reduce_t<DT, EPI>(s, P, S, g);
}

template <bool A4, bool B4, int EPI, int DT>
hipError_t run(hipStream_t s, const GemmArgs& g, int splits, int32_t* partial, int id) {
  if (splits <= 1) return gemm_t<tile_m<A4>(), kBN, A4, B4, EPI, DT>(s, g, 1, id);
  GemmArgs p = g;
  p.out = partial;
  p.ldo = g.N;
  hipError_t e = gemm_t<tile_m<A4>(), kBN, A4, B4, kEpiPartial, DT>(s, p, splits, id);
  if (e != hipSuccess) return e;
  GemmArgs r = g;
  return reduce_dt<EPI, DT>(s, partial, splits, r);
}

template <bool A4, bool B4, int EPI>
hipError_t run_dt(hipStream_t s, int dt, const GemmArgs& g, int splits, int32_t* partial, int id) {
  switch (dt) {
    case kF32: return run<A4, B4, EPI, kF32>(s, g, splits, partial, id);
    case kF16: return run<A4, B4, EPI, kF16>(s, g, splits, partial, id);
    case kBF16: return run<A4, B4, EPI, kBF16>(s, g, splits, partial, id);
  }
  return hipErrorInvalidValue;
}

}  // namespace

static int g_split_override = 0;
void gemm_set_split_override(int splits) { g_split_override = splits < 0 ? 0 : splits; }

int gemm_splits(int64_t M, int64_t N, int64_t K, bool a_int4, bool b_int4) {
  (void)b_int4;
  if (g_split_override) return g_split_override;
  const int64_t bm = a_int4 ? 256 : 128, slots = a_int4 ? 256 : 512;  // workgroups in flight
  const int64_t tiles = ((M + bm - 1) / bm) * ((N + kBN - 1) / kBN);
  const int64_t stages = (K + 127) / 128;  // in units of 128 k
  if (2 * tiles >= slots || stages < 16) return 1;
  int64_t s = (slots + tiles - 1) / tiles;  // about one workgroup per slot
  const int64_t smax = stages / 8;          // keep >= 8 stages per split
  if (s > smax) s = smax;
  return (int)(s < 1 ? 1 : s);
}

size_t gemm_partial_bytes(int64_t M, int64_t N, int splits) {
  return splits > 1 ? (size_t)splits * M * N * 4 : 0;
}

hipError_t launch_gemm(hipStream_t s, int epi, int dt, bool a_int4, bool b_int4, const GemmArgs& g,
                       int splits, int32_t* partial) {
  if (a_int4 && b_int4) {
    if (epi == kEpiFwd) return run_dt<true, true, kEpiFwd>(s, dt, g, splits, partial, kKGemmFwd);
    if (epi == kEpiAcc) return run<true, true, kEpiAcc, kF32>(s, g, splits, partial, kKGemmAcc);
  } else if (!a_int4 && b_int4) {
    if (epi == kEpiDx) return run_dt<false, true, kEpiDx>(s, dt, g, splits, partial, kKGemmDx);
    if (epi == kEpiDw) return run_dt<false, true, kEpiDw>(s, dt, g, splits, partial, kKGemmDw);
    if (epi == kEpiAcc) return run<false, true, kEpiAcc, kF32>(s, g, splits, partial, kKGemmAcc);
  }
  return hipErrorInvalidValue;
}

}  // namespace hqlss
