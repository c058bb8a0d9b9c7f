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
#include "common.h"
#include "launch.h"

namespace hqlss {

namespace {

typedef int v4i __attribute__((ext_vector_type(4)));
typedef int v16i __attribute__((ext_vector_type(16)));
typedef __attribute__((address_space(3))) void lds_void;

constexpr int kBN = 256;  // workgroup tile width (n)
constexpr int kNarrowBN = 64;  // tile width of the gradient GEMMs for outputs <= 64 wide
constexpr int kMidBN = 128;    // tile width of gradient GEMMs with few 256-wide tiles
// Split-K gradient GEMMs wider than 64 columns run 128-wide tiles: twice the tiles, so
// about half the splits fill the device and half the int32 partials are written and
// summed (and a GEMM whose 128-wide tiles fill one round alone is not split at all).
constexpr bool split_mid(bool a_int4, int64_t N) { return !a_int4 && N > kNarrowBN; }
constexpr int kKS = 128;  // K elements per stage
#ifndef HQLSS_GEMM_FWD_BM
#define HQLSS_GEMM_FWD_BM 128
#endif
#ifndef HQLSS_GEMM_GRAD_BM
#define HQLSS_GEMM_GRAD_BM 128
#endif
template <bool A4> constexpr int tile_m() { return A4 ? HQLSS_GEMM_FWD_BM : HQLSS_GEMM_GRAD_BM; }

template <int BM, bool A4, int WN_ = 128, int BN_ = kBN>
struct Cfg {
  static constexpr int BN = BN_;
  static constexpr int WAVES = BM / 32, THREADS = 64 * WAVES;
  static constexpr int WN = WN_, WGN = BN / WN, WGM = WAVES / WGN;
  static constexpr int WM = BM / WGM, TI = WM / 32, TJ = WN / 32;
  static constexpr int RA = A4 ? kKS / 2 : kKS;  // bytes of an A row per stage
  static constexpr int RB = kKS / 2;             // B is always INT4
  static constexpr int CPA = RA / 16, CPB = RB / 16;
  static constexpr int A_BYTES = BM * RA, B_BYTES = BN * RB, STAGE = A_BYTES + B_BYTES;
  static constexpr int A_BPW = A_BYTES / 1024 / WAVES, B_BPW = B_BYTES / 1024 / WAVES;
  static constexpr int DMA = A_BPW + B_BPW;  // 1 KB LDS-DMA loads per wave per stage
  static constexpr int OCC = BM == 128 ? 2 : 1;  // workgroups per CU
  static constexpr int NBUF = (OCC == 2 && !A4) ? 2 : 3;
  static constexpr int LDS_MAIN = NBUF * STAGE;
  static constexpr int SHIFT = (A4 ? 4 : 0) + 4;
  static_assert(A_BYTES % (1024 * WAVES) == 0 && B_BYTES % (1024 * WAVES) == 0, "DMA split");
};

// 16-byte chunk of row r that holds data chunk c (XOR swizzle; see the file comment).
template <int RB>
__device__ __forceinline__ int swz(int r) {
  return RB == 64 ? ((r >> 2) & 3) : ((r >> 1) & 7);
}

// B-tile LDS slot s -> tile row n_t (slot order puts a lane's 16 accumulators on 16
// consecutive n): within the WN rows of a wave, slot 32 j + t holds
// n = 16 j + 4 (t / 8) + (t % 4) + (WN / 2) ((t / 4) % 2).
template <int WN>
__device__ __forceinline__ int b_row_of_slot(int s) {
  const int wn = s / WN, rem = s % WN, j = rem >> 5, t = rem & 31;
  return wn * WN + 16 * j + 4 * (t >> 3) + (t & 3) + (WN / 2) * ((t >> 2) & 1);
}

// Widen k step `half` of a 16-byte INT4 raw read to an int8 fragment (16 x the code).
__device__ __forceinline__ v4i widen(const uint4& w, int half) {
  const uint32_t a = half ? w.z : w.x, b = half ? w.w : w.y;
  v4i f;
  f[0] = (int)((a << 4) & 0xF0F0F0F0u);
  f[1] = (int)(a & 0xF0F0F0F0u);
  f[2] = (int)((b << 4) & 0xF0F0F0F0u);
  f[3] = (int)(b & 0xF0F0F0F0u);
  return f;
}
__device__ __forceinline__ v4i as_frag(const uint4& w) {
  v4i f;
  f[0] = (int)w.x; f[1] = (int)w.y; f[2] = (int)w.z; f[3] = (int)w.w;
  return f;
}

// In-register Hadamard transform (block 2^LOG2B <= 2 NV) of one lane's NV n values of one
// m row: v[16 j + r] is n = 16 j + r + NV h (h = lane / 32).  Strides below NV run in
// registers, the stride NV pairs lanes l and l ^ 32.
template <int LOG2B, int NV>
__device__ __forceinline__ void fwht_lane(int* v, int lane) {
  constexpr int b = 1 << LOG2B;
  static_assert(b <= 2 * NV, "Hadamard block wider than a wave tile");
#pragma unroll
  for (int h = 1; h < NV && h < b; h <<= 1) {
#pragma unroll
    for (int e = 0; e < NV; ++e)
      if ((e & h) == 0) {
        const int a = v[e], c = v[e + h];
        v[e] = a + c;
        v[e + h] = a - c;
      }
  }
  if constexpr (b > NV) {
    const bool upper = (lane & 32) != 0;
#pragma unroll
    for (int e = 0; e < NV; ++e) {
      const int p = __shfl_xor(v[e], 32);
      v[e] = upper ? (p - v[e]) : (v[e] + p);
    }
  }
}

// XCD-aware tile order.  The hardware dispatches workgroups to the 8 XCDs round-robin by
// linear id, so workgroup b runs on XCD b % 8.  The T tiles (row-major, n fastest) are cut
// into 8 contiguous chunks, one per XCD, and the j-th workgroup of XCD x takes the j-th
// tile of chunk x.  T counts only the tiles with rows below M (the device-side row count
// of dX), so that the tiles past it do not all fall on the last XCDs; workgroups beyond
// their chunk get no tile.  Returns false for those.  Small grids keep the plain order.
// In a grid with a z extent (split-K index or batch) the XCD of workgroup (b, z) is
// (b + z gridDim.x) % 8: every class b % 8 still sits on one XCD within its z slice, so
// the chunks hold there too.
//
// Within a chunk, the whole tile rows are walked in column groups of G tiles: all rows of
// the chunk for columns [0, G), then for [G, 2G), ...  The workgroups resident on one XCD
// at a time (about 64) then cover a block of about 64 / G rows by G columns, so they share
// G operand panels of one side and 64 / G of the other in that XCD's L2, instead of the
// two rows by all columns of the plain order.  The chunk's partial first and last rows
// come after its whole rows, in the plain order.
template <int G>
__device__ __forceinline__ int grouped_tile(int j, int s, int len, int tiles_n) {
  const int rf = (s + tiles_n - 1) / tiles_n, rl = (s + len) / tiles_n;
  if (rl - rf < 2) return s + j;
  const int R = rl - rf, nfull = R * tiles_n, head = rf * tiles_n - s;
  if (j < nfull) {
    const int nfg = tiles_n / G;
    if (j < nfg * R * G) {
      const int g = j / (R * G), inner = j - g * (R * G);
      return (rf + inner / G) * tiles_n + g * G + inner % G;
    }
    const int rem = j - nfg * R * G, gl = tiles_n - nfg * G;
    return (rf + rem / gl) * tiles_n + nfg * G + rem % gl;
  }
  if (j < nfull + head) return s + (j - nfull);
  return rl * tiles_n + (j - nfull - head);
}

template <int G>
__device__ __forceinline__ bool tile_of(int T, int tiles_n, int& tm, int& tn) {
  const int b = blockIdx.x;
  int L = b;
  if (T >= 16) {
    const int x = b & 7, j = b >> 3, q = T >> 3, r = T & 7;
    const int len = q + (x < r ? 1 : 0);
    if (j >= len) return false;
    L = grouped_tile<G>(j, x * q + min(x, r), len, tiles_n);
  } else if (b >= T) {
    return false;
  }
  tm = L / tiles_n;
  tn = L % tiles_n;
  return true;
}

// 16-byte LDS-DMA load (global_load_lds_dwordx4): each lane's 16 bytes at g land at
// lds_base + 16 * lane.  Issued as inline assembly with a memory clobber: the compiler
// keeps it in program order with every other memory access, but does not treat it as a
// pending LDS write; it would otherwise wait for every such load before any later LDS
// read, including the loads just issued for a later stage.  The stage pipeline waits for
// exactly the loads each stage needs.
__device__ __forceinline__ void dma16(const void* g, void* lds_base) {
  const uint32_t l = (uint32_t)(uintptr_t)(lds_void*)lds_base;
  asm volatile("global_load_lds_dwordx4 %0, off" ::"v"(g), "{m0}"(l) : "memory");
}

// s_waitcnt: vector-memory count <= n, LDS count 0 (gfx9 encoding: vmcnt [3:0] and
// [15:14], expcnt [6:4] left at its maximum, lgkmcnt [11:8]).
template <int n>
__device__ __forceinline__ void wait_vm_lgkm0() {
  __builtin_amdgcn_s_waitcnt((n & 15) | ((n >> 4) << 14) | (7 << 4));
}

// alpha = fl(fl(s1 s2) / denom); an operand flagged in steps_mask is a step itself,
// otherwise a tensor maximum a with s = fl(a / 7).
__device__ __forceinline__ float scale_of(const GemmArgs& g) {
  const uint32_t a1 = *g.amax1, a2 = *g.amax2;
  const float s1 = (g.steps_mask & 1) ? __uint_as_float(a1) : step_of(a1);
  const float s2 = (g.steps_mask & 2) ? __uint_as_float(a2) : step_of(a2);
  return (s1 * s2) / g.denom;
}

__device__ __forceinline__ double f16_bits_to_double(uint32_t h) {
  return (double)__builtin_bit_cast(_Float16, (uint16_t)h);
}
// clip indicator of the learned-step-size mode from an fp16 delta: |delta| <= 1/2
__device__ __forceinline__ bool inside_of(uint32_t h) { return (h & 0x7FFFu) <= 0x3800u; }

// Sum over the workgroup of one double per thread (fixed order); thread 0 gets the total.
template <int THREADS>
__device__ __forceinline__ double block_sum_f64(double v, double* red) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o);
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = v;
  __syncthreads();
  double t = 0.0;
  if (threadIdx.x == 0) {
#pragma unroll
    for (int w = 0; w < THREADS / 64; ++w) t += red[w];
  }
  return t;
}

template <int BM, bool A4, int WN, int EPI, int DT, int LOG2B, int BN_>
__global__ __launch_bounds__((Cfg<BM, A4, WN, BN_>::THREADS), (Cfg<BM, A4, WN, BN_>::OCC)) void gemm_kernel(GemmArgs g) {
  using C_ = Cfg<BM, A4, WN, BN_>;
  constexpr int TI = C_::TI, TJ = C_::TJ, BN = C_::BN;
  constexpr bool RAW = (EPI == kEpiAcc || EPI == kEpiPartial);
  constexpr bool LSQ = (EPI == kEpiDxL || EPI == kEpiDwL);
  constexpr bool GRAD = (EPI == kEpiDx || EPI == kEpiDw || LSQ);
  constexpr bool ROWMAP = (EPI == kEpiDx || EPI == kEpiDxL);  // rows scatter through out_rows
  constexpr int ES = (RAW || DT == kF32) ? 4 : 2;
  constexpr int E_PITCH = BN * ES + 16;
  constexpr int E_ROWS = (BM * E_PITCH <= C_::LDS_MAIN) ? BM
                         : (BM / 2 * E_PITCH <= C_::LDS_MAIN) ? BM / 2
                         : (BM / 4 * E_PITCH <= C_::LDS_MAIN) ? BM / 4 : BM / 8;
  static_assert(E_ROWS >= 32 && E_ROWS * E_PITCH <= C_::LDS_MAIN, "epilogue staging");
  __shared__ __attribute__((aligned(1024))) uint8_t smem[C_::LDS_MAIN];

  const int tid = threadIdx.x, lane = tid & 63;
  // wave index as a scalar: the LDS-DMA destinations (M0) then need no lane-to-scalar moves
  const int wid = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wid / C_::WGN, wn = wid % C_::WGN;
  // grid z: the batch of a batched launch, else the split-K index
  const int nsplit = g.batch > 0 ? 1 : (int)gridDim.z;
  const int zsplit = g.batch > 0 ? 0 : (int)blockIdx.z;
  if (g.batch > 0) {
    const int64_t b = blockIdx.z;
    g.A = static_cast<const uint8_t*>(g.A) + b * g.bs_a;
    g.B = static_cast<const uint8_t*>(g.B) + b * g.bs_b;
    g.out = static_cast<char*>(g.out) + b * g.bs_out * ES;
    if (g.out_rows) g.out_rows += b * g.bs_rows;
    if (g.m_dev) g.m_dev += b;
    if (g.k_dev) g.k_dev += b;
    if (g.amax1) g.amax1 += b;
    if (g.amax2) g.amax2 += b;
    if (g.delta) g.delta += b * g.bs_delta;
    if (g.ds_part) g.ds_part += b * gridDim.x;
  }

  int64_t M = g.M;
  if (g.m_dev) {
    const int64_t md = *g.m_dev;
    M = md < M ? md : M;
  }
  const int tiles_n = (int)((g.N + BN - 1) / BN);
  const int t_valid = tiles_n * (int)((M + BM - 1) / BM);  // tiles with rows below M
  int tm, tn;
  // column groups: 4 tiles for INT4 x INT4 (the 256-wide B panels are twice the A panels),
  // 8 for int8 x INT4 (equal panels)
  if (!tile_of<A4 ? 4 : 8>(t_valid, tiles_n, tm, tn)) {  // uniform exit before any barrier
    if constexpr (LSQ) {
      if (tid == 0) g.ds_part[blockIdx.x] = 0.0;
    }
    return;
  }
  const int64_t m0 = (int64_t)tm * BM, n0 = (int64_t)tn * BN;
  // the scale is read up front so that its latency hides behind the main loop
  float alpha = 0.f;
  if constexpr (EPI == kEpiFwd) {
    // fl(alpha 2^-SHIFT * fl(acc)) == fl(alpha * fl(acc >> SHIFT)): acc is a multiple of
    // 2^SHIFT and both scalings by powers of two are exact
    alpha = scale_of(g) * (1.0f / (float)(1 << C_::SHIFT));
  } else if constexpr (GRAD) {
    alpha = scale_of(g);
  }
  int64_t K = g.K;
  if (g.k_dev) K = ((int64_t)*g.k_dev + 127) / 128 * 128;
  // split-K range of this workgroup (whole stages)
  const int nst_all = (int)((K + kKS - 1) / kKS);
  const int per = (nst_all + nsplit - 1) / nsplit;
  const int st0 = zsplit * per;
  const int nst = max(0, min(nst_all, st0 + per) - st0);
  const int64_t Ka = A4 ? K / 2 : K, Kb = K / 2;  // row extents in bytes

  // per-lane source pointers of this wave's DMA blocks (stage 0 of this split); rows past
  // the end re-read the last row (their results are never stored)
  const uint8_t* pa[C_::A_BPW];
  const uint8_t* pb[C_::B_BPW];
  int ca[C_::A_BPW], cb[C_::B_BPW];
#pragma unroll
  for (int x = 0; x < C_::A_BPW; ++x) {
    const int r = (wid * C_::A_BPW + x) * (1024 / C_::RA) + lane / C_::CPA;
    const int c = (lane % C_::CPA) ^ swz<C_::RA>(r);
    int64_t gm = m0 + r;
    gm = gm < M ? gm : M - 1;
    ca[x] = c * 16;
    pa[x] = static_cast<const uint8_t*>(g.A) + gm * g.lda + (int64_t)st0 * C_::RA + c * 16;
  }
#pragma unroll
  for (int x = 0; x < C_::B_BPW; ++x) {
    const int s = (wid * C_::B_BPW + x) * (1024 / C_::RB) + lane / C_::CPB;
    const int c = (lane % C_::CPB) ^ swz<C_::RB>(s);
    int64_t gn = n0 + b_row_of_slot<C_::WN>(s);
    gn = gn < g.N ? gn : g.N - 1;
    cb[x] = c * 16;
    pb[x] = static_cast<const uint8_t*>(g.B) + gn * g.ldb + (int64_t)st0 * C_::RB + c * 16;
  }
  // issue the loads of local stage st into buffer st % NBUF; chunks past K are zeroed
  auto issue = [&](int st) {
    uint8_t* sa = smem + (st % C_::NBUF) * C_::STAGE;
    uint8_t* sb = sa + C_::A_BYTES;
    const int64_t ka = (int64_t)(st0 + st) * C_::RA, kb = (int64_t)(st0 + st) * C_::RB;
    if (ka + C_::RA <= Ka && kb + C_::RB <= Kb) {  // whole stage inside K: straight line
#pragma unroll
      for (int x = 0; x < C_::A_BPW; ++x)
        dma16(pa[x] + (int64_t)st * C_::RA, sa + (wid * C_::A_BPW + x) * 1024);
#pragma unroll
      for (int x = 0; x < C_::B_BPW; ++x)
        dma16(pb[x] + (int64_t)st * C_::RB, sb + (wid * C_::B_BPW + x) * 1024);
      return;
    }
#pragma unroll
    for (int x = 0; x < C_::A_BPW; ++x) {
      uint8_t* dst = sa + (wid * C_::A_BPW + x) * 1024;
      if (ka + ca[x] < Ka)
        dma16(pa[x] + (int64_t)st * C_::RA, dst);
      else
        *reinterpret_cast<uint4*>(dst + lane * 16) = make_uint4(0u, 0u, 0u, 0u);
    }
#pragma unroll
    for (int x = 0; x < C_::B_BPW; ++x) {
      uint8_t* dst = sb + (wid * C_::B_BPW + x) * 1024;
      if (kb + cb[x] < Kb)
        dma16(pb[x] + (int64_t)st * C_::RB, dst);
      else
        *reinterpret_cast<uint4*>(dst + lane * 16) = make_uint4(0u, 0u, 0u, 0u);
    }
  };

  v16i acc[TI][TJ];
#pragma unroll
  for (int i = 0; i < TI; ++i)
#pragma unroll
    for (int j = 0; j < TJ; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0;

  // fragment rows of this lane and their swizzles
  const int frow = lane & 31, fg = lane >> 5;
  int offa[TI], sza[TI], offb[TJ], szb[TJ];
#pragma unroll
  for (int i = 0; i < TI; ++i) {
    const int r = wm * C_::WM + 32 * i + frow;
    offa[i] = r * C_::RA;
    sza[i] = swz<C_::RA>(r);
  }
#pragma unroll
  for (int j = 0; j < TJ; ++j) {
    const int r = wn * C_::WN + 32 * j + frow;
    offb[j] = r * C_::RB;
    szb[j] = swz<C_::RB>(r);
  }

  // Software pipeline over the four 32-k MFMA steps of a stage.  While the 8 MFMAs of
  // step t run, the next step's fragments are widened and the LDS reads of the pair after
  // are issued, interleaved one MFMA at a time (the wave issues in order, so a burst of
  // MFMAs would otherwise hold back its own VALU and LDS work).  Raw reads cover a pair
  // of steps (16 bytes of INT4 per lane) and sit in slot 0 (steps 0, 1) or slot 1 (2, 3);
  // the wait for the next stage's loads and the barrier come after step 1, when every
  // read of the current stage has been issued, and that barrier frees the current buffer
  // for the next load.
  constexpr int RA_PAIR = A4 ? 1 : 2;  // 16-byte A reads per row per pair
  uint4 rb[2][TJ], ra[2][RA_PAIR][TI];
  v4i fb[2][TJ], fa[2][TI];
  auto read_pair = [&](int slot, int st, int pp) {
    const uint8_t* sa = smem + (st % C_::NBUF) * C_::STAGE;
    const uint8_t* sb = sa + C_::A_BYTES;
#pragma unroll
    for (int j = 0; j < TJ; ++j)
      rb[slot][j] = *reinterpret_cast<const uint4*>(sb + offb[j] + (((2 * pp + fg) ^ szb[j]) << 4));
#pragma unroll
    for (int h = 0; h < RA_PAIR; ++h)
#pragma unroll
      for (int i = 0; i < TI; ++i) {
        const int c = A4 ? 2 * pp + fg : 4 * pp + 2 * fg + h;
        ra[slot][h][i] = *reinterpret_cast<const uint4*>(sa + offa[i] + ((c ^ sza[i]) << 4));
      }
  };
  auto widen_step = [&](int f, int slot, int h) {
#pragma unroll
    for (int j = 0; j < TJ; ++j) fb[f][j] = widen(rb[slot][j], h);
#pragma unroll
    for (int i = 0; i < TI; ++i) fa[f][i] = A4 ? widen(ra[slot][0][i], h) : as_frag(ra[slot][h][i]);
  };
  auto mfma_step = [&](int f) {
#pragma unroll
    for (int i = 0; i < TI; ++i)
#pragma unroll
      for (int j = 0; j < TJ; ++j)
        acc[i][j] = __builtin_amdgcn_mfma_i32_32x32x32_i8(fb[f][j], fa[f][i], acc[i][j], 0, 0, 0);
  };
  auto interleave = [&]() {
#pragma unroll
    for (int q = 0; q < TI * TJ; ++q) {
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);  // 1 MFMA
      __builtin_amdgcn_sched_group_barrier(0x002, 5, 0);  // up to 5 VALU
      __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);  // up to 1 LDS read
    }
  };
#ifndef HQLSS_LSQ_PREFETCH
#define HQLSS_LSQ_PREFETCH 1
#endif
  // Learned-step epilogues read this tile's deltas (2 B per output) after the main loop.
  // The deltas are fetched into the caches during the main loop by LDS-DMA loads into a
  // 1 KB sink (no registers held): each lane touches one 128-byte line of one row.
  constexpr bool PREFETCH = LSQ && HQLSS_LSQ_PREFETCH;
  // with two stage buffers every stage wait drains all loads, the prefetch included
  static_assert(!PREFETCH || C_::NBUF == 2, "partial stage waits would not count the prefetch");
  __shared__ __attribute__((aligned(1024))) uint8_t pf_sink[PREFETCH ? 1024 : 16];
  int pf_row[2] = {0, 0};
  if constexpr (PREFETCH) {
#pragma unroll
    for (int x = 0; x < 2; ++x) {
      int64_t gm = m0 + (wid * 2 + x) * 16 + (lane >> 2);
      gm = gm < M ? gm : M - 1;
      pf_row[x] = ROWMAP ? g.out_rows[gm] : (int)gm;
    }
  }
  auto prefetch_delta = [&]() {
    if constexpr (PREFETCH) {
      int64_t col = n0 + (int64_t)(lane & 3) * 64;  // one 128-byte line of fp16
      col = col < g.N ? col : n0;
#pragma unroll
      for (int x = 0; x < 2; ++x) dma16(g.delta + (int64_t)pf_row[x] * g.ldo + col, pf_sink);
    }
  };
  auto stage_ready = [&](int st) {  // this wave's loads of stage st landed, then all waves'
    // loads of later stages may stay in flight: min(NBUF - 2, nst - 1 - st) of them
    const int later = nst - 1 - st;
    if (C_::NBUF >= 4 && later >= 2) wait_vm_lgkm0<2 * C_::DMA>();
    else if (C_::NBUF >= 3 && later >= 1) wait_vm_lgkm0<C_::DMA>();
    else wait_vm_lgkm0<0>();
    __builtin_amdgcn_s_barrier();
    if (st + C_::NBUF - 1 < nst) issue(st + C_::NBUF - 1);
    if (st == 0) prefetch_delta();
  };
#pragma unroll
  for (int p = 0; p < C_::NBUF - 1; ++p)
    if (p < nst) issue(p);
  if (nst > 0) {
    stage_ready(0);
    read_pair(0, 0, 0);
    widen_step(0, 0, 0);
  }
  for (int st = 0; st + 1 < nst; ++st) {  // stages with a successor: branch-free steps
    // step 0: MFMAs on F0 || widen step 1, read pair 1
    mfma_step(0);
    widen_step(1, 0, 1);
    read_pair(1, st, 1);
    interleave();
    // step 1: MFMAs on F1 || widen step 2 (pair 1 landed during step 0)
    mfma_step(1);
    widen_step(0, 1, 0);
    interleave();
    stage_ready(st + 1);
    // step 2: MFMAs on F0 || widen step 3, read pair 0 of the next stage
    mfma_step(0);
    widen_step(1, 1, 1);
    read_pair(0, st + 1, 0);
    interleave();
    // step 3: MFMAs on F1 || widen step 0 of the next stage
    mfma_step(1);
    widen_step(0, 0, 0);
    interleave();
  }
  if (nst > 0) {  // last stage
    mfma_step(0);
    widen_step(1, 0, 1);
    read_pair(1, nst - 1, 1);
    interleave();
    mfma_step(1);
    widen_step(0, 1, 0);
    interleave();
    mfma_step(0);
    widen_step(1, 1, 1);
    interleave();
    mfma_step(1);
  }
  wait_vm_lgkm0<0>();
  __builtin_amdgcn_s_barrier();  // every wave is done with the stage buffers

  // ---------------------------------------------------------------- epilogue
  // values of (i, j): row m = wm*WM + 32 i + (lane % 32), columns n = wn*WN + 16 j +
  // (WN/2) (lane / 32) + r.  They go through LDS so that every store writes whole rows.
  const int ml = lane & 31;
  const int nh = (C_::WN / 2) * (lane >> 5);
  double lsq_sum = 0.0;
  if constexpr (LSQ) {
    // sum of acc * delta over this workgroup's valid entries, then the clip mask (App. A.3):
    // both use the integer accumulator before the transform H^T.  Rows past M hold
    // re-read data and are skipped; N is a multiple of the block, so the mask never mixes
    // valid and invalid columns inside one transform.
#pragma unroll
    for (int i = 0; i < TI; ++i) {
      const int64_t gm = m0 + wm * C_::WM + 32 * i + ml;
      if (gm >= M) continue;
      const int64_t drow = ROWMAP ? (int64_t)g.out_rows[gm] : gm;
      const uint16_t* dp = g.delta + drow * g.ldo + n0 + wn * C_::WN + nh;
#pragma unroll
      for (int j = 0; j < TJ; ++j) {
        if (n0 + wn * C_::WN + 16 * j + nh >= g.N) continue;
        const uint4 d0 = ld_stream<true>(dp + 16 * j), d1 = ld_stream<true>(dp + 16 * j + 8);
        const uint32_t dw[8] = {d0.x, d0.y, d0.z, d0.w, d1.x, d1.y, d1.z, d1.w};
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const uint32_t h = (dw[r >> 1] >> (16 * (r & 1))) & 0xFFFFu;
          const int a = acc[i][j][r];
          lsq_sum += (double)(a >> C_::SHIFT) * f16_bits_to_double(h);
          acc[i][j][r] = inside_of(h) ? a : 0;
        }
      }
    }
  }
  if constexpr (GRAD) {
#pragma unroll
    for (int i = 0; i < TI; ++i) {
      int v[TJ * 16];
#pragma unroll
      for (int j = 0; j < TJ; ++j)
#pragma unroll
        for (int r = 0; r < 16; ++r) v[16 * j + r] = acc[i][j][r] >> C_::SHIFT;
      fwht_lane<LOG2B, TJ * 16>(v, lane);
#pragma unroll
      for (int j = 0; j < TJ; ++j)
#pragma unroll
        for (int r = 0; r < 16; ++r) acc[i][j][r] = v[16 * j + r];
    }
  }
  constexpr int PIECES = BN * ES / 16;  // 16-byte pieces per output row
  char* const out = static_cast<char*>(g.out);
  const int64_t out_plane = (EPI == kEpiPartial) ? (int64_t)zsplit * g.M * g.ldo : 0;
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
              if constexpr (RAW) w[t] = (uint32_t)(a >> C_::SHIFT);
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
    // every LDS read (and, for dX, every destination-row lookup) of the chunk is issued
    // before the first store, so their latencies overlap instead of adding up
    constexpr int ITER = E_ROWS * PIECES / C_::THREADS;
    static_assert(ITER * C_::THREADS == E_ROWS * PIECES, "whole store rounds");
    uint4 val[ITER];
    int orow[ITER];  // destination row (rows < 2^30), -1 past the end
#pragma unroll
    for (int it = 0; it < ITER; ++it) {
      const int idx = tid + it * C_::THREADS;
      const int r = idx / PIECES, pc = idx % PIECES;
      const int64_t gm = m0 + r_lo + r;
      val[it] = *reinterpret_cast<const uint4*>(smem + r * E_PITCH + pc * 16);
      orow[it] = gm < M ? (ROWMAP ? g.out_rows[gm] : (int)gm) : -1;
    }
#pragma unroll
    for (int it = 0; it < ITER; ++it) {
      const int idx = tid + it * C_::THREADS;
      const int pc = idx % PIECES;
      const int64_t gn = n0 + (int64_t)pc * (16 / ES);
      if (orow[it] >= 0 && gn < g.N)
        st_stream<(EPI == kEpiPartial) ? (bool)HQ_NT_P_ST : (bool)HQ_NT_G_ST>(
            out + (out_plane + (int64_t)orow[it] * g.ldo + gn) * ES, val[it]);
    }
    __syncthreads();
  }
  if constexpr (LSQ) {
    __shared__ double red[C_::WAVES];
    const double t = block_sum_f64<C_::THREADS>(lsq_sum, red);
    if (tid == 0) g.ds_part[blockIdx.x] = t;
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
template <bool A4, int LOG2B> constexpr int wave_n() { return (A4 || LOG2B >= 6) ? 128 : 64; }

// workgroups of reduce_epilogue for an M x N output (four waves, one (row, 512-column
// chunk) item per wave at a time)
int64_t reduce_grid(int64_t M, int64_t N) {
  const int64_t items = M * ((N + 511) / 512);
  int64_t wg = (items + 3) / 4;
  if (wg > 2048) wg = 2048;
  return wg < 1 ? 1 : wg;
}

// BN_: workgroup tile width; kNarrowBN for outputs at most that wide (attention head
// dimensions), which would otherwise leave most of a 256-wide tile idle
template <int BM, bool A4, int EPI, int DT, int LOG2B, int BN_ = kBN>
hipError_t gemm_t(hipStream_t s, const GemmArgs& g, int splits, int id) {
  // 128-wide INT4 x INT4 tiles: 64 x 64 wave tiles (one widened fragment per MFMA)
  constexpr int WN = (A4 && BN_ == kMidBN) ? 64 : wave_n<A4, LOG2B>() < BN_ ? wave_n<A4, LOG2B>() : BN_;
  using C_ = Cfg<BM, A4, WN, BN_>;
  // one workgroup per tile of the M x N output (M the host-side bound; see tile_of)
  dim3 grid((unsigned)(((g.N + BN_ - 1) / BN_) * ((g.M + BM - 1) / BM)), 1u,
            (unsigned)(g.batch > 0 ? g.batch : splits));
  timing_begin(s);
  gemm_kernel<BM, A4, WN, EPI, DT, LOG2B, BN_><<<grid, C_::THREADS, 0, s>>>(g);
  timing_end(s, id);
  return hipGetLastError();
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
template <int BM, bool A4, int EPI, int DT>
hipError_t gemm_b(hipStream_t s, const GemmArgs& g, int splits, int id) {
  if constexpr (EPI == kEpiDx || EPI == kEpiDw || EPI == kEpiDxL || EPI == kEpiDwL) {
    const int bn = grad_bn(g.M, g.N, splits);
    if (bn == kMidBN) {
      switch (g.log2b) {
        case 0: return gemm_t<BM, A4, EPI, DT, 0, kMidBN>(s, g, splits, id);
        case 1: return gemm_t<BM, A4, EPI, DT, 1, kMidBN>(s, g, splits, id);
        case 2: return gemm_t<BM, A4, EPI, DT, 2, kMidBN>(s, g, splits, id);
        case 3: return gemm_t<BM, A4, EPI, DT, 3, kMidBN>(s, g, splits, id);
        case 4: return gemm_t<BM, A4, EPI, DT, 4, kMidBN>(s, g, splits, id);
        case 5: return gemm_t<BM, A4, EPI, DT, 5, kMidBN>(s, g, splits, id);
        case 6: return gemm_t<BM, A4, EPI, DT, 6, kMidBN>(s, g, splits, id);
        case 7: return gemm_t<BM, A4, EPI, DT, 7, kMidBN>(s, g, splits, id);
      }
      return hipErrorInvalidValue;
    }
    if (bn == kNarrowBN) {  // narrow output: blocks of at most 64 columns
      switch (g.log2b) {
        case 0: return gemm_t<BM, A4, EPI, DT, 0, kNarrowBN>(s, g, splits, id);
        case 1: return gemm_t<BM, A4, EPI, DT, 1, kNarrowBN>(s, g, splits, id);
        case 2: return gemm_t<BM, A4, EPI, DT, 2, kNarrowBN>(s, g, splits, id);
        case 3: return gemm_t<BM, A4, EPI, DT, 3, kNarrowBN>(s, g, splits, id);
        case 4: return gemm_t<BM, A4, EPI, DT, 4, kNarrowBN>(s, g, splits, id);
        case 5: return gemm_t<BM, A4, EPI, DT, 5, kNarrowBN>(s, g, splits, id);
        case 6: return gemm_t<BM, A4, EPI, DT, 6, kNarrowBN>(s, g, splits, id);
      }
      return hipErrorInvalidValue;
    }
    switch (g.log2b) {
      case 0: return gemm_t<BM, A4, EPI, DT, 0>(s, g, splits, id);
      case 1: return gemm_t<BM, A4, EPI, DT, 1>(s, g, splits, id);
      case 2: return gemm_t<BM, A4, EPI, DT, 2>(s, g, splits, id);
      case 3: return gemm_t<BM, A4, EPI, DT, 3>(s, g, splits, id);
      case 4: return gemm_t<BM, A4, EPI, DT, 4>(s, g, splits, id);
      case 5: return gemm_t<BM, A4, EPI, DT, 5>(s, g, splits, id);
      case 6: return gemm_t<BM, A4, EPI, DT, 6>(s, g, splits, id);
      case 7: return gemm_t<BM, A4, EPI, DT, 7>(s, g, splits, id);
    }
    return hipErrorInvalidValue;
  } else {
    if (fwd_bn(g.M, g.N, splits, g.batch) == kMidBN) return gemm_t<BM, A4, EPI, DT, 0, kMidBN>(s, g, splits, id);
    return gemm_t<BM, A4, EPI, DT, 0>(s, g, splits, id);
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

template <bool A4, int EPI, int DT>
hipError_t run(hipStream_t s, const GemmArgs& g, int splits, int32_t* partial, int id) {
  constexpr int BM = tile_m<A4>();
  if (splits <= 1) return gemm_b<BM, A4, EPI, DT>(s, g, 1, id);
  GemmArgs p = g;
  p.out = partial;
  p.ldo = g.N;
  hipError_t e = split_mid(A4, g.N) ? gemm_t<BM, A4, kEpiPartial, DT, 0, kMidBN>(s, p, splits, id)
                                     : gemm_t<BM, A4, kEpiPartial, DT, 0>(s, p, splits, id);
  if (e != hipSuccess) return e;
  return reduce_t<DT, EPI>(s, partial, splits, g);
}

template <bool A4, int EPI>
hipError_t run_dt(hipStream_t s, int dt, const GemmArgs& g, int splits, int32_t* partial, int id) {
  switch (dt) {
    case kF32: return run<A4, EPI, kF32>(s, g, splits, partial, id);
    case kF16: return run<A4, EPI, kF16>(s, g, splits, partial, id);
    case kBF16: return run<A4, EPI, kBF16>(s, g, splits, partial, id);
  }
  return hipErrorInvalidValue;
}

}  // namespace

static thread_local int g_split_override = 0;
void gemm_set_split_override(int splits) { g_split_override = splits < 0 ? 0 : splits; }
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
