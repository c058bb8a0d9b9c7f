// Device side of the integer and FP6 GEMMs of HQ-MM / LSS-MM (internal to libhqlss):
// operand layouts, the tile order, the kernel template with its main loops and fused
// epilogues, and its launcher.  Included by the translation units that instantiate it
// (gemm.hip: int8 MFMA route; gemm6.hip: FP6 MFMA route); see gemm.hip for the design.
#pragma once
#include "common.h"
#include "launch.h"

namespace hqlss {

namespace {


typedef int v4i __attribute__((ext_vector_type(4)));
typedef int v16i __attribute__((ext_vector_type(16)));
typedef int v8i __attribute__((ext_vector_type(8)));
typedef int v2i __attribute__((ext_vector_type(2)));
typedef float v16f __attribute__((ext_vector_type(16)));
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
// FP6 256-row tiles: K per stage and stage buffers (128 KB of LDS either way)
#ifndef HQLSS_F6_KS256
#define HQLSS_F6_KS256 128
#endif
#ifndef HQLSS_F6_NBUF256
#define HQLSS_F6_NBUF256 (HQLSS_F6_KS256 == 128 ? 2 : 4)
#endif

// F6: both operands hold FP6 (e2m3) codes in the padded layout of fp6.hip (one byte per
// code: every 32 codes are 24 bytes of 6-bit fields and 8 zero bytes), run on the FP6 MFMA
// (v_mfma_f32_32x32x64_f8f6f4) with fp32 accumulation.  A stage is then 64 k, i.e. 64 bytes
// per row: the LDS geometry of the INT4 x INT4 configuration (A4).
template <int BM, bool A4, int WN_ = 128, int BN_ = kBN, bool F6 = false>
struct Cfg {
  static_assert(!F6 || A4, "the FP6 route uses the INT4 x INT4 geometry");
  // K elements per stage: FP6 128-row tiles (two workgroups per CU) take 64 k, FP6 256-row
  // tiles (one workgroup per CU) 128 k in two 64-k MFMA steps
  static constexpr int KS = F6 ? (BM == 256 ? HQLSS_F6_KS256 : 64) : kKS;
  static constexpr int BN = BN_;
  static constexpr int WAVES = BM / 32, THREADS = 64 * WAVES;
  static constexpr int WN = WN_, WGN = BN / WN, WGM = WAVES / WGN;
  static constexpr int WM = BM / WGM, TI = WM / 32, TJ = WN / 32;
  static constexpr int RA = F6 ? KS : A4 ? kKS / 2 : kKS;  // bytes of an A row per stage
  static constexpr int RB = F6 ? KS : kKS / 2;             // B: INT4, or FP6 (a byte per code)
  static constexpr int CPA = RA / 16, CPB = RB / 16;
  static constexpr int A_BYTES = BM * RA, B_BYTES = BN * RB, STAGE = A_BYTES + B_BYTES;
  static constexpr int A_BPW = A_BYTES / 1024 / WAVES, B_BPW = B_BYTES / 1024 / WAVES;
  static constexpr int DMA = A_BPW + B_BPW;  // 1 KB LDS-DMA loads per wave per stage
  static constexpr int OCC = BM == 128 ? 2 : 1;  // workgroups per CU
  static constexpr int NBUF = (F6 && BM == 256) ? HQLSS_F6_NBUF256 : (OCC == 2 && !A4) ? 2 : 3;
  static constexpr int LDS_MAIN = NBUF * STAGE;
  static constexpr int SHIFT = F6 ? 0 : (A4 ? 4 : 0) + 4;
  static_assert(A_BYTES % (1024 * WAVES) == 0 && B_BYTES % (1024 * WAVES) == 0, "DMA split");
};

// Position p of a group of 8 int8 k in the K-interleaved order holds k = nu8(p):
// 0,2,4,6,1,3,5,7 (the order in which a packed INT4 word widens, see widen()).
__device__ __forceinline__ constexpr int nu8(int p) { return ((p & 3) << 1) | (p >> 2); }

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
    // v_permlane32_swap exchanges the upper half-wave of its first register with the lower
    // half-wave of its second: after one swap of (v[e], v[e + 1]) every lane holds both
    // partners of one butterfly (lanes 0-31 those of element e, lanes 32-63 those of
    // e + 1), and a second swap returns the sum to the lower and the difference to the
    // upper lanes
    static_assert(NV % 2 == 0, "pairs of elements");
#pragma unroll
    for (int e = 0; e < NV; e += 2) {
      const v2i s = __builtin_amdgcn_permlane32_swap(v[e], v[e + 1], false, false);
      const v2i t = __builtin_amdgcn_permlane32_swap(s[0] + s[1], s[0] - s[1], false, false);
      v[e] = t[0];
      v[e + 1] = t[1];
    }
    (void)lane;
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

// F6K (FP6 route): 0 the plain product (forward), kF6Dx the dX product (two K passes for tiles
// holding upper tokens, row weights), kF6Dw the dW product (weight classes along K)
constexpr int kF6Dx = 1, kF6Dw = 2;
// TRA (int8 x INT4 only): A is stored k-major, A[k][m] with pitch lda and its m positions
// K-interleaved in groups of 8 (the dX operand A_T read as the dW operand A_T^T).  A stage
// of it lands in LDS as 128 k rows of BM m bytes, and the gfx950 transposing read
// ds_read_b64_tr_b8 forms the k-contiguous MFMA fragments out of it: in each group of 16
// lanes, byte b of lane j comes from byte j % 8 of the 8 bytes addressed by lane
// 2 b + j / 8.  Output row m' of the tile is then the interleaved position, i.e. row
// (m' & ~7) | nu8(m' & 7) of the result.  K must be whole stages.
template <int BM, bool A4, int WN, int EPI, int DT, int LOG2B, int BN_, bool F6 = false, int F6K = 0,
          bool TRA = false>
__global__ __launch_bounds__((Cfg<BM, A4, WN, BN_, F6>::THREADS), (Cfg<BM, A4, WN, BN_, F6>::OCC)) void gemm_kernel(GemmArgs g) {
  using C_ = Cfg<BM, A4, WN, BN_, F6>;
  constexpr int TI = C_::TI, TJ = C_::TJ, BN = C_::BN;
  constexpr bool RAW = (EPI == kEpiAcc || EPI == kEpiPartial);
  constexpr bool LSQ = (EPI == kEpiDxL || EPI == kEpiDwL);
  constexpr bool GRAD = (EPI == kEpiDx || EPI == kEpiDw || LSQ);
  constexpr bool ROWMAP = (EPI == kEpiDx || EPI == kEpiDxL);  // rows scatter through out_rows
  constexpr int ES = (RAW || DT == kF32) ? 4 : 2;
  constexpr int E_PITCH = BN * ES + 16;
  // Two workgroups per CU leave up to 80 KB of LDS each: the epilogue stages all BM rows in
  // one round when they fit there, even past the stage buffers (the 128 x 256 gradient
  // tiles with 2-byte outputs: 66 KB against 64 KB of stages).
  constexpr int SMEM = (C_::OCC == 2 && BM * E_PITCH > C_::LDS_MAIN && BM * E_PITCH <= 78 * 1024)
                           ? BM * E_PITCH : C_::LDS_MAIN;
  constexpr int E_ROWS = (BM * E_PITCH <= SMEM) ? BM
                         : (BM / 2 * E_PITCH <= SMEM) ? BM / 2
                         : (BM / 4 * E_PITCH <= SMEM) ? BM / 4 : BM / 8;
  static_assert(E_ROWS >= 32 && E_ROWS * E_PITCH <= SMEM, "epilogue staging");
  static_assert(!(F6 && LSQ), "the learned-step epilogues run on the int8 route");
  static_assert(!TRA || (!A4 && !F6 && !ROWMAP && C_::RA == 128 && C_::KS == 128),
                "k-major A: int8 A, 128-byte rows of 128 k per stage, plain output rows");
  // result row of tile row gm (k-major A: the K-interleaved position gm)
  auto res_row = [](int64_t gm) -> int64_t { return TRA ? ((gm & ~int64_t(7)) | nu8((int)(gm & 7))) : gm; };
  __shared__ __attribute__((aligned(1024))) uint8_t smem[SMEM];

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
  // FP6 dX tiles holding upper-row tokens (rows below *m2_dev) run two K passes, first over
  // the upper codes (A2), then the lower ones (A), each of npass stages
  int npass = 0;
  bool two = false;
  if constexpr (F6 && F6K == kF6Dx) {
    npass = (int)((K + C_::KS - 1) / C_::KS);
    two = m0 < (int64_t)*g.m2_dev;
  }
  // split-K range of this workgroup (whole stages)
  const int nst_all = two ? 2 * npass : (int)((K + C_::KS - 1) / C_::KS);
  const int per = (nst_all + nsplit - 1) / nsplit;
  const int st0 = zsplit * per;
  const int nst = max(0, min(nst_all, st0 + per) - st0);
  const int64_t Ka = F6 ? K : A4 ? K / 2 : K, Kb = F6 ? K : K / 2;  // row extents in bytes

  // per-lane source pointers of this wave's DMA blocks (stage 0 of this split); rows past
  // the end re-read the last row (their results are never stored)
  const uint8_t* pa[C_::A_BPW];
  const uint8_t* pb[C_::B_BPW];
  int ca[C_::A_BPW], cb[C_::B_BPW];
#pragma unroll
  for (int x = 0; x < C_::A_BPW; ++x) {
    const int r = (wid * C_::A_BPW + x) * (1024 / C_::RA) + lane / C_::CPA;
    if constexpr (TRA) {  // r: k row of the stage; chunks past M re-read the last 16 m
      const int c = (lane % C_::CPA) ^ (r & 7);
      int64_t col = m0 + c * 16;
      col = col + 16 <= M ? col : M - 16;
      ca[x] = c * 16;
      pa[x] = static_cast<const uint8_t*>(g.A) + ((int64_t)st0 * C_::KS + r) * g.lda + col;
      continue;
    }
    const int c = (lane % C_::CPA) ^ swz<C_::RA>(r);
    int64_t gm = m0 + r;
    gm = gm < M ? gm : M - 1;
    ca[x] = c * 16;
    pa[x] = static_cast<const uint8_t*>(g.A) + gm * g.lda + (F6 ? 0 : (int64_t)st0 * C_::RA) + c * 16;
  }
#pragma unroll
  for (int x = 0; x < C_::B_BPW; ++x) {
    const int s = (wid * C_::B_BPW + x) * (1024 / C_::RB) + lane / C_::CPB;
    const int c = (lane % C_::CPB) ^ swz<C_::RB>(s);
    int64_t gn = n0 + b_row_of_slot<C_::WN>(s);
    gn = gn < g.N ? gn : g.N - 1;
    cb[x] = c * 16;
    pb[x] = static_cast<const uint8_t*>(g.B) + gn * g.ldb + (F6 ? 0 : (int64_t)st0 * C_::RB) + c * 16;
  }
  // issue the loads of local stage st into buffer st % NBUF; chunks past K are zeroed
  // FP6: the byte offset of global stage gs in the rows (a byte per code, same for A and B),
  // and for two-pass tiles the upper operand A2 in the first pass
  const int64_t dA2 = (F6K == kF6Dx && two) ? static_cast<const uint8_t*>(g.A2) - static_cast<const uint8_t*>(g.A) : 0;
  auto issue = [&](int st) {
    uint8_t* sa = smem + (st % C_::NBUF) * C_::STAGE;
    uint8_t* sb = sa + C_::A_BYTES;
    if constexpr (F6) {
      const int gs = st0 + st;
      const bool upper = two && gs < npass;
      const int64_t kin = (int64_t)(two && !upper ? gs - npass : gs) * C_::RA;
      const int64_t da = upper ? dA2 : 0;
      if (kin + C_::RA <= K) {
#pragma unroll
        for (int x = 0; x < C_::A_BPW; ++x) dma16(pa[x] + da + kin, sa + (wid * C_::A_BPW + x) * 1024);
#pragma unroll
        for (int x = 0; x < C_::B_BPW; ++x) dma16(pb[x] + kin, sb + (wid * C_::B_BPW + x) * 1024);
        return;
      }
#pragma unroll
      for (int x = 0; x < C_::A_BPW; ++x) {
        uint8_t* dst = sa + (wid * C_::A_BPW + x) * 1024;
        if (kin + ca[x] < K)
          dma16(pa[x] + da + kin, dst);
        else
          *reinterpret_cast<uint4*>(dst + lane * 16) = make_uint4(0u, 0u, 0u, 0u);
      }
#pragma unroll
      for (int x = 0; x < C_::B_BPW; ++x) {
        uint8_t* dst = sb + (wid * C_::B_BPW + x) * 1024;
        if (kin + cb[x] < K)
          dma16(pb[x] + kin, dst);
        else
          *reinterpret_cast<uint4*>(dst + lane * 16) = make_uint4(0u, 0u, 0u, 0u);
      }
      return;
    }
    if constexpr (TRA) {  // whole stages (K a multiple of 128): A advances by 128 rows
#pragma unroll
      for (int x = 0; x < C_::A_BPW; ++x)
        dma16(pa[x] + (int64_t)st * C_::KS * g.lda, sa + (wid * C_::A_BPW + x) * 1024);
#pragma unroll
      for (int x = 0; x < C_::B_BPW; ++x)
        dma16(pb[x] + (int64_t)st * C_::RB, sb + (wid * C_::B_BPW + x) * 1024);
      return;
    }
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

  // int32 accumulators; the FP6 route accumulates in fp32 (accf, exact integers) and its
  // epilogues read those directly (the gradient ones convert a row block at a time)
  v16i acc[TI][TJ];
  v16f accf[TI][TJ];
  if constexpr (!F6) {
#pragma unroll
    for (int i = 0; i < TI; ++i)
#pragma unroll
      for (int j = 0; j < TJ; ++j)
#pragma unroll
        for (int r = 0; r < 16; ++r) acc[i][j][r] = 0;
  }

  // fragment rows of this lane and their swizzles
  const int frow = lane & 31, fg = lane >> 5;
  int offa[TI], sza[TI], offb[TJ], szb[TJ];
#pragma unroll
  for (int i = 0; i < TI; ++i) {
    const int r = wm * C_::WM + 32 * i + frow;
    offa[i] = r * C_::RA;
    sza[i] = swz<C_::RA>(r);
    if constexpr (TRA) {
      // lane j of 16-lane group q (m half q % 2, k half fg = q / 2) supplies the 8 bytes
      // of k row 32 fg + nu8(j / 2) (+ the step's offset) at m bytes 16 (q % 2) + 8 (j % 2)
      // of the fragment's 32; that row's chunks are swizzled by its k % 8 = nu8(j / 2)
      const int j = lane & 15, q = lane >> 4, kr = nu8(j >> 1);
      const int chunk = (wm * C_::WM + 32 * i) / 16 + (q & 1);
      offa[i] = (32 * (q >> 1) + kr) * C_::RA + ((chunk ^ kr) << 4) + 8 * (j & 1);
    }
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
        if constexpr (TRA) {
          // k step 2 pp + h: bytes 0-7 of the fragment from k rows 64 pp + 16 h + 0..7 (+ 32 fg),
          // bytes 8-15 from the next 8 rows
          typedef __attribute__((address_space(3))) v2i lds_v2i;
          const uint8_t* p = sa + offa[i] + (64 * pp + 16 * h) * C_::RA;
          const v2i lo = __builtin_amdgcn_ds_read_tr8_b64_v2i32((lds_v2i*)(lds_void*)p);
          const v2i hi = __builtin_amdgcn_ds_read_tr8_b64_v2i32((lds_v2i*)(lds_void*)(p + 8 * C_::RA));
          ra[slot][h][i] = make_uint4((uint32_t)lo[0], (uint32_t)lo[1], (uint32_t)hi[0], (uint32_t)hi[1]);
          continue;
        }
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
      __builtin_amdgcn_sched_group_barrier(0x002, 3, 0);  // up to 3 VALU
      __builtin_amdgcn_sched_group_barrier(0x100, TRA ? 2 : 1, 0);  // LDS reads
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
      pf_row[x] = ROWMAP ? g.out_rows[gm] : (int)res_row(gm);
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
  // The main loop runs at wave priority 1 and the epilogue at 0: when the two workgroups
  // of a CU share a SIMD, the one feeding the matrix core wins the issue slots over the
  // other's conversion and Hadamard arithmetic.
  __builtin_amdgcn_s_setprio(1);
  if constexpr (F6) {
    // FP6 main loop: one stage is one 64-k MFMA step.  A lane's fragment of a row is the
    // 32-byte group of its 32 k (24 bytes of fields, then the 8 zero bytes the instruction
    // does not read): two 16-byte LDS reads of chunks 2 fg and 2 fg + 1.  While the 8 MFMAs
    // of stage st run, the fragments of stage st + 1 are read, interleaved one MFMA at a
    // time; the stage wait and barrier come first, when this wave's reads of stage st have
    // landed, and that barrier frees stage st's buffer for the load NBUF - 1 stages ahead.
    // Products of codes |q| <= 7 and their sums are integers far below 2^24, so the fp32
    // accumulation is exact and the result equals the integer GEMM's.
#pragma unroll
    for (int i = 0; i < TI; ++i)
#pragma unroll
      for (int j = 0; j < TJ; ++j)
#pragma unroll
        for (int r = 0; r < 16; ++r) accf[i][j][r] = 0.f;
    v8i f6a[2][TI], f6b[2][TJ];
    constexpr int KST = C_::KS / 64;  // 64-k MFMA steps per stage
    // 16 + 8 bytes of group (2 ks + fg) of the stage: the zero bytes are not read
    auto frag6 = [&](const uint8_t* row, int sz, int ks) {
      const uint4 lo = *reinterpret_cast<const uint4*>(row + (((4 * ks + 2 * fg) ^ sz) << 4));
      const uint2 hi = *reinterpret_cast<const uint2*>(row + (((4 * ks + 2 * fg + 1) ^ sz) << 4));
      v8i f;
      f[0] = (int)lo.x; f[1] = (int)lo.y; f[2] = (int)lo.z; f[3] = (int)lo.w;
      f[4] = (int)hi.x; f[5] = (int)hi.y; f[6] = 0; f[7] = 0;
      return f;
    };
    auto read6 = [&](int f, int st, int ks) {
      const uint8_t* sa = smem + (st % C_::NBUF) * C_::STAGE;
      const uint8_t* sb = sa + C_::A_BYTES;
#pragma unroll
      for (int j = 0; j < TJ; ++j) f6b[f][j] = frag6(sb + offb[j], szb[j], ks);
#pragma unroll
      for (int i = 0; i < TI; ++i) f6a[f][i] = frag6(sa + offa[i], sza[i], ks);
    };
    auto mfma6 = [&](int f) {
#pragma unroll
      for (int i = 0; i < TI; ++i)
#pragma unroll
        for (int j = 0; j < TJ; ++j)  // formats 2, 2: e2m3 x e2m3; zero scales: unscaled form
          accf[i][j] = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(f6b[f][j], f6a[f][i], accf[i][j],
                                                                       2, 2, 0, 0, 0, 0);
    };
    auto interleave6 = [&]() {
#pragma unroll
      for (int q = 0; q < TI * TJ; ++q) {
        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);  // 1 MFMA
        __builtin_amdgcn_sched_group_barrier(0x100, 2, 0);  // up to 2 LDS reads
      }
    };
    // Weights the GEMM applies to its fp32 accumulators (all exact: powers of two, and for
    // dX 14 / w_dn in {14, 7, 3.5} on half-integers below 2^23).
    //   dX: row m of token t accumulates f1 x (upper pass) + lower pass, times f2, with
    //   f1 = 14 / w_dn (14 if w_dn = 0, whose lower row is zero) and f2 = max(w_dn, 1),
    //   giving 14 w_up acc_up + w_dn acc_dn.
    //   dW: the K entries come in classes of weight 2^4 .. 2^0 (class bounds kcls); crossing
    //   from class e to e' doubles the sum e - e' times (Horner), and the sum ends times
    //   2^(class of the last stage).
    // The K loop runs in segments between the stages where a weight is due, so the loop
    // body itself never touches the accumulators outside the MFMAs.
    int b3 = 0, b2 = 0, b1 = 0, b0 = 0;
    if constexpr (F6K == kF6Dw) {
      b3 = g.kcls[0]; b2 = g.kcls[1]; b1 = g.kcls[2]; b0 = g.kcls[3];
    }
    auto cls_of = [&](int gs) {  // weight class of global stage gs (128 entries)
      const int e = gs * C_::KS;
      return 4 - (e >= b3) - (e >= b2) - (e >= b1) - (e >= b0);
    };
    auto next_bound = [&](int gs) {  // first global stage after gs where a weight is due
      int nb = 1 << 30;
      if constexpr (F6K == kF6Dx) {
        if (two && gs < npass) nb = npass;
      } else if constexpr (F6K == kF6Dw) {
        const int bs[4] = {b3, b2, b1, b0};
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const int b = bs[q] / C_::KS;
          if (b > gs && b < nb) nb = b;
        }
      }
      return nb;
    };
    auto row_weights = [&](bool up_pass) {  // dX: f1 (up_pass) or f2 of this lane's rows
#pragma unroll
      for (int i = 0; i < TI; ++i) {
        const int64_t m = m0 + wm * C_::WM + 32 * i + (lane & 31);
        float f = 1.f;
        if (m < M) {
          const int t = g.out_rows[m];
          const int wu = g.w_up[t], wd = g.w_dn[t];
          f = up_pass ? (wu ? (wd ? 14.f / (float)wd : 14.f) : 1.f) : (wd ? (float)wd : 1.f);
        }
#pragma unroll
        for (int j = 0; j < TJ; ++j)
#pragma unroll
          for (int r = 0; r < 16; ++r) accf[i][j][r] *= f;
      }
    };
    auto scale_all = [&](int sh) {
      const float f = (float)(1 << sh);
#pragma unroll
      for (int i = 0; i < TI; ++i)
#pragma unroll
        for (int j = 0; j < TJ; ++j)
#pragma unroll
          for (int r = 0; r < 16; ++r) accf[i][j][r] *= f;
    };
    auto rescale6 = [&](int gs) {  // before global stage gs (gs > st0) runs
      if constexpr (F6K == kF6Dx) {
        if (two && gs == npass) row_weights(true);
      } else if constexpr (F6K == kF6Dw) {
        const int d = cls_of(gs - 1) - cls_of(gs);
        if (d > 0) scale_all(d);
      }
    };
#pragma unroll
    for (int p = 0; p < C_::NBUF - 1; ++p)
      if (p < nst) issue(p);
    if constexpr (KST == 1) {
      if (nst > 0) {
        stage_ready(0);
        read6(0, 0, 0);
      }
      int st = 0;
      for (; st + 2 < nst; st += 2) {
        stage_ready(st + 1);
        read6(1, st + 1, 0);
        mfma6(0);
        interleave6();
        stage_ready(st + 2);
        read6(0, st + 2, 0);
        mfma6(1);
        interleave6();
      }
      if (st + 1 < nst) {
        stage_ready(st + 1);
        read6(1, st + 1, 0);
        mfma6(0);
        interleave6();
        mfma6(1);
      } else if (st < nst) {
        mfma6(0);
      }
    } else {  // two steps per stage: the wait and barrier sit between them
      static_assert(KST == 2, "FP6 stages of one or two MFMA steps");
      if (nst > 0) {
        stage_ready(0);
        read6(0, 0, 0);
      }
      int st = 0;
      while (st < nst) {
        const int seg = min(nst, next_bound(st0 + st) - st0);
        for (; st < seg; ++st) {
          read6(1, st, 1);
          mfma6(0);
          interleave6();
          if (st + 1 < nst) {
            stage_ready(st + 1);
            read6(0, st + 1, 0);
          }
          mfma6(1);
          interleave6();
        }
        if (st < nst) rescale6(st0 + st);
      }
    }
    if (nst > 0) {  // the weights still due at the end of this split's K range
      const int gl = st0 + nst - 1;
      if constexpr (F6K == kF6Dx) {
        if (two && gl < npass) row_weights(true);
        row_weights(false);
      } else if constexpr (F6K == kF6Dw) {
        const int e = cls_of(gl);
        if (e > 0) scale_all(e);
      }
    }
  } else {
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
  }
  wait_vm_lgkm0<0>();
  __builtin_amdgcn_s_barrier();  // every wave is done with the stage buffers
  __builtin_amdgcn_s_setprio(0);

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
    // valid and invalid columns inside one transform.  Four partial sums (by r % 4) keep
    // the fp64 additions out of one dependent chain; each product is exact in fp64.
    double part[4] = {0.0, 0.0, 0.0, 0.0};
#pragma unroll
    for (int i = 0; i < TI; ++i) {
      const int64_t gm = m0 + wm * C_::WM + 32 * i + ml;
      if (gm >= M) continue;
      const int64_t drow = ROWMAP ? (int64_t)g.out_rows[gm] : res_row(gm);
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
          part[r & 3] = __builtin_fma((double)(a >> C_::SHIFT), f16_bits_to_double(h), part[r & 3]);
          acc[i][j][r] = inside_of(h) ? a : 0;
        }
      }
    }
    lsq_sum = (part[0] + part[1]) + (part[2] + part[3]);
  }
  if constexpr (GRAD) {
#pragma unroll
    for (int i = 0; i < TI; ++i) {
      int v[TJ * 16];
#pragma unroll
      for (int j = 0; j < TJ; ++j)
#pragma unroll
        for (int r = 0; r < 16; ++r) v[16 * j + r] = F6 ? (int)accf[i][j][r] : acc[i][j][r] >> C_::SHIFT;
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
              if constexpr (F6 && !GRAD) {
                const float a = accf[i][j][4 * q + t];
                if constexpr (RAW) w[t] = (uint32_t)(int)a;
                else w[t] = __float_as_uint(alpha * a);
              } else {
                const int a = acc[i][j][4 * q + t];
                if constexpr (RAW) w[t] = (uint32_t)(a >> C_::SHIFT);
                else w[t] = __float_as_uint(alpha * (float)a);
              }
            }
            p[q] = make_uint4(w[0], w[1], w[2], w[3]);
          }
        } else {
          float f[16];
#pragma unroll
          for (int r = 0; r < 16; ++r)
            f[r] = alpha * ((F6 && !GRAD) ? accf[i][j][r] : (float)acc[i][j][r]);
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
      orow[it] = gm < M ? (ROWMAP ? g.out_rows[gm] : (int)res_row(gm)) : -1;
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
template <bool A4, int LOG2B> constexpr int wave_n() { return (A4 || LOG2B >= 6) ? 128 : 64; }

// workgroups of reduce_epilogue for an M x N output (four waves, one (row, 512-column
// chunk) item per wave at a time)
// BN_: workgroup tile width; kNarrowBN for outputs at most that wide (attention head
// dimensions), which would otherwise leave most of a 256-wide tile idle
template <int BM, bool A4, int EPI, int DT, int LOG2B, int BN_ = kBN, bool F6 = false, int F6K = 0,
          bool TRA = false>
hipError_t gemm_t(hipStream_t s, const GemmArgs& g, int splits, int id) {
  // 128-wide INT4 x INT4 tiles: 64 x 64 wave tiles (one widened fragment per MFMA)
  constexpr int WN = (A4 && BN_ == kMidBN) ? 64 : wave_n<A4, LOG2B>() < BN_ ? wave_n<A4, LOG2B>() : BN_;
  using C_ = Cfg<BM, A4, WN, BN_, F6>;
  // one workgroup per tile of the M x N output (M the host-side bound; see tile_of)
  dim3 grid((unsigned)(((g.N + BN_ - 1) / BN_) * ((g.M + BM - 1) / BM)), 1u,
            (unsigned)(g.batch > 0 ? g.batch : splits));
  timing_begin(s);
  if (TRA && (g.K % kKS != 0 || g.M % 16 != 0)) return hipErrorInvalidValue;  // whole stages, 16 m
  gemm_kernel<BM, A4, WN, EPI, DT, LOG2B, BN_, F6, F6K, TRA><<<grid, C_::THREADS, 0, s>>>(g);
  timing_end(s, id);
  return hipGetLastError();
}

}  // namespace

}  // namespace hqlss
