// bf16 implicit-GEMM convolutions on gfx950 MFMA (v_mfma_f32_32x32x16_bf16),
// fp32 accumulation, NHWC activations, KRSC weights.
//
// Forward (and data gradient, which is the same contraction on the rotated,
// transposed weight):  Y^T[co][p] = sum_k W[co][k] * im2col(X)[p][k],
// k = (tap, ci) so that every 64-wide K slice is one filter tap and 64
// contiguous channels: both operands are K-contiguous 128-byte rows that are
// staged into LDS with 16-byte loads.  Each block computes a BN x BM
// (channels x pixels) tile with 4 waves; bias + ReLU + bf16 rounding are fused
// into the epilogue.
//
// Weight gradient:  dW[co][tap][ci] = sum_p dZ[p][co] * X[p + off(tap)][ci],
// K = pixels.  In NHWC both operands are channel-contiguous, so each thread
// loads an 8-pixel x 8-channel block with 16-byte loads and transposes it in
// registers before writing pixel-contiguous rows to LDS.  The pixel range is
// split over grid.z; each split writes its fp32 partial tile and a second
// kernel sums the splits in fixed order (deterministic, no atomics).
#include "common.h"
#include "kernels.h"
#include "prof.h"

namespace tgpk {
namespace {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));
// 16-byte chunk as a native vector (HIP's u32x4 wraps a union that keeps
// arrays of it out of registers)
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

// XOR swizzle of the eight 16-byte chunks of a 128-byte LDS row, so that
// eight consecutive rows read at the same logical chunk, and rows eight apart
// written at the same chunk, hit distinct banks.
__device__ __forceinline__ int swz(int row, int q) { return q ^ ((row ^ (row >> 3)) & 7); }

__device__ __forceinline__ bf16x8_t as_bf16x8(u32x4 v) { return __builtin_bit_cast(bf16x8_t, v); }

__device__ __forceinline__ f32x16_t mfma32(bf16x8_t a, bf16x8_t b, f32x16_t c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

// Global -> register prefetch of one 64-wide K step of the forward GEMM:
// A = weight rows (16-byte chunk q of each of A_CH rows), B = im2col rows
// (the pixel's neighbour at this step's tap, zero outside the image).
template <int A_CH, int B_CH, int TAPS>
__device__ __forceinline__ void fwd_gload(u32x4 (&ra)[A_CH], u32x4 (&rb)[B_CH], int ks, int cpt,
                                          int Cin, int K, int W, int H,
                                          const bf16_t* __restrict__ wbase,
                                          const bf16_t* __restrict__ xbase,
                                          const int (&ph)[B_CH], const int (&pw)[B_CH],
                                          const bool (&pok)[B_CH]) {
  const int tap = ks / cpt;
  const int c0 = (ks - tap * cpt) * 64;
  const int dr = (TAPS == 9) ? tap / 3 - 1 : 0;
  const int dc = (TAPS == 9) ? tap % 3 - 1 : 0;
#pragma unroll
  for (int u = 0; u < A_CH; ++u)
    ra[u] = *(const u32x4*)(wbase + (long)32 * u * K + tap * Cin + c0);
  const long shift = ((long)dr * W + dc) * Cin + c0;
#pragma unroll
  for (int u = 0; u < B_CH; ++u) {
    const int hh = ph[u] + dr, ww = pw[u] + dc;
    const bool ok = pok[u] && (unsigned)hh < (unsigned)H && (unsigned)ww < (unsigned)W;
    u32x4 v = u32x4{0, 0, 0, 0};
    if (ok) v = *(const u32x4*)(xbase + (long)32 * u * Cin + shift);
    rb[u] = v;
  }
}

template <int A_CH, int B_CH>
__device__ __forceinline__ void fwd_lstore(const u32x4 (&ra)[A_CH], const u32x4 (&rb)[B_CH],
                                           u32x4* As, u32x4* Bs, int tid, int q) {
#pragma unroll
  for (int u = 0; u < A_CH; ++u) {
    const int row = (tid >> 3) + 32 * u;
    As[row * 8 + swz(row, q)] = ra[u];
  }
#pragma unroll
  for (int u = 0; u < B_CH; ++u) {
    const int row = (tid >> 3) + 32 * u;
    Bs[row * 8 + swz(row, q)] = rb[u];
  }
}

// ---------------------------------------------------------------- forward

// WCO x WP waves; each wave owns TM x TN MFMA tiles of 32 x 32.
template <int WCO, int WP, int TM, int TN, int TAPS>
__global__ __launch_bounds__(256) void conv_fwd_mfma(
    const bf16_t* __restrict__ X, const bf16_t* __restrict__ Wt,
    const float* __restrict__ bias, bf16_t* __restrict__ Y, int P, int H, int W, int Cin,
    int Cout, int relu) {
  static_assert(WCO * WP == 4, "4 waves");
  constexpr int BN = WCO * TM * 32;  // output channels per block
  constexpr int BM = WP * TN * 32;   // pixels per block
  constexpr int BK = 64;
  constexpr int A_CH = BN * 8 / 256;  // 16-byte chunks per thread per K step
  constexpr int B_CH = BM * 8 / 256;
  static_assert(A_CH >= 1 && B_CH >= 1, "tile too small");
  __shared__ u32x4 smem[2][(BN + BM) * 8];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wco = wave / WP, wp = wave % WP;
  const int p0 = blockIdx.x * BM, co0 = blockIdx.y * BN;
  const int K = TAPS * Cin;
  const int cpt = Cin / BK;
  const int nk = TAPS * cpt;
  const int q = tid & 7;
  const int HW = H * W;

  int ph[B_CH], pw[B_CH];
  bool pok[B_CH];
#pragma unroll
  for (int u = 0; u < B_CH; ++u) {
    int p = p0 + (tid >> 3) + 32 * u;
    pok[u] = p < P;
    int pp = pok[u] ? p : 0;
    int rem = pp % HW;
    ph[u] = rem / W;
    pw[u] = rem - ph[u] * W;
  }
  const bf16_t* xbase = X + (long)(p0 + (tid >> 3)) * Cin + q * 8;
  const bf16_t* wbase = Wt + (long)(co0 + (tid >> 3)) * K + q * 8;

  u32x4 ra[A_CH], rb[B_CH];
  f32x16_t acc[TM][TN];
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j) acc[i][j] = f32x16_t{};

  fwd_gload<A_CH, B_CH, TAPS>(ra, rb, 0, cpt, Cin, K, W, H, wbase, xbase, ph, pw, pok);
  fwd_lstore<A_CH, B_CH>(ra, rb, smem[0], smem[0] + BN * 8, tid, q);
  __syncthreads();
  for (int ks = 0; ks < nk; ++ks) {
    const int buf = ks & 1;
    if (ks + 1 < nk)
      fwd_gload<A_CH, B_CH, TAPS>(ra, rb, ks + 1, cpt, Cin, K, W, H, wbase, xbase, ph, pw, pok);
    const u32x4* As = smem[buf];
    const u32x4* Bs = smem[buf] + BN * 8;
#pragma unroll
    for (int kk = 0; kk < BK / 16; ++kk) {
      const int qq = 2 * kk + (lane >> 5);
      bf16x8_t a[TM], b[TN];
#pragma unroll
      for (int i = 0; i < TM; ++i) {
        int row = wco * TM * 32 + i * 32 + (lane & 31);
        a[i] = as_bf16x8(As[row * 8 + swz(row, qq)]);
      }
#pragma unroll
      for (int j = 0; j < TN; ++j) {
        int row = wp * TN * 32 + j * 32 + (lane & 31);
        b[j] = as_bf16x8(Bs[row * 8 + swz(row, qq)]);
      }
#pragma unroll
      for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j) acc[i][j] = mfma32(a[i], b[j], acc[i][j]);
    }
    if (ks + 1 < nk) fwd_lstore<A_CH, B_CH>(ra, rb, smem[buf ^ 1], smem[buf ^ 1] + BN * 8, tid, q);
    __syncthreads();
  }

  // Epilogue: lane holds pixel (lane & 31) of each 32x32 tile and, per group
  // g, four consecutive channels 8g + 4*(lane>>5) + 0..3.
#pragma unroll
  for (int i = 0; i < TM; ++i) {
#pragma unroll
    for (int j = 0; j < TN; ++j) {
      int p = p0 + wp * TN * 32 + j * 32 + (lane & 31);
      if (p >= P) continue;
      bf16_t* yrow = Y + (long)p * Cout;
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        int co = co0 + wco * TM * 32 + i * 32 + 8 * g + 4 * (lane >> 5);
        float v[4];
#pragma unroll
        for (int t = 0; t < 4; ++t) {
          v[t] = acc[i][j][4 * g + t];
          if (bias) v[t] += bias[co + t];
          if (relu) v[t] = fmaxf(v[t], 0.0f);
        }
        uint2 o;
        o.x = f2bf(v[0]) | (f2bf(v[1]) << 16);
        o.y = f2bf(v[2]) | (f2bf(v[3]) << 16);
        *(uint2*)(yrow + co) = o;
      }
    }
  }
}

// ---------------------------------------------------------------- forward (LDS DMA)

// Sixteen zero bytes in device memory: the source of every im2col chunk that
// falls outside the image (the zero padding), so that all tile loads can be
// direct global -> LDS copies.
__device__ __attribute__((aligned(16))) unsigned int g_zero16[4];

#define TGP_LDS(p) ((__attribute__((address_space(3))) void*)(p))

// s_waitcnt with only the vector-memory counter limited to N (gfx9 encoding:
// vmcnt in bits 3:0 and 15:14; expcnt and lgkmcnt left at their maxima).
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | 0x70 | 0xF00);
}

// Waits until at most `ahead` stages of LPS loads each are still in flight.
template <int NS, int LPS>
__device__ __forceinline__ void wait_stages(int ahead) {
  if constexpr (NS >= 4) {
    if (ahead >= 2) { wait_vmcnt<2 * LPS>(); return; }
  }
  if constexpr (NS >= 3) {
    if (ahead >= 1) { wait_vmcnt<LPS>(); return; }
  }
  wait_vmcnt<0>();
}

// Implicit-GEMM forward with an NS-stage ring of LDS tiles filled by
// global_load_lds_dwordx4: each wave instruction copies 8 rows of 128 bytes;
// lane l fills physical chunk l & 7 of row l >> 3 with the logical chunk that
// the XOR swizzle puts there.  Loads run NS - 1 K steps ahead of the MFMAs.
// Block index remapped so that consecutive pixel tiles (which share halo
// rows and read the same weights) run on the same XCD: the dispatcher deals
// blocks round-robin over the 8 XCDs, each with its own L2.
__device__ __forceinline__ int xcd_remap(int bid, int nb) {
  const int per = nb / 8, rem = nb % 8;
  const int x = bid % 8, i = bid / 8;
  return x < rem ? x * (per + 1) + i : rem * (per + 1) + (x - rem) * per + i;
}

template <int WCO, int WP, int TM, int TN, int TAPS, int NS>
__global__ __launch_bounds__(WCO * WP * 64) void conv_fwd_dma(
    const bf16_t* __restrict__ X, const bf16_t* __restrict__ Wt,
    const float* __restrict__ bias, bf16_t* __restrict__ Y, int P, int H, int W, int Cin,
    int Cout, int relu, int co_major) {
  constexpr int NW = WCO * WP;       // waves per block
  constexpr int BN = WCO * TM * 32;  // output channels per block
  constexpr int BM = WP * TN * 32;   // pixels per block
  constexpr int ROWS = BN + BM;
  constexpr int LPS = ROWS / (8 * NW);  // DMA instructions per wave per stage
  static_assert(BN % 64 == 0 && ROWS % (8 * NW) == 0, "tile shape");
  __shared__ u32x4 smem[NS][ROWS * 8];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wco = wave / WP, wp = wave % WP;
  // The grid is (pixel tiles x channel tiles) flattened.  Each XCD gets a
  // contiguous range of it: pixel-tile-major when the activations are the
  // larger operand (an XCD then holds a slice of the image plus all weights
  // in its L2), channel-tile-major when the weights are (a slice of the
  // weights plus the whole activation tile set).
  const int nct = Cout / BN;
  const int npt = gridDim.x / nct;
  const int lb = xcd_remap(blockIdx.x, gridDim.x);
  const int p0 = (co_major ? lb % npt : lb / nct) * BM;
  const int co0 = (co_major ? lb / npt : lb % nct) * BN;
  const int K = TAPS * Cin;
  const int cpt = Cin / 64;
  const int nk = TAPS * cpt;
  const int HW = H * W;

  // Source of each row this lane fills, per stage instruction u.
  const bf16_t* src[LPS];
  int ph[LPS], pw[LPS];
  bool pok[LPS];
#pragma unroll
  for (int u = 0; u < LPS; ++u) {
    const int r = (wave + NW * u) * 8 + (lane >> 3);
    const int c = (lane & 7) ^ ((r ^ (r >> 3)) & 7);
    if ((wave + NW * u) * 8 < BN) {
      src[u] = Wt + (long)(co0 + r) * K + c * 8;
      ph[u] = pw[u] = 0;
      pok[u] = true;
    } else {
      const int p = p0 + r - BN;
      pok[u] = p < P;
      const int pp = pok[u] ? p : 0;
      const int rem = pp % HW;
      ph[u] = rem / W;
      pw[u] = rem - ph[u] * W;
      src[u] = X + (long)pp * Cin + c * 8;
    }
  }
  const bf16_t* zero = (const bf16_t*)g_zero16;

  auto issue = [&](int ks, int slot) __attribute__((always_inline)) {
    const int tap = ks / cpt;
    const int c0 = (ks - tap * cpt) * 64;
    const int dr = (TAPS == 9) ? tap / 3 - 1 : 0;
    const int dc = (TAPS == 9) ? tap % 3 - 1 : 0;
    const long shift = ((long)dr * W + dc) * Cin + c0;
#pragma unroll
    for (int u = 0; u < LPS; ++u) {
      const bf16_t* g;
      if ((wave + NW * u) * 8 < BN) {
        g = src[u] + tap * Cin + c0;
      } else {
        const int hh = ph[u] + dr, ww = pw[u] + dc;
        const bool ok = pok[u] && (unsigned)hh < (unsigned)H && (unsigned)ww < (unsigned)W;
        g = ok ? src[u] + shift : zero;
      }
      __builtin_amdgcn_global_load_lds((const void*)g,
                                       TGP_LDS(&smem[slot][(wave + NW * u) * 64]), 16, 0, 0);
    }
  };

  f32x16_t acc[TM][TN];
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j) acc[i][j] = f32x16_t{};

#pragma unroll
  for (int s = 0; s < NS - 1; ++s)
    if (s < nk) issue(s, s);
  for (int ks = 0; ks < nk; ++ks) {
    const int ahead = min(NS - 2, nk - 1 - ks);
    wait_stages<NS, LPS>(ahead);
    __builtin_amdgcn_s_barrier();
    if (ks + NS - 1 < nk) issue(ks + NS - 1, (ks + NS - 1) % NS);
    const u32x4* As = smem[ks % NS];
    const u32x4* Bs = smem[ks % NS] + BN * 8;
    // the fragments of K sub-step kk + 1 are read while the MFMAs of kk run
    bf16x8_t a[2][TM], b[2][TN];
    auto load = [&](int kk, int buf) __attribute__((always_inline)) {
      const int qq = 2 * kk + (lane >> 5);
#pragma unroll
      for (int i = 0; i < TM; ++i) {
        const int row = wco * TM * 32 + i * 32 + (lane & 31);
        a[buf][i] = as_bf16x8(As[row * 8 + swz(row, qq)]);
      }
#pragma unroll
      for (int j = 0; j < TN; ++j) {
        const int row = wp * TN * 32 + j * 32 + (lane & 31);
        b[buf][j] = as_bf16x8(Bs[row * 8 + swz(row, qq)]);
      }
    };
    load(0, 0);
#pragma unroll
    for (int kk = 0; kk < 4; ++kk) {
      if (kk + 1 < 4) load(kk + 1, (kk + 1) & 1);
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j) acc[i][j] = mfma32(a[kk & 1][i], b[kk & 1][j], acc[i][j]);
      __builtin_amdgcn_sched_barrier(0);
    }
  }

#pragma unroll
  for (int i = 0; i < TM; ++i) {
#pragma unroll
    for (int j = 0; j < TN; ++j) {
      const int p = p0 + wp * TN * 32 + j * 32 + (lane & 31);
      if (p >= P) continue;
      bf16_t* yrow = Y + (long)p * Cout;
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        const int co = co0 + wco * TM * 32 + i * 32 + 8 * g + 4 * (lane >> 5);
        float v[4];
#pragma unroll
        for (int t = 0; t < 4; ++t) {
          v[t] = acc[i][j][4 * g + t];
          if (bias) v[t] += bias[co + t];
          if (relu) v[t] = fmaxf(v[t], 0.0f);
        }
        uint2 o;
        o.x = f2bf(v[0]) | (f2bf(v[1]) << 16);
        o.y = f2bf(v[2]) | (f2bf(v[3]) << 16);
        *(uint2*)(yrow + co) = o;
      }
    }
  }
}

// ---------------------------------------------------------------- forward, row-stage 3x3

// 3x3 implicit GEMM whose K loop runs over stages (64-channel chunk c, filter
// row r).  A stage holds, for a block of BM consecutive output pixels
// [p0, p0 + BM), the BM + 2 input pixel rows q = p0 + (r-1) W - 1 + j
// (j = 0 .. BM+1) and the weights of the three taps (r, 0..2); the three
// column taps then read the pixel rows at offsets 0, 1, 2 from LDS, so each
// input row is fetched once per filter row instead of once per tap.  A B
// fragment whose source pixel (h + r - 1, w + s - 1) lies outside the image
// is zeroed after the LDS read (that covers the left / right padding and the
// rows that belong to the neighbouring sample).  K order (chunk, r, s,
// channel) is fixed by the shape, so recomputation is bit-identical.
//
// SPLIT: the stages are divided over gridDim.x / tiles splits; each split
// writes fp32 partials part[split][p][co] and conv_rows_epilogue sums them
// in split order and applies bias, ReLU and the bf16 rounding.
template <int WCO, int WP, int TM, int TN, int NS, bool SPLIT>
__global__ __launch_bounds__(WCO * WP * 64) void conv_fwd_rows(
    const bf16_t* __restrict__ X, const bf16_t* __restrict__ Wt,
    const float* __restrict__ bias, bf16_t* __restrict__ Y, float* __restrict__ part, int P,
    int H, int W, int Cin, int Cout, int relu, int co_major, int tiles, int st_per_split) {
  constexpr int NW = WCO * WP;
  constexpr int BN = WCO * TM * 32;
  constexpr int BM = WP * TN * 32;
  constexpr int RA = 3 * BN;                               // weight rows per stage
  constexpr int ROWS = (RA + BM + 2 + 8 * NW - 1) / (8 * NW) * (8 * NW);
  constexpr int LPS = ROWS / (8 * NW);                     // DMA instructions per wave per stage
  static_assert(BN % 64 == 0, "weight rows must keep the swizzle phase");
  __shared__ u32x4 smem[NS][ROWS * 8];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wco = wave / WP, wp = wave % WP;
  const int nct = Cout / BN;
  const int npt = tiles / nct;
  int lb = xcd_remap(blockIdx.x, gridDim.x);
  const int split = lb / tiles;
  lb -= split * tiles;
  const int p0 = (co_major ? lb % npt : lb / nct) * BM;
  const int co0 = (co_major ? lb / npt : lb % nct) * BN;
  const int nst = 3 * (Cin / 64);
  const int s_begin = SPLIT ? split * st_per_split : 0;
  const int s_end = SPLIT ? min(nst, s_begin + st_per_split) : nst;
  const int HW = H * W;

  // DMA sources: row rr of the stage (A: weight row of tap (r, rr / BN),
  // B: input pixel row rr - RA); logical chunk from the swizzle.
  const bf16_t* abase[LPS];
  int brow[LPS];
#pragma unroll
  for (int u = 0; u < LPS; ++u) {
    const int r = (wave + NW * u) * 8 + (lane >> 3);
    const int c = (lane & 7) ^ ((r ^ (r >> 3)) & 7);
    if ((wave + NW * u) * 8 < RA) {
      const int t3 = r / BN, co = co0 + r % BN;
      abase[u] = Wt + ((long)co * 9 + t3) * Cin + c * 8;   // + 3 * rfilt * Cin + c0
      brow[u] = 0;
    } else {
      abase[u] = X + c * 8;
      brow[u] = r - RA;                                   // j
    }
  }
  const bf16_t* zero = (const bf16_t*)g_zero16;

  // Validity of the B fragment of tile j for filter row rf, column tap t3.
  unsigned vmask[TN];
#pragma unroll
  for (int j = 0; j < TN; ++j) {
    const int p = p0 + wp * TN * 32 + j * 32 + (lane & 31);
    unsigned m = 0;
    if (p < P) {
      const int rem = p % HW, h = rem / W, w = rem - (rem / W) * W;
#pragma unroll
      for (int rf = 0; rf < 3; ++rf)
#pragma unroll
        for (int t3 = 0; t3 < 3; ++t3)
          if ((unsigned)(h + rf - 1) < (unsigned)H && (unsigned)(w + t3 - 1) < (unsigned)W)
            m |= 1u << (rf * 3 + t3);
    }
    vmask[j] = m;
  }

  auto issue = [&](int st, int slot) __attribute__((always_inline)) {
    const int chunk = st / 3, rf = st - chunk * 3;
    const int c0 = chunk * 64;
    const long qbase = (long)p0 + (long)(rf - 1) * W - 1;
#pragma unroll
    for (int u = 0; u < LPS; ++u) {
      const bf16_t* g;
      if ((wave + NW * u) * 8 < RA) {
        g = abase[u] + (long)rf * 3 * Cin + c0;
      } else {
        const long q = qbase + brow[u];
        const bool ok = brow[u] < BM + 2 && q >= 0 && q < P;
        g = ok ? abase[u] + q * Cin + c0 : zero;
      }
      __builtin_amdgcn_global_load_lds((const void*)g,
                                       TGP_LDS(&smem[slot][(wave + NW * u) * 64]), 16, 0, 0);
    }
  };

  f32x16_t acc[TM][TN];
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j) acc[i][j] = f32x16_t{};

  const int n = s_end - s_begin;
#pragma unroll
  for (int k = 0; k < NS - 1; ++k)
    if (k < n) issue(s_begin + k, k);
  for (int k = 0; k < n; ++k) {
    const int ahead = min(NS - 2, n - 1 - k);
    wait_stages<NS, LPS>(ahead);
    __builtin_amdgcn_s_barrier();
    if (k + NS - 1 < n) issue(s_begin + k + NS - 1, (k + NS - 1) % NS);
    const int st = s_begin + k;
    const int rf = st % 3;
    const u32x4* As = smem[k % NS];
    const u32x4* Bs = smem[k % NS] + RA * 8;
    // 12 steps (3 column taps x 4 K sub-steps); the fragments of step t + 1
    // are read from LDS while the MFMAs of step t run.
    bf16x8_t fa[2][TM];
    u32x4 fb[2][TN];
    auto load = [&](int t, int buf) __attribute__((always_inline)) {
      const int t3 = t >> 2, kk = t & 3;
      const int qq = 2 * kk + (lane >> 5);
#pragma unroll
      for (int i = 0; i < TM; ++i) {
        const int row = t3 * BN + wco * TM * 32 + i * 32 + (lane & 31);
        fa[buf][i] = as_bf16x8(As[row * 8 + swz(row, qq)]);
      }
#pragma unroll
      for (int j = 0; j < TN; ++j) {
        const int row = wp * TN * 32 + j * 32 + (lane & 31) + t3;
        fb[buf][j] = Bs[row * 8 + swz(row, qq)];
      }
    };
    load(0, 0);
#pragma unroll
    for (int t = 0; t < 12; ++t) {
      const int cur = t & 1;
      // the B rows of a column tap that falls outside the image are zeroed
      // here, at use, so that the wait for the LDS read sits after the
      // previous step's MFMAs
      bf16x8_t bm[TN];
#pragma unroll
      for (int j = 0; j < TN; ++j) {
        const bool ok = (vmask[j] >> (rf * 3 + (t >> 2))) & 1u;
        bm[j] = as_bf16x8(ok ? fb[cur][j] : u32x4{0, 0, 0, 0});
      }
      if (t + 1 < 12) load(t + 1, cur ^ 1);
      // fence: the reads above are issued before the MFMAs below, which
      // then cover their latency
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j) acc[i][j] = mfma32(fa[cur][i], bm[j], acc[i][j]);
      __builtin_amdgcn_sched_barrier(0);
    }
  }

#pragma unroll
  for (int i = 0; i < TM; ++i) {
#pragma unroll
    for (int j = 0; j < TN; ++j) {
      const int p = p0 + wp * TN * 32 + j * 32 + (lane & 31);
      if (p >= P) continue;
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        const int co = co0 + wco * TM * 32 + i * 32 + 8 * g + 4 * (lane >> 5);
        if constexpr (SPLIT) {
          float4 o = make_float4(acc[i][j][4 * g], acc[i][j][4 * g + 1], acc[i][j][4 * g + 2],
                                 acc[i][j][4 * g + 3]);
          *(float4*)(part + ((long)split * P + p) * Cout + co) = o;
        } else {
          float v[4];
#pragma unroll
          for (int t = 0; t < 4; ++t) {
            v[t] = acc[i][j][4 * g + t];
            if (bias) v[t] += bias[co + t];
            if (relu) v[t] = fmaxf(v[t], 0.0f);
          }
          uint2 o;
          o.x = f2bf(v[0]) | (f2bf(v[1]) << 16);
          o.y = f2bf(v[2]) | (f2bf(v[3]) << 16);
          *(uint2*)(Y + (long)p * Cout + co) = o;
        }
      }
    }
  }
}

// y[p][co] = bf16(act(sum_{s < S} part[s][p][co] + b[co])), s ascending.
__global__ __launch_bounds__(256) void conv_rows_epilogue(const float* __restrict__ part,
                                                          const float* __restrict__ bias,
                                                          bf16_t* __restrict__ Y, long P,
                                                          int Cout, int S, int relu) {
  const long e = ((long)blockIdx.x * 256 + threadIdx.x) * 8;
  const long n = P * Cout;
  if (e >= n) return;
  float v[8];
  const float4 a0 = *(const float4*)(part + e), a1 = *(const float4*)(part + e + 4);
  v[0] = a0.x; v[1] = a0.y; v[2] = a0.z; v[3] = a0.w;
  v[4] = a1.x; v[5] = a1.y; v[6] = a1.z; v[7] = a1.w;
  for (int s = 1; s < S; ++s) {
    const float4 b0 = *(const float4*)(part + (long)s * n + e);
    const float4 b1 = *(const float4*)(part + (long)s * n + e + 4);
    v[0] += b0.x; v[1] += b0.y; v[2] += b0.z; v[3] += b0.w;
    v[4] += b1.x; v[5] += b1.y; v[6] += b1.z; v[7] += b1.w;
  }
  const int co = e % Cout;
  u32x4 o;
#pragma unroll
  for (int t = 0; t < 8; t += 2) {
    float x0 = v[t], x1 = v[t + 1];
    if (bias) { x0 += bias[co + t]; x1 += bias[co + t + 1]; }
    if (relu) { x0 = fmaxf(x0, 0.f); x1 = fmaxf(x1, 0.f); }
    o[t / 2] = f2bf(x0) | (f2bf(x1) << 16);
  }
  *(u32x4*)(Y + e) = o;
}

// ---------------------------------------------------------------- wgrad

// 8x8 transpose of bfloat16: in[j] holds 8 channels of pixel j; out[c] gets
// 8 pixels of channel c.
__device__ __forceinline__ void transpose8x8(const u32x4 (&in)[8], u32x4 (&out)[8]) {
#pragma unroll
  for (int c = 0; c < 8; ++c) {
    uint32_t d[4];
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      uint32_t lo = in[2 * e][c >> 1];
      uint32_t hi = in[2 * e + 1][c >> 1];
      d[e] = (c & 1) ? ((lo >> 16) | (hi & 0xffff0000u)) : ((lo & 0xffffu) | (hi << 16));
    }
    out[c] = u32x4{d[0], d[1], d[2], d[3]};
  }
}

template <int WM, int WN, int TM, int TN, int TAPS>
__global__ __launch_bounds__(256) void conv_wgrad_mfma(
    const bf16_t* __restrict__ X, const bf16_t* __restrict__ dZ, float* __restrict__ part,
    int P, int H, int W, int Cin, int Cout, int pix_per_split) {
  static_assert(WM * WN == 4, "4 waves");
  constexpr int BMc = WM * TM * 32;  // output channels (co) per block
  constexpr int BNc = WN * TN * 32;  // input channels (ci) per block
  constexpr int BK = 64;             // pixels per K step
  static_assert(BMc + BNc <= 256, "one 8x8 block per thread");
  __shared__ u32x4 smem[2][(BMc + BNc) * 8];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave / WN, wn = wave % WN;
  const int ncb = Cin / BNc;
  const int tap = blockIdx.x / ncb;
  const int ci0 = (blockIdx.x - tap * ncb) * BNc;
  const int co0 = blockIdx.y * BMc;
  const int split = blockIdx.z;
  const int ps = split * pix_per_split;
  const int pe = min(P, ps + pix_per_split);
  const int nk = (pe - ps + BK - 1) / BK;
  const int dr = (TAPS == 9) ? tap / 3 - 1 : 0;
  const int dc = (TAPS == 9) ? tap % 3 - 1 : 0;

  // Load role: threads [0, BMc) load dZ blocks, [BMc, BMc+BNc) load X blocks.
  const bool isA = tid < BMc;
  const bool active = tid < BMc + BNc;
  const int t2 = isA ? tid : tid - BMc;
  const int nchunk = isA ? BMc / 8 : BNc / 8;
  const int cc = t2 % nchunk;      // 8-channel chunk
  const int pc = t2 / nchunk;      // 8-pixel chunk within the K step (0..7)

  u32x4 v[8];
  auto gload = [&](int ks) {
    int pbase = ps + ks * BK + pc * 8;
    if (!active) return;
    if (isA) {
      const bf16_t* src = dZ + (long)pbase * Cout + co0 + cc * 8;
#pragma unroll
      for (int j = 0; j < 8; ++j)
        v[j] = (pbase + j < pe) ? *(const u32x4*)(src + (long)j * Cout) : u32x4{0, 0, 0, 0};
    } else {
      int HW = H * W;
      int pp = pbase < P ? pbase : 0;
      int rem = pp % HW;
      int h = rem / W, w = rem - h * W;
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        int hh = h + dr, ww = w + dc;
        bool ok = (pbase + j < pe) && (unsigned)hh < (unsigned)H && (unsigned)ww < (unsigned)W;
        v[j] = ok ? *(const u32x4*)(X + ((long)(pbase + j) + (long)dr * W + dc) * Cin + ci0 + cc * 8)
                  : u32x4{0, 0, 0, 0};
        if (++w == W) { w = 0; if (++h == H) h = 0; }
      }
    }
  };
  auto lstore = [&](int buf) {
    if (!active) return;
    u32x4 o[8];
    transpose8x8(v, o);
    u32x4* dst = smem[buf] + (isA ? 0 : BMc * 8);
#pragma unroll
    for (int c = 0; c < 8; ++c) {
      int row = cc * 8 + c;
      dst[row * 8 + swz(row, pc)] = o[c];
    }
  };

  f32x16_t acc[TM][TN];
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j) acc[i][j] = f32x16_t{};

  if (nk > 0) {
    gload(0);
    lstore(0);
  }
  __syncthreads();
  for (int ks = 0; ks < nk; ++ks) {
    const int buf = ks & 1;
    if (ks + 1 < nk) gload(ks + 1);
    const u32x4* As = smem[buf];
    const u32x4* Bs = smem[buf] + BMc * 8;
    // the fragments of K sub-step kk + 1 are read while the MFMAs of kk run
    bf16x8_t a[2][TM], b[2][TN];
    auto load = [&](int kk, int fb) __attribute__((always_inline)) {
      const int qq = 2 * kk + (lane >> 5);
#pragma unroll
      for (int i = 0; i < TM; ++i) {
        const int row = wm * TM * 32 + i * 32 + (lane & 31);
        a[fb][i] = as_bf16x8(As[row * 8 + swz(row, qq)]);
      }
#pragma unroll
      for (int j = 0; j < TN; ++j) {
        const int row = wn * TN * 32 + j * 32 + (lane & 31);
        b[fb][j] = as_bf16x8(Bs[row * 8 + swz(row, qq)]);
      }
    };
    load(0, 0);
#pragma unroll
    for (int kk = 0; kk < BK / 16; ++kk) {
      if (kk + 1 < BK / 16) load(kk + 1, (kk + 1) & 1);
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j) acc[i][j] = mfma32(a[kk & 1][i], b[kk & 1][j], acc[i][j]);
      __builtin_amdgcn_sched_barrier(0);
    }
    if (ks + 1 < nk) lstore(buf ^ 1);
    __syncthreads();
  }

  float* out = part + (long)split * Cout * TAPS * Cin;
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j) {
      int ci = ci0 + wn * TN * 32 + j * 32 + (lane & 31);
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        int co = co0 + wm * TM * 32 + i * 32 + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
        out[((long)co * TAPS + tap) * Cin + ci] = acc[i][j][r];
      }
    }
}

// dw[e] = sum_{s < S} part[s][e] in a fixed order: split-lane l of a block
// sums s = l, l + 16, l + 32, ... serially, then lanes 0..15 are added in
// order.  Each block covers 16 float4 columns (64 elements).
__global__ __launch_bounds__(256) void splitk_reduce(const float* __restrict__ part,
                                                     float* __restrict__ dw, long E, int S) {
  __shared__ float4 red[16][16];
  const int col = threadIdx.x & 15, lane = threadIdx.x >> 4;
  const long e4 = ((long)blockIdx.x * 16 + col) * 4;
  const bool vec = (E & 3) == 0;
  float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
  if (e4 < E) {
    for (int k = lane; k < S; k += 16) {
      const float* p = part + (long)k * E + e4;
      if (vec) {
        float4 t = *(const float4*)p;
        acc.x += t.x; acc.y += t.y; acc.z += t.z; acc.w += t.w;
      } else {
        acc.x += p[0];
        if (e4 + 1 < E) acc.y += p[1];
        if (e4 + 2 < E) acc.z += p[2];
        if (e4 + 3 < E) acc.w += p[3];
      }
    }
  }
  red[lane][col] = acc;
  __syncthreads();
  if (lane == 0 && e4 < E) {
    float4 s = red[0][col];
    for (int l = 1; l < 16; ++l) {
      float4 t = red[l][col];
      s.x += t.x; s.y += t.y; s.z += t.z; s.w += t.w;
    }
    if (vec) {
      *(float4*)(dw + e4) = s;
    } else {
      dw[e4] = s.x;
      if (e4 + 1 < E) dw[e4 + 1] = s.y;
      if (e4 + 2 < E) dw[e4 + 2] = s.z;
      if (e4 + 3 < E) dw[e4 + 3] = s.w;
    }
  }
}

// wt[ci][tap'][co] = w[co][taps-1-tap'][ci]: the data gradient of a
// cross-correlation is a cross-correlation with the 180-degree rotated,
// channel-transposed filter.
template <typename T>
__global__ void wtransform_kernel(const T* __restrict__ w, T* __restrict__ wt, int cout, int cin,
                                  int taps) {
  long e = (long)blockIdx.x * 256 + threadIdx.x;
  long n = (long)cout * cin * taps;
  if (e >= n) return;
  int co = e % cout;
  long r = e / cout;
  int tp = r % taps;
  int ci = r / taps;
  wt[e] = w[((long)co * taps + (taps - 1 - tp)) * cin + ci];
}

struct WgradPlan {
  int S, pix_per_split;
};

// Split count for the weight gradient: enough blocks to fill the chip
// (~512), at least 256 pixels per split, and at most ~8 MB of fp32 partials
// (their write + fixed-order re-read otherwise costs more than the extra
// parallelism gains).
template <int TM, int TN>
WgradPlan wgrad_plan(long P, int tiles, long E) {
  const int BK = 64;
  int S = cdiv(512, tiles);
  int maxS = cdiv(P, 256);
  if (S > maxS) S = maxS;
  long cap = (8L << 20) / (4 * E);
  if (S > cap) S = (int)cap;
  if (S < 1) S = 1;
  int pps = cdiv(cdiv(P, S), BK) * BK;
  S = cdiv(P, pps);
  return {S, pps};
}

}  // namespace

// ---------------------------------------------------------------- dispatch

hipError_t splitk_reduce_launch(const float* part, float* out, long E, int S, hipStream_t st);

bool mfma_conv_ok(int dt, int cin, int cout) {
  return dt == 0 && cin % 64 == 0 && cout % 64 == 0;
}

// Forward tile configurations.  A configuration is chosen per shape by
// fwd_config() (a pure function of the shape, so recomputation reuses the
// exact same kernel); g_fwd_variant > 0 forces one for measurement sweeps.
int g_fwd_variant = 0;
int g_fwd_order = -1;   // -1: by operand size; 0/1 forced (measurement only)

template <int WCO, int WP, int TM, int TN, int NS>
hipError_t launch_fwd_dma(const char* name, const bf16_t* X, const bf16_t* Wt, const float* b,
                          bf16_t* Y, long P, const ConvShape& s, int relu, hipStream_t st) {
  constexpr int BN = WCO * TM * 32, BM = WP * TN * 32;
  if (s.cout % BN) return hipErrorInvalidValue;
  dim3 grid(cdiv(P, BM) * (s.cout / BN));
  double flops = 2.0 * P * s.cout * s.taps * s.cin;
  double bytes = 2.0 * ((double)P * s.cin + (double)s.cout * s.taps * s.cin + (double)P * s.cout);
  ProfScope ps(name, flops, bytes, st);
  const double xbytes = 2.0 * P * s.cin, wbytes = 2.0 * s.cout * s.taps * s.cin;
  const int co_major = g_fwd_order >= 0 ? g_fwd_order : (wbytes > xbytes ? 1 : 0);
  if (s.taps == 9)
    hipLaunchKernelGGL((conv_fwd_dma<WCO, WP, TM, TN, 9, NS>), grid, dim3(WCO * WP * 64), 0, st, X,
                       Wt, b, Y, (int)P, s.H, s.W, s.cin, s.cout, relu, co_major);
  else
    hipLaunchKernelGGL((conv_fwd_dma<WCO, WP, TM, TN, 1, NS>), grid, dim3(WCO * WP * 64), 0, st, X,
                       Wt, b, Y, (int)P, s.H, s.W, s.cin, s.cout, relu, co_major);
  return hipGetLastError();
}

#define TGP_FWD_CFG(WCO, WP, TM, TN, NS) \
  launch_fwd_dma<WCO, WP, TM, TN, NS>("conv_fwd_dma<" #WCO "," #WP "," #TM "," #TN "," #NS ">", X, Wt, b, Y, P, s, relu, st)

// Row-stage forward launches.  S > 1 splits the stages over S blocks per
// tile; the partials live in `part` (capacity part_cap floats; S is reduced
// to fit, which only happens under measurement overrides).
template <int WCO, int WP, int TM, int TN, int NS>
hipError_t launch_fwd_rows(const char* name, const bf16_t* X, const bf16_t* Wt, const float* b,
                           bf16_t* Y, float* part, size_t part_cap, long P, const ConvShape& s,
                           int relu, int S, hipStream_t st) {
  constexpr int BN = WCO * TM * 32, BM = WP * TN * 32;
  if (s.cout % BN || s.cin % 64 || s.taps != 9) return hipErrorInvalidValue;
  const int tiles = cdiv(P, BM) * (s.cout / BN);
  const int nst = 3 * (s.cin / 64);
  if (S > nst) S = nst;
  while (S > 1 && (size_t)S * P * s.cout > part_cap) --S;
  const int sps = cdiv(nst, S > 1 ? S : 1);
  S = cdiv(nst, sps);
  const double flops = 2.0 * P * s.cout * 9 * s.cin;
  const double xbytes = 2.0 * P * s.cin, wbytes = 2.0 * s.cout * 9 * s.cin;
  const int co_major = g_fwd_order >= 0 ? g_fwd_order : (wbytes > xbytes ? 1 : 0);
  dim3 grid(tiles * S), block(WCO * WP * 64);
  if (S == 1) {
    ProfScope ps(name, flops, xbytes + wbytes + 2.0 * P * s.cout, st);
    hipLaunchKernelGGL((conv_fwd_rows<WCO, WP, TM, TN, NS, false>), grid, block, 0, st, X, Wt, b,
                       Y, part, (int)P, s.H, s.W, s.cin, s.cout, relu, co_major, tiles, sps);
    return hipGetLastError();
  }
  {
    ProfScope ps(name, flops, xbytes + wbytes + 4.0 * S * P * s.cout, st);
    hipLaunchKernelGGL((conv_fwd_rows<WCO, WP, TM, TN, NS, true>), grid, block, 0, st, X, Wt, b,
                       Y, part, (int)P, s.H, s.W, s.cin, s.cout, relu, co_major, tiles, sps);
  }
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  ProfScope ps2("conv_rows_epilogue", 0.0, 4.0 * S * P * s.cout + 2.0 * P * s.cout, st);
  hipLaunchKernelGGL(conv_rows_epilogue, dim3(cdiv(P * s.cout, 2048)), dim3(256), 0, st, part, b,
                     Y, P, s.cout, S, relu);
  return hipGetLastError();
}

#define TGP_ROWS_CFG(WCO, WP, TM, TN, NS, S)                                               \
  launch_fwd_rows<WCO, WP, TM, TN, NS>("conv_fwd_rows<" #WCO "," #WP "," #TM "," #TN "," #NS ">", \
                                       X, Wt, b, Y, part, part_cap, P, s, relu, S, st)

int g_fwd_split = 0;   // > 0 forces the split count (measurement only)

struct FwdPlan {
  int cfg;   // 1..: row-stage configurations; 100+: per-tap configurations
  int S;
};

// Pure function of the shape (plus the measurement overrides).
FwdPlan fwd_plan(const ConvShape& s) {
  const long P = s.pixels();
  FwdPlan pl{0, 1};
  // Row-stage tiles pay off only on the deep, small-image layers (few pixel
  // tiles, long K); elsewhere the per-tap kernel keeps more blocks per CU.
  if (s.taps == 9 && s.cin % 64 == 0 && s.cin >= 256 && P <= 4096) {
    pl.cfg = 3;    // 64 x 256, 8 waves
  } else {
    pl.cfg = 100;
  }
  if (g_fwd_variant > 0) pl.cfg = g_fwd_variant;
  if ((pl.cfg == 2 || pl.cfg == 5) && s.cout % 128) pl.cfg = pl.cfg == 2 ? 1 : 3;  // 128-wide tiles need cout % 128 == 0
  if (pl.cfg < 100) {
    const int BN = (pl.cfg == 2 || pl.cfg == 5) ? 128 : 64;
    const int BM = (pl.cfg == 2 || pl.cfg == 5 || pl.cfg == 6 || pl.cfg == 7) ? 128 : 256;
    const long tiles = cdiv(P, BM) * (s.cout / BN);
    const int nst = 3 * (s.cin / 64);
    int S = tiles > 0 ? (int)cdiv(512, tiles) : 1;
    if (S > nst / 3) S = nst / 3 > 0 ? nst / 3 : 1;   // at least one channel chunk per split
    if (S < 1) S = 1;
    pl.S = g_fwd_split > 0 ? g_fwd_split : S;
  }
  return pl;
}

size_t conv_forward_partial_floats(int dt, const ConvShape& s) {
  if (!mfma_conv_ok(dt, s.cin, s.cout)) return 0;
  FwdPlan pl = fwd_plan(s);
  return pl.cfg < 100 && pl.S > 1 ? (size_t)pl.S * s.pixels() * s.cout : 0;
}

hipError_t conv_forward_mfma(const void* x, const void* w, const float* b, void* y,
                             const ConvShape& s, int relu, float* part, size_t part_cap,
                             hipStream_t st) {
  long P = s.pixels();
  const bf16_t* X = (const bf16_t*)x;
  const bf16_t* Wt = (const bf16_t*)w;
  bf16_t* Y = (bf16_t*)y;
  const FwdPlan pl = fwd_plan(s);
  const bool wide = s.cout % 128 == 0;
  switch (pl.cfg) {
    case 1: return TGP_ROWS_CFG(1, 4, 2, 2, 2, pl.S);                 // 64 x 256, 4 waves
    case 2: return wide ? TGP_ROWS_CFG(2, 2, 2, 2, 2, pl.S)           // 128 x 128, 4 waves
                        : TGP_ROWS_CFG(1, 4, 2, 2, 2, pl.S);
    case 3: return TGP_ROWS_CFG(1, 8, 2, 1, 2, pl.S);                 // 64 x 256, 8 waves
    case 4: return TGP_ROWS_CFG(2, 4, 1, 2, 2, pl.S);                 // 64 x 256, 8 waves
    case 5: return wide ? TGP_ROWS_CFG(2, 4, 2, 1, 2, pl.S)           // 128 x 128, 8 waves
                        : TGP_ROWS_CFG(1, 8, 2, 1, 2, pl.S);
    case 6: return TGP_ROWS_CFG(1, 4, 2, 1, 2, pl.S);                 // 64 x 128, 4 waves
    case 7: return TGP_ROWS_CFG(1, 4, 2, 1, 3, pl.S);                 // 64 x 128, 4 waves, 3 stages
    default: break;
  }
  // per-tap kernel (1x1 convolutions, and reference configurations)
  const int v = pl.cfg >= 100 ? pl.cfg - 100 : 0;
  switch (v) {
    case 1: return TGP_FWD_CFG(2, 2, 1, 1, 2);          // 64 x 64, 4 waves
    case 2: return TGP_FWD_CFG(2, 4, 1, 1, 2);          // 64 x 128, 8 waves
    default: return P >= 32768 && s.cout <= 128 ? TGP_FWD_CFG(2, 4, 1, 1, 2)
                                                 : TGP_FWD_CFG(2, 2, 1, 1, 2);
  }
}

hipError_t weight_transform(int dt, const void* w, void* wt, int cout, int cin, int taps,
                            hipStream_t st) {
  long n = (long)cout * cin * taps;
  ProfScope ps("wtransform", 0.0, 2.0 * n * (dt == 0 ? 2 : 4), st);
  if (dt == 0)
    hipLaunchKernelGGL(wtransform_kernel<bf16_t>, dim3(cdiv(n, 256)), dim3(256), 0, st,
                       (const bf16_t*)w, (bf16_t*)wt, cout, cin, taps);
  else
    hipLaunchKernelGGL(wtransform_kernel<float>, dim3(cdiv(n, 256)), dim3(256), 0, st,
                       (const float*)w, (float*)wt, cout, cin, taps);
  return hipGetLastError();
}

size_t wgrad_mfma_partial_floats(const ConvShape& s) {
  int tiles = s.taps * (s.cin / 64) * (s.cout / 64);
  if (s.cin % 128 == 0 && s.cout % 128 == 0) tiles = s.taps * (s.cin / 128) * (s.cout / 128);
  long E = (long)s.cout * s.taps * s.cin;
  WgradPlan pl = wgrad_plan<2, 2>(s.pixels(), tiles, E);
  return (size_t)pl.S * E;
}

hipError_t conv_wgrad_mfma(const void* x, const void* dz, float* dw, float* partial,
                           const ConvShape& s, hipStream_t st) {
  long P = s.pixels();
  const bf16_t* X = (const bf16_t*)x;
  const bf16_t* DZ = (const bf16_t*)dz;
  bool big = s.cin % 128 == 0 && s.cout % 128 == 0;
  int bm = big ? 128 : 64, bn = big ? 128 : 64;
  int tiles = s.taps * (s.cin / bn) * (s.cout / bm);
  long E = (long)s.cout * s.taps * s.cin;
  WgradPlan pl = wgrad_plan<2, 2>(P, tiles, E);
  dim3 grid(s.taps * (s.cin / bn), s.cout / bm, pl.S);
  double flops = 2.0 * P * E;
  double bytes = 2.0 * ((double)P * s.cin + (double)P * s.cout) + 4.0 * pl.S * E;
  {
    const char* nm = big ? (s.taps == 9 ? "conv_wgrad_mfma<2,2,2,2,9>" : "conv_wgrad_mfma<2,2,2,2,1>")
                         : (s.taps == 9 ? "conv_wgrad_mfma<2,2,1,1,9>" : "conv_wgrad_mfma<2,2,1,1,1>");
    ProfScope ps(nm, flops, bytes, st);
    if (pl.S == 1) partial = dw;   // a single split writes the gradient itself
    if (big) {
      if (s.taps == 9)
        hipLaunchKernelGGL((conv_wgrad_mfma<2, 2, 2, 2, 9>), grid, dim3(256), 0, st, X, DZ,
                           partial, (int)P, s.H, s.W, s.cin, s.cout, pl.pix_per_split);
      else
        hipLaunchKernelGGL((conv_wgrad_mfma<2, 2, 2, 2, 1>), grid, dim3(256), 0, st, X, DZ,
                           partial, (int)P, s.H, s.W, s.cin, s.cout, pl.pix_per_split);
    } else {
      if (s.taps == 9)
        hipLaunchKernelGGL((conv_wgrad_mfma<2, 2, 1, 1, 9>), grid, dim3(256), 0, st, X, DZ,
                           partial, (int)P, s.H, s.W, s.cin, s.cout, pl.pix_per_split);
      else
        hipLaunchKernelGGL((conv_wgrad_mfma<2, 2, 1, 1, 1>), grid, dim3(256), 0, st, X, DZ,
                           partial, (int)P, s.H, s.W, s.cin, s.cout, pl.pix_per_split);
    }
  }
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  return pl.S == 1 ? hipSuccess : splitk_reduce_launch(partial, dw, E, pl.S, st);
}

hipError_t splitk_reduce_launch(const float* part, float* out, long E, int S, hipStream_t st) {
  ProfScope ps("splitk_reduce", 0.0, 4.0 * E * (S + 1), st);
  hipLaunchKernelGGL(splitk_reduce, dim3(cdiv(E, 64)), dim3(256), 0, st, part, out, E, S);
  return hipGetLastError();
}

}  // namespace tgpk
