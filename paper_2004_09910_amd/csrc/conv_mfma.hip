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
#include "mfma_util.h"
#include "prof.h"

namespace tgpk {
namespace {

// XOR swizzle of the eight 16-byte chunks of a 128-byte LDS row, so that
// eight consecutive rows read at the same logical chunk, and rows eight apart
// written at the same chunk, hit distinct banks.
__device__ __forceinline__ int swz(int row, int q) { return q ^ ((row ^ (row >> 3)) & 7); }

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

// Implicit-GEMM forward with an NS-stage ring of LDS tiles filled by
// global_load_lds_dwordx4: each wave instruction copies 8 rows of 128 bytes;
// lane l fills physical chunk l & 7 of row l >> 3 with the logical chunk that
// the XOR swizzle puts there.  Loads run NS - 1 K steps ahead of the MFMAs.
// Block index remapped (xcd_remap) so that consecutive pixel tiles, which
// share halo rows and read the same weights, run on the same XCD.

// X2 / Y2 (both null or both set): a second micro-batch of P pixels; the
// grid then holds both micro-batches' tiles, the second half for it.
template <int WCO, int WP, int TM, int TN, int TAPS, int NS>
__global__ __launch_bounds__(WCO * WP * 64) void conv_fwd_dma(
    const bf16_t* __restrict__ X0, const bf16_t* __restrict__ X2, const bf16_t* __restrict__ Wt,
    const float* __restrict__ bias, bf16_t* __restrict__ Y0, bf16_t* __restrict__ Y2, int P,
    int H, int W, int Cin, int Cout, int relu, int co_major) {
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
  const int per = X2 ? gridDim.x / 2 : gridDim.x;              // blocks per micro-batch
  const int npt = per / nct;
  const int lb0 = xcd_remap(blockIdx.x, gridDim.x);
  const bool g1 = lb0 >= per;                                   // second micro-batch (uniform)
  const int lb = g1 ? lb0 - per : lb0;
  const bf16_t* __restrict__ X = g1 ? X2 : X0;
  bf16_t* __restrict__ Y = g1 ? Y2 : Y0;
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
  // this lane's bias values for the epilogue, loaded up front as 16-byte
  // vectors (channels co0 + wco TM 32 + 32 i + 8 g + 4 (lane / 32) + t);
  // loaded one by one at the epilogue they held up every store
  f32x4_t bv[TM][4];
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int g = 0; g < 4; ++g)
      bv[i][g] = bias ? *(const f32x4_t*)(bias + co0 + wco * TM * 32 + i * 32 + 8 * g +
                                          4 * (lane >> 5))
                      : f32x4_t{};
  for (int ks = 0; ks < nk; ++ks) {
    const int ahead = min(NS - 2, nk - 1 - ks);
    wait_stages<NS, LPS>(ahead);
    ring_barrier();
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

  // Epilogue: lanes l and l + 32 hold channels 8 g + 0..3 and 8 g + 4..7
  // of pixel l % 32.  Swapping the halves of groups 2 h and 2 h + 1 across
  // the two half-waves leaves lane l with channels 16 h + 0..7 and lane
  // l + 32 with 16 h + 8..15, so each lane stores 16 contiguous bytes
  // (scattered 8-byte stores cost a memory-pipeline cycle per lane).
#pragma unroll
  for (int i = 0; i < TM; ++i) {
#pragma unroll
    for (int j = 0; j < TN; ++j) {
      const int p = p0 + wp * TN * 32 + j * 32 + (lane & 31);
      unsigned pk[4][2];
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        float v[4];
#pragma unroll
        for (int t = 0; t < 4; ++t) {
          v[t] = acc[i][j][4 * g + t] + bv[i][g][t];
          if (relu) v[t] = fmaxf(v[t], 0.0f);
        }
        pk[g][0] = f2bf(v[0]) | (f2bf(v[1]) << 16);
        pk[g][1] = f2bf(v[2]) | (f2bf(v[3]) << 16);
      }
#pragma unroll
      for (int h = 0; h < 2; ++h) {
#pragma unroll
        for (int r = 0; r < 2; ++r) {
          const auto sw = __builtin_amdgcn_permlane32_swap(pk[2 * h][r], pk[2 * h + 1][r], false,
                                                           false);
          pk[2 * h][r] = sw[0];
          pk[2 * h + 1][r] = sw[1];
        }
        const int co = co0 + wco * TM * 32 + i * 32 + 16 * h + 8 * (lane >> 5);
        if (p < P)
          *(u32x4*)(Y + (long)p * Cout + co) =
              u32x4{pk[2 * h][0], pk[2 * h][1], pk[2 * h + 1][0], pk[2 * h + 1][1]};
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
  // this lane's bias values for the epilogue, loaded up front (channels
  // co0 + wco TM 32 + 32 i + 8 g + 4 (lane / 32) + t)
  f32x4_t bv[TM][4];
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int g = 0; g < 4; ++g)
      bv[i][g] = (!SPLIT && bias) ? *(const f32x4_t*)(bias + co0 + wco * TM * 32 + i * 32 +
                                                     8 * g + 4 * (lane >> 5))
                                  : f32x4_t{};

  const int n = s_end - s_begin;
#pragma unroll
  for (int k = 0; k < NS - 1; ++k)
    if (k < n) issue(s_begin + k, k);
  for (int k = 0; k < n; ++k) {
    const int ahead = min(NS - 2, n - 1 - k);
    wait_stages<NS, LPS>(ahead);
    ring_barrier();
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
            v[t] = acc[i][j][4 * g + t] + bv[i][g][t];
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

// ---------------------------------------------------------------- 1x1, resident weights

// 1x1 convolution y[p][co] = act(sum_ci x[p][ci] w[co][ci] + b[co]) with
// Cout = 256 and Cin a multiple of 64 up to 256 (the depthwise/pointwise
// cells): a GEMM whose K is short, so a block with a tile of weights has
// little work per byte of weights it loads.  Here each block loads the
// whole weight matrix into LDS once (256 rows of Cin channels, in the
// 64-channel stage blocks and 16-byte-chunk swizzle of conv_fwd_dma) and
// then streams tiles of 64 pixels through an NS-deep ring of 64-channel
// stages.  Wave w computes output channels 32 w .. 32 w + 31 of the tile's
// 64 pixels (two 32 x 32 MFMA tiles), so every pixel row is read once.
// The K order (64-channel stages, 16-channel MFMA steps, increasing
// channel) is conv_fwd_dma's, so both kernels give the same bits.  Blocks
// are persistent over the tiles of all ng micro-batches of the launch (each
// of P pixels, micro-batch k's tiles after those of k - 1).
struct Mb1x1 {
  const bf16_t* x[kMaxGroup];
  bf16_t* y[kMaxGroup];
};
template <int NS>
__global__ __launch_bounds__(512) void conv1x1_res(Mb1x1 io, int ng,
                                                   const bf16_t* __restrict__ Wt,
                                                   const float* __restrict__ bias, int P, int Cin,
                                                   int relu) {
  constexpr int COUT = 256, BM = 64, NW = 8;
  __shared__ u32x4 smem[(4 * COUT + NS * BM) * 8];             // weights, then the ring
  u32x4* const ring = smem + 4 * COUT * 8;

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int nks = Cin / 64;                                     // stages per tile
  const int T1 = (P + BM - 1) / BM;                             // tiles per micro-batch
  const int T = ng * T1;
  const int G = gridDim.x;
  const int lb = xcd_remap(blockIdx.x, G);
  const int n_mine = lb < T ? (T - lb + G - 1) / G : 0;
  const int total = n_mine * nks;

  // DMA: one wave instruction fills 8 rows of 128 bytes; lane l the 16
  // bytes of physical chunk l & 7 of row l >> 3, holding logical chunk c.
  const int rsub = lane >> 3;
  // weights: row R = 256 s + co of stage block s
  for (int u = 0; u < nks * COUT / 8 / NW; ++u) {
    const int R = (wave + NW * u) * 8 + rsub;
    const int sblk = R / COUT, co = R - sblk * COUT;
    const int c = (lane & 7) ^ ((R ^ (R >> 3)) & 7);
    __builtin_amdgcn_global_load_lds((const void*)(Wt + (long)co * Cin + sblk * 64 + c * 8),
                                     TGP_LDS(&smem[(wave + NW * u) * 64]), 16, 0, 0);
  }
  // the X ring: stage idx of this block is tile lb + (idx / nks) G, stage
  // idx % nks; row r = wave * 8 + rsub of the slot is pixel p0 + r
  const int xr = wave * 8 + rsub;
  const int xc = (lane & 7) ^ ((xr ^ (xr >> 3)) & 7);
  auto issue = [&](int idx) __attribute__((always_inline)) {
    const int tt = lb + (idx / nks) * G, ks = idx - (idx / nks) * nks;
    const int gi = tt / T1;                                     // micro-batch (uniform)
    const bf16_t* X = pickg(io.x, gi);
    const int p = min((tt - gi * T1) * BM + xr, P - 1);         // rows past P: any pixel
    __builtin_amdgcn_global_load_lds((const void*)(X + (long)p * Cin + ks * 64 + xc * 8),
                                     TGP_LDS(&ring[(idx % NS) * BM * 8 + wave * 64]), 16, 0, 0);
  };
#pragma unroll
  for (int k = 0; k < NS - 1; ++k)
    if (k < total) issue(k);

  // this lane's bias values (channels 32 wave + 8 g + 4 (lane / 32) + t)
  f32x4_t bv[4];
#pragma unroll
  for (int g = 0; g < 4; ++g)
    bv[g] = bias ? *(const f32x4_t*)(bias + 32 * wave + 8 * g + 4 * (lane >> 5)) : f32x4_t{};

  int idx = 0;
  for (int it = 0; it < n_mine; ++it) {
    const int tt = lb + it * G;
    const int gi = tt / T1;
    bf16_t* __restrict__ Y = pickg(io.y, gi);
    const int p0 = (tt - gi * T1) * BM;
    f32x16_t acc[2] = {f32x16_t{}, f32x16_t{}};
    for (int ks = 0; ks < nks; ++ks, ++idx) {
      // loads complete in order (the weights first); epilogue stores only
      // lengthen this wait
      wait_stages<NS, 1>(min(NS - 2, total - 1 - idx));
      ring_barrier();
      if (idx + NS - 1 < total) issue(idx + NS - 1);
      const u32x4* As = smem + ks * COUT * 8;
      const u32x4* Bs = ring + (idx % NS) * BM * 8;
      bf16x8_t a[2], b[2][2];
      auto load = [&](int kk, int buf) __attribute__((always_inline)) {
        const int qq = 2 * kk + (lane >> 5);
        const int ra = 32 * wave + (lane & 31);
        a[buf] = as_bf16x8(As[ra * 8 + swz(ra, qq)]);
#pragma unroll
        for (int j = 0; j < 2; ++j) {
          const int rb = 32 * j + (lane & 31);
          b[buf][j] = as_bf16x8(Bs[rb * 8 + swz(rb, qq)]);
        }
      };
      load(0, 0);
#pragma unroll
      for (int kk = 0; kk < 4; ++kk) {
        if (kk + 1 < 4) load(kk + 1, (kk + 1) & 1);
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int j = 0; j < 2; ++j) acc[j] = mfma32(a[kk & 1], b[kk & 1][j], acc[j]);
        __builtin_amdgcn_sched_barrier(0);
      }
    }
    // Epilogue: lanes l and l + 32 hold channels 8 g + 0..3 and 8 g + 4..7
    // of pixel l % 32; swapping the halves of groups 2 h and 2 h + 1 across
    // the half-waves leaves each lane 8 consecutive channels, one 16-byte
    // store.
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      const int p = p0 + 32 * j + (lane & 31);
      unsigned pk[4][2];
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        float v[4];
#pragma unroll
        for (int t = 0; t < 4; ++t) {
          v[t] = acc[j][4 * g + t] + bv[g][t];
          if (relu) v[t] = fmaxf(v[t], 0.0f);
        }
        pk[g][0] = f2bf(v[0]) | (f2bf(v[1]) << 16);
        pk[g][1] = f2bf(v[2]) | (f2bf(v[3]) << 16);
      }
#pragma unroll
      for (int h = 0; h < 2; ++h) {
#pragma unroll
        for (int r = 0; r < 2; ++r) {
          const auto sw = __builtin_amdgcn_permlane32_swap(pk[2 * h][r], pk[2 * h + 1][r], false,
                                                           false);
          pk[2 * h][r] = sw[0];
          pk[2 * h + 1][r] = sw[1];
        }
        if (p < P)
          *(u32x4*)(Y + (long)p * COUT + 32 * wave + 16 * h + 8 * (lane >> 5)) =
              u32x4{pk[2 * h][0], pk[2 * h][1], pk[2 * h + 1][0], pk[2 * h + 1][1]};
      }
    }
  }
}

// ---------------------------------------------------------------- forward, persistent row-stage 3x3

// XOR swizzle of the four 16-byte chunks of a 64-byte LDS row: eight
// consecutive rows read at one logical chunk land on eight distinct 16-byte
// slots of a 128-byte bank cycle.
__device__ __forceinline__ int swz4(int row, int q) { return q ^ ((row >> 1) & 3); }

// Persistent 3x3 implicit GEMM.  The K loop of an output tile (BN channels x
// BM consecutive pixels) runs over stages (32-channel chunk c, filter row r):
// a stage holds the weights of taps (r, 0..2) for the tile's channels and the
// BM + 2 input pixel rows q = p0 + (r - 1) W - 1 + j, so each input row is
// fetched once per filter row and read by the three column taps at row
// offsets 0, 1, 2.  A B fragment whose source pixel lies outside the image
// (left / right padding, or a row of the neighbouring sample) is zeroed at
// use.  Work items are (split, pixel tile, channel tile); block lb of G takes
// items lb, lb + G, ... and streams all their stages through one NS-deep LDS
// ring, so the next item's loads are in flight while the current item
// finishes and writes its tile.  Each wave owns TM x TN MFMA tiles of 32 x 32.
// The K order (chunk, r, s, channel) is fixed by the shape and the split
// count, so a recomputation is bit-identical.
//
// SPLIT: item split s covers stages [s * nk, (s + 1) * nk) and writes fp32
// partials part[s][p][co]; conv_rows_epilogue sums them in split order.
template <int WCO, int WP, int TM, int TN, int NS, bool SPLIT>
__global__ __launch_bounds__(WCO * WP * 64) void conv_rows_pers(
    const bf16_t* __restrict__ X, const bf16_t* __restrict__ Wt,
    const float* __restrict__ bias, bf16_t* __restrict__ Y, float* __restrict__ part, int P,
    int H, int W, int Cin, int Cout, int relu, int co_major, int npt, int S) {
  constexpr int NW = WCO * WP;
  constexpr int BN = WCO * TM * 32;                        // output channels per tile
  constexpr int BM = WP * TN * 32;                         // output pixels per tile
  constexpr int RA = 3 * BN;                               // weight rows per stage
  constexpr int RB = BM + 2;                               // input pixel rows per stage
  constexpr int RPI = 16 * NW;                             // LDS rows per DMA round
  constexpr int ROWS = (RA + RB + RPI - 1) / RPI * RPI;
  constexpr int L = ROWS / RPI;                            // DMA instructions per wave per stage
  constexpr int LA = RA / RPI;                             // ... of which weight rows
  static_assert(RA % RPI == 0, "weight rows must fill whole DMA rounds");
  __shared__ u32x4 smem[NS][ROWS * 4];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wco = wave / WP, wp = wave % WP;
  const int wcu = __builtin_amdgcn_readfirstlane(wco);
  const int nct = Cout / BN;
  const int tiles = npt * nct;
  const int G = gridDim.x;
  const int lb = xcd_remap(blockIdx.x, G);
  const int items = tiles * S;
  const int n_items = lb < items ? (items - lb + G - 1) / G : 0;
  const int nk = 3 * (Cin / 32) / S;                       // stages per item
  const int total = n_items * nk;
  const int HW = H * W;

  // Buffer descriptors: a byte offset at or past the end (or negative, read
  // as unsigned) returns zeros, which is the zero padding of pixels outside
  // [0, P).  Sizes are below 2^31 (checked by the launcher).
  const u32x4 rx = make_rsrc(X, P * Cin * 2);
  const u32x4 rw = make_rsrc(Wt, Cout * 9 * Cin * 2);

  // Per-lane byte offsets of the rows this lane fills (loop invariant).
  // Weight row of instruction u < LA: channel co (within the tile), column
  // tap t3; pixel row of instruction u >= LA: j (0 .. BM + 1, or padding).
  int aoff[LA], boff[L - LA];
#pragma unroll
  for (int u = 0; u < L; ++u) {
    const int row = (wave + NW * u) * 16 + (lane >> 2);
    const int c = (lane & 3) ^ ((row >> 1) & 3);
    if (u < LA) {
      const int t3 = row / BN, co = row - t3 * BN;
      aoff[u < LA ? u : 0] = ((co * 9 + t3) * Cin + c * 8) * 2;
    } else {
      boff[u < LA ? 0 : u - LA] = ((row - RA) * Cin + c * 8) * 2;
    }
  }

  auto coords = [&](int it, int& split, int& p0, int& co0) __attribute__((always_inline)) {
    const int item = lb + it * G;
    split = item / tiles;
    const int t = item - split * tiles;
    p0 = (co_major ? t % npt : t / nct) * BM;
    co0 = (co_major ? t / npt : t % nct) * BN;
  };

  // issue side: the item whose stage is loaded next
  int i_it = 0, i_ks = 0, i_split = 0, i_p0 = 0, i_co0 = 0;
  if (total > 0) coords(0, i_split, i_p0, i_co0);
  auto issue = [&](int slot) __attribute__((always_inline)) {
    const int stg = i_split * nk + i_ks;
    const int chunk = stg / 3, rf = stg - 3 * chunk;
    const int c0 = chunk * 32;
    const int soff_a = ((i_co0 * 9 + 3 * rf) * Cin + c0) * 2;
    const int base_b = ((i_p0 + (rf - 1) * W - 1) * Cin + c0) * 2;
#pragma unroll
    for (int u = 0; u < L; ++u) {
      auto* dst = TGP_LDS(&smem[slot][(wave + NW * u) * 64]);
      if (u < LA)
        dma16(rw, dst, aoff[u < LA ? u : 0], soff_a);
      else
        dma16(rx, dst, base_b + boff[u < LA ? 0 : u - LA], 0);
    }
    if (++i_ks == nk) {
      i_ks = 0;
      if (++i_it < n_items) coords(i_it, i_split, i_p0, i_co0);
    }
  };

#pragma unroll
  for (int k = 0; k < NS - 1; ++k)
    if (k < total) issue(k);

  // compute side: one item at a time, its stages streamed through the ring
  int idx = 0;
  for (int c_it = 0; c_it < n_items; ++c_it) {
    int c_split, c_p0, c_co0;
    coords(c_it, c_split, c_p0, c_co0);
    unsigned vmask[TN];
#pragma unroll
    for (int j = 0; j < TN; ++j) {
      const int p = c_p0 + wp * TN * 32 + j * 32 + (lane & 31);
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

    f32x16_t acc[TM][TN];
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
      for (int j = 0; j < TN; ++j) acc[i][j] = f32x16_t{};

    for (int c_ks = 0; c_ks < nk; ++c_ks, ++idx) {
      // Loads complete in order, so stage idx is in when at most the stages
      // issued after it are pending (stores of a tile epilogue only make
      // this wait longer).
      wait_stages<NS, L>(min(NS - 2, total - 1 - idx));
      ring_barrier();
      if (idx + NS - 1 < total) issue((idx + NS - 1) % NS);
      const int rf = (c_split * nk + c_ks) % 3;
      const u32x4* As = smem[idx % NS];
      const u32x4* Bs = smem[idx % NS] + RA * 4;
      // 6 steps (3 column taps x 2 K sub-steps of 16 channels).  Step t + 1's
      // fragments are read while step t's MFMAs run, and its B fragments
      // are masked between them.
      bf16x8_t fa[2][TM], bm[2][TN];
      u32x4 fb[TN];
      auto load = [&](int t, int buf) __attribute__((always_inline)) {
        const int t3 = t >> 1, kk = t & 1;
        const int qq = 2 * kk + (lane >> 5);
#pragma unroll
        for (int i = 0; i < TM; ++i) {
          const int row = t3 * BN + wco * TM * 32 + i * 32 + (lane & 31);
          fa[buf][i] = as_bf16x8(As[row * 4 + swz4(row, qq)]);
        }
#pragma unroll
        for (int j = 0; j < TN; ++j) {
          const int row = wp * TN * 32 + j * 32 + (lane & 31) + t3;
          fb[j] = Bs[row * 4 + swz4(row + RA, qq)];
        }
      };
      auto mask = [&](int t, int buf) __attribute__((always_inline)) {
#pragma unroll
        for (int j = 0; j < TN; ++j) {
          const bool ok = (vmask[j] >> (rf * 3 + (t >> 1))) & 1u;
          bm[buf][j] = as_bf16x8(ok ? fb[j] : u32x4{0, 0, 0, 0});
        }
      };
      load(0, 0);
      mask(0, 0);
#pragma unroll
      for (int t = 0; t < 6; ++t) {
        const int cur = t & 1;
        if (t + 1 < 6) load(t + 1, cur ^ 1);
#pragma unroll
        for (int i = 0; i < TM; ++i)
#pragma unroll
          for (int j = 0; j < TN; ++j) acc[i][j] = mfma32(fa[cur][i], bm[cur][j], acc[i][j]);
        if (t + 1 < 6) {
          mask(t + 1, cur ^ 1);
          // reads first, half the MFMAs (covering the read latency), the
          // masking, then the other half
          __builtin_amdgcn_sched_group_barrier(0x100, TM + TN, 0);
          __builtin_amdgcn_sched_group_barrier(0x008, (TM * TN + 1) / 2, 0);
          __builtin_amdgcn_sched_group_barrier(0x002, 4 * TN + 8, 0);
          __builtin_amdgcn_sched_group_barrier(0x008, TM * TN / 2, 0);
        }
        __builtin_amdgcn_sched_barrier(0);
      }
    }

    // tile epilogue; the bias goes through the constant address space so its
    // (wave-uniform) loads are scalar and do not wait on the DMA ring
    const __attribute__((address_space(4))) float* cbias =
        (const __attribute__((address_space(4))) float*)bias;
#pragma unroll
    for (int i = 0; i < TM; ++i) {
#pragma unroll
      for (int j = 0; j < TN; ++j) {
        const int p = c_p0 + wp * TN * 32 + j * 32 + (lane & 31);
#pragma unroll
        for (int g = 0; g < 4; ++g) {
          const int cob = c_co0 + wcu * TM * 32 + i * 32 + 8 * g;
          const int co = cob + 4 * (lane >> 5);
          if constexpr (SPLIT) {
            const float4 o = make_float4(acc[i][j][4 * g], acc[i][j][4 * g + 1],
                                         acc[i][j][4 * g + 2], acc[i][j][4 * g + 3]);
            if (p < P) *(float4*)(part + ((long)c_split * P + p) * Cout + co) = o;
          } else {
            float v[4];
#pragma unroll
            for (int e = 0; e < 4; ++e) {
              v[e] = acc[i][j][4 * g + e];
              if (bias) {
                const float b0 = cbias[cob + e], b1 = cbias[cob + 4 + e];
                v[e] += (lane >> 5) ? b1 : b0;
              }
              if (relu) v[e] = fmaxf(v[e], 0.0f);
            }
            uint2 o;
            o.x = f2bf(v[0]) | (f2bf(v[1]) << 16);
            o.y = f2bf(v[2]) | (f2bf(v[3]) << 16);
            if (p < P) *(uint2*)(Y + (long)p * Cout + co) = o;
          }
        }
      }
    }
  }
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

// The ng micro-batches of one launch: micro-batch k's blocks form the k-th
// of ng equal parts of the grid.
struct MbWg {
  const bf16_t* x[kMaxGroup];
  const bf16_t* dz[kMaxGroup];
  float* part[kMaxGroup];
};
template <int WM, int WN, int TM, int TN, int TAPS>
__global__ __launch_bounds__(256) void conv_wgrad_mfma(MbWg io, int ng, int P, int H, int W,
                                                       int Cin, int Cout, int pix_per_split) {
  static_assert(WM * WN == 4, "4 waves");
  constexpr int BMc = WM * TM * 32;  // output channels (co) per block
  constexpr int BNc = WN * TN * 32;  // input channels (ci) per block
  constexpr int BK = 64;             // pixels per K step
  static_assert(BMc + BNc <= 256, "one 8x8 block per thread");
  __shared__ u32x4 smem[2][(BMc + BNc) * 8];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave / WN, wn = wave % WN;
  const int ncb = Cin / BNc;
  // 1-D grid of (split, tap, ci tile, co tile), split slowest.  The
  // dispatcher deals blocks round-robin over the 8 XCDs; remapped, each XCD
  // runs a contiguous range of splits with all their tiles, so the pixel rows
  // of X and dZ a split reads are fetched into one L2 only.
  const int T = TAPS * ncb * (Cout / BMc);
  const int per = gridDim.x / ng;                               // blocks per micro-batch
  const int lb0 = xcd_remap(blockIdx.x, gridDim.x);
  const int gi = lb0 / per;                                     // micro-batch (uniform)
  const int lb = lb0 - gi * per;
  const bf16_t* __restrict__ X = pickg(io.x, gi);
  const bf16_t* __restrict__ dZ = pickg(io.dz, gi);
  float* __restrict__ part = pickg(io.part, gi);
  const int split = lb / T;
  const int t = lb - split * T;
  const int tx = t % (TAPS * ncb);
  const int tap = tx / ncb;
  const int ci0 = (tx - tap * ncb) * BNc;
  const int co0 = (t / (TAPS * ncb)) * BMc;
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

// out[e] = sum_{s < S} part[s][e] in a fixed order: a block of 1024 threads
// covers C4 float4 columns with LANES = 1024 / C4 split lanes; lane l sums
// s = l, l + LANES, ... in ascending order, then lanes 0 .. LANES - 1 are
// added in order.  (C4, LANES) is a function of S only, so the order is a
// function of the shape.  E must be a multiple of 4.
// Blocks from nblk1 on run a second, independent sum (part2, out2, E2, S2)
// in the same launch.
template <int C4>
__global__ __launch_bounds__(1024) void splitk_reduce(const float* __restrict__ part,
                                                      float* __restrict__ out, long E, int S,
                                                      const float* __restrict__ part2,
                                                      float* __restrict__ out2, long E2, int S2,
                                                      int nblk1) {
  constexpr int LANES = 1024 / C4;
  __shared__ float4 red[LANES][C4];
  int bx = blockIdx.x;
  if (bx >= nblk1) {   // block-uniform
    bx -= nblk1;
    part = part2; out = out2; E = E2; S = S2;
  }
  const int col = threadIdx.x % C4, lane = threadIdx.x / C4;
  const long e4 = ((long)bx * C4 + col) * 4;
  float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
  if (e4 < E) {
    int k = lane;
    // eight independent loads in flight per step
    for (; k + 7 * LANES < S; k += 8 * LANES) {
      float4 t[8];
#pragma unroll
      for (int u = 0; u < 8; ++u) t[u] = *(const float4*)(part + (long)(k + u * LANES) * E + e4);
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        acc.x += t[u].x; acc.y += t[u].y; acc.z += t[u].z; acc.w += t[u].w;
      }
    }
    for (; k < S; k += LANES) {
      const float4 t = *(const float4*)(part + (long)k * E + e4);
      acc.x += t.x; acc.y += t.y; acc.z += t.z; acc.w += t.w;
    }
  }
  red[lane][col] = acc;
  __syncthreads();
  if (lane == 0 && e4 < E) {
    float4 r = red[0][col];
    for (int l = 1; l < LANES; ++l) {
      const float4 t = red[l][col];
      r.x += t.x; r.y += t.y; r.z += t.z; r.w += t.w;
    }
    *(float4*)(out + e4) = r;
  }
}

// The same sum for E not a multiple of 4 (e.g. the bias of a one-channel
// head), one element per thread, s ascending.
__global__ __launch_bounds__(256) void splitk_reduce_scalar(const float* __restrict__ part,
                                                            float* __restrict__ out, long E,
                                                            int S) {
  const long e = (long)blockIdx.x * 256 + threadIdx.x;
  if (e >= E) return;
  float acc = 0.f;
  for (int k = 0; k < S; ++k) acc += part[(long)k * E + e];
  out[e] = acc;
}

// wt[ci][tap'][co] = w[co][taps-1-tap'][ci]: the data gradient of a
// cross-correlation is a cross-correlation with the 180-degree rotated,
// channel-transposed filter.  A batch of tensors in one launch: blocks
// blk0[k] .. blk0[k + 1] - 1 serve tensor k.
template <typename T>
__global__ void wtransform_batch_kernel(WtBatch b) {
  int k = 0;
  while (k + 1 < b.count && (int)blockIdx.x >= b.blk0[k + 1]) ++k;
  const long e = (long)(blockIdx.x - b.blk0[k]) * 256 + threadIdx.x;
  const int cout = b.cout[k], cin = b.cin[k], taps = b.taps[k];
  if (e >= (long)cout * cin * taps) return;
  const int co = e % cout;
  const long r = e / cout;
  const int tp = r % taps;
  const int ci = r / taps;
  ((T*)b.wt[k])[e] = ((const T*)b.w[k])[((long)co * taps + (taps - 1 - tp)) * cin + ci];
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

bool mfma_conv_ok(int dt, int cin, int cout) {
  return dt == 0 && cin % 64 == 0 && cout % 64 == 0;
}

// Forward tile configurations.  A configuration is chosen per shape by
// fwd_config() (a pure function of the shape, so recomputation reuses the
// exact same kernel); g_fwd_variant > 0 forces one for measurement sweeps.
int g_fwd_variant = 0;
int g_fwd_order = -1;   // -1: by operand size; 0/1 forced (measurement only)

template <int WCO, int WP, int TM, int TN, int NS>
hipError_t launch_fwd_dma(const char* name9, const char* name1, const bf16_t* X, const bf16_t* Wt,
                          const float* b, bf16_t* Y, long P, const ConvShape& s, int relu,
                          hipStream_t st, const bf16_t* X2 = nullptr, bf16_t* Y2 = nullptr) {
  const char* name = s.taps == 9 ? name9 : name1;
  constexpr int BN = WCO * TM * 32, BM = WP * TN * 32;
  if (s.cout % BN || (X2 == nullptr) != (Y2 == nullptr)) return hipErrorInvalidValue;
  const int ng = X2 ? 2 : 1;
  dim3 grid(ng * cdiv(P, BM) * (s.cout / BN));
  double flops = 2.0 * ng * P * s.cout * s.taps * s.cin;
  double bytes = 2.0 * ((double)ng * P * s.cin + (double)s.cout * s.taps * s.cin +
                        (double)ng * P * s.cout);
  ProfScope ps(name, flops, bytes, st);
  const double xbytes = 2.0 * P * s.cin, wbytes = 2.0 * s.cout * s.taps * s.cin;
  const int co_major = g_fwd_order >= 0 ? g_fwd_order : (wbytes > xbytes ? 1 : 0);
  if (s.taps == 9)
    TGP_LAUNCH(ps, (conv_fwd_dma<WCO, WP, TM, TN, 9, NS>), grid, dim3(WCO * WP * 64), 0, st, X,
                       X2, Wt, b, Y, Y2, (int)P, s.H, s.W, s.cin, s.cout, relu, co_major);
  else
    TGP_LAUNCH(ps, (conv_fwd_dma<WCO, WP, TM, TN, 1, NS>), grid, dim3(WCO * WP * 64), 0, st, X,
                       X2, Wt, b, Y, Y2, (int)P, s.H, s.W, s.cin, s.cout, relu, co_major);
  return launch_status();
}

#define TGP_FWD_CFG(WCO, WP, TM, TN, NS)                                                        \
  launch_fwd_dma<WCO, WP, TM, TN, NS>("conv_fwd_dma<" #WCO "," #WP "," #TM "," #TN ",9," #NS ">", \
                                      "conv_fwd_dma<" #WCO "," #WP "," #TM "," #TN ",1," #NS ">", \
                                      X, Wt, b, Y, P, s, relu, st, X2, Y2)

// Row-stage forward launches.  S > 1 splits the stages over S blocks per
// tile; the partials live in `part` (capacity part_cap floats; S is reduced
// to fit, which only happens under measurement overrides).
template <int WCO, int WP, int TM, int TN, int NS>
hipError_t launch_fwd_rows(const char* name_f, const char* name_t, const bf16_t* X,
                           const bf16_t* Wt, const float* b,
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
    ProfScope ps(name_f, flops, xbytes + wbytes + 2.0 * P * s.cout, st);
    TGP_LAUNCH(ps, (conv_fwd_rows<WCO, WP, TM, TN, NS, false>), grid, block, 0, st, X, Wt, b,
                       Y, part, (int)P, s.H, s.W, s.cin, s.cout, relu, co_major, tiles, sps);
    return launch_status();
  }
  {
    ProfScope ps(name_t, flops, xbytes + wbytes + 4.0 * S * P * s.cout, st);
    TGP_LAUNCH(ps, (conv_fwd_rows<WCO, WP, TM, TN, NS, true>), grid, block, 0, st, X, Wt, b,
                       Y, part, (int)P, s.H, s.W, s.cin, s.cout, relu, co_major, tiles, sps);
  }
  hipError_t e = launch_status();
  if (e != hipSuccess) return e;
  ProfScope ps2("conv_rows_epilogue", 0.0, 4.0 * S * P * s.cout + 2.0 * P * s.cout, st);
  TGP_LAUNCH(ps2, conv_rows_epilogue, dim3(cdiv(P * s.cout, 2048)), dim3(256), 0, st, part, b,
                     Y, P, s.cout, S, relu);
  return launch_status();
}

#define TGP_ROWS_CFG(WCO, WP, TM, TN, NS, S)                                                   \
  launch_fwd_rows<WCO, WP, TM, TN, NS>(                                                        \
      "conv_fwd_rows<" #WCO "," #WP "," #TM "," #TN "," #NS ",false>",                          \
      "conv_fwd_rows<" #WCO "," #WP "," #TM "," #TN "," #NS ",true>", X, Wt, b, Y, part, part_cap, \
      P, s, relu, S, st)

// Persistent row-stage launches.  S (a divisor of the 3 * Cin / 32 stages,
// reduced to fit part_cap) splits every tile's K range; the grid is the
// number of blocks that fit on the chip at once, capped by the item count.
constexpr int rows_pers_lds(int WCO, int WP, int TM, int TN, int NS) {
  return NS * ((3 * WCO * TM * 32 + WP * TN * 32 + 2 + 16 * WCO * WP - 1) / (16 * WCO * WP) *
               (16 * WCO * WP)) * 64;
}

template <int WCO, int WP, int TM, int TN, int NS>
hipError_t launch_rows_pers(const char* name_f, const char* name_t, const bf16_t* X,
                            const bf16_t* Wt, const float* b,
                            bf16_t* Y, float* part, size_t part_cap, long P, const ConvShape& s,
                            int relu, int S, hipStream_t st) {
  constexpr int BN = WCO * TM * 32, BM = WP * TN * 32, NW = WCO * WP;
  constexpr int LDS = rows_pers_lds(WCO, WP, TM, TN, NS);
  static_assert(LDS <= 160 * 1024, "LDS ring too large");
  if (s.cout % BN || s.cin % 32 || s.taps != 9) return hipErrorInvalidValue;
  // byte offsets into X and W are 32-bit, negative ones must read as out of range
  if ((double)(P + BM + 2L * s.W + 2) * s.cin * 2 >= 2147483648.0 ||
      (double)s.cout * 9 * s.cin * 2 >= 2147483648.0)
    return hipErrorInvalidValue;
  const int nst = 3 * (s.cin / 32);
  if (S < 1) S = 1;
  if (S > nst) S = nst;
  while (S > 1 && (nst % S || (size_t)S * P * s.cout > part_cap)) --S;
  const int npt = cdiv(P, BM);
  const long items = (long)npt * (s.cout / BN) * S;
  int occ = (160 * 1024) / LDS;
  if (occ * NW > 16) occ = 16 / NW;
  if (occ < 1) occ = 1;
  const int G = (int)(items < 256L * occ ? items : 256L * occ);
  const double flops = 2.0 * P * s.cout * 9 * s.cin;
  const double xbytes = 2.0 * P * s.cin, wbytes = 2.0 * s.cout * 9 * s.cin;
  const int co_major = g_fwd_order >= 0 ? g_fwd_order : (wbytes > xbytes ? 1 : 0);
  if (G == 0) return hipSuccess;
  if (S == 1) {
    ProfScope ps(name_f, flops, xbytes + wbytes + 2.0 * P * s.cout, st);
    TGP_LAUNCH(ps, (conv_rows_pers<WCO, WP, TM, TN, NS, false>), dim3(G), dim3(NW * 64), 0, st,
                       X, Wt, b, Y, part, (int)P, s.H, s.W, s.cin, s.cout, relu, co_major, npt, 1);
    return launch_status();
  }
  {
    ProfScope ps(name_t, flops, xbytes + wbytes + 4.0 * S * P * s.cout, st);
    TGP_LAUNCH(ps, (conv_rows_pers<WCO, WP, TM, TN, NS, true>), dim3(G), dim3(NW * 64), 0, st,
                       X, Wt, b, Y, part, (int)P, s.H, s.W, s.cin, s.cout, relu, co_major, npt, S);
  }
  hipError_t e = launch_status();
  if (e != hipSuccess) return e;
  ProfScope ps2("conv_rows_epilogue", 0.0, 4.0 * S * P * s.cout + 2.0 * P * s.cout, st);
  TGP_LAUNCH(ps2, conv_rows_epilogue, dim3(cdiv(P * s.cout, 2048)), dim3(256), 0, st, part, b,
                     Y, P, s.cout, S, relu);
  return launch_status();
}

#define TGP_PERS_CFG(WCO, WP, TM, TN, NS, S)                                                    \
  launch_rows_pers<WCO, WP, TM, TN, NS>(                                                        \
      "conv_rows_pers<" #WCO "," #WP "," #TM "," #TN "," #NS ",false>",                          \
      "conv_rows_pers<" #WCO "," #WP "," #TM "," #TN "," #NS ",true>", X, Wt, b, Y, part, part_cap, \
      P, s, relu, S, st)

int g_fwd_split = 0;   // > 0 forces the split count (measurement only)
// Measurement only: bit 0 allows the row-tiled kernel for forward calls, bit
// 1 for data-gradient calls, bit 2 the row-blocked weight gradient, bit 3
// the nine-tap row kernel.
int g_rowtile_mask = 15;
thread_local int t_in_dgrad = 0;

struct FwdPlan {
  int cfg;   // 1..: row-stage configurations; 100+: per-tap (150: 1x1 with resident
             // weights); 200+: persistent row-stage
  int S;
};

// The resident-weight 1x1 kernel's shapes (its static LDS holds 256 x 256
// weights) and its launch.
static bool conv1x1_res_ok(const ConvShape& s) {
  return s.taps == 1 && s.cout == 256 && s.cin % 64 == 0 && s.cin <= 256 && s.pixels() > 0;
}

// n micro-batches x[k] -> y[k] in one launch.
static hipError_t launch_1x1_res(int n, const void* const* x, const bf16_t* Wt, const float* b,
                                 void* const* y, const ConvShape& s, int relu, hipStream_t st) {
  if (!conv1x1_res_ok(s) || n < 1 || n > kMaxGroup) return hipErrorInvalidValue;
  const long P = s.pixels();
  if (P > (1L << 30)) return hipErrorInvalidValue;              // pixel index is an int
  Mb1x1 io;
  for (int k = 0; k < kMaxGroup; ++k) {   // unused entries repeat the first
    io.x[k] = (const bf16_t*)x[k < n ? k : 0];
    io.y[k] = (bf16_t*)y[k < n ? k : 0];
  }
  const long T = n * ((P + 63) / 64);
  const int G = (int)(T < 256 ? T : 256);
  ProfScope ps("conv1x1_res", 2.0 * n * P * s.cout * s.cin,
               2.0 * ((double)n * P * (s.cin + s.cout) + (double)s.cout * s.cin), st);
  TGP_LAUNCH(ps, conv1x1_res<4>, dim3(G), dim3(512), 0, st, io, n, Wt, b, (int)P, s.cin, relu);
  return launch_status();
}

struct PersTile { int BN, BM; };
PersTile pers_tile(int cfg) {
  switch (cfg) {
    case 202: return {128, 256};
    case 203: return {64, 256};
    case 204: return {128, 128};
    case 205: return {64, 640};
    case 206: return {128, 256};
    case 207: return {128, 256};
    default: return {64, 512};
  }
}

// Pure function of the per-sample shape (H, W, Cin, Cout, taps), plus the
// measurement overrides: the kernel family and the split count fix the K
// summation order, so keeping them independent of the number of samples
// keeps every sample's output bit-identical whatever the micro-batch size.
// The tile-count heuristics use a nominal micro-batch of 4 samples.
FwdPlan fwd_plan(const ConvShape& s) {
  const long P = 4L * s.H * s.W;
  FwdPlan pl{0, 1};
  // Measured per shape (3x3, kernel time in a step): the nine-tap
  // whole-row kernel is fastest on images of 48 x 48 and up, and from 24 x 24
  // where one micro-batch gives it at least 48 tiles (at 24 x 24 a paired
  // launch of it takes 27 us where the split-K row-stage kernel and its
  // epilogue take 40; with fewer tiles, as at one or two samples, most CUs
  // idle); the persistent row-stage kernel with split K on the other small,
  // deep layers (few pixel tiles, long K); the per-tap kernel for the rest.
  const bool k3 = s.taps == 9 && s.cin % 64 == 0;
  const long hw = (long)s.H * s.W;
  if (k3 && (hw >= 48 * 48 || (hw >= 24 * 24 && conv_rows32_tiles(s) >= 48)) &&
      (g_rowtile_mask >> 3 & 1) && conv_rows32_ok(s)) {
    pl.cfg = 400;  // whole-row tiles, nine taps per stage, 32x32x16
  } else if (k3 && (long)s.H * s.W >= 96 * 96 && conv_rowtile_ok(s) &&
      (g_rowtile_mask >> (t_in_dgrad ? 1 : 0) & 1)) {
    pl.cfg = 300;  // row-tiled 16x16x32
  } else if (k3 && P <= 4096) {
    pl.cfg = 203;  // persistent row-stage, 64 x 256
  } else if (k3 && P <= 16384 && s.cin >= 256 && s.cout % 128 == 0) {
    pl.cfg = 207;  // persistent row-stage, 128 x 256, 8 waves
  } else if (conv1x1_res_ok(s)) {
    pl.cfg = 150;  // 1x1, all weights resident in LDS
  } else {
    pl.cfg = 100;
  }
  if (g_fwd_variant > 0) pl.cfg = g_fwd_variant;
  if (pl.cfg == 150 && !conv1x1_res_ok(s)) pl.cfg = 100;
  if (pl.cfg >= 400) {
    g_rows32_cfg = pl.cfg >= 401 ? pl.cfg - 401 : -1;
    if (!conv_rows32_ok(s)) pl.cfg = 100;
    g_rows32_cfg = -1;
    return pl;
  }
  if (pl.cfg >= 300) {
    if (!conv_rowtile_ok(s)) pl.cfg = 100;
    return pl;
  }
  if ((pl.cfg == 2 || pl.cfg == 5) && s.cout % 128) pl.cfg = pl.cfg == 2 ? 1 : 3;  // 128-wide tiles need cout % 128 == 0
  if (pl.cfg >= 200) {
    if (s.taps != 9 || s.cin % 32) { pl.cfg = 100; return pl; }
    const PersTile t = pers_tile(pl.cfg);
    if (s.cout % t.BN) pl.cfg = 201;                   // 64-channel tiles fit every shape here
    const PersTile u = pers_tile(pl.cfg);
    const long tiles = cdiv(P, u.BM) * (long)(s.cout / u.BN);
    const int nst = 3 * (s.cin / 32);
    int S = 1;
    // split K only when the tiles alone leave most of the chip idle
    while (tiles * S < 192 && S < 8) {
      int n = S + 1;
      while (n <= nst && nst % n) ++n;
      if (n > nst) break;
      S = n;
    }
    pl.S = g_fwd_split > 0 ? g_fwd_split : S;
    return pl;
  }
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
  const bool splits = pl.cfg < 100 || (pl.cfg >= 200 && pl.cfg < 300);   // per-tap and row-tiled never split
  return splits && pl.S > 1 ? (size_t)pl.S * s.pixels() * s.cout : 0;
}

hipError_t conv_forward_mfma(const void* x, const void* w, const float* b, void* y,
                             const ConvShape& s, int relu, float* part, size_t part_cap,
                             hipStream_t st) {
  long P = s.pixels();
  const bf16_t* X = (const bf16_t*)x;
  const bf16_t* Wt = (const bf16_t*)w;
  bf16_t* Y = (bf16_t*)y;
  const bf16_t* X2 = nullptr;   // per-tap configurations: one micro-batch
  bf16_t* Y2 = nullptr;
  const FwdPlan pl = fwd_plan(s);
  const bool wide = s.cout % 128 == 0;
  if (pl.cfg == 150) return launch_1x1_res(1, &x, Wt, b, &y, s, relu, st);
  if (pl.cfg >= 400) {
    g_rows32_cfg = pl.cfg >= 401 ? pl.cfg - 401 : -1;
    const hipError_t e = conv_forward_rows32(1, &x, w, b, &y, s, relu, st);
    g_rows32_cfg = -1;
    return e;
  }
  if (pl.cfg >= 300) {
    g_rowtile_cfg = pl.cfg >= 301 ? pl.cfg - 301 : -1;
    const hipError_t e = conv_forward_rowtile(x, w, b, y, s, relu, st);
    g_rowtile_cfg = -1;
    return e;
  }
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
    case 201: return TGP_PERS_CFG(1, 4, 2, 4, 3, pl.S);               // 64 x 512
    case 202: return TGP_PERS_CFG(2, 2, 2, 4, 3, pl.S);               // 128 x 256
    case 203: return TGP_PERS_CFG(1, 4, 2, 2, 4, pl.S);               // 64 x 256
    case 204: return TGP_PERS_CFG(2, 2, 2, 2, 4, pl.S);               // 128 x 128
    case 205: return TGP_PERS_CFG(1, 4, 2, 5, 2, pl.S);               // 64 x 640
    case 206: return TGP_PERS_CFG(2, 2, 2, 4, 2, pl.S);               // 128 x 256, 2 stages
    case 207: return TGP_PERS_CFG(2, 4, 2, 2, 3, pl.S);               // 128 x 256, 8 waves
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

hipError_t weight_transform_batch(int dt, WtBatch b, hipStream_t st) {
  if (b.count < 0 || b.count > kMaxWt) return hipErrorInvalidValue;
  long blocks = 0;
  double bytes = 0;
  for (int k = 0; k < b.count; ++k) {
    const long n = (long)b.cout[k] * b.cin[k] * b.taps[k];
    if (n <= 0) return hipErrorInvalidValue;
    b.blk0[k] = (int)blocks;
    blocks += cdiv(n, 256);
    bytes += 2.0 * n * (dt == 0 ? 2 : 4);
  }
  if (b.count == 0) return hipSuccess;
  if (blocks >= (1L << 31)) return hipErrorInvalidValue;
  ProfScope ps("wtransform", 0.0, bytes, st);
  if (dt == 0)
    TGP_LAUNCH(ps, wtransform_batch_kernel<bf16_t>, dim3((unsigned)blocks), dim3(256), 0, st, b);
  else
    TGP_LAUNCH(ps, wtransform_batch_kernel<float>, dim3((unsigned)blocks), dim3(256), 0, st, b);
  return launch_status();
}

// Bit 2 of g_rowtile_mask selects the row-blocked weight-gradient kernel.
static bool use_wgrad_rows(const ConvShape& s) {
  return (g_rowtile_mask >> 2 & 1) && wgrad_rows_ok(s);
}

size_t wgrad_mfma_partial_floats(const ConvShape& s) {
  if (use_wgrad_rows(s)) return wgrad_rows_partial_floats(s);
  int tiles = s.taps * (s.cin / 64) * (s.cout / 64);
  if (s.cin % 128 == 0 && s.cout % 128 == 0) tiles = s.taps * (s.cin / 128) * (s.cout / 128);
  long E = (long)s.cout * s.taps * s.cin;
  WgradPlan pl = wgrad_plan<2, 2>(s.pixels(), tiles, E);
  return (size_t)pl.S * E;
}

// The per-tap weight gradient of n micro-batches in one grid; the split plan
// is the single micro-batch's either way.  Where the plan has one split,
// part[k] is set to dw[k] (the kernel writes the gradient itself).
static hipError_t launch_wgrad_mfma(int n, const void* const* x, const void* const* dz,
                                    float* const* dw, float** part, const ConvShape& s,
                                    WgradPlan& pl, hipStream_t st) {
  if (n < 1 || n > kMaxGroup) return hipErrorInvalidValue;
  long P = s.pixels();
  bool big = s.cin % 128 == 0 && s.cout % 128 == 0;
  int bm = big ? 128 : 64, bn = big ? 128 : 64;
  int tiles = s.taps * (s.cin / bn) * (s.cout / bm);
  long E = (long)s.cout * s.taps * s.cin;
  pl = wgrad_plan<2, 2>(P, tiles, E);
  if (pl.S == 1)   // a single split writes the gradient itself
    for (int k = 0; k < n; ++k) part[k] = dw[k];
  MbWg io;
  for (int k = 0; k < kMaxGroup; ++k) {   // unused entries repeat the first
    const int q = k < n ? k : 0;
    io.x[k] = (const bf16_t*)x[q];
    io.dz[k] = (const bf16_t*)dz[q];
    io.part[k] = part[q];
  }
  dim3 grid(n * s.taps * (s.cin / bn) * (s.cout / bm) * pl.S);
  double flops = 2.0 * n * P * E;
  double bytes = n * (2.0 * ((double)P * s.cin + (double)P * s.cout) + 4.0 * pl.S * E);
  const char* nm = big ? (s.taps == 9 ? "conv_wgrad_mfma<2,2,2,2,9>" : "conv_wgrad_mfma<2,2,2,2,1>")
                       : (s.taps == 9 ? "conv_wgrad_mfma<2,2,1,1,9>" : "conv_wgrad_mfma<2,2,1,1,1>");
  ProfScope ps(nm, flops, bytes, st);
  if (big) {
    if (s.taps == 9)
      TGP_LAUNCH(ps, (conv_wgrad_mfma<2, 2, 2, 2, 9>), grid, dim3(256), 0, st, io, n, (int)P, s.H,
                 s.W, s.cin, s.cout, pl.pix_per_split);
    else
      TGP_LAUNCH(ps, (conv_wgrad_mfma<2, 2, 2, 2, 1>), grid, dim3(256), 0, st, io, n, (int)P, s.H,
                 s.W, s.cin, s.cout, pl.pix_per_split);
  } else {
    if (s.taps == 9)
      TGP_LAUNCH(ps, (conv_wgrad_mfma<2, 2, 1, 1, 9>), grid, dim3(256), 0, st, io, n, (int)P, s.H,
                 s.W, s.cin, s.cout, pl.pix_per_split);
    else
      TGP_LAUNCH(ps, (conv_wgrad_mfma<2, 2, 1, 1, 1>), grid, dim3(256), 0, st, io, n, (int)P, s.H,
                 s.W, s.cin, s.cout, pl.pix_per_split);
  }
  return launch_status();
}

hipError_t conv_wgrad_mfma(const void* x, const void* dz, float* dw, float* partial,
                           const ConvShape& s, hipStream_t st, const ReduceJob* extra,
                           ReduceJob* defer) {
  if (use_wgrad_rows(s)) return conv_wgrad_rows_launch(x, dz, dw, partial, s, st, extra, defer);
  long E = (long)s.cout * s.taps * s.cin;
  WgradPlan pl;
  hipError_t e = launch_wgrad_mfma(1, &x, &dz, &dw, &partial, s, pl, st);
  if (e != hipSuccess) return e;
  if (defer) {
    *defer = ReduceJob{partial, dw, E, pl.S};   // partial == dw when S == 1
    return extra ? hipErrorInvalidValue : hipSuccess;
  }
  if (pl.S == 1)
    return extra ? splitk_reduce_launch(extra->part, extra->out, extra->E, extra->S, st) : hipSuccess;
  return splitk_reduce_launch(partial, dw, E, pl.S, st, extra);
}

hipError_t splitk_reduce_launch(const float* part, float* out, long E, int S, hipStream_t st,
                               const ReduceJob* extra) {
  if (extra && (E % 4 || extra->E % 4)) {   // scalar sums run on their own
    const hipError_t e = splitk_reduce_launch(extra->part, extra->out, extra->E, extra->S, st);
    if (e != hipSuccess) return e;
    extra = nullptr;
  }
  ProfScope ps("splitk_reduce", 0.0,
               4.0 * E * (S + 1) + (extra ? 4.0 * extra->E * (extra->S + 1) : 0.0), st);
  if (E % 4) {
    TGP_LAUNCH(ps, splitk_reduce_scalar, dim3(cdiv(E, 256)), dim3(256), 0, st, part, out, E, S);
    return launch_status();
  }
  // many splits of few columns: 16 columns x 64 split lanes; few splits:
  // 256 columns x 4 lanes (chosen by the first sum's S; the second, if any,
  // uses the same layout)
  const int C4 = S >= 64 ? 16 : (S >= 16 ? 64 : 256);
  const int nb1 = (int)cdiv(E, 4L * C4);
  const int nb2 = extra ? (int)cdiv(extra->E, 4L * C4) : 0;
  const float* p2 = extra ? extra->part : nullptr;
  float* o2 = extra ? extra->out : nullptr;
  const long E2 = extra ? extra->E : 0;
  const int S2 = extra ? extra->S : 0;
  if (C4 == 16)
    TGP_LAUNCH(ps, splitk_reduce<16>, dim3(nb1 + nb2), dim3(1024), 0, st, part, out, E, S, p2, o2,
               E2, S2, nb1);
  else if (C4 == 64)
    TGP_LAUNCH(ps, splitk_reduce<64>, dim3(nb1 + nb2), dim3(1024), 0, st, part, out, E, S, p2, o2,
               E2, S2, nb1);
  else
    TGP_LAUNCH(ps, splitk_reduce<256>, dim3(nb1 + nb2), dim3(1024), 0, st, part, out, E, S, p2,
               o2, E2, S2, nb1);
  return launch_status();
}

// Two micro-batches of one layer where the planned kernel takes two tensors
// (the per-tap kernel), else one launch each; the same values as two
// conv_forward_mfma calls either way.
static hipError_t conv_forward_mfma_pair(const void* x0, const void* x1, const void* w,
                                         const float* b, void* y0, void* y1, const ConvShape& s,
                                         int relu, float* part0, float* part1, size_t part_cap,
                                         hipStream_t st) {
  const FwdPlan pl = fwd_plan(s);
  if (pl.cfg >= 100 && pl.cfg < 200) {
    // the per-tap kernel: both micro-batches' tiles in one grid
    const long P = s.pixels();
    const bf16_t* X = (const bf16_t*)x0;
    const bf16_t* X2 = (const bf16_t*)x1;
    const bf16_t* Wt = (const bf16_t*)w;
    bf16_t* Y = (bf16_t*)y0;
    bf16_t* Y2 = (bf16_t*)y1;
    switch (pl.cfg - 100) {
      case 1: return TGP_FWD_CFG(2, 2, 1, 1, 2);
      case 2: return TGP_FWD_CFG(2, 4, 1, 1, 2);
      default: return P >= 32768 && s.cout <= 128 ? TGP_FWD_CFG(2, 4, 1, 1, 2)
                                                   : TGP_FWD_CFG(2, 2, 1, 1, 2);
    }
  }
  hipError_t e = conv_forward_mfma(x0, w, b, y0, s, relu, part0, part_cap, st);
  if (e != hipSuccess) return e;
  return conv_forward_mfma(x1, w, b, y1, s, relu, part1, part_cap, st);
}

// n micro-batches of one layer: one launch of the nine-tap or resident-
// weight 1x1 kernel where it is planned, else pairs (and a single for odd n).
hipError_t conv_forward_mfma_n(int n, const void* const* x, const void* w, const float* b,
                               void* const* y, const ConvShape& s, int relu, float* const* part,
                               size_t part_cap, hipStream_t st) {
  if (n < 1 || n > kMaxGroup) return hipErrorInvalidValue;
  const FwdPlan pl = fwd_plan(s);
  if (pl.cfg == 150) return launch_1x1_res(n, x, (const bf16_t*)w, b, y, s, relu, st);
  if (pl.cfg >= 400) {
    g_rows32_cfg = pl.cfg >= 401 ? pl.cfg - 401 : -1;
    const hipError_t e = conv_forward_rows32(n, x, w, b, y, s, relu, st);
    g_rows32_cfg = -1;
    return e;
  }
  for (int k = 0; k < n; k += 2) {
    const hipError_t e =
        k + 1 < n ? conv_forward_mfma_pair(x[k], x[k + 1], w, b, y[k], y[k + 1], s, relu, part[k],
                                           part[k + 1], part_cap, st)
                  : conv_forward_mfma(x[k], w, b, y[k], s, relu, part[k], part_cap, st);
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

// The weight gradients of n micro-batches in one launch, every sum left
// pending: the row-blocked kernel where it applies, else the per-tap one.
hipError_t conv_wgrad_mfma_n(int n, const void* const* x, const void* const* dz,
                             float* const* dw, float* const* part, const ConvShape& s,
                             hipStream_t st, ReduceJob* const* defer) {
  if (n < 1 || n > kMaxGroup) return hipErrorInvalidValue;
  if (use_wgrad_rows(s)) return conv_wgrad_rows_launch_n(n, x, dz, dw, part, s, st, defer);
  const long E = (long)s.cout * s.taps * s.cin;
  WgradPlan pl;
  float* pp[kMaxGroup];
  for (int k = 0; k < n; ++k) pp[k] = part[k];
  hipError_t e = launch_wgrad_mfma(n, x, dz, dw, pp, s, pl, st);
  if (e != hipSuccess) return e;
  for (int k = 0; k < n; ++k) *defer[k] = ReduceJob{pp[k], dw[k], E, pl.S};   // pp == dw when S == 1
  return hipSuccess;
}

}  // namespace tgpk
