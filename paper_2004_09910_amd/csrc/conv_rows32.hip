// bf16 3x3 convolution (forward, and data gradient on the rotated,
// transposed weights) on 32 x 32 x 16 MFMA with whole-row pixel tiles and
// all nine taps per stage.
//
// An output tile is 64 output channels x R whole image rows of one sample
// (R W pixels, a multiple of 32).  Its K loop runs over 16-channel chunks
// of the input; a stage holds in LDS, for one chunk:
//   - the weights of all nine taps for the 64 channels: 576 rows, tap-major;
//   - the R + 2 input rows h0 - 1 .. h0 + R, each as a block of BWP LDS rows
//     (BWP = W + 2 rounded up to a multiple of 16): row 0 and row W + 1 of a
//     block are the zero padding of the convolution, the rest are pixels.
// Every LDS row is 16 channels (32 bytes), its two 16-byte halves swapped
// when bit 3 of the row index is set.  With that swizzle a fragment read of
// 32 consecutive rows at one half is free of bank conflicts from any start
// row, and since BWP is a multiple of 16 a filter-row shift of the input is
// an immediate offset: output pixel (rho, w) at tap (r, s) reads block row
// rho + r, LDS row w + s.  So the input rows are loaded once per chunk for
// all three filter rows, and no fragment is masked: the zero padding and the
// rows outside the image are buffer reads at out-of-range offsets.
//
// The tile's R W / 32 pixel fragments are dealt to 4 pixel groups, FW each
// (the last groups may hold fewer real ones and compute on a clamped copy);
// with 4 waves each wave is a pixel group over all 64 channels (2 x FW MFMA
// tiles), with 8 waves two waves share a group, one per 32-channel half.  Blocks are persistent
// over tiles, their stages streamed through one NS-deep LDS ring.  Bias and
// ReLU are applied in the epilogue, which transposes each fragment through
// LDS into whole pixel rows.  The K
// order (chunk, tap, channel) is fixed by the per-sample shape, so a
// recomputation is bit-identical.
#include "common.h"
#include "kernels.h"
#include "mfma_util.h"
#include "prof.h"

namespace tgpk {
namespace {

constexpr int R32_OOB = (int)0x80000000;   // byte offset that reads as out of range
constexpr int R32_AROWS = 9 * 64;          // weight rows per stage

typedef __bf16 bf16x2_r32 __attribute__((ext_vector_type(2)));

__device__ __forceinline__ unsigned pack2_bf16(float a, float b) {
  const bf16x2_r32 h = {(__bf16)a, (__bf16)b};
  return __builtin_bit_cast(unsigned, h);
}

// RK > 0: the weights of all RK stages (Cin = 16 RK, one 64-channel output
// tile) stay resident in LDS ahead of the ring, loaded once per block, and
// a ring slot holds only the input rows.
template <int W, int R, int RK = 0>
struct Rows32Geom {
  static constexpr int BWP = (W + 2 + 15) / 16 * 16;           // LDS rows per input row
  static constexpr int BROWS = (R + 2) * BWP;
  static constexpr int AR = RK ? 0 : R32_AROWS;                 // weight rows per slot
  static constexpr int SB = ((AR + BROWS) * 32 + 4095) / 4096 * 4096;  // stage (slot) bytes
  static constexpr int RB = RK * R32_AROWS * 32;                // resident weight bytes
  static constexpr int L = SB / 4096;                           // DMA instructions per wave
  static constexpr int F = R * W / 32;                          // pixel fragments per tile
  static_assert(R * W % 32 == 0, "whole fragments per tile");
  static_assert(R32_AROWS * 32 % 1024 == 0, "weight region ends on a DMA chunk");
};

// CH is the number of 32-channel halves a wave covers: CH = 2 runs 4 waves
// (one per SIMD), each over all 64 channels; CH = 1 runs 8 waves (two per
// SIMD), the two waves of a SIMD on the two channel halves of the same
// pixels, so that one wave's MFMAs run while the other waits on its DMA
// issue or its LDS reads.
//
// The micro-batches of one launch (ng of them, nb samples each, the same
// weights): the tiles of micro-batch k follow those of k - 1 (sample index
// k nb .. k nb + nb - 1), so one launch covers them all and a block streams
// tiles of several through its ring.
// At most eight per launch (a larger group runs as launches of eight): a
// select over more pointers cost the U-Net stage's launches about 1%.
constexpr int kR32Group = 8;
struct R32Io {
  const bf16_t* x[kR32Group];
  bf16_t* y[kR32Group];
};

template <int W, int R, int FW, int NS, int CH, int RK>
__global__ __launch_bounds__(CH == 2 ? 256 : 512) void conv3x3_rows32(
    R32Io io, int ng, const bf16_t* __restrict__ Wt, const float* __restrict__ bias, int nb,
    int H, int Cin, int Cout, int relu) {
  typedef Rows32Geom<W, R, RK> G_;
  constexpr int BWP = G_::BWP, SB = G_::SB, F = G_::F, AR = G_::AR, RB = G_::RB;
  constexpr int NW = CH == 2 ? 4 : 8;                           // waves
  constexpr int NCH = SB / 1024;                                // DMA chunks per stage
  constexpr int LW = (NCH + NW - 1) / NW;                       // ... per wave, at most
  constexpr int ACH = AR * 32 / 1024;                           // DMA chunks of weights per stage
  constexpr int WCH = R32_AROWS * 32 / 1024;                    // ... of one stage's weights
  static_assert(F <= 4 * FW, "fragments per pixel group");
  static_assert(RB + NS * SB <= 160 * 1024, "LDS ring");
  __shared__ __attribute__((aligned(16))) unsigned char smem[RB + NS * SB];
  unsigned char* const ring = smem + RB;

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int pg = wave & 3;                                      // pixel group (the SIMD)
  const int chf = CH == 2 ? 0 : wave >> 2;                      // channel half (CH = 1)
  const int nrb = (H + R - 1) / R;                              // row blocks per sample
  const int nct = Cout / 64;
  const int items = ng * nb * nrb * nct;
  const int G = gridDim.x;
  const int lb = xcd_remap(blockIdx.x, G);
  const int n_items = lb < items ? (items - lb + G - 1) / G : 0;
  const int nk = Cin / 16;                                      // stages per tile
  const int total = n_items * nk;
  // DMA instructions of this wave per stage (waits count them)
  const bool full = NCH % NW == 0 || wave < NCH % NW;
  auto wait_ring = [&](int ahead) __attribute__((always_inline)) {
    if constexpr (NCH % NW == 0) {
      wait_stages<NS, LW>(ahead);
    } else {
      if (full) wait_stages<NS, LW>(ahead);
      else wait_stages<NS, LW - 1>(ahead);
    }
  };

  const int xbytes = nb * H * W * Cin * 2;                      // one micro-batch's input
  const u32x4 rw = make_rsrc(Wt, Cout * 9 * Cin * 2);

  // DMA: instruction u of this wave fills stage chunk k = NW u + wave
  // (1 KiB); lane l the 16 bytes at + 16 l: row k * 32 + l / 2, physical half
  // l % 2, which holds logical half (l % 2) ^ bit 3 of the row.  Chunks below
  // ACH are weight rows (tap, channel), the rest input rows (block row,
  // pixel).
  int doff[LW], drow[LW];
#pragma unroll
  for (int u = 0; u < LW; ++u) {
    const int k = NW * u + wave;
    const int row = k * 32 + (lane >> 1);
    const int lh = (lane & 1) ^ ((row >> 3) & 1);
    if (k < ACH) {
      const int tap = row >> 6, co = row & 63;
      doff[u] = ((co * 9 + tap) * Cin + 8 * lh) * 2;
      drow[u] = 0;
    } else {
      const int q = row - AR;
      const int rr = q / BWP, wp = q - rr * BWP;
      const bool ok = rr < R + 2 && wp >= 1 && wp <= W;
      doff[u] = ok ? ((rr * W + wp - 1) * Cin + 8 * lh) * 2 : 0;
      drow[u] = ok ? rr : -1;
    }
  }

  // Fragment addresses (bytes within a stage).  A: weight row tap * 64 +
  // 32 (channel half) + l % 32 at logical half l / 32, tap as an immediate.
  // B: for each fragment j of the pixel group and column tap s, LDS row
  // rho BWP + w + s of the input region (filter row r adds r BWP rows as an
  // immediate).
  const int abase = (lane & 31) * 32 + (((lane >> 5) ^ ((lane >> 3) & 1)) << 4) + chf * 32 * 32;
  int bq[FW][3];
#pragma unroll
  for (int j = 0; j < FW; ++j) {
    const int f = pg * FW + j;
    int tp = f * 32 + (lane & 31);
    if (tp >= R * W) tp = R * W - 1;                            // clamped copy for padding fragments
    const int rho = tp / W, w = tp - rho * W;
#pragma unroll
    for (int s = 0; s < 3; ++s) {
      const int q = rho * BWP + w + s;
      bq[j][s] = AR * 32 + q * 32 + (((lane >> 5) ^ ((q >> 3) & 1)) << 4);
    }
  }

  // item -> micro-batch gi, its sample n, first row h0, output channels co0
  auto coords = [&](int it, int& gi, int& n, int& h0, int& co0) __attribute__((always_inline)) {
    const int item = lb + it * G;
    const int ct = item % nct, rest = item / nct;
    const int rb = rest % nrb;
    n = rest / nrb;
    gi = n / nb;
    n -= gi * nb;
    h0 = rb * R;
    co0 = ct * 64;
  };

  // issue side: a stage's DMA is issued in parts (u in [u0, u1)) so that
  // inside the stage loop it is spread over the nine taps; the instruction
  // issue stalls while the memory pipeline is full, and spread out those
  // stalls overlap the MFMAs already queued
  int i_it = 0, i_ks = 0, i_gi = 0, i_n = 0, i_h0 = 0, i_co0 = 0;
  if (total > 0) coords(0, i_gi, i_n, i_h0, i_co0);
  u32x4 rxg = make_rsrc(pickg(io.x, i_gi), xbytes);            // the issuing item's input
  auto issue_part = [&](int slot, int u0, int u1) __attribute__((always_inline)) {
    const int c0 = i_ks * 16;
    const int soff_a = (i_co0 * 9 * Cin + c0) * 2;
    const int hb = i_h0 - 1;                                    // input row of block row 0
    const int base_b = ((i_n * H + hb) * W * Cin + c0) * 2;    // negative for hb = -1
    const bool interior = hb >= 0 && hb + R + 2 <= H;
#pragma unroll
    for (int u = 0; u < LW; ++u) {
      if (u < u0 || u >= u1) continue;
      const int k = NW * u + wave;
      if (NCH % NW != 0 && k >= NCH) continue;                  // wave-uniform
      auto* dst = TGP_LDS(ring + slot * SB + k * 1024);
      if (k < ACH) {
        dma16(rw, dst, doff[u], soff_a);
      } else {
        const bool ok = drow[u] >= 0 && (interior || (unsigned)(hb + drow[u]) < (unsigned)H);
        dma16(rxg, dst, ok ? base_b + doff[u] : R32_OOB, 0);
      }
    }
  };
  auto issue_done = [&]() __attribute__((always_inline)) {
    if (++i_ks == nk) {
      i_ks = 0;
      if (++i_it < n_items) {
        coords(i_it, i_gi, i_n, i_h0, i_co0);
        rxg = make_rsrc(pickg(io.x, i_gi), xbytes);
      }
    }
  };

  if constexpr (RK > 0) {
    // every stage's weights of the block's single output-channel tile, once,
    // in the slot layout (chunk c: stage c / WCH, weight chunk c % WCH); the
    // ring's waits cover them since loads complete in order
    if (total > 0) {
#pragma unroll
      for (int u = 0; u < (RK * WCH + NW - 1) / NW; ++u) {
        const int c = NW * u + wave;
        if (c >= RK * WCH) continue;                             // wave-uniform
        const int row = (c % WCH) * 32 + (lane >> 1);
        const int lh = (lane & 1) ^ ((row >> 3) & 1);
        const int tap = row >> 6, co = row & 63;
        dma16(rw, TGP_LDS(smem + c * 1024), ((co * 9 + tap) * Cin + 8 * lh) * 2,
              (c / WCH) * 16 * 2);
      }
    }
  }
#pragma unroll
  for (int k = 0; k < NS - 1; ++k)
    if (k < total) {
      issue_part(k, 0, LW);
      issue_done();
    }

  int idx = 0;
  for (int c_it = 0; c_it < n_items; ++c_it) {
    int gi, n, h0, co0;
    coords(c_it, gi, n, h0, co0);
    // this lane's bias values for the epilogue, loaded up front: channel
    // co0 + 32 (half) + 8 g + 4 (l / 32) + e is bv[i][g][e], half = i (CH = 2)
    // or chf (CH = 1)
    f32x4_t bv[CH][4];
#pragma unroll
    for (int i = 0; i < CH; ++i)
#pragma unroll
      for (int g = 0; g < 4; ++g)
        bv[i][g] = bias ? *(const f32x4_t*)(bias + co0 + 32 * (i + chf) + 8 * g + 4 * (lane >> 5))
                        : f32x4_t{};
    f32x16_t acc[CH][FW];
#pragma unroll
    for (int i = 0; i < CH; ++i)
#pragma unroll
      for (int j = 0; j < FW; ++j) acc[i][j] = f32x16_t{};

    for (int ks = 0; ks < nk; ++ks, ++idx) {
      // loads complete in order: stage idx is in once at most the stages
      // issued after it are pending (epilogue stores only lengthen the wait)
      wait_ring(min(NS - 2, total - 1 - idx));
      ring_barrier();
      const bool fill = idx + NS - 1 < total;                   // refill the slot freed last stage
      const int fslot = (idx + NS - 1) % NS;
      const unsigned char* st = ring + (idx % NS) * SB;
      const unsigned char* sa = RK ? smem + ks * R32_AROWS * 32 : st;   // weights of this stage
      // nine taps; tap t + 1's fragments are read while tap t's MFMAs run
      bf16x8_t fa[2][CH], fb[2][FW];
      auto load = [&](int t, int buf) __attribute__((always_inline)) {
        const int r = t / 3, s = t - 3 * (t / 3);
#pragma unroll
        for (int i = 0; i < CH; ++i)
          fa[buf][i] = as_bf16x8(*(const u32x4*)(sa + abase + (t * 64 + 32 * i) * 32));
#pragma unroll
        for (int j = 0; j < FW; ++j)
          fb[buf][j] = as_bf16x8(*(const u32x4*)(st + bq[j][s] + r * BWP * 32));
      };
      load(0, 0);
      constexpr int NQ = CH * FW;                               // MFMAs per tap
#pragma unroll
      for (int t = 0; t < 9; ++t) {
        // reads for tap t + 1, half of tap t's MFMAs, this tap's share of the
        // next stage's DMA, the other half of the MFMAs
        if (t + 1 < 9) load(t + 1, (t + 1) & 1);
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int q = 0; q < NQ; ++q)
          if (q < NQ / 2)
            acc[q % CH][q / CH] = mfma32(fa[t & 1][q % CH], fb[t & 1][q / CH], acc[q % CH][q / CH]);
        __builtin_amdgcn_sched_barrier(0);
        if (fill) issue_part(fslot, t * LW / 9, (t + 1) * LW / 9);
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int q = 0; q < NQ; ++q)
          if (q >= NQ / 2)
            acc[q % CH][q / CH] = mfma32(fa[t & 1][q % CH], fb[t & 1][q / CH], acc[q % CH][q / CH]);
        __builtin_amdgcn_sched_barrier(0);
      }
      if (fill) issue_done();
    }

    // Epilogue, staged through LDS so that every store writes whole runs of
    // one pixel's channels (scattered 8-byte stores cost a memory-pipeline
    // cycle per lane).  The slot of the stage just consumed is free once
    // every wave is past its last MFMAs; its DMA refill is issued only after
    // the next stage's barrier.  Per fragment j each wave uses its own 4 KiB
    // (CH = 2: 32 pixel rows of 64 channels, 16-byte chunk c of row p at
    // position c ^ (p % 8)) or 2 KiB (CH = 1: rows of 32 channels, chunk c at
    // c ^ (p % 4)).  Element v of lane l of acc[i][j] is channel 32 (half) +
    // 8 (v / 4) + 4 (l / 32) + v % 4 of pixel l % 32.
    ring_barrier();
    constexpr int ROWB = 64 * CH;                               // staged bytes per pixel
    constexpr int NCK = 4 * CH;                                 // 16-byte chunks per pixel
    unsigned char* ep = ring + ((idx - 1) % NS) * SB + wave * 32 * ROWB;
    static_assert(NW * 32 * ROWB <= SB, "epilogue staging fits a slot");
    bf16_t* const Yg = pickg(io.y, gi);
    const long pix0 = (long)(n * H + h0) * W;
    const int pw = lane & 31, hw = lane >> 5;
#pragma unroll
    for (int j = 0; j < FW; ++j) {
#pragma unroll
      for (int i = 0; i < CH; ++i) {
#pragma unroll
        for (int g = 0; g < 4; ++g) {
          float v[4];
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            v[e] = acc[i][j][4 * g + e] + bv[i][g][e];
            if (relu) v[e] = fmaxf(v[e], 0.0f);
          }
          uint2 o;
          o.x = pack2_bf16(v[0], v[1]);
          o.y = pack2_bf16(v[2], v[3]);
          *(uint2*)(ep + pw * ROWB + (((4 * i + g) ^ (pw & (NCK - 1))) << 4) + 8 * hw) = o;
        }
      }
      constexpr int PPI = 64 / NCK;                             // pixels per read
#pragma unroll
      for (int q = 0; q < 32 / PPI; ++q) {
        const int p = lane / NCK + PPI * q, c = lane % NCK;
        const u32x4 val = *(const u32x4*)(ep + p * ROWB + ((c ^ (p & (NCK - 1))) << 4));
        const int tp = (pg * FW + j) * 32 + p;
        if (pg * FW + j < F && h0 + tp / W < H)
          *(u32x4*)(Yg + (pix0 + tp) * Cout + co0 + 32 * chf + 8 * c) = val;
      }
    }
  }
}

struct R32Cfg { int W, R, FW, NS, CH, RK; };
constexpr R32Cfg kR32Cfgs[] = {
    {192, 3, 5, 3, 2, 0}, {192, 1, 2, 4, 2, 0},
    {96, 6, 5, 3, 2, 0},  {96, 3, 3, 4, 2, 0},  {96, 2, 2, 4, 2, 0},
    {48, 12, 5, 3, 2, 0}, {48, 6, 3, 4, 2, 0},  {48, 4, 2, 4, 2, 0},
    {24, 24, 5, 3, 2, 0}, {24, 12, 3, 4, 2, 0}, {24, 8, 2, 4, 2, 0},
    // eight waves, two per SIMD
    {192, 3, 5, 3, 1, 0}, {96, 3, 3, 4, 1, 0}, {96, 2, 2, 4, 1, 0}, {48, 4, 2, 4, 1, 0},
    {24, 8, 2, 4, 1, 0},
    // eight waves, weights of 64 input channels resident (Cin = 64, Cout = 64)
    {192, 2, 3, 3, 1, 4}, {192, 3, 5, 2, 1, 4},
    // widths 64 and 32 (the 6-level U-Net's deeper levels)
    {64, 4, 2, 4, 1, 0}, {64, 6, 3, 3, 2, 0}, {32, 8, 2, 4, 1, 0}, {32, 12, 3, 3, 2, 0},
    // eight waves, twelve whole fragments per tile
    {48, 8, 3, 3, 1, 0}, {96, 4, 3, 3, 1, 0},
};
constexpr int kR32N = sizeof(kR32Cfgs) / sizeof(kR32Cfgs[0]);

}  // namespace

// Configuration for a per-sample shape and ng micro-batches per launch:
// among those for its width, the one with the fewest rounds of 256 tiles
// (for a nominal 4 ng samples) times fragments per wave, a four-wave
// configuration's fragments weighted 1.1 (measured: at equal rounds and
// fragments it runs about 10% slower than the eight-wave layout).  The
// summation order of every output is the same in all configurations, so
// the choice does not change values.  Returns an index into kR32Cfgs, or -1.
int g_rows32_cfg = -1;   // >= 0 forces a configuration (measurement only)
int g_rows32_ch = 0;     // 1 or 2: only that wave layout (measurement); 0: both

static int rows32_pick(const ConvShape& s, int ng = 1) {
  if (s.taps != 9 || s.cin % 16 || s.cout % 64) return -1;
  int best = -1;
  long best_cost = 0;
  for (int c = 0; c < kR32N; ++c) {
    const R32Cfg k = kR32Cfgs[c];
    if (k.W != s.W || k.R > s.H) continue;
    if (k.RK && (s.cin != 16 * k.RK || s.cout != 64)) continue;
    if (g_rows32_cfg < 0 && g_rows32_ch && k.CH != g_rows32_ch) continue;
    const long items = 4L * ng * ((s.H + k.R - 1) / k.R) * (s.cout / 64);
    const long cost = (items + 255) / 256 * k.FW * (k.RK ? 8 : (k.CH == 2 ? 11 : 10));
    if (g_rows32_cfg == c || (g_rows32_cfg < 0 && (best < 0 || cost < best_cost))) {
      best = c;
      best_cost = cost;
    }
  }
  return best;
}

// Tiles of one micro-batch in the configuration a single launch takes.
int conv_rows32_tiles(const ConvShape& s) {
  const int c = rows32_pick(s);
  if (c < 0) return 0;
  return s.nb * ((s.H + kR32Cfgs[c].R - 1) / kR32Cfgs[c].R) * (s.cout / 64);
}

bool conv_rows32_ok(const ConvShape& s) {
  return rows32_pick(s) >= 0 && (double)s.pixels() * s.cin * 2 < 2147483648.0 &&
         (double)s.cout * 9 * s.cin * 2 < 2147483648.0;
}

template <int W, int R, int FW, int NS, int CH, int RK>
static hipError_t launch_rows32(const R32Io& io, int ng, const bf16_t* Wt, const float* b,
                                const ConvShape& s, int relu, hipStream_t st) {
  static const char* name = nullptr;
  static char buf[64];
  if (!name) {
    snprintf(buf, sizeof buf, "conv3x3_rows32<%d,%d,%d,%d%s%s>", W, R, FW, NS,
             CH == 2 ? "" : ",8w", RK ? ",rk" : "");
    name = buf;
  }
  if (RK && (s.cin != 16 * RK || s.cout != 64)) return hipErrorInvalidValue;
  const long items = (long)ng * s.nb * ((s.H + R - 1) / R) * (s.cout / 64);
  const int G = (int)(items < 256 ? items : 256);
  if (G == 0) return hipSuccess;
  const long P = (long)ng * s.pixels();
  ProfScope ps(name, 2.0 * P * s.cout * 9 * s.cin,
               2.0 * ((double)P * s.cin + 9.0 * s.cin * s.cout + (double)P * s.cout), st);
  TGP_LAUNCH(ps, (conv3x3_rows32<W, R, FW, NS, CH, RK>), dim3(G), dim3(CH == 2 ? 256 : 512), 0, st,
             io, ng, Wt, b, s.nb, s.H, s.cin, s.cout, relu);
  return launch_status();
}

hipError_t conv_forward_rows32(int n, const void* const* x, const void* w, const float* b,
                               void* const* y, const ConvShape& s, int relu, hipStream_t st) {
  if (n < 1 || n > kMaxGroup) return hipErrorInvalidValue;
  if (n > kR32Group) {
    for (int k0 = 0; k0 < n; k0 += kR32Group) {
      const int c = n - k0 < kR32Group ? n - k0 : kR32Group;
      const hipError_t e = conv_forward_rows32(c, x + k0, w, b, y + k0, s, relu, st);
      if (e != hipSuccess) return e;
    }
    return hipSuccess;
  }
  const int c = rows32_pick(s, n);
  if (c < 0 || !conv_rows32_ok(s)) return hipErrorInvalidValue;
  R32Io io{};
  for (int k = 0; k < kR32Group; ++k) {   // unused entries repeat micro-batch 0
    io.x[k] = (const bf16_t*)x[k < n ? k : 0];
    io.y[k] = (bf16_t*)y[k < n ? k : 0];
    if (!io.x[k] || !io.y[k]) return hipErrorInvalidValue;
  }
  const bf16_t* Wt = (const bf16_t*)w;
  switch (c) {
#define R32_CASE(i)                                                                      \
  case i:                                                                                \
    return launch_rows32<kR32Cfgs[i].W, kR32Cfgs[i].R, kR32Cfgs[i].FW, kR32Cfgs[i].NS,   \
                         kR32Cfgs[i].CH, kR32Cfgs[i].RK>(io, n, Wt, b, s, relu, st);
    R32_CASE(0) R32_CASE(1) R32_CASE(2) R32_CASE(3) R32_CASE(4) R32_CASE(5)
    R32_CASE(6) R32_CASE(7) R32_CASE(8) R32_CASE(9) R32_CASE(10) R32_CASE(11)
    R32_CASE(12) R32_CASE(13) R32_CASE(14) R32_CASE(15) R32_CASE(16) R32_CASE(17)
    R32_CASE(18) R32_CASE(19) R32_CASE(20) R32_CASE(21) R32_CASE(22) R32_CASE(23)
#undef R32_CASE
    default: return hipErrorInvalidValue;
  }
}

}  // namespace tgpk
