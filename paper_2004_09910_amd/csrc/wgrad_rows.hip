// bf16 3x3 weight gradient on 32 x 32 x 16 MFMA, operands read from LDS
// with the gfx950 transpose loads.
//
// dW[co][r][s][ci] = sum_p dZ[p][co] X[p + (r - 1) W + (s - 1)][ci]: a GEMM
// with M = co, N = ci, K = pixels, one per tap.  Both operands live in
// NHWC, where a pixel's channels are contiguous but an MFMA fragment needs
// 8 consecutive pixels of one channel; ds_read_b64_tr_b16 gathers exactly
// that from pixel-major LDS rows, so the tiles go global -> LDS by buffer
// DMA and are never transposed in registers.
//
// A work item is (K range, filter row r, 64 output channels, 64 input
// channels): it accumulates the three column taps s = 0..2 of filter row r
// over the K range, a block of whole image rows of one sample.  A stage
// holds RPS image rows h.. of dZ (RPS W pixels) and the RPS input rows
// h + r - 1.. each padded with a zero pixel on either side (in a block of
// W + 4 LDS rows, so every block starts at a multiple of 4 rows), so tap s
// of pixel (h, w) reads padded row w + s; the padding pixels and rows outside the image are
// buffer reads at out-of-range offsets and hold zeros.  Rows are 64 channels
// (128 bytes) with their 16-byte chunks XOR-swizzled by 2 (row & 3), which
// keeps the transpose reads of four consecutive rows on distinct banks.
//
// Each wave owns a 32 x 32 (co x ci) quarter of the item for all three
// taps.  Blocks are persistent over items, their stages streamed through
// one NS-deep LDS ring.  Each item writes its fp32 partial dW slice for its
// K range; the slices are summed in K-range order by splitk_reduce (or, with
// one K range, the item writes dW directly).  The summation order is fixed
// by the shape.
#include "common.h"
#include "kernels.h"
#include "mfma_util.h"
#include "prof.h"

namespace tgpk {
namespace {

constexpr int WG_OOB = (int)0x80000000;

typedef short s16x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) s16x4 lds_s16x4;

// Transpose read: within each group of 16 lanes, lane i receives element
// i % 4 of the 8-byte blocks addressed by lanes 4 e + i / 4, e = 0..3.
__device__ __forceinline__ s16x4 tr16(const unsigned char* p) {
  return __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4*)TGP_LDS(p));
}

__device__ __forceinline__ bf16x8_t frag2(s16x4 lo, s16x4 hi) {
  const u32x4 v = {__builtin_bit_cast(unsigned, (short __attribute__((ext_vector_type(2)))){lo[0], lo[1]}),
                   __builtin_bit_cast(unsigned, (short __attribute__((ext_vector_type(2)))){lo[2], lo[3]}),
                   __builtin_bit_cast(unsigned, (short __attribute__((ext_vector_type(2)))){hi[0], hi[1]}),
                   __builtin_bit_cast(unsigned, (short __attribute__((ext_vector_type(2)))){hi[2], hi[3]})};
  return as_bf16x8(v);
}

constexpr int round32(int v) { return (v + 31) / 32 * 32; }

// Barrier after LDS writes (or before LDS writes over data) that other waves
// of the block read (or wrote) on the other side: this wave's LDS accesses
// have completed when it arrives, and the compiler moves none across it.
__device__ __forceinline__ void lds_handoff_barrier() {
  asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
}

// The micro-batches of one launch (ng of them, nb samples each): the K
// ranges of micro-batch k follow those of k - 1 and its slices go to
// out[k], so one launch covers them all.
// At most eight per launch (a larger group runs as launches of eight).
constexpr int kWgGroup = 8;
struct WgIo {
  const bf16_t* x[kWgGroup];
  const bf16_t* dz[kWgGroup];
  float* out[kWgGroup];
};
//
// KS is the number of waves per SIMD: with KS = 2 the two waves of a SIMD
// own the same 32 x 32 quarter and take alternate k steps, and the second's
// sums are added to the first's through LDS before the store, so one wave's
// MFMAs run while the other waits on its DMA issue or LDS reads.  With
// KS = 3 the three take every third k step, all of them issue DMA, and the
// first adds the second's and then the third's sums before storing.
template <int W, int RPS, int NS, int KS>
__global__ __launch_bounds__(256 * KS) void conv_wgrad_rows(WgIo io, int ng, int nb, int H,
                                                            int Cin, int Cout, int R) {
  constexpr int AR = round32(RPS * W);          // dZ rows per stage
  constexpr int BW = W + 4;                     // LDS rows per padded input row
  constexpr int BR = round32(RPS * BW);         // padded X rows per stage
  constexpr int SB = (AR + BR) * 128;           // stage bytes
  constexpr int NW = 4 * KS;                    // waves
  constexpr int AC = AR / 8, BC = BR / 8;       // DMA chunks (8 rows, 1 KiB) per region
  // With KS = 2 only the four waves of phase 1 issue the DMA (each twice
  // its share): an issuing wave stalls while the memory pipeline is full,
  // and meanwhile its SIMD's phase-0 wave keeps the MFMAs busy.
  constexpr int ND = KS == 2 ? 4 : NW;          // waves that issue the DMA
  constexpr int LA = (AC + ND - 1) / ND, LB = (BC + ND - 1) / ND;   // per issuing wave, at most
  constexpr int KT = RPS * W / 16;               // k steps per stage
  static_assert(RPS * W % 16 == 0 && W % 8 == 0, "k steps of 16 pixels, halves within a row");
  static_assert(KT % KS == 0, "k steps shared evenly");
  static_assert(NW * 2048 <= SB && (KS != 3 || 8 * 4096 <= SB), "exchange of the sums fits a slot");
  __shared__ __attribute__((aligned(16))) unsigned char smem[NS * SB];

  // the wave index is uniform: readfirstlane lets the compiler branch on it
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int qw = wave & 3, kh = wave >> 2;      // quarter of the item, k-step phase
  const int cw = qw >> 1, nw = qw & 1;          // this wave's co / ci halves
  const int nct = Cout / 64, ncit = Cin / 64;
  // R = 0: one K range per micro-batch spanning all nb samples' whole
  // images (sample-major stages, each stage within one sample)
  const bool merged = R == 0;
  const int nrb = merged ? 1 : (H + R - 1) / R;
  const int kpg = merged ? 1 : nb * nrb;          // K ranges per micro-batch
  const int sps = (H + RPS - 1) / RPS;            // stages per sample image (merged)
  const int per_k = 3 * nct * ncit;             // items per K range
  const int items = ng * kpg * per_k;
  const int G = gridDim.x;
  const int lb = xcd_remap(blockIdx.x, G);
  const int n_items = lb < items ? (items - lb + G - 1) / G : 0;
  const long E = (long)Cout * 9 * Cin;

  const int zbytes = nb * H * W * Cout * 2, xbytes = nb * H * W * Cin * 2;

  // DMA lane constants: instruction u of issuing wave d fills chunk c = ND u
  // + d of the A (dZ) or B (padded X) region, rows 8 c + lane / 8, physical
  // chunk lane % 8, which holds logical chunk (lane % 8) ^ (2 (row & 3)).
  // Chunks past a region's end are not issued (wave-uniform).
  const int dwi = KS == 2 ? qw : wave;          // index among the issuing waves
  const bool issuer = KS != 2 || kh == 1;
  int aoff[LA], arow[LA], boff[LB], brow[LB];
#pragma unroll
  for (int u = 0; u < LA; ++u) {
    const int row = (ND * u + dwi) * 8 + (lane >> 3);
    const int lc = (lane & 7) ^ (2 * (row & 3));
    const int rr = row / W, w = row - rr * W;
    const bool ok = row < RPS * W;
    aoff[u] = ok ? ((rr * W + w) * Cout + 8 * lc) * 2 : WG_OOB;
    arow[u] = ok ? rr : -1;
  }
#pragma unroll
  for (int u = 0; u < LB; ++u) {
    const int row = (ND * u + dwi) * 8 + (lane >> 3);
    const int lc = (lane & 7) ^ (2 * (row & 3));
    const int rr = row / BW, q = row - rr * BW;
    const bool ok = rr < RPS && q >= 1 && q <= W;
    boff[u] = ok ? ((rr * W + q - 1) * Cin + 8 * lc) * 2 : WG_OOB;
    brow[u] = ok ? rr : -1;
  }
  // DMA instructions an issuing wave issues per stage (the waits count
  // them); the other waves find the stage complete after the ring barrier,
  // which the issuers reach only once their loads have landed
  const int na = (AC - dwi + ND - 1) / ND, nbq = (BC - dwi + ND - 1) / ND;
  const int mine = na + nbq;
  auto wait_ring = [&](int ahead) __attribute__((always_inline)) {
    if (!issuer) return;
    if constexpr (AC % ND == 0 && BC % ND == 0) {
      wait_stages<NS, LA + LB>(ahead);
    } else {
      if (mine == LA + LB) wait_stages<NS, LA + LB>(ahead);
      else if (mine == LA + LB - 1) wait_stages<NS, LA + LB - 1>(ahead);
      else wait_stages<NS, LA + LB - 2>(ahead);
    }
  };

  // Fragment lane constants (byte offsets in a stage).  Lane group g = lane /
  // 16 holds MFMA rows / columns 16 (g % 2) .. + 15 and k 8 (g / 2) .. + 7;
  // lane j = lane % 16 addresses pixel k + j / 4, channels + 4 (j % 4).
  const int g = lane >> 4, j = lane & 15;
  const int kb = 8 * (g >> 1) + (j >> 2);
  const int cha = (cw * 32 + 16 * (g & 1) + 4 * (j & 3)) * 2;   // byte within a row
  const int chb = (nw * 32 + 16 * (g & 1) + 4 * (j & 3)) * 2;
  const int fa = kb * 128 + (((cha >> 4) ^ (2 * (kb & 3))) << 4) + (cha & 15);
  int fb[3];
#pragma unroll
  for (int s = 0; s < 3; ++s)
    fb[s] = AR * 128 + (kb + s) * 128 + (((chb >> 4) ^ (2 * ((kb + s) & 3))) << 4) + (chb & 15);
  // k step t covers stage pixels 16 t .. + 15; this lane group's 8 of them,
  // 16 t + 8 (g / 2) .., lie in stage row rr = (16 t + 8 (g / 2)) / W, whose
  // padded X block starts 4 rr rows after its pixels' own index (the B row
  // of pixel q at column tap s is q + 4 rr + s).  With W a multiple of 16 the
  // row is the same for the whole step and the offset is an immediate.
  auto xoff = [&](int t) __attribute__((always_inline)) {
    if constexpr (W % 16 == 0) return (16 * t + 4 * ((16 * t) / W)) * 128;
    else return (16 * t + 4 * ((16 * t + 8 * (g >> 1)) / W)) * 128;
  };

  auto coords = [&](int it, int& kr, int& r, int& co0, int& ci0) __attribute__((always_inline)) {
    const int item = lb + it * G;
    kr = item / per_k;
    int t = item - kr * per_k;
    r = t / (nct * ncit);
    t -= r * nct * ncit;
    co0 = (t / ncit) * 64;
    ci0 = (t % ncit) * 64;
  };
  auto stages_of = [&](int kr) __attribute__((always_inline)) {
    if (merged) return nb * sps;
    const int rb = kr % nrb;
    const int rows = min(R, H - rb * R);
    return (rows + RPS - 1) / RPS;
  };

  // issue side; the issuing item's micro-batch gi (K range krl within it)
  int i_it = 0, i_st = 0, i_kr = 0, i_r = 0, i_co0 = 0, i_ci0 = 0, i_ns = 0, i_krl = 0;
  u32x4 rzg = {}, rxg = {};
  auto issue_item = [&]() __attribute__((always_inline)) {
    i_ns = stages_of(i_kr);
    const int gi = i_kr / kpg;
    i_krl = i_kr - gi * kpg;
    rzg = make_rsrc(pickg(io.dz, gi), zbytes);
    rxg = make_rsrc(pickg(io.x, gi), xbytes);
  };
  if (n_items > 0) {
    coords(0, i_kr, i_r, i_co0, i_ci0);
    issue_item();
  }
  // A stage's DMA is issued all at once, right after the ring barrier of
  // the stage NS - 1 before it.  (Spread over the k steps between the
  // MFMAs, the memory pipeline's issue stalls held up the MFMAs: 25 to 60%
  // slower.)
  auto issue = [&](int slot) __attribute__((always_inline)) {
    const int krl = i_krl;
    const int n = merged ? i_st / sps : krl / nrb;
    const int h = merged ? (i_st - (i_st / sps) * sps) * RPS
                         : (krl - (krl / nrb) * nrb) * R + i_st * RPS;   // first image row
    const int zsoff = (((n * H + h) * W) * Cout + i_co0) * 2;
    const int hb = h + i_r - 1;                              // input row of stage row 0
    const int xsoff = (((n * H + hb) * W) * Cin + i_ci0) * 2;
#pragma unroll
    for (int u = 0; u < LA; ++u) {
      const int c = ND * u + dwi;
      if (!issuer || (AC % ND != 0 && c >= AC)) continue;   // wave-uniform
      auto* dst = TGP_LDS(smem + slot * SB + c * 1024);
      const bool ok = arow[u] >= 0 && h + arow[u] < H;
      dma16(rzg, dst, ok ? aoff[u] + zsoff : WG_OOB, 0);
    }
#pragma unroll
    for (int u = 0; u < LB; ++u) {
      const int c = ND * u + dwi;
      if (!issuer || (BC % ND != 0 && c >= BC)) continue;   // wave-uniform
      auto* dst = TGP_LDS(smem + slot * SB + AR * 128 + c * 1024);
      const bool ok = brow[u] >= 0 && (unsigned)(hb + brow[u]) < (unsigned)H && h + brow[u] < H;
      // the row offset can be negative for filter row 0 (rows above are out
      // of range there), so it goes into the per-lane offset
      dma16(rxg, dst, ok ? boff[u] + xsoff : WG_OOB, 0);
    }
    if (++i_st == i_ns) {
      i_st = 0;
      if (++i_it < n_items) {
        coords(i_it, i_kr, i_r, i_co0, i_ci0);
        issue_item();
      }
    }
  };

  // total stages of this block
  int total = 0;
  for (int it = 0; it < n_items; ++it) {
    int kr, r, co0, ci0;
    coords(it, kr, r, co0, ci0);
    total += stages_of(kr);
  }

#pragma unroll
  for (int k = 0; k < NS - 1; ++k)
    if (k < total) issue(k);

  int idx = 0;
  for (int c_it = 0; c_it < n_items; ++c_it) {
    int kr, r, co0, ci0;
    coords(c_it, kr, r, co0, ci0);
    const int ns = stages_of(kr);
    f32x16_t acc[3] = {f32x16_t{}, f32x16_t{}, f32x16_t{}};
    for (int st = 0; st < ns; ++st, ++idx) {
      // loads complete in order: stage idx is in once at most the stages
      // issued after it are pending (epilogue stores only lengthen this wait)
      wait_ring(min(NS - 2, total - 1 - idx));
      ring_barrier();
      if (idx + NS - 1 < total) issue((idx + NS - 1) % NS);   // the slot freed last stage
      const unsigned char* sp = smem + (idx % NS) * SB;
      // k step t: stage pixels 16 t .. 16 t + 15 (dZ rows are the pixel
      // index); with KS = 2 this wave takes every other step.  Step tt + 1's
      // fragments are read while step tt's MFMAs run (left to itself the
      // compiler waited for each MFMA's own reads right before it).
      constexpr int NT = KT / KS;                               // this wave's k steps
      bf16x8_t a[2], b[2][3];
      auto load = [&](int tt, int buf) __attribute__((always_inline)) {
        const int t = KS * tt + (KS == 1 ? 0 : kh);
        const int ka = 16 * t * 128;
        int kx;
        if constexpr (KS == 1) kx = xoff(t);
        else if constexpr (KS == 2) kx = kh ? xoff(KS * tt + 1) : xoff(KS * tt);
        else kx = xoff(KS * tt + kh);
        a[buf] = frag2(tr16(sp + fa + ka), tr16(sp + fa + ka + 4 * 128));
#pragma unroll
        for (int s = 0; s < 3; ++s)
          b[buf][s] = frag2(tr16(sp + fb[s] + kx), tr16(sp + fb[s] + kx + 4 * 128));
      };
      load(0, 0);
#pragma unroll
      for (int tt = 0; tt < NT; ++tt) {
        if (tt + 1 < NT) load(tt + 1, (tt + 1) & 1);
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int s = 0; s < 3; ++s) acc[s] = mfma32(a[tt & 1], b[tt & 1][s], acc[s]);
        __builtin_amdgcn_sched_barrier(0);
      }
    }
    if constexpr (KS == 2) {
      // the two waves of a SIMD swap halves of their sums through the slot
      // just consumed (free once every wave is past its last MFMAs; its
      // refill is issued only after the next stage's barrier): wave kh keeps
      // elements 8 kh .. 8 kh + 7 of each tap and adds the partner's.  The
      // sum is the same from either side, so the order is fixed.  2 KiB per
      // wave per tap, 16-byte chunk c of lane l at c * 64 + l.
      f32x4_t* xo = (f32x4_t*)(smem + ((idx - 1) % NS) * SB) + wave * 128 + lane;
      const f32x4_t* xi = (const f32x4_t*)(smem + ((idx - 1) % NS) * SB) + (wave ^ 4) * 128 + lane;
#pragma unroll
      for (int s = 0; s < 3; ++s) {
        lds_handoff_barrier();
        if (kh) {
          xo[0] = f32x4_t{acc[s][0], acc[s][1], acc[s][2], acc[s][3]};
          xo[64] = f32x4_t{acc[s][4], acc[s][5], acc[s][6], acc[s][7]};
        } else {
          xo[0] = f32x4_t{acc[s][8], acc[s][9], acc[s][10], acc[s][11]};
          xo[64] = f32x4_t{acc[s][12], acc[s][13], acc[s][14], acc[s][15]};
        }
        lds_handoff_barrier();
        const f32x4_t v0 = xi[0], v1 = xi[64];
        if (kh) {
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            acc[s][8 + e] += v0[e];
            acc[s][12 + e] += v1[e];
          }
        } else {
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            acc[s][e] += v0[e];
            acc[s][4 + e] += v1[e];
          }
        }
      }
      // the exchange reads are done before the slot's refill is issued
      asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
    }
    if constexpr (KS == 3) {
      // waves kh = 1, 2 of a quarter pass their sums to wave 0 through the
      // slot just consumed (4 KiB per wave and tap), which adds them in the
      // order kh = 1, 2
      f32x4_t* xs = (f32x4_t*)(smem + ((idx - 1) % NS) * SB);
#pragma unroll
      for (int s = 0; s < 3; ++s) {
        lds_handoff_barrier();
        if (kh) {
#pragma unroll
          for (int c = 0; c < 4; ++c)
            xs[((kh - 1) * 4 + qw) * 256 + c * 64 + lane] =
                f32x4_t{acc[s][4 * c], acc[s][4 * c + 1], acc[s][4 * c + 2], acc[s][4 * c + 3]};
        }
        lds_handoff_barrier();
        if (!kh) {
#pragma unroll
          for (int p2 = 0; p2 < 2; ++p2)
#pragma unroll
            for (int c = 0; c < 4; ++c) {
              const f32x4_t v = xs[(p2 * 4 + qw) * 256 + c * 64 + lane];
#pragma unroll
              for (int e = 0; e < 4; ++e) acc[s][4 * c + e] += v[e];
            }
        }
      }
      asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
    }
    // epilogue: element v of lane l is co 8 (v / 4) + 4 (l / 32) + v % 4, ci
    // l % 32 of this wave's quarter; with KS = 2 wave kh stores v = 8 kh ..
    // 8 kh + 7
    const int gi = kr / kpg;
    float* o = pickg(io.out, gi) + (long)(kr - gi * kpg) * E;
    const int ci = ci0 + nw * 32 + (lane & 31);
    auto store = [&](int v0, int v1) __attribute__((always_inline)) {
#pragma unroll
      for (int s = 0; s < 3; ++s)
#pragma unroll
        for (int v = v0; v < v1; ++v) {
          const int co = co0 + cw * 32 + 8 * (v >> 2) + 4 * (lane >> 5) + (v & 3);
          o[((long)co * 9 + 3 * r + s) * Cin + ci] = acc[s][v];
        }
    };
    if (KS == 1 || (KS == 3 && kh == 0)) store(0, 16);
    else if (KS == 2 && kh) store(8, 16);
    else if (KS == 2) store(0, 8);
  }
}

// The same weight gradient with all three filter rows in one item.  The
// twelve waves of a block are (filter row fr = w / 4, quarter w % 4), three
// per SIMD, so a stage holds the RPS dZ rows once and the RPS + 2 input rows
// h - 1 .. h + RPS that the three filter rows read (filter row fr of stage
// row t reads input block t + fr, an immediate offset).  A stage moves
// RPS W + (RPS + 2)(W + 4) LDS rows for three filter rows, where the kernel
// above moves RPS W + RPS (W + 4) for one, and every wave issues its share
// of the DMA while the two others on its SIMD run MFMAs.  Each wave sums
// its k steps in order, as the kernel above does with one wave per SIMD.
template <int W, int RPS, int NS>
__global__ __launch_bounds__(768) void conv_wgrad_rows3(WgIo io, int ng, int nb, int H, int Cin,
                                                        int Cout, int R) {
  constexpr int AR = round32(RPS * W);          // dZ rows per stage
  constexpr int BW = W + 4;                     // LDS rows per padded input row
  constexpr int BR = round32((RPS + 2) * BW);   // padded X rows per stage
  constexpr int SB = (AR + BR) * 128;           // stage bytes
  constexpr int NW = 12;                        // waves
  constexpr int AC = AR / 8, BC = BR / 8;       // DMA chunks (8 rows, 1 KiB) per region
  constexpr int LA = (AC + NW - 1) / NW, LB = (BC + NW - 1) / NW;   // per wave, at most
  constexpr int KT = RPS * W / 16;              // k steps per stage
  static_assert(RPS * W % 16 == 0 && W % 8 == 0, "k steps of 16 pixels, halves within a row");
  static_assert(NS * SB <= 160 * 1024, "LDS ring");
  static_assert((NS - 2) * (LA + LB) < 64, "vmcnt range");
  __shared__ __attribute__((aligned(16))) unsigned char smem[NS * SB];

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int qw = wave & 3, fr = wave >> 2;      // quarter of the item, filter row
  const int cw = qw >> 1, nw = qw & 1;          // this wave's co / ci halves
  const int nct = Cout / 64, ncit = Cin / 64;
  const bool merged = R == 0;
  const int nrb = merged ? 1 : (H + R - 1) / R;
  const int kpg = merged ? 1 : nb * nrb;          // K ranges per micro-batch
  const int sps = (H + RPS - 1) / RPS;            // stages per sample image (merged)
  const int per_k = nct * ncit;                   // items per K range
  const int items = ng * kpg * per_k;
  const int G = gridDim.x;
  const int lb = xcd_remap(blockIdx.x, G);
  const int n_items = lb < items ? (items - lb + G - 1) / G : 0;
  const long E = (long)Cout * 9 * Cin;

  const int zbytes = nb * H * W * Cout * 2, xbytes = nb * H * W * Cin * 2;

  // DMA lane constants: instruction u of wave w fills chunk c = NW u + w of
  // the A (dZ) or B (padded X) region, as in the kernel above.  B block rr
  // of a stage is input row h - 1 + rr.
  int aoff[LA], arow[LA], boff[LB], brow[LB];
#pragma unroll
  for (int u = 0; u < LA; ++u) {
    const int row = (NW * u + wave) * 8 + (lane >> 3);
    const int lc = (lane & 7) ^ (2 * (row & 3));
    const int rr = row / W, w = row - rr * W;
    const bool ok = row < RPS * W;
    aoff[u] = ok ? ((rr * W + w) * Cout + 8 * lc) * 2 : WG_OOB;
    arow[u] = ok ? rr : -1;
  }
#pragma unroll
  for (int u = 0; u < LB; ++u) {
    const int row = (NW * u + wave) * 8 + (lane >> 3);
    const int lc = (lane & 7) ^ (2 * (row & 3));
    const int rr = row / BW, q = row - rr * BW;
    const bool ok = rr < RPS + 2 && q >= 1 && q <= W;
    boff[u] = ok ? ((rr * W + q - 1) * Cin + 8 * lc) * 2 : WG_OOB;
    brow[u] = ok ? rr : -1;
  }
  // DMA instructions this wave issues per stage (the waits count them)
  const int na = (AC - wave + NW - 1) / NW, nbq = (BC - wave + NW - 1) / NW;
  const int mine = na + nbq;
  auto wait_ring = [&](int ahead) __attribute__((always_inline)) {
    if constexpr (AC % NW == 0 && BC % NW == 0) {
      wait_stages<NS, LA + LB>(ahead);
    } else {
      if (mine == LA + LB) wait_stages<NS, LA + LB>(ahead);
      else if (mine == LA + LB - 1) wait_stages<NS, LA + LB - 1>(ahead);
      else wait_stages<NS, LA + LB - 2>(ahead);
    }
  };

  // Fragment lane constants, as in the kernel above; filter row fr's input
  // blocks start fr blocks further on.
  const int g = lane >> 4, j = lane & 15;
  const int kb = 8 * (g >> 1) + (j >> 2);
  const int cha = (cw * 32 + 16 * (g & 1) + 4 * (j & 3)) * 2;
  const int chb = (nw * 32 + 16 * (g & 1) + 4 * (j & 3)) * 2;
  const int fa = kb * 128 + (((cha >> 4) ^ (2 * (kb & 3))) << 4) + (cha & 15);
  int fb[3];
#pragma unroll
  for (int s = 0; s < 3; ++s)
    fb[s] = AR * 128 + fr * BW * 128 + (kb + s) * 128 +
            (((chb >> 4) ^ (2 * ((kb + s) & 3))) << 4) + (chb & 15);
  auto xoff = [&](int t) __attribute__((always_inline)) {
    if constexpr (W % 16 == 0) return (16 * t + 4 * ((16 * t) / W)) * 128;
    else return (16 * t + 4 * ((16 * t + 8 * (g >> 1)) / W)) * 128;
  };

  auto coords = [&](int it, int& kr, int& co0, int& ci0) __attribute__((always_inline)) {
    const int item = lb + it * G;
    kr = item / per_k;
    const int t = item - kr * per_k;
    co0 = (t / ncit) * 64;
    ci0 = (t % ncit) * 64;
  };
  auto stages_of = [&](int kr) __attribute__((always_inline)) {
    if (merged) return nb * sps;
    const int rb = kr % nrb;
    const int rows = min(R, H - rb * R);
    return (rows + RPS - 1) / RPS;
  };

  int i_it = 0, i_st = 0, i_kr = 0, i_co0 = 0, i_ci0 = 0, i_ns = 0, i_krl = 0;
  u32x4 rzg = {}, rxg = {};
  auto issue_item = [&]() __attribute__((always_inline)) {
    i_ns = stages_of(i_kr);
    const int gi = i_kr / kpg;
    i_krl = i_kr - gi * kpg;
    rzg = make_rsrc(pickg(io.dz, gi), zbytes);
    rxg = make_rsrc(pickg(io.x, gi), xbytes);
  };
  if (n_items > 0) {
    coords(0, i_kr, i_co0, i_ci0);
    issue_item();
  }
  auto issue = [&](int slot) __attribute__((always_inline)) {
    const int krl = i_krl;
    const int n = merged ? i_st / sps : krl / nrb;
    const int h = merged ? (i_st - (i_st / sps) * sps) * RPS
                         : (krl - (krl / nrb) * nrb) * R + i_st * RPS;   // first image row
    const int zsoff = (((n * H + h) * W) * Cout + i_co0) * 2;
    const int hb = h - 1;                                    // input row of B block 0
    const int xsoff = (((n * H + hb) * W) * Cin + i_ci0) * 2;
#pragma unroll
    for (int u = 0; u < LA; ++u) {
      const int c = NW * u + wave;
      if (AC % NW != 0 && c >= AC) continue;                 // wave-uniform
      auto* dst = TGP_LDS(smem + slot * SB + c * 1024);
      const bool ok = arow[u] >= 0 && h + arow[u] < H;
      dma16(rzg, dst, ok ? aoff[u] + zsoff : WG_OOB, 0);
    }
#pragma unroll
    for (int u = 0; u < LB; ++u) {
      const int c = NW * u + wave;
      if (BC % NW != 0 && c >= BC) continue;                 // wave-uniform
      auto* dst = TGP_LDS(smem + slot * SB + AR * 128 + c * 1024);
      // rows outside the sample's image (above it for h = 0) read zeros; the
      // row offset can be negative, so it goes into the per-lane offset
      const bool ok = brow[u] >= 0 && (unsigned)(hb + brow[u]) < (unsigned)H;
      dma16(rxg, dst, ok ? boff[u] + xsoff : WG_OOB, 0);
    }
    if (++i_st == i_ns) {
      i_st = 0;
      if (++i_it < n_items) {
        coords(i_it, i_kr, i_co0, i_ci0);
        issue_item();
      }
    }
  };

  int total = 0;
  for (int it = 0; it < n_items; ++it) {
    int kr, co0, ci0;
    coords(it, kr, co0, ci0);
    total += stages_of(kr);
  }

#pragma unroll
  for (int k = 0; k < NS - 1; ++k)
    if (k < total) issue(k);

  int idx = 0;
  for (int c_it = 0; c_it < n_items; ++c_it) {
    int kr, co0, ci0;
    coords(c_it, kr, co0, ci0);
    const int ns = stages_of(kr);
    f32x16_t acc[3] = {f32x16_t{}, f32x16_t{}, f32x16_t{}};
    for (int st = 0; st < ns; ++st, ++idx) {
      wait_ring(min(NS - 2, total - 1 - idx));
      ring_barrier();
      if (idx + NS - 1 < total) issue((idx + NS - 1) % NS);   // the slot freed last stage
      const unsigned char* sp = smem + (idx % NS) * SB;
      bf16x8_t a[2], b[2][3];
      auto load = [&](int t, int buf) __attribute__((always_inline)) {
        const int ka = 16 * t * 128;
        const int kx = xoff(t);
        a[buf] = frag2(tr16(sp + fa + ka), tr16(sp + fa + ka + 4 * 128));
#pragma unroll
        for (int s = 0; s < 3; ++s)
          b[buf][s] = frag2(tr16(sp + fb[s] + kx), tr16(sp + fb[s] + kx + 4 * 128));
      };
      load(0, 0);
#pragma unroll
      for (int tt = 0; tt < KT; ++tt) {
        if (tt + 1 < KT) load(tt + 1, (tt + 1) & 1);
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int s = 0; s < 3; ++s) acc[s] = mfma32(a[tt & 1], b[tt & 1][s], acc[s]);
        __builtin_amdgcn_sched_barrier(0);
      }
    }
    // epilogue: element v of lane l is co 8 (v / 4) + 4 (l / 32) + v % 4, ci
    // l % 32 of this wave's quarter, tap (fr, s)
    const int gi = kr / kpg;
    float* o = pickg(io.out, gi) + (long)(kr - gi * kpg) * E;
    const int ci = ci0 + nw * 32 + (lane & 31);
#pragma unroll
    for (int s = 0; s < 3; ++s)
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        const int co = co0 + cw * 32 + 8 * (v >> 2) + 4 * (lane >> 5) + (v & 3);
        o[((long)co * 9 + 3 * fr + s) * Cin + ci] = acc[s][v];
      }
  }
}

struct WgPlan { int R, nK; };   // image rows per K range (0: whole micro-batch), K ranges

}  // namespace

// Image rows per stage and ring depth per width: stages of 128 to 256
// pixels, ring within the 160 KiB of LDS.
struct WgCfg { int W, RPS, NS; };
constexpr WgCfg kWgCfgs[] = {{256, 1, 2}, {192, 1, 3}, {128, 1, 4}, {96, 2, 3}, {64, 3, 3},
                             {48, 4, 3},  {32, 6, 3},  {24, 4, 5},  {16, 8, 4}, {8, 8, 4}};
static_assert(sizeof(kWgCfgs) / sizeof(kWgCfgs[0]) == 10, "one launch case per width");

static int wgrad_rows_rps(int W) {
  for (const WgCfg& c : kWgCfgs)
    if (c.W == W) return c.RPS;
  return 0;
}

// Rows per K range: the fewest (a multiple of the rows per stage) that keep
// one micro-batch's item count within 128 for micro-batches of four or more
// samples, so that a launch over two micro-batches fills one round of 256
// blocks, and within 256 for smaller ones, which the pipelined schedule
// launches one at a time.  (Measured: on the U-Net stage at four samples a
// bound of 256 writes twice the partial slices and was 2.5% slower per
// step, 192 leaves 1.5 rounds; on the 6-level network at two samples, one
// micro-batch per launch, 128 halved the weight gradient's rate at widths
// 256 and 128.)
static WgPlan wgrad_rows_plan(const ConvShape& s) {
  const long per_k = 3L * (s.cout / 64) * (s.cin / 64);
  const int rps = wgrad_rows_rps(s.W);
  int R = rps;
  const long cap = s.nb >= 4 ? 128 : 256;
  while (R < s.H && (long)s.nb * ((s.H + R - 1) / R) * per_k > cap) R += rps;
  if (R > s.H) R = s.H;
  // Deep layers whose items fill the chip even with one K range per
  // micro-batch: let it span all samples (R = 0), so the kernel writes the
  // gradient itself and no partial slices are written or summed.  From four
  // samples on, 64 items per micro-batch are enough: a launch over four
  // micro-batches then fills a round of blocks (on the U-Net stage the
  // 256 -> 512 layer at 24 x 24 drops 19 MB of partial slices per
  // micro-batch, 0.7% of the step; a launch over one micro-batch runs on
  // fewer blocks).
  if (R == s.H && s.nb > 1 && (per_k >= 128 || (s.nb >= 4 && per_k >= 64))) return {0, 1};
  return {R, s.nb * ((s.H + R - 1) / R)};
}

// waves per SIMD of the row-blocked weight gradient (0: chosen by width)
int g_wgrad_ks = 0;

bool wgrad_rows_ok(const ConvShape& s) {
  return s.taps == 9 && wgrad_rows_rps(s.W) > 0 && s.cin % 64 == 0 &&
         s.cout % 64 == 0 && (double)s.pixels() * (s.cin > s.cout ? s.cin : s.cout) * 2 < 2147483648.0;
}

size_t wgrad_rows_partial_floats(const ConvShape& s) {
  const WgPlan p = wgrad_rows_plan(s);
  return p.nK > 1 ? (size_t)p.nK * s.cout * 9 * s.cin : 0;
}

template <int W, int RPS, int NS, int KS>
static hipError_t launch_wgrad_rows(const WgIo& io, int ng, const ConvShape& s, const WgPlan& p,
                                    hipStream_t st) {
  const long items = (long)ng * p.nK * 3 * (s.cout / 64) * (s.cin / 64);
  const int G = (int)(items < 256 ? items : 256);
  const double flops = 2.0 * ng * s.pixels() * s.cout * 9 * s.cin;
  const double bytes = ng * (2.0 * s.pixels() * (s.cin + s.cout) + 4.0 * p.nK * s.cout * 9 * s.cin);
  static char name[48];
  if (!name[0])
    snprintf(name, sizeof name, "conv_wgrad_rows<%d,%d,%d%s>", W, RPS, NS,
             KS == 2 ? ",8w" : KS == 3 ? ",12w" : "");
  ProfScope ps(name, flops, bytes, st);
  TGP_LAUNCH(ps, (conv_wgrad_rows<W, RPS, NS, KS>), dim3(G), dim3(256 * KS), 0, st, io, ng, s.nb,
             s.H, s.cin, s.cout, p.R);
  return launch_status();
}

template <int W, int RPS, int NS>
static hipError_t launch_wgrad_rows_ks(const WgIo& io, int ng, const ConvShape& s,
                                       const WgPlan& p, hipStream_t st, bool one_wave) {
  // two waves per SIMD, the phase-1 waves issuing the DMA, pay off where a
  // stage has many k steps (on the U-Net stage: 192 and 48 7-11% faster
  // than with every wave issuing, 96 7% faster than one wave per SIMD; 24
  // 14% slower); at 192 three waves per SIMD are 5% faster again
  const int ks = one_wave ? 1 : g_wgrad_ks ? g_wgrad_ks
                                           : W == 192 ? 3 : ((W == 96 || W == 48) ? 2 : 1);
  if constexpr (W == 192)
    if (ks == 3) return launch_wgrad_rows<W, RPS, NS, 3>(io, ng, s, p, st);
  return ks == 2 ? launch_wgrad_rows<W, RPS, NS, 2>(io, ng, s, p, st)
                 : launch_wgrad_rows<W, RPS, NS, 1>(io, ng, s, p, st);
}

// The three-filter-row kernel: its widths with the ring depth that fits
// (rows per stage as in kWgCfgs), and the shapes it serves: micro-batches
// of at least kWg3MinNb samples at the widths wg3_use_width names (measured
// faster there).  It has a third of the one-row kernel's items, so a launch
// of few micro-batches would leave CUs idle: such a launch runs the one-row
// kernel with one wave per SIMD instead, which sums every K range in the
// same order (the same bits).  g_wgrad_rows3 = 0 turns it off (measurement
// and tests).
struct Wg3Cfg { int W, RPS, NS; };
constexpr Wg3Cfg kWg3Cfgs[] = {{128, 1, 2}, {96, 2, 2}, {64, 3, 2}, {48, 4, 2},
                               {32, 6, 2},  {24, 4, 4}, {16, 8, 3}, {8, 8, 4}};
constexpr int kWg3MinNb = 4;
constexpr long kWg3MinItems = 128;   // items of a launch below which it runs the one-row kernel
constexpr bool wg3_use_width(int W) { return W == 96 || W == 48 || W == 24; }
int g_wgrad_rows3 = 1;
static bool use_rows3(const ConvShape& s) {
  return g_wgrad_rows3 && s.nb >= kWg3MinNb && wg3_use_width(s.W);
}

template <int W, int RPS, int NS>
static hipError_t launch_wgrad_rows3(const WgIo& io, int ng, const ConvShape& s, const WgPlan& p,
                                     hipStream_t st) {
  if (wgrad_rows_rps(W) != RPS) return hipErrorInvalidValue;   // the plan's rows per stage
  const long items = (long)ng * p.nK * (s.cout / 64) * (s.cin / 64);
  const int G = (int)(items < 256 ? items : 256);
  const double flops = 2.0 * ng * s.pixels() * s.cout * 9 * s.cin;
  const double bytes = ng * (2.0 * s.pixels() * (s.cin + s.cout) + 4.0 * p.nK * s.cout * 9 * s.cin);
  static char name[48];
  if (!name[0]) snprintf(name, sizeof name, "conv_wgrad_rows3<%d,%d,%d>", W, RPS, NS);
  ProfScope ps(name, flops, bytes, st);
  TGP_LAUNCH(ps, (conv_wgrad_rows3<W, RPS, NS>), dim3(G), dim3(768), 0, st, io, ng, s.nb, s.H,
             s.cin, s.cout, p.R);
  return launch_status();
}

static hipError_t launch_wgrad_rows_w(const WgIo& io, int ng, const ConvShape& s,
                                      const WgPlan& p, hipStream_t st) {
  const bool rows3 = use_rows3(s);
  if (rows3 && (long)ng * p.nK * (s.cout / 64) * (s.cin / 64) >= kWg3MinItems) {
    switch (s.W) {
#define WG3_CASE(i)                                                                          \
  case kWg3Cfgs[i].W:                                                                        \
    return launch_wgrad_rows3<kWg3Cfgs[i].W, kWg3Cfgs[i].RPS, kWg3Cfgs[i].NS>(io, ng, s, p, st);
      WG3_CASE(0) WG3_CASE(1) WG3_CASE(2) WG3_CASE(3) WG3_CASE(4) WG3_CASE(5) WG3_CASE(6)
      WG3_CASE(7)
#undef WG3_CASE
      default: return hipErrorInvalidValue;
    }
  }
  switch (s.W) {
#define WG_CASE(i)                                                                           \
  case kWgCfgs[i].W:                                                                         \
    return launch_wgrad_rows_ks<kWgCfgs[i].W, kWgCfgs[i].RPS, kWgCfgs[i].NS>(io, ng, s, p, st, \
                                                                             rows3);
    WG_CASE(0) WG_CASE(1) WG_CASE(2) WG_CASE(3) WG_CASE(4)
    WG_CASE(5) WG_CASE(6) WG_CASE(7) WG_CASE(8) WG_CASE(9)
#undef WG_CASE
    default: return hipErrorInvalidValue;
  }
}

hipError_t conv_wgrad_rows_launch(const void* x, const void* dz, float* dw, float* partial,
                                  const ConvShape& s, hipStream_t st, const ReduceJob* extra,
                                  ReduceJob* defer) {
  if (!wgrad_rows_ok(s)) return hipErrorInvalidValue;
  const WgPlan p = wgrad_rows_plan(s);
  float* out = p.nK > 1 ? partial : dw;
  WgIo io{};
  for (int k = 0; k < kWgGroup; ++k) {
    io.x[k] = (const bf16_t*)x;
    io.dz[k] = (const bf16_t*)dz;
    io.out[k] = out;
  }
  hipError_t e = launch_wgrad_rows_w(io, 1, s, p, st);
  if (e != hipSuccess) return e;
  if (defer) {
    *defer = ReduceJob{out, dw, (long)s.cout * 9 * s.cin, p.nK};
    return extra ? hipErrorInvalidValue : hipSuccess;
  }
  if (p.nK == 1)
    return extra ? splitk_reduce_launch(extra->part, extra->out, extra->E, extra->S, st) : e;
  return splitk_reduce_launch(partial, dw, (long)s.cout * 9 * s.cin, p.nK, st, extra);
}

// n micro-batches in one launch, each sum left pending (*defer[k]): the
// same slices as n conv_wgrad_rows_launch calls with `defer`.
hipError_t conv_wgrad_rows_launch_n(int n, const void* const* x, const void* const* dz,
                                    float* const* dw, float* const* partial, const ConvShape& s,
                                    hipStream_t st, ReduceJob* const* defer) {
  if (n < 1 || n > kMaxGroup || !wgrad_rows_ok(s)) return hipErrorInvalidValue;
  if (n > kWgGroup) {
    for (int k0 = 0; k0 < n; k0 += kWgGroup) {
      const int c = n - k0 < kWgGroup ? n - k0 : kWgGroup;
      const hipError_t e =
          conv_wgrad_rows_launch_n(c, x + k0, dz + k0, dw + k0, partial + k0, s, st, defer + k0);
      if (e != hipSuccess) return e;
    }
    return hipSuccess;
  }
  const WgPlan p = wgrad_rows_plan(s);
  WgIo io{};
  for (int k = 0; k < kWgGroup; ++k) {   // unused entries repeat micro-batch 0
    const int q = k < n ? k : 0;
    io.x[k] = (const bf16_t*)x[q];
    io.dz[k] = (const bf16_t*)dz[q];
    io.out[k] = p.nK > 1 ? partial[q] : dw[q];
    if (!io.x[k] || !io.dz[k] || !io.out[k] || !defer[q]) return hipErrorInvalidValue;
  }
  hipError_t e = launch_wgrad_rows_w(io, n, s, p, st);
  if (e != hipSuccess) return e;
  const long E = (long)s.cout * 9 * s.cin;
  for (int k = 0; k < n; ++k) *defer[k] = ReduceJob{io.out[k], dw[k], E, p.nK};
  return hipSuccess;
}

}  // namespace tgpk
