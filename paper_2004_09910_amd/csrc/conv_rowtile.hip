// bf16 3x3 convolution (forward, and data gradient on the rotated,
// transposed weights) on 16 x 16 x 32 MFMA with row-aligned pixel tiles.
//
// An output tile is 64 output channels x R whole image rows of one sample
// (R W pixels).  Its K loop runs over stages (32-channel chunk c, filter row
// r), 3 Cin / 32 of them.  A stage holds in LDS:
//   - the weights of taps (r, 0..2) for the 64 channels: 192 rows;
//   - input rows h0 + r - 1 .. h0 + r - 2 + R, each padded to W + 2 pixels
//     with a zero pixel on either side: R (W + 2) rows.
// Every row is 32 channels (64 bytes) at an 80-byte pitch, which makes the
// MFMA fragment reads (16 consecutive rows at one 16-byte chunk)
// bank-conflict-free without a swizzle.  Output pixel (rho, w) at column tap
// s reads padded row rho (W + 2) + w + s, so the zero padding of the
// convolution is real zeros in LDS and no fragment is masked; every fragment
// address is a per-lane constant plus an immediate offset.  The padding
// pixels, the rows above and below the image and the 16-byte pad of each row
// are filled by buffer loads at out-of-range offsets, which return zeros.
//
// Each of the 4 waves owns TN 16-pixel sub-tiles of the tile for all 64
// channels (4 x TN MFMA tiles).  Blocks are persistent: block lb of G takes
// tiles lb, lb + G, ... and streams all their stages through one NS-deep
// LDS ring, so the next tile's loads are in flight while the current one
// finishes.  Bias and ReLU are applied in the epilogue from an LDS copy of
// the bias, with the hardware bf16 conversion (round to nearest even).  The
// K order (chunk, r, s, channel) is fixed by the per-sample shape, so a
// recomputation is bit-identical.
#include "common.h"
#include "kernels.h"
#include "mfma_util.h"
#include "prof.h"

namespace tgpk {
namespace {

constexpr int RT_PITCH = 80;                    // bytes per LDS row (32 channels + pad)
constexpr int RT_AREG = 16384;                  // weight region: 192 rows, rounded to 16 KiB
constexpr int RT_MAXC = 1024;                   // output channels whose bias fits in LDS
constexpr int RT_OOB = (int)0x80000000;         // byte offset that reads as out of range

typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));

__device__ __forceinline__ unsigned pack_bf16(float a, float b) {
  const bf16x2_t h = {(__bf16)a, (__bf16)b};
  return __builtin_bit_cast(unsigned, h);
}

template <int TN, int NS, int SKB>
__global__ __launch_bounds__(256) void conv3x3_rowtile(
    const bf16_t* __restrict__ X, const bf16_t* __restrict__ Wt,
    const float* __restrict__ bias, bf16_t* __restrict__ Y, int nb, int H, int W, int Cin,
    int Cout, int relu, int R) {
  constexpr int SB = SKB * 1024;                // stage bytes
  constexpr int L = SB / 4096;                  // DMA instructions per wave per stage
  constexpr int LA = RT_AREG / 4096;            // ... of which weight rows
  static_assert(SB % 4096 == 0 && L > LA, "stage layout");
  __shared__ __attribute__((aligned(16))) unsigned char smem[NS * SB];
  __shared__ __attribute__((aligned(16))) float sbias[RT_MAXC];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int WP2 = W + 2;
  const int nrb = (H + R - 1) / R;              // row blocks per sample
  const int nct = Cout / 64;
  const int items = nb * nrb * nct;
  const int G = gridDim.x;
  const int lb = xcd_remap(blockIdx.x, G);
  const int n_items = lb < items ? (items - lb + G - 1) / G : 0;
  const int nk = 3 * (Cin / 32);                // stages per tile
  const int total = n_items * nk;

  // the bias of every output channel, read once before the first DMA
  if (bias)
    for (int c = tid; c < Cout; c += 256) sbias[c] = bias[c];
  __syncthreads();   // the stage loop's barriers do not wait for LDS writes

  const u32x4 rx = make_rsrc(X, nb * H * W * Cin * 2);
  const u32x4 rw = make_rsrc(Wt, Cout * 9 * Cin * 2);

  // DMA: instruction u of this wave fills stage bytes [(4 u + wave) KiB, + 1
  // KiB); lane l the 16 bytes at + 16 l, i.e. row off / 80, chunk
  // (off % 80) / 16 (chunk 4 is the row's pad).
  int aoff[LA];                                 // weight row byte offset, or out of range
  int boff[L - LA];                             // pixel byte offset within the row block
  int brow[L - LA];                             // its row in the block, -1 for no pixel
#pragma unroll
  for (int u = 0; u < L; ++u) {
    const int off = ((u * 4 + wave) * 64 + lane) * 16;
    if (u < LA) {
      const int a = off / RT_PITCH, piece = (off % RT_PITCH) / 16;
      const int t3 = a / 64, co = a % 64;
      aoff[u < LA ? u : 0] = a < 192 && piece < 4 ? ((co * 9 + t3) * Cin + piece * 8) * 2 : RT_OOB;
    } else {
      const int ob = off - RT_AREG;
      const int q = ob / RT_PITCH, piece = (ob % RT_PITCH) / 16;
      const int rho = q / WP2, wp = q - rho * WP2;
      const bool ok = rho < R && piece < 4 && wp >= 1 && wp <= W;
      boff[u < LA ? 0 : u - LA] = ok ? ((rho * W + wp - 1) * Cin + piece * 8) * 2 : 0;
      brow[u < LA ? 0 : u - LA] = ok ? rho : -1;
    }
  }

  // MFMA fragment bases (byte offsets within a stage) and output pixels
  const int abase = (lane & 15) * RT_PITCH + (lane >> 4) * 16;
  int bbase[TN], orow[TN], opix[TN];
#pragma unroll
  for (int j = 0; j < TN; ++j) {
    const int t = (wave * TN + j) * 16 + (lane & 15);    // pixel within the tile
    const int rho = t / W, w = t - (t / W) * W;
    const bool ok = t < R * W;
    bbase[j] = RT_AREG + (ok ? rho * WP2 + w : 0) * RT_PITCH + (lane >> 4) * 16;
    orow[j] = ok ? rho : 1 << 20;
    opix[j] = ok ? t : 0;
  }

  auto coords = [&](int it, int& n, int& h0, int& co0) __attribute__((always_inline)) {
    const int item = lb + it * G;
    const int ct = item % nct, rest = item / nct;
    const int rb = rest % nrb;
    n = rest / nrb;
    h0 = rb * R;
    co0 = ct * 64;
  };

  // issue side
  int i_it = 0, i_ks = 0, i_n = 0, i_h0 = 0, i_co0 = 0;
  if (total > 0) coords(0, i_n, i_h0, i_co0);
  auto issue = [&](int slot) __attribute__((always_inline)) {
    const int chunk = i_ks / 3, r = i_ks - 3 * chunk;
    const int c0 = chunk * 32;
    const int soff_a = ((i_co0 * 9 + 3 * r) * Cin + c0) * 2;
    const int hb = i_h0 + r - 1;                             // input row of block row 0
    const int base_b = ((i_n * H + hb) * W * Cin + c0) * 2;
    const bool interior = hb >= 0 && hb + R <= H;
#pragma unroll
    for (int u = 0; u < L; ++u) {
      auto* dst = TGP_LDS(smem + slot * SB + (u * 4 + wave) * 1024);
      if (u < LA) {
        dma16(rw, dst, aoff[u < LA ? u : 0], soff_a);
      } else {
        const int k = u < LA ? 0 : u - LA;
        const bool ok = brow[k] >= 0 && (interior || (unsigned)(hb + brow[k]) < (unsigned)H);
        dma16(rx, dst, ok ? base_b + boff[k] : RT_OOB, 0);
      }
    }
    if (++i_ks == nk) {
      i_ks = 0;
      if (++i_it < n_items) coords(i_it, i_n, i_h0, i_co0);
    }
  };

#pragma unroll
  for (int k = 0; k < NS - 1; ++k)
    if (k < total) issue(k);

  int idx = 0;
  for (int c_it = 0; c_it < n_items; ++c_it) {
    int n, h0, co0;
    coords(c_it, n, h0, co0);
    f32x4_t acc[4][TN];
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int j = 0; j < TN; ++j) acc[i][j] = f32x4_t{};

    for (int ks = 0; ks < nk; ++ks, ++idx) {
      // loads complete in order: stage idx is in once at most the stages
      // issued after it are pending (stores of an epilogue only make this
      // wait longer)
      wait_stages<NS, L>(min(NS - 2, total - 1 - idx));
      ring_barrier();
      if (idx + NS - 1 < total) issue((idx + NS - 1) % NS);
      const unsigned char* st = smem + (idx % NS) * SB;
      // 3 column taps; tap s + 1's fragments are read while tap s's MFMAs run
      bf16x8_t fa[2][4], fb[2][TN];
      auto load = [&](int s, int buf) __attribute__((always_inline)) {
#pragma unroll
        for (int i = 0; i < 4; ++i)
          fa[buf][i] = as_bf16x8(*(const u32x4*)(st + abase + (s * 64 + i * 16) * RT_PITCH));
#pragma unroll
        for (int j = 0; j < TN; ++j)
          fb[buf][j] = as_bf16x8(*(const u32x4*)(st + bbase[j] + s * RT_PITCH));
      };
      load(0, 0);
#pragma unroll
      for (int s = 0; s < 3; ++s) {
        if (s + 1 < 3) load(s + 1, (s + 1) & 1);
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int i = 0; i < 4; ++i)
#pragma unroll
          for (int j = 0; j < TN; ++j) acc[i][j] = mfma16(fa[s & 1][i], fb[s & 1][j], acc[i][j]);
        __builtin_amdgcn_sched_barrier(0);
      }
    }

    // epilogue: lane holds output channels co0 + 16 i + 4 (lane / 16) + 0..3
    // of tile pixel opix[j]
    const long pix0 = (long)(n * H + h0) * W;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int co = co0 + i * 16 + 4 * (lane >> 4);
      f32x4_t b4 = f32x4_t{};
      if (bias) b4 = *(const f32x4_t*)(sbias + co);
#pragma unroll
      for (int j = 0; j < TN; ++j) {
        f32x4_t v = acc[i][j] + b4;
        if (relu) {
#pragma unroll
          for (int e = 0; e < 4; ++e) v[e] = fmaxf(v[e], 0.0f);
        }
        if (h0 + orow[j] < H) {
          uint2 o;
          o.x = pack_bf16(v[0], v[1]);
          o.y = pack_bf16(v[2], v[3]);
          *(uint2*)(Y + (pix0 + opix[j]) * Cout + co) = o;
        }
      }
    }
  }
}

struct RtCfg { int TN, NS, SKB; };
constexpr RtCfg kRtCfgs[] = {{9, 2, 64}, {5, 3, 40}, {3, 4, 32}};

}  // namespace

// Tile shape for a per-sample shape: R rows per tile for each sub-tile count
// TN that fits (the stage must fit its LDS slot), scored by the rounds of
// 256 tiles a nominal 4-sample micro-batch needs times TN.  Returns the
// index into kRtCfgs, or -1 when the shape is not supported.
int g_rowtile_cfg = -1;   // >= 0 forces a configuration (measurement only)

static int rowtile_pick(const ConvShape& s, int& R) {
  if (s.taps != 9 || s.cin % 32 || s.cout % 64 || s.cout > RT_MAXC) return -1;
  int best = -1;
  long best_cost = 0;
  for (int c = 0; c < 3; ++c) {
    const RtCfg k = kRtCfgs[c];
    int r = (64 * k.TN) / s.W;
    if (r > s.H) r = s.H;
    while (r >= 1 && RT_AREG + (long)r * (s.W + 2) * RT_PITCH > k.SKB * 1024L) --r;
    if (r < 1) continue;
    const long items = 4L * ((s.H + r - 1) / r) * (s.cout / 64);
    const long cost = (items + 255) / 256 * k.TN;
    if (g_rowtile_cfg == c || (g_rowtile_cfg < 0 && (best < 0 || cost < best_cost))) {
      best = c;
      best_cost = cost;
      R = r;
    }
  }
  return best;
}

bool conv_rowtile_ok(const ConvShape& s) {
  int R;
  return rowtile_pick(s, R) >= 0 && (double)s.pixels() * s.cin * 2 < 2147483648.0 &&
         (double)s.cout * 9 * s.cin * 2 < 2147483648.0;
}

template <int TN, int NS, int SKB>
static hipError_t launch_rowtile(const char* name, const bf16_t* X, const bf16_t* Wt,
                                 const float* b, bf16_t* Y, const ConvShape& s, int R, int relu,
                                 hipStream_t st) {
  const long items = (long)s.nb * ((s.H + R - 1) / R) * (s.cout / 64);
  const int G = (int)(items < 256 ? items : 256);
  if (G == 0) return hipSuccess;
  const long P = s.pixels();
  ProfScope ps(name, 2.0 * P * s.cout * 9 * s.cin,
               2.0 * ((double)P * s.cin + 9.0 * s.cin * s.cout + (double)P * s.cout), st);
  TGP_LAUNCH(ps, (conv3x3_rowtile<TN, NS, SKB>), dim3(G), dim3(256), 0, st, X, Wt, b, Y, s.nb,
             s.H, s.W, s.cin, s.cout, relu, R);
  return launch_status();
}

hipError_t conv_forward_rowtile(const void* x, const void* w, const float* b, void* y,
                                const ConvShape& s, int relu, hipStream_t st) {
  int R = 0;
  const int c = rowtile_pick(s, R);
  if (c < 0 || !conv_rowtile_ok(s)) return hipErrorInvalidValue;
  const bf16_t* X = (const bf16_t*)x;
  const bf16_t* Wt = (const bf16_t*)w;
  bf16_t* Y = (bf16_t*)y;
  switch (c) {
    case 0: return launch_rowtile<9, 2, 64>("conv3x3_rowtile<9,2,64>", X, Wt, b, Y, s, R, relu, st);
    case 1: return launch_rowtile<5, 3, 40>("conv3x3_rowtile<5,3,40>", X, Wt, b, Y, s, R, relu, st);
    default: return launch_rowtile<3, 4, 32>("conv3x3_rowtile<3,4,32>", X, Wt, b, Y, s, R, relu, st);
  }
}

}  // namespace tgpk
