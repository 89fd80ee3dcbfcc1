// Non-MFMA kernels: direct convolutions for float32 runs and for shapes the
// MFMA tiles do not cover (e.g. a 1-channel head), depthwise 3x3, ReLU
// backward, bias gradient, max-pool, upsample-concat, MSE and gradient
// accumulation.  All reductions run in a fixed order (per-thread serial sums,
// fixed LDS trees, fixed split order), so results are bit-reproducible.
#include "common.h"
#include "kernels.h"
#include "prof.h"

namespace tgpk {

bool mfma_conv_ok(int dt, int cin, int cout);
hipError_t conv_forward_mfma(const void* x, const void* w, const float* b, void* y,
                             const ConvShape& s, int relu, float* part, size_t part_cap,
                             hipStream_t st);
size_t wgrad_mfma_partial_floats(const ConvShape& s);
hipError_t conv_wgrad_mfma(const void* x, const void* dz, float* dw, float* partial,
                           const ConvShape& s, hipStream_t st, const ReduceJob* extra,
                           ReduceJob* defer);
hipError_t conv_forward_mfma_n(int n, const void* const* x, const void* w, const float* b,
                               void* const* y, const ConvShape& s, int relu, float* const* part,
                               size_t part_cap, hipStream_t st);
hipError_t conv_wgrad_mfma_n(int n, const void* const* x, const void* const* dz,
                             float* const* dw, float* const* part, const ConvShape& s,
                             hipStream_t st, ReduceJob* const* defer);

namespace {


// ---------------------------------------------------------------- 16-byte packs

template <typename T> struct Pk;
template <> struct Pk<bf16_t> {
  static constexpr int N = 8;
  static __device__ __forceinline__ void un(uint4 v, float* f) {
    const uint32_t* d = &v.x;
#pragma unroll
    for (int i = 0; i < 4; ++i) { f[2 * i] = bf2f(d[i] & 0xffffu); f[2 * i + 1] = bf2f(d[i] >> 16); }
  }
  static __device__ __forceinline__ uint4 pk(const float* f) {
    uint4 v;
    uint32_t* d = &v.x;
#pragma unroll
    for (int i = 0; i < 4; ++i) d[i] = f2bf(f[2 * i]) | (f2bf(f[2 * i + 1]) << 16);
    return v;
  }
};
template <> struct Pk<float> {
  static constexpr int N = 4;
  static __device__ __forceinline__ void un(uint4 v, float* f) {
    f[0] = __uint_as_float(v.x); f[1] = __uint_as_float(v.y);
    f[2] = __uint_as_float(v.z); f[3] = __uint_as_float(v.w);
  }
  static __device__ __forceinline__ uint4 pk(const float* f) {
    return make_uint4(__float_as_uint(f[0]), __float_as_uint(f[1]), __float_as_uint(f[2]),
                      __float_as_uint(f[3]));
  }
};

template <typename T> __device__ __forceinline__ uint4 ld16(const T* p) { return *(const uint4*)p; }
template <typename T> __device__ __forceinline__ void st16(T* p, uint4 v) { *(uint4*)p = v; }

// ---------------------------------------------------------------- direct conv

template <typename T>
__global__ __launch_bounds__(256) void conv_fwd_direct(const T* __restrict__ x,
                                                       const T* __restrict__ w,
                                                       const float* __restrict__ b,
                                                       T* __restrict__ y, long P, int H, int W,
                                                       int Cin, int Cout, int taps, int relu) {
  long e = (long)blockIdx.x * 256 + threadIdx.x;
  if (e >= P * Cout) return;
  int co = e % Cout;
  long p = e / Cout;
  int HW = H * W;
  int rem = p % HW, h = rem / W, wq = rem - h * W;
  float acc = 0.f;
  for (int t = 0; t < taps; ++t) {
    int dr = taps == 9 ? t / 3 - 1 : 0, dc = taps == 9 ? t % 3 - 1 : 0;
    int hh = h + dr, ww = wq + dc;
    if ((unsigned)hh >= (unsigned)H || (unsigned)ww >= (unsigned)W) continue;
    const T* xr = x + (p + (long)dr * W + dc) * Cin;
    const T* wr = w + ((long)co * taps + t) * Cin;
    for (int ci = 0; ci < Cin; ++ci) acc += Elt<T>::ld(xr + ci) * Elt<T>::ld(wr + ci);
  }
  if (b) acc += b[co];
  if (relu) acc = fmaxf(acc, 0.f);
  Elt<T>::st(y + e, acc);
}

template <typename T>
__global__ __launch_bounds__(256) void conv_dgrad_direct(const T* __restrict__ dz,
                                                         const T* __restrict__ w,
                                                         T* __restrict__ dx, long P, int H,
                                                         int W, int Cin, int Cout, int taps) {
  long e = (long)blockIdx.x * 256 + threadIdx.x;
  if (e >= P * Cin) return;
  int ci = e % Cin;
  long p = e / Cin;
  int HW = H * W;
  int rem = p % HW, h = rem / W, wq = rem - h * W;
  float acc = 0.f;
  for (int t = 0; t < taps; ++t) {
    int dr = taps == 9 ? t / 3 - 1 : 0, dc = taps == 9 ? t % 3 - 1 : 0;
    // output pixel (h - dr, w - dc) read input pixel (h, w) through tap t
    int hh = h - dr, ww = wq - dc;
    if ((unsigned)hh >= (unsigned)H || (unsigned)ww >= (unsigned)W) continue;
    const T* dr_ = dz + (p - (long)dr * W - dc) * Cout;
    for (int co = 0; co < Cout; ++co)
      acc += Elt<T>::ld(dr_ + co) * Elt<T>::ld(w + ((long)co * taps + t) * Cin + ci);
  }
  Elt<T>::st(dx + e, acc);
}

// partial[s][co][tap][ci] = sum over pixels of split s of dz[p][co] * x[p+off][ci]
template <typename T>
__global__ __launch_bounds__(256) void conv_wgrad_direct(const T* __restrict__ x,
                                                         const T* __restrict__ dz,
                                                         float* __restrict__ part, long P,
                                                         int H, int W, int Cin, int Cout,
                                                         int taps, long pps) {
  long E = (long)Cout * taps * Cin;
  long e = (long)blockIdx.x * 256 + threadIdx.x;
  if (e >= E) return;
  int ci = e % Cin;
  long r = e / Cin;
  int t = r % taps;
  int co = r / taps;
  int dr = taps == 9 ? t / 3 - 1 : 0, dc = taps == 9 ? t % 3 - 1 : 0;
  long ps = (long)blockIdx.y * pps, pe = ps + pps < P ? ps + pps : P;
  int HW = H * W;
  float acc = 0.f;
  for (long p = ps; p < pe; ++p) {
    int rem = p % HW, h = rem / W, wq = rem - h * W;
    int hh = h + dr, ww = wq + dc;
    if ((unsigned)hh >= (unsigned)H || (unsigned)ww >= (unsigned)W) continue;
    acc += Elt<T>::ld(dz + p * Cout + co) * Elt<T>::ld(x + (p + (long)dr * W + dc) * Cin + ci);
  }
  part[(long)blockIdx.y * E + e] = acc;
}

// 1x1 convolution with at most kSmallCo output channels (the network head):
// one thread per pixel reads its channels in 16-byte packs.
constexpr int kSmallCo = 4;

template <typename T>
__global__ __launch_bounds__(256) void conv1x1_small_fwd_k(const T* __restrict__ x,
                                                           const T* __restrict__ w,
                                                           const float* __restrict__ b,
                                                           T* __restrict__ y, long P, int Cin,
                                                           int Cout, int relu) {
  constexpr int N = Pk<T>::N;
  const long p = (long)blockIdx.x * 256 + threadIdx.x;
  if (p >= P) return;
  float acc[kSmallCo];
#pragma unroll
  for (int co = 0; co < kSmallCo; ++co) acc[co] = (co < Cout && b) ? b[co] : 0.f;
  for (int c0 = 0; c0 < Cin; c0 += N) {
    float xv[N];
    Pk<T>::un(ld16(x + p * Cin + c0), xv);
#pragma unroll
    for (int co = 0; co < kSmallCo; ++co) {
      if (co >= Cout) break;
#pragma unroll
      for (int i = 0; i < N; ++i) acc[co] += xv[i] * Elt<T>::ld(w + (long)co * Cin + c0 + i);
    }
  }
#pragma unroll
  for (int co = 0; co < kSmallCo; ++co) {
    if (co >= Cout) break;
    Elt<T>::st(y + p * Cout + co, relu ? fmaxf(acc[co], 0.f) : acc[co]);
  }
}

// Its weight gradient dW[co][ci] = sum_p dz[p][co] x[p][ci]: block b covers
// pixels [b*rows, (b+1)*rows); thread t takes channel pack t % CP of pixels
// t / CP, t / CP + 256 / CP, ... in order; row lanes are then added in order
// in LDS and part[b][co][ci] is written.  Needs 256 % CP == 0 (CP = Cin / pack).
template <typename T>
__global__ __launch_bounds__(256) void wgrad1x1_small_k(const T* __restrict__ x,
                                                        const T* __restrict__ dz,
                                                        float* __restrict__ part, long P,
                                                        int Cin, int Cout, long rows) {
  constexpr int N = Pk<T>::N;
  __shared__ float red[256 * N];
  const int CP = Cin / N;
  const int cp = threadIdx.x % CP, rl = threadIdx.x / CP, nl = 256 / CP;
  const long p0 = (long)blockIdx.x * rows, p1 = p0 + rows < P ? p0 + rows : P;
  float acc[kSmallCo][N];
#pragma unroll
  for (int co = 0; co < kSmallCo; ++co)
#pragma unroll
    for (int i = 0; i < N; ++i) acc[co][i] = 0.f;
  for (long p = p0 + rl; p < p1; p += nl) {
    float xv[N];
    Pk<T>::un(ld16(x + p * Cin + cp * N), xv);
#pragma unroll
    for (int co = 0; co < kSmallCo; ++co) {
      if (co >= Cout) break;
      const float g = Elt<T>::ld(dz + p * Cout + co);
#pragma unroll
      for (int i = 0; i < N; ++i) acc[co][i] += g * xv[i];
    }
  }
  const long E = (long)Cout * Cin;
#pragma unroll
  for (int co = 0; co < kSmallCo; ++co) {   // one output channel at a time through LDS
    if (co >= Cout) break;                  // block-uniform
    __syncthreads();
#pragma unroll
    for (int i = 0; i < N; ++i) red[threadIdx.x * N + i] = acc[co][i];
    __syncthreads();
    if (rl == 0) {
      float sum[N];
#pragma unroll
      for (int i = 0; i < N; ++i) sum[i] = red[cp * N + i];
      for (int l = 1; l < nl; ++l)
#pragma unroll
        for (int i = 0; i < N; ++i) sum[i] += red[(l * CP + cp) * N + i];
#pragma unroll
      for (int i = 0; i < N; ++i) part[(long)blockIdx.x * E + (long)co * Cin + cp * N + i] = sum[i];
    }
  }
}

long direct_wgrad_pps(long P) { return P < 256 ? 256 : (P + 63) / 64; }
int direct_wgrad_splits(long P) { return (int)((P + direct_wgrad_pps(P) - 1) / direct_wgrad_pps(P)); }

// ---------------------------------------------------------------- depthwise

template <typename T>
__global__ __launch_bounds__(256) void dw_fwd(const T* __restrict__ x, const T* __restrict__ w,
                                              const float* __restrict__ b, T* __restrict__ y,
                                              long P, int H, int W, int C, int relu) {
  long e = (long)blockIdx.x * 256 + threadIdx.x;
  if (e >= P * C) return;
  int c = e % C;
  long p = e / C;
  int HW = H * W, rem = p % HW, h = rem / W, wq = rem - h * W;
  float acc = 0.f;
#pragma unroll
  for (int t = 0; t < 9; ++t) {
    int hh = h + t / 3 - 1, ww = wq + t % 3 - 1;
    if ((unsigned)hh < (unsigned)H && (unsigned)ww < (unsigned)W)
      acc += Elt<T>::ld(w + c * 9 + t) * Elt<T>::ld(x + (p + (long)(t / 3 - 1) * W + (t % 3 - 1)) * C + c);
  }
  if (b) acc += b[c];
  if (relu) acc = fmaxf(acc, 0.f);
  Elt<T>::st(y + e, acc);
}

template <typename T>
__global__ __launch_bounds__(256) void dw_dgrad_k(const T* __restrict__ dz, const T* __restrict__ w,
                                                  T* __restrict__ dx, long P, int H, int W, int C) {
  long e = (long)blockIdx.x * 256 + threadIdx.x;
  if (e >= P * C) return;
  int c = e % C;
  long p = e / C;
  int HW = H * W, rem = p % HW, h = rem / W, wq = rem - h * W;
  float acc = 0.f;
#pragma unroll
  for (int t = 0; t < 9; ++t) {
    int dr = t / 3 - 1, dc = t % 3 - 1;
    int hh = h - dr, ww = wq - dc;
    if ((unsigned)hh < (unsigned)H && (unsigned)ww < (unsigned)W)
      acc += Elt<T>::ld(w + c * 9 + t) * Elt<T>::ld(dz + (p - (long)dr * W - dc) * C + c);
  }
  Elt<T>::st(dx + e, acc);
}

// Depthwise 3x3 over bf16 NHWC with C % 8 == 0 and C / 8 dividing 256.
// Thread q of block (chunk, strip) owns column wc = q / CP and channel pack
// cp = q % CP (CP = C / 8, eight channels per 16-byte pack) and produces the
// output rows [h0, h0 + RS) of that column: the 3 x 3 window of input packs
// slides down the rows, three new packs per output row, so each input pack
// is fetched about (RS + 2) / RS times per column and its horizontal
// neighbours come from the same block's loads.  The nine filter taps of the
// thread's eight channels are one contiguous 144-byte run (w is [C][9]).
// FLIP applies the filter rotated by 180 degrees, which is the data
// gradient (dx = dz correlated with the flipped filter); the sum runs over
// the window in row-major order.
// gridDim.z (1 .. kMaxGroup) micro-batches: blockIdx.z selects x[k] / y[k].
// MASK (data gradient only): the result stored is the ReLU backward of the
// layer below, whose output m[k] masks it (its dz), and the block's column
// sums of the stored values go to part[k] (row blockIdx.y gridDim.x +
// blockIdx.x, C floats): that layer's bias-gradient partials.  It needs every
// thread of a block inside the image (W C / 8 a multiple of 256).
struct DwIo {
  const bf16_t* x[kMaxGroup];
  bf16_t* y[kMaxGroup];
  const bf16_t* m[kMaxGroup];
  float* part[kMaxGroup];
};
template <int RS, bool FLIP, bool MASK = false>
__global__ __launch_bounds__(256) void dw3_rows_k(DwIo io, const bf16_t* __restrict__ w,
                                                  const float* __restrict__ b, int H, int W, int C,
                                                  int relu) {
  const bf16_t* __restrict__ x = pickg(io.x, blockIdx.z);
  bf16_t* __restrict__ y = pickg(io.y, blockIdx.z);
  const int CP = C >> 3;
  const int q = blockIdx.x * 256 + threadIdx.x;
  const int wc = q / CP, cp = q - (q / CP) * CP;
  if (wc >= W) return;
  const int strips = (H + RS - 1) / RS;
  const int n = blockIdx.y / strips, h0 = (blockIdx.y - n * strips) * RS;
  float wt[9][8];
  {
    const uint4* wp = (const uint4*)(w + (long)cp * 72);
#pragma unroll
    for (int u = 0; u < 9; ++u) {
      float f[8];
      Pk<bf16_t>::un(wp[u], f);
#pragma unroll
      for (int v = 0; v < 8; ++v) {
        const int e = u * 8 + v, c = e / 9, t = e - (e / 9) * 9;
        wt[FLIP ? 8 - t : t][c] = f[v];
      }
    }
  }
  float bias[8];
#pragma unroll
  for (int i = 0; i < 8; ++i) bias[i] = b ? b[cp * 8 + i] : 0.f;
  // buffer loads over the sample's image: an offset outside it reads zeros,
  // so the halo needs no branches and the next row's loads stay in flight
  // while this row's products run
  const __amdgpu_buffer_rsrc_t rx = __builtin_amdgcn_make_buffer_rsrc(
      (void*)(x + (long)n * H * W * C), (short)0, H * W * C * 2, 0x00020000);
  auto ld = [&](int hh, int ww) __attribute__((always_inline)) {
    const bool ok = (unsigned)hh < (unsigned)H && (unsigned)ww < (unsigned)W;
    const int off = ok ? ((hh * W + ww) * C + cp * 8) * 2 : (int)0x80000000;
    return __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(rx, off, 0, 0));
  };
  uint4 win[3][3], nxt[3];
#pragma unroll
  for (int s = 0; s < 3; ++s) {
    win[0][s] = ld(h0 - 1, wc + s - 1);
    win[1][s] = ld(h0, wc + s - 1);
    win[2][s] = ld(h0 + 1, wc + s - 1);
  }
  const int h1 = min(h0 + RS, H);
  float bsum[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};   // MASK: this thread's column sums
  for (int h = h0; h < h1; ++h) {
#pragma unroll
    for (int s = 0; s < 3; ++s) nxt[s] = ld(h + 2, wc + s - 1);
    float acc[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) acc[i] = 0.f;
#pragma unroll
    for (int r = 0; r < 3; ++r)
#pragma unroll
      for (int s = 0; s < 3; ++s) {
        float f[8];
        Pk<bf16_t>::un(win[r][s], f);
#pragma unroll
        for (int i = 0; i < 8; ++i) acc[i] = fmaf(wt[r * 3 + s][i], f[i], acc[i]);
      }
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      acc[i] += bias[i];
      if (relu) acc[i] = fmaxf(acc[i], 0.f);
    }
    const long eo = (long)n * H * W * C + ((long)h * W + wc) * C + cp * 8;
    if constexpr (MASK) {
      float mv[8];
      Pk<bf16_t>::un(ld16(pickg(io.m, blockIdx.z) + eo), mv);
#pragma unroll
      for (int i = 0; i < 8; ++i) acc[i] = mv[i] > 0.f ? acc[i] : 0.f;
      const uint4 o = Pk<bf16_t>::pk(acc);
      st16(y + eo, o);
      Pk<bf16_t>::un(o, acc);   // the bias gradient sums the stored (rounded) dz
#pragma unroll
      for (int i = 0; i < 8; ++i) bsum[i] += acc[i];
    } else {
      st16(y + eo, Pk<bf16_t>::pk(acc));
    }
#pragma unroll
    for (int s = 0; s < 3; ++s) {
      win[0][s] = win[1][s];
      win[1][s] = win[2][s];
      win[2][s] = nxt[s];
    }
  }
  if constexpr (MASK) {
    // the block's column sums: lanes of one channel pack added in order of
    // their column
    __shared__ float red[256 * 8];
#pragma unroll
    for (int i = 0; i < 8; ++i) red[threadIdx.x * 8 + i] = bsum[i];
    __syncthreads();
    if ((int)threadIdx.x < CP) {
      float s8[8];
#pragma unroll
      for (int i = 0; i < 8; ++i) s8[i] = red[threadIdx.x * 8 + i];
      for (int l = 1; l < 256 / CP; ++l)
#pragma unroll
        for (int i = 0; i < 8; ++i) s8[i] += red[(l * CP + threadIdx.x) * 8 + i];
      float* pr = pickg(io.part, blockIdx.z) + ((long)blockIdx.y * gridDim.x + blockIdx.x) * C +
                  cp * 8;
#pragma unroll
      for (int i = 0; i < 8; ++i) pr[i] = s8[i];
    }
  }
}

// Depthwise 3x3 weight-gradient partials over bf16 NHWC (same shape rules
// as dw3_rows_k).  Thread (column, pack) of block (chunk, strip) sums
// dz[p] * x[p + tap] over the rows [h0, h0 + RS) of its column for its
// eight channels and nine taps (x through the sliding window, the next
// row's window and dz loaded while the current row's products run); the
// block then adds its 256 / CP column groups in order in LDS, taps 0-4 and
// then 5-8 through one buffer of a 41-float row per thread (the odd row
// length keeps both the writes and the reads free of bank conflicts), and
// writes part[blk][c * 9 + t], blk = strip block * chunks + chunk.  The partials are summed in block order
// afterwards, so the result is deterministic.
// gridDim.z (1 .. kMaxGroup) micro-batches: blockIdx.z selects (x[k],
// dz[k], part[k]).
struct DwWgIo {
  const bf16_t* x[kMaxGroup];
  const bf16_t* dz[kMaxGroup];
  float* part[kMaxGroup];
};
template <int RS>
__global__ __launch_bounds__(256) void dw3_wgrad_rows_k(DwWgIo io, int H, int W, int C) {
  const bf16_t* __restrict__ x = pickg(io.x, blockIdx.z);
  const bf16_t* __restrict__ dz = pickg(io.dz, blockIdx.z);
  float* __restrict__ part = pickg(io.part, blockIdx.z);
  constexpr int TH = 5;                      // taps per reduction pass
  constexpr int RW = TH * 8 + 1;             // floats per thread row
  __shared__ float red[256][RW];
  const int CP = C >> 3;
  const int q = blockIdx.x * 256 + threadIdx.x;
  const int wc = q / CP, cp = q - (q / CP) * CP;
  const int strips = (H + RS - 1) / RS;
  const int n = blockIdx.y / strips, h0 = (blockIdx.y - n * strips) * RS;
  float acc[9][8];
#pragma unroll
  for (int t = 0; t < 9; ++t)
#pragma unroll
    for (int i = 0; i < 8; ++i) acc[t][i] = 0.f;
  if (wc < W) {
    // buffer loads over the sample's image: an offset outside it reads
    // zeros, so the halo needs no branches (a branch per load made the
    // compiler wait for every load in flight, the prefetch included)
    const int img = H * W * C * 2;                              // bytes per sample image
    const long sb = (long)n * H * W * C;
    const __amdgpu_buffer_rsrc_t rx = __builtin_amdgcn_make_buffer_rsrc(
        (void*)(x + sb), (short)0, img, 0x00020000);
    const __amdgpu_buffer_rsrc_t rz = __builtin_amdgcn_make_buffer_rsrc(
        (void*)(dz + sb), (short)0, img, 0x00020000);
    auto ld = [&](int hh, int ww) __attribute__((always_inline)) {
      const bool ok = (unsigned)hh < (unsigned)H && (unsigned)ww < (unsigned)W;
      const int off = ok ? ((hh * W + ww) * C + cp * 8) * 2 : (int)0x80000000;
      return __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(rx, off, 0, 0));
    };
    auto ldz = [&](int hh) __attribute__((always_inline)) {
      const int off = hh < H ? ((hh * W + wc) * C + cp * 8) * 2 : (int)0x80000000;
      return __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(rz, off, 0, 0));
    };
    const int h1 = min(h0 + RS, H);
    uint4 win[3][3], nxt[3], dzc = ldz(h0);
#pragma unroll
    for (int s = 0; s < 3; ++s) {
      win[0][s] = ld(h0 - 1, wc + s - 1);
      win[1][s] = ld(h0, wc + s - 1);
      win[2][s] = ld(h0 + 1, wc + s - 1);
    }
    for (int h = h0; h < h1; ++h) {
      // next row's loads first: they arrive while this row's products run
#pragma unroll
      for (int s = 0; s < 3; ++s) nxt[s] = ld(h + 2, wc + s - 1);
      const uint4 dzn = ldz(h + 1);
      float d[8];
      Pk<bf16_t>::un(dzc, d);
#pragma unroll
      for (int r = 0; r < 3; ++r)
#pragma unroll
        for (int s = 0; s < 3; ++s) {
          float f[8];
          Pk<bf16_t>::un(win[r][s], f);
#pragma unroll
          for (int i = 0; i < 8; ++i) acc[r * 3 + s][i] = fmaf(d[i], f[i], acc[r * 3 + s][i]);
        }
#pragma unroll
      for (int s = 0; s < 3; ++s) {
        win[0][s] = win[1][s];
        win[1][s] = win[2][s];
        win[2][s] = nxt[s];
      }
      dzc = dzn;
    }
  }
  const int E = C * 9, NG = 256 / CP;
  float* out = part + ((long)blockIdx.y * gridDim.x + blockIdx.x) * E;
#pragma unroll
  for (int pass = 0; pass < 2; ++pass) {
    const int t0 = pass * TH, nt = pass ? 9 - TH : TH;
    if (pass) __syncthreads();                 // the first pass's reads are done
#pragma unroll
    for (int t = 0; t < TH; ++t)
      if (t < nt)
#pragma unroll
        for (int i = 0; i < 8; ++i) red[threadIdx.x][t * 8 + i] = acc[t0 + t][i];
    __syncthreads();
    for (int e = threadIdx.x; e < C * nt; e += 256) {
      const int c = e / nt, t = e - (e / nt) * nt, pk = c >> 3, i = c & 7;
      float s = 0.f;
      for (int g = 0; g < NG; ++g) s += red[g * CP + pk][t * 8 + i];
      out[c * 9 + t0 + t] = s;
    }
  }
}

constexpr int kDwRows = 8;       // output rows per thread, forward and data gradient
constexpr int kDwWgradRows = 8;  // rows per thread of the weight gradient

// The row-window depthwise kernels apply: bf16, whole 16-byte packs, a pack
// count dividing the block, 16-byte aligned tensors and weights, and a
// sample image under 2 GiB (their buffer loads take 32-bit offsets).
static bool dw3_rows_ok(int dt, int nb, int H, int W, int C, const void* a, const void* b2,
                        const void* c2) {
  auto al = [](const void* p) { return ((uintptr_t)p & 15) == 0; };
  return dt == 0 && C > 0 && C % 8 == 0 && 256 % (C / 8) == 0 && al(a) && al(b2) && al(c2) &&
         (long)nb * cdiv(H, kDwRows) <= 65535 && 2.0 * H * W * C < 2147483648.0;
}

static int dw3_wgrad_blocks(int nb, int H, int W, int C) {
  return (int)cdiv((long)W * (C / 8), 256) * nb * (int)cdiv(H, kDwWgradRows);
}

// ---------------------------------------------------------------- elementwise

template <typename T>
__global__ __launch_bounds__(256) void relu_bwd_k(const T* __restrict__ dy, const T* __restrict__ ds,
                                                  const T* __restrict__ y, T* __restrict__ dz,
                                                  int relu, long n, int vec) {
  constexpr int N = Pk<T>::N;
  long e0 = ((long)blockIdx.x * 256 + threadIdx.x) * N;
  if (e0 >= n) return;
  if (vec && e0 + N <= n) {
    float a[N], s[N], m[N];
    Pk<T>::un(ld16(dy + e0), a);
    if (ds) {
      Pk<T>::un(ld16(ds + e0), s);
#pragma unroll
      for (int i = 0; i < N; ++i) a[i] += s[i];
    }
    if (relu) {
      Pk<T>::un(ld16(y + e0), m);
#pragma unroll
      for (int i = 0; i < N; ++i) a[i] = m[i] > 0.f ? a[i] : 0.f;
    }
    st16(dz + e0, Pk<T>::pk(a));
  } else {
    for (long e = e0; e < n && e < e0 + N; ++e) {
      float a = Elt<T>::ld(dy + e);
      if (ds) a += Elt<T>::ld(ds + e);
      if (relu && !(Elt<T>::ld(y + e) > 0.f)) a = 0.f;
      Elt<T>::st(dz + e, a);
    }
  }
}

// dz = (dy [+ dskip]) * [y > 0] with the bias gradient's column partial sums
// fused in: block b covers rows [b*rows, (b+1)*rows); thread t handles the
// 16-byte channel pack t % CP for rows t / CP, t / CP + 256 / CP, ...
// (serial, fixed order); row lanes are then added in order in LDS and
// part[b][c] is written.  Needs 256 % CP == 0 (CP = C / pack).  A launch
// covers gridDim.y (1 .. kMaxGroup) micro-batches of the same shape;
// blockIdx.y selects the pointer set.
template <typename T>
struct RbPtrs {
  const T* dy;   // the incoming gradient (the pool gradient for the pooled kernel)
  const T* ds;
  const T* y;
  T* dz;
  float* part;
};
template <typename T>
struct RbGroup {   // pointer set k of each field is micro-batch k's
  const T* dy[kMaxGroup];
  const T* ds[kMaxGroup];
  const T* y[kMaxGroup];
  T* dz[kMaxGroup];
  float* part[kMaxGroup];
};
// The pointer set of group entry blockIdx.y.
template <typename T>
__device__ __forceinline__ RbPtrs<T> rb_pick(const RbGroup<T>& a) {
  const int k = blockIdx.y;
  return RbPtrs<T>{pickg(a.dy, k), pickg(a.ds, k), pickg(a.y, k), pickg(a.dz, k), pickg(a.part, k)};
}

template <typename T>
__global__ __launch_bounds__(256) void relu_bwd_bias_k(RbGroup<T> ga, int relu, long P, int C,
                                                       long rows) {
  const RbPtrs<T> g = rb_pick(ga);
  const T* __restrict__ dy = g.dy;
  const T* __restrict__ ds = g.ds;
  const T* __restrict__ y = g.y;
  T* __restrict__ dz = g.dz;
  float* __restrict__ part = g.part;
  constexpr int N = Pk<T>::N;
  __shared__ float red[256 * N];
  const int CP = C / N;
  const int cp = threadIdx.x % CP, rl = threadIdx.x / CP, nl = 256 / CP;
  const long p0 = (long)blockIdx.x * rows, p1 = p0 + rows < P ? p0 + rows : P;
  float sum[N];
#pragma unroll
  for (int i = 0; i < N; ++i) sum[i] = 0.f;
  for (long p = p0 + rl; p < p1; p += nl) {
    const long e = p * C + cp * N;
    float a[N], s2[N], m[N];
    Pk<T>::un(ld16(dy + e), a);
    if (ds) {
      Pk<T>::un(ld16(ds + e), s2);
#pragma unroll
      for (int i = 0; i < N; ++i) a[i] += s2[i];
    }
    if (relu) {
      Pk<T>::un(ld16(y + e), m);
#pragma unroll
      for (int i = 0; i < N; ++i) a[i] = m[i] > 0.f ? a[i] : 0.f;
    }
    uint4 o = Pk<T>::pk(a);
    st16(dz + e, o);
    Pk<T>::un(o, a);   // the bias gradient sums the stored (rounded) dz
#pragma unroll
    for (int i = 0; i < N; ++i) sum[i] += a[i];
  }
#pragma unroll
  for (int i = 0; i < N; ++i) red[threadIdx.x * N + i] = sum[i];
  __syncthreads();
  if (rl == 0) {
    for (int l = 1; l < nl; ++l)
#pragma unroll
      for (int i = 0; i < N; ++i) sum[i] += red[(l * CP + cp) * N + i];
#pragma unroll
    for (int i = 0; i < N; ++i) part[(long)blockIdx.x * C + cp * N + i] = sum[i];
  }
}

// relu_bwd_bias_k for a layer whose output feeds a 2x2/2 max pool: dy is
// the pool gradient dp routed to the first maximal element of each window
// of y.  Block b covers pooled pixels [b*rows, (b+1)*rows); thread t handles
// channel pack t % CP of windows t / CP, t / CP + 256 / CP, ... (the four
// pixels of a window in row-major order), then row lanes are added in order
// in LDS and part[b][c] is written.
template <typename T>
__global__ __launch_bounds__(256) void pool_relu_bwd_bias_k(RbGroup<T> ga, int relu, int nb,
                                                            int H, int W, int C, long rows) {
  const RbPtrs<T> gp = rb_pick(ga);
  const T* __restrict__ dp = gp.dy;
  const T* __restrict__ ds = gp.ds;
  const T* __restrict__ y = gp.y;
  T* __restrict__ dz = gp.dz;
  float* __restrict__ part = gp.part;
  constexpr int N = Pk<T>::N;
  __shared__ float red[256 * N];
  const int CP = C / N;
  const int cp = threadIdx.x % CP, rl = threadIdx.x / CP, nl = 256 / CP;
  const int H2 = H / 2, W2 = W / 2;
  const long P2 = (long)nb * H2 * W2;
  const long q0 = (long)blockIdx.x * rows, q1 = q0 + rows < P2 ? q0 + rows : P2;
  float sum[N];
#pragma unroll
  for (int i = 0; i < N; ++i) sum[i] = 0.f;
  for (long q = q0 + rl; q < q1; q += nl) {
    const int w2 = q % W2;
    const long r = q / W2;
    const int h2 = r % H2, n = r / H2;
    const long o = (((long)n * H + 2 * h2) * W + 2 * w2) * C + cp * N;
    const long off[4] = {0, C, (long)W * C, (long)W * C + C};
    float v[4][N], g[N], a[4][N];
#pragma unroll
    for (int k = 0; k < 4; ++k) Pk<T>::un(ld16(y + o + off[k]), v[k]);
    Pk<T>::un(ld16(dp + q * C + cp * N), g);
#pragma unroll
    for (int i = 0; i < N; ++i) {
      int arg = 0;
      float best = v[0][i];
#pragma unroll
      for (int k = 1; k < 4; ++k)
        if (v[k][i] > best) { best = v[k][i]; arg = k; }
#pragma unroll
      for (int k = 0; k < 4; ++k) a[k][i] = k == arg ? g[i] : 0.f;
    }
    if (ds) {
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        float s2[N];
        Pk<T>::un(ld16(ds + o + off[k]), s2);
#pragma unroll
        for (int i = 0; i < N; ++i) a[k][i] += s2[i];
      }
    }
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      if (relu) {
#pragma unroll
        for (int i = 0; i < N; ++i) a[k][i] = v[k][i] > 0.f ? a[k][i] : 0.f;
      }
      const uint4 o16 = Pk<T>::pk(a[k]);
      st16(dz + o + off[k], o16);
      Pk<T>::un(o16, a[k]);   // the bias gradient sums the stored (rounded) dz
#pragma unroll
      for (int i = 0; i < N; ++i) sum[i] += a[k][i];
    }
  }
#pragma unroll
  for (int i = 0; i < N; ++i) red[threadIdx.x * N + i] = sum[i];
  __syncthreads();
  if (rl == 0) {
    for (int l = 1; l < nl; ++l)
#pragma unroll
      for (int i = 0; i < N; ++i) sum[i] += red[(l * CP + cp) * N + i];
#pragma unroll
    for (int i = 0; i < N; ++i) part[(long)blockIdx.x * C + cp * N + i] = sum[i];
  }
}

// Column sums of a P x C matrix: block (cg, pb) sums rows [pb*rows, ...) for
// channels cg*64 .. +63; 4 row lanes, combined in fixed order.
template <typename T>
__global__ __launch_bounds__(256) void colsum_k(const T* __restrict__ a, float* __restrict__ part,
                                                long P, int C, long rows) {
  __shared__ float red[4][64];
  int c = blockIdx.x * 64 + (threadIdx.x & 63);
  int lane = threadIdx.x >> 6;
  long p0 = (long)blockIdx.y * rows, p1 = p0 + rows < P ? p0 + rows : P;
  float s = 0.f;
  if (c < C)
    for (long p = p0 + lane; p < p1; p += 4) s += Elt<T>::ld(a + p * C + c);
  red[lane][threadIdx.x & 63] = s;
  __syncthreads();
  if (lane == 0 && c < C) {
    int k = threadIdx.x & 63;
    part[(long)blockIdx.y * C + c] = ((red[0][k] + red[1][k]) + red[2][k]) + red[3][k];
  }
}

// depthwise wgrad partials: thread (c, tap) of split s
template <typename T>
__global__ __launch_bounds__(256) void dw_wgrad_k(const T* __restrict__ x, const T* __restrict__ dz,
                                                  float* __restrict__ part, long P, int H, int W,
                                                  int C, long pps) {
  long E = (long)C * 9;
  long e = (long)blockIdx.x * 256 + threadIdx.x;
  if (e >= E) return;
  int t = e % 9, c = e / 9;
  int dr = t / 3 - 1, dc = t % 3 - 1;
  long ps = (long)blockIdx.y * pps, pe = ps + pps < P ? ps + pps : P;
  int HW = H * W;
  float acc = 0.f;
  for (long p = ps; p < pe; ++p) {
    int rem = p % HW, h = rem / W, wq = rem - h * W;
    int hh = h + dr, ww = wq + dc;
    if ((unsigned)hh >= (unsigned)H || (unsigned)ww >= (unsigned)W) continue;
    acc += Elt<T>::ld(dz + p * C + c) * Elt<T>::ld(x + (p + (long)dr * W + dc) * C + c);
  }
  part[(long)blockIdx.y * E + e] = acc;
}

// ---------------------------------------------------------------- pool

// 2x2/2 max pool of gridDim.y (1 .. kMaxGroup) micro-batches (blockIdx.y
// selects x[k] / y[k]).
template <typename T>
struct PoolGroup {
  const T* x[kMaxGroup];
  T* y[kMaxGroup];
};
template <typename T>
__global__ __launch_bounds__(256) void maxpool_fwd_k(PoolGroup<T> pg, int nb, int H, int W, int C) {
  const T* __restrict__ x = pickg(pg.x, blockIdx.y);
  T* __restrict__ y = pickg(pg.y, blockIdx.y);
  constexpr int N = Pk<T>::N;
  int CP = C / N, H2 = H / 2, W2 = W / 2;
  long e = (long)blockIdx.x * 256 + threadIdx.x;
  long total = (long)nb * H2 * W2 * CP;
  if (e >= total) return;
  int cp = e % CP;
  long r = e / CP;
  int w2 = r % W2;
  r /= W2;
  int h2 = r % H2;
  int n = r / H2;
  const T* base = x + (((long)n * H + 2 * h2) * W + 2 * w2) * C + cp * N;
  float m[N], v[N];
  Pk<T>::un(ld16(base), m);
  const long off[3] = {C, (long)W * C, (long)W * C + C};
#pragma unroll
  for (int k = 0; k < 3; ++k) {
    Pk<T>::un(ld16(base + off[k]), v);
#pragma unroll
    for (int i = 0; i < N; ++i) m[i] = v[i] > m[i] ? v[i] : m[i];
  }
  st16(y + e * N, Pk<T>::pk(m));
}

template <typename T>
__global__ __launch_bounds__(256) void maxpool_bwd_k(const T* __restrict__ x, const T* __restrict__ dy,
                                                     T* __restrict__ dx, int nb, int H, int W, int C) {
  constexpr int N = Pk<T>::N;
  int CP = C / N, H2 = H / 2, W2 = W / 2;
  long e = (long)blockIdx.x * 256 + threadIdx.x;
  long total = (long)nb * H2 * W2 * CP;
  if (e >= total) return;
  int cp = e % CP;
  long r = e / CP;
  int w2 = r % W2;
  r /= W2;
  int h2 = r % H2;
  int n = r / H2;
  long o = (((long)n * H + 2 * h2) * W + 2 * w2) * C + cp * N;
  const long off[4] = {0, C, (long)W * C, (long)W * C + C};
  float v[4][N], g[N];
#pragma unroll
  for (int k = 0; k < 4; ++k) Pk<T>::un(ld16(x + o + off[k]), v[k]);
  Pk<T>::un(ld16(dy + e * N), g);
  float out[4][N];
#pragma unroll
  for (int i = 0; i < N; ++i) {
    int arg = 0;
    float best = v[0][i];
#pragma unroll
    for (int k = 1; k < 4; ++k)
      if (v[k][i] > best) { best = v[k][i]; arg = k; }
#pragma unroll
    for (int k = 0; k < 4; ++k) out[k][i] = (k == arg) ? g[i] : 0.f;
  }
#pragma unroll
  for (int k = 0; k < 4; ++k) st16(dx + o + off[k], Pk<T>::pk(out[k]));
}

// ---------------------------------------------------------------- upsample-concat

template <typename T>
__global__ __launch_bounds__(256) void upcat_fwd_k(const T* __restrict__ prev, const T* __restrict__ skip,
                                                   T* __restrict__ out, int nb, int H, int W, int C1,
                                                   int C2) {
  constexpr int N = Pk<T>::N;
  int C = C1 + C2, CP = C / N;
  long e = (long)blockIdx.x * 256 + threadIdx.x;
  long total = (long)nb * H * W * CP;
  if (e >= total) return;
  int cp = e % CP;
  long p = e / CP;
  int w = p % W;
  long r = p / W;
  int h = r % H;
  int n = r / H;
  int c = cp * N;
  uint4 v;
  if (c < C1)
    v = ld16(prev + (((long)n * (H / 2) + h / 2) * (W / 2) + w / 2) * C1 + c);
  else
    v = ld16(skip + p * C2 + (c - C1));
  st16(out + p * C + c, v);
}

template <typename T>
__global__ __launch_bounds__(256) void upcat_bwd_prev_k(const T* __restrict__ dcat, T* __restrict__ dprev,
                                                        int nb, int H, int W, int C1, int C2) {
  constexpr int N = Pk<T>::N;
  int C = C1 + C2, CP = C1 / N, H2 = H / 2, W2 = W / 2;
  long e = (long)blockIdx.x * 256 + threadIdx.x;
  long total = (long)nb * H2 * W2 * CP;
  if (e >= total) return;
  int cp = e % CP;
  long r = e / CP;
  int w2 = r % W2;
  r /= W2;
  int h2 = r % H2;
  int n = r / H2;
  long o = (((long)n * H + 2 * h2) * W + 2 * w2) * C + cp * N;
  const long off[4] = {0, C, (long)W * C, (long)W * C + C};
  float s[N], v[N];
  Pk<T>::un(ld16(dcat + o), s);
#pragma unroll
  for (int k = 1; k < 4; ++k) {
    Pk<T>::un(ld16(dcat + o + off[k]), v);
#pragma unroll
    for (int i = 0; i < N; ++i) s[i] += v[i];
  }
  st16(dprev + e * N, Pk<T>::pk(s));
}

template <typename T>
__global__ __launch_bounds__(256) void upcat_bwd_skip_k(const T* __restrict__ dcat, T* __restrict__ dskip,
                                                        long P, int C1, int C2) {
  constexpr int N = Pk<T>::N;
  int CP = C2 / N;
  long e = (long)blockIdx.x * 256 + threadIdx.x;
  if (e >= P * CP) return;
  int cp = e % CP;
  long p = e / CP;
  st16(dskip + p * C2 + cp * N, ld16(dcat + p * (C1 + C2) + C1 + cp * N));
}

// ---------------------------------------------------------------- loss / accumulate

template <typename T>
__global__ __launch_bounds__(256) void mse_k(const T* __restrict__ y, const T* __restrict__ t,
                                             T* __restrict__ dy, float* __restrict__ part, long n,
                                             float inv_numel, long per_block) {
  __shared__ float red[256];
  long b0 = (long)blockIdx.x * per_block, b1 = b0 + per_block < n ? b0 + per_block : n;
  float s = 0.f;
  for (long e = b0 + threadIdx.x; e < b1; e += 256) {
    float d = Elt<T>::ld(y + e) - Elt<T>::ld(t + e);
    s += d * d;
    Elt<T>::st(dy + e, 2.0f * d * inv_numel);
  }
  red[threadIdx.x] = s;
  __syncthreads();
  for (int k = 128; k > 0; k >>= 1) {
    if (threadIdx.x < k) red[threadIdx.x] += red[threadIdx.x + k];
    __syncthreads();
  }
  if (threadIdx.x == 0) part[blockIdx.x] = red[0];
}

__global__ void serial_sum_k(const float* __restrict__ a, int n, float scale,
                             float* __restrict__ out) {
  if (threadIdx.x != 0 || blockIdx.x != 0) return;
  float s = 0.f;
  for (int i = 0; i < n; ++i) s += a[i];
  *out = s * scale;
}

__global__ __launch_bounds__(256) void accumulate_k(float* __restrict__ acc, const float* __restrict__ g,
                                                    long n, int overwrite) {
  long e0 = ((long)blockIdx.x * 256 + threadIdx.x) * 4;
  if (e0 >= n) return;
  if (e0 + 4 <= n) {
    float4 v = *(const float4*)(g + e0);
    if (!overwrite) {
      float4 a = *(const float4*)(acc + e0);
      v.x = a.x + v.x; v.y = a.y + v.y; v.z = a.z + v.z; v.w = a.w + v.w;
    }
    *(float4*)(acc + e0) = v;
  } else {
    for (long e = e0; e < n; ++e) acc[e] = overwrite ? g[e] : acc[e] + g[e];
  }
}

// acc_k = r_k or acc_k + r_k with r_k = sum_{s < S_k} g_k[s n_k + e], every
// entry in one launch.  Tiles blk0[k] .. blk0[k + 1] - 1 serve entry k.  A
// tile of 1024 threads covers C4 float4 columns with LANES = 1024 / C4
// split lanes; lane l sums s = l, l + LANES, .. in ascending order, then the
// lanes are added pairwise in LDS (lane l takes lane l + h for h = LANES / 2,
// .., 1), with (C4, LANES) a function of S only, so the sum is fixed by the
// shape.  An entry with n not a multiple of 4 takes one element per thread,
// s ascending.
__host__ __device__ __forceinline__ int acc_c4(int S) {
  // about four slices per split lane: C4 = 4096 / S rounded down to a power
  // of two, within 1 .. 1024 (a bias gradient's hundreds of block sums then
  // spread over several tiles instead of one long one)
  int c = 1024;
  while (c > 1 && (long)c * S > 4096) c >>= 1;
  return c;
}

// NG: micro-batches per entry as a template constant (1) or b.ng (0).
template <int NG>
__global__ __launch_bounds__(1024) void reduce_accumulate_k(AccBatch b, int overwrite,
                                                            int ntiles) {
  // blocks are persistent over tiles (tile = the block of the layout above),
  // so the entry lookup and the block start are paid once per block
  __shared__ float4 red[1024];
  const int ng = NG ? NG : b.ng;
  int k = 0;   // entry of the current tile (tiles only increase)
  for (int tile = blockIdx.x; tile < ntiles; tile += gridDim.x) {
    while (k + 1 < b.count && tile >= b.blk0[k + 1]) ++k;
    const long bx = (long)tile - b.blk0[k];
    const long E = b.n[k];
    const int S = b.S[k];
    float* __restrict__ acc = b.acc[k];
    if (E % 4) {   // tile-uniform
      const long e = bx * 1024 + threadIdx.x;
      if (e < E) {
        float cur = 0.f;
        for (int q = 0; q < ng; ++q) {
          const float* __restrict__ part = b.g[k] + q * b.gstride[k];
          float r = 0.f;
          for (int s = 0; s < S; ++s) r += part[(long)s * E + e];
          cur = q > 0 ? cur + r : overwrite ? r : acc[e] + r;
        }
        acc[e] = cur;
      }
      continue;
    }
    const int C4 = acc_c4(S), LANES = 1024 / C4;
    const int col = threadIdx.x % C4, lane = threadIdx.x / C4;
    const long e4 = (bx * C4 + col) * 4;
    float4 cur = make_float4(0.f, 0.f, 0.f, 0.f);   // the running sum (lane 0)
    for (int q = 0; q < ng; ++q) {
      const float* __restrict__ part = b.g[k] + q * b.gstride[k];
      float4 a = make_float4(0.f, 0.f, 0.f, 0.f);
      if (e4 < E) {
        // up to eight loads in flight per step; slices past S add zeros
        for (int s = lane; s < S; s += 8 * LANES) {
          float4 t[8];
#pragma unroll
          for (int u = 0; u < 8; ++u)
            t[u] = s + u * LANES < S ? *(const float4*)(part + (long)(s + u * LANES) * E + e4)
                                     : make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll
          for (int u = 0; u < 8; ++u) {
            a.x += t[u].x; a.y += t[u].y; a.z += t[u].z; a.w += t[u].w;
          }
        }
      }
      float4 r = a;
      if (LANES > 1) {   // tile-uniform
        red[lane * C4 + col] = a;
        __syncthreads();
        for (int h = LANES >> 1; h > 0; h >>= 1) {
          if (lane < h) {
            const float4 t = red[(lane + h) * C4 + col];
            r.x += t.x; r.y += t.y; r.z += t.z; r.w += t.w;
            red[lane * C4 + col] = r;
          }
          __syncthreads();
        }
        if (NG != 1) __syncthreads();   // red is rewritten by the next micro-batch
      }
      if (lane == 0 && e4 < E) {
        if (q > 0) {
          cur.x = cur.x + r.x; cur.y = cur.y + r.y; cur.z = cur.z + r.z; cur.w = cur.w + r.w;
        } else if (overwrite) {
          cur = r;
        } else {
          const float4 o = *(const float4*)(acc + e4);
          cur.x = o.x + r.x; cur.y = o.y + r.y; cur.z = o.z + r.z; cur.w = o.w + r.w;
        }
      }
    }
    if (lane == 0 && e4 < E) *(float4*)(acc + e4) = cur;
    if (NG == 1 && LANES > 1) __syncthreads();   // red is rewritten by the next tile
  }
}

inline bool al16(const void* p) { return ((uintptr_t)p & 15) == 0; }

}  // namespace

// ---------------------------------------------------------------- dispatch

static long relu_bias_rows(long P, int C, int N);

// The 1x1 path for few output channels (the network head).
static bool small1x1_ok(int dt, const ConvShape& s, const void* x) {
  const int N = dt == 0 ? 8 : 4;
  if (s.taps != 1 || s.cout > kSmallCo || s.cin % N || !al16(x)) return false;
  const int CP = s.cin / N;
  return CP <= 256 && 256 % CP == 0;
}

hipError_t conv_forward(int dt, const void* x, const void* w, const float* b, void* y,
                        const ConvShape& s, int relu, float* part, size_t part_cap,
                        hipStream_t st) {
  if (mfma_conv_ok(dt, s.cin, s.cout))
    return conv_forward_mfma(x, w, b, y, s, relu, part, part_cap, st);
  if (small1x1_ok(dt, s, x)) {
    const long P = s.pixels();
    ProfScope ps("conv1x1_small_fwd", 2.0 * P * s.cout * s.cin,
                 (dt == 0 ? 2.0 : 4.0) * P * (s.cin + s.cout), st);
    if (dt == 0)
      TGP_LAUNCH(ps, conv1x1_small_fwd_k<bf16_t>, dim3(cdiv(P, 256)), dim3(256), 0, st,
                 (const bf16_t*)x, (const bf16_t*)w, b, (bf16_t*)y, P, s.cin, s.cout, relu);
    else
      TGP_LAUNCH(ps, conv1x1_small_fwd_k<float>, dim3(cdiv(P, 256)), dim3(256), 0, st,
                 (const float*)x, (const float*)w, b, (float*)y, P, s.cin, s.cout, relu);
    return launch_status();
  }
  long P = s.pixels();
  dim3 g(cdiv(P * s.cout, 256));
  int esz = dt == 0 ? 2 : 4;
  ProfScope ps("conv_fwd_direct", 2.0 * P * s.cout * s.taps * s.cin,
               (double)esz * (P * s.cin + (double)s.cout * s.taps * s.cin + P * s.cout), st);
  if (dt == 0)
    TGP_LAUNCH(ps, conv_fwd_direct<bf16_t>, g, dim3(256), 0, st, (const bf16_t*)x,
                       (const bf16_t*)w, b, (bf16_t*)y, P, s.H, s.W, s.cin, s.cout, s.taps, relu);
  else
    TGP_LAUNCH(ps, conv_fwd_direct<float>, g, dim3(256), 0, st, (const float*)x,
                       (const float*)w, b, (float*)y, P, s.H, s.W, s.cin, s.cout, s.taps, relu);
  return launch_status();
}

bool conv_dgrad_uses_wt(int dt, const ConvShape& s) { return mfma_conv_ok(dt, s.cout, s.cin); }

hipError_t conv_dgrad(int dt, const void* dz, const void* w, const void* wt, void* dx,
                      const ConvShape& s, float* part, size_t part_cap, hipStream_t st) {
  if (conv_dgrad_uses_wt(dt, s)) {
    ConvShape t{s.nb, s.H, s.W, s.cout, s.cin, s.taps};
    t_in_dgrad = 1;
    const hipError_t e = conv_forward_mfma(dz, wt, nullptr, dx, t, 0, part, part_cap, st);
    t_in_dgrad = 0;
    return e;
  }
  long P = s.pixels();
  dim3 g(cdiv(P * s.cin, 256));
  int esz = dt == 0 ? 2 : 4;
  ProfScope ps("conv_dgrad_direct", 2.0 * P * s.cout * s.taps * s.cin,
               (double)esz * (P * s.cin + (double)s.cout * s.taps * s.cin + P * s.cout), st);
  if (dt == 0)
    TGP_LAUNCH(ps, conv_dgrad_direct<bf16_t>, g, dim3(256), 0, st, (const bf16_t*)dz,
                       (const bf16_t*)w, (bf16_t*)dx, P, s.H, s.W, s.cin, s.cout, s.taps);
  else
    TGP_LAUNCH(ps, conv_dgrad_direct<float>, g, dim3(256), 0, st, (const float*)dz,
                       (const float*)w, (float*)dx, P, s.H, s.W, s.cin, s.cout, s.taps);
  return launch_status();
}

size_t conv_wgrad_partial_floats(int dt, const ConvShape& s) {
  if (mfma_conv_ok(dt, s.cin, s.cout)) return wgrad_mfma_partial_floats(s);
  const int N = dt == 0 ? 8 : 4;
  if (small1x1_ok(dt, s, (const void*)16)) {   // (alignment is checked per call)
    const size_t direct = (size_t)direct_wgrad_splits(s.pixels()) * s.cout * s.taps * s.cin;
    const size_t small = (size_t)cdiv(s.pixels(), relu_bias_rows(s.pixels(), s.cin, N)) * s.cout * s.cin;
    return direct > small ? direct : small;
  }
  return (size_t)direct_wgrad_splits(s.pixels()) * s.cout * s.taps * s.cin;
}

hipError_t conv_wgrad(int dt, const void* x, const void* dz, float* dw, float* partial,
                      const ConvShape& s, hipStream_t st, const ReduceJob* extra,
                      ReduceJob* defer) {
  if (defer && extra) return hipErrorInvalidValue;
  if (mfma_conv_ok(dt, s.cin, s.cout))
    return conv_wgrad_mfma(x, dz, dw, partial, s, st, extra, defer);
  if (small1x1_ok(dt, s, x)) {
    const long P = s.pixels(), E = (long)s.cout * s.cin;
    const long rows = relu_bias_rows(P, s.cin, dt == 0 ? 8 : 4);
    const int nbk = cdiv(P, rows);
    {
      ProfScope ps("wgrad1x1_small", 2.0 * P * E,
                   (dt == 0 ? 2.0 : 4.0) * P * (s.cin + s.cout) + 4.0 * nbk * E, st);
      if (dt == 0)
        TGP_LAUNCH(ps, wgrad1x1_small_k<bf16_t>, dim3(nbk), dim3(256), 0, st, (const bf16_t*)x,
                   (const bf16_t*)dz, partial, P, s.cin, s.cout, rows);
      else
        TGP_LAUNCH(ps, wgrad1x1_small_k<float>, dim3(nbk), dim3(256), 0, st, (const float*)x,
                   (const float*)dz, partial, P, s.cin, s.cout, rows);
    }
    const hipError_t e = launch_status();
    if (e != hipSuccess) return e;
    if (defer) {
      *defer = ReduceJob{partial, dw, E, nbk};
      return hipSuccess;
    }
    return splitk_reduce_launch(partial, dw, E, nbk, st, extra);
  }
  long P = s.pixels();
  long E = (long)s.cout * s.taps * s.cin;
  long pps = direct_wgrad_pps(P);
  int S = direct_wgrad_splits(P);
  dim3 g(cdiv(E, 256), S);
  {
  int esz = dt == 0 ? 2 : 4;
  ProfScope ps("conv_wgrad_direct", 2.0 * P * E, (double)esz * P * (s.cin + s.cout) + 4.0 * S * E, st);
  if (dt == 0)
    TGP_LAUNCH(ps, conv_wgrad_direct<bf16_t>, g, dim3(256), 0, st, (const bf16_t*)x,
                       (const bf16_t*)dz, partial, P, s.H, s.W, s.cin, s.cout, s.taps, pps);
  else
    TGP_LAUNCH(ps, conv_wgrad_direct<float>, g, dim3(256), 0, st, (const float*)x,
                       (const float*)dz, partial, P, s.H, s.W, s.cin, s.cout, s.taps, pps);
  }
  hipError_t e = launch_status();
  if (e != hipSuccess) return e;
  if (defer) {
    *defer = ReduceJob{partial, dw, E, S};
    return hipSuccess;
  }
  return splitk_reduce_launch(partial, dw, E, S, st, extra);
}

hipError_t conv_forward_n(int dt, int n, const void* const* x, const void* w, const float* b,
                          void* const* y, const ConvShape& s, int relu, float* const* part,
                          size_t part_cap, hipStream_t st) {
  if (n < 1 || n > kMaxGroup) return hipErrorInvalidValue;
  if (mfma_conv_ok(dt, s.cin, s.cout))
    return conv_forward_mfma_n(n, x, w, b, y, s, relu, part, part_cap, st);
  for (int k = 0; k < n; ++k) {
    const hipError_t e = conv_forward(dt, x[k], w, b, y[k], s, relu, part[k], part_cap, st);
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

hipError_t conv_dgrad_n(int dt, int n, const void* const* dz, const void* w, const void* wt,
                        void* const* dx, const ConvShape& s, float* const* part,
                        size_t part_cap, hipStream_t st) {
  if (n < 1 || n > kMaxGroup) return hipErrorInvalidValue;
  if (conv_dgrad_uses_wt(dt, s)) {
    ConvShape t{s.nb, s.H, s.W, s.cout, s.cin, s.taps};
    t_in_dgrad = 1;
    const hipError_t e = conv_forward_mfma_n(n, dz, wt, nullptr, dx, t, 0, part, part_cap, st);
    t_in_dgrad = 0;
    return e;
  }
  for (int k = 0; k < n; ++k) {
    const hipError_t e = conv_dgrad(dt, dz[k], w, wt, dx[k], s, part[k], part_cap, st);
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

hipError_t conv_wgrad_n(int dt, int n, const void* const* x, const void* const* dz,
                        float* const* dw, float* const* part, const ConvShape& s, hipStream_t st,
                        ReduceJob* const* defer) {
  if (n < 1 || n > kMaxGroup) return hipErrorInvalidValue;
  for (int k = 0; k < n; ++k)
    if (!defer[k]) return hipErrorInvalidValue;
  if (mfma_conv_ok(dt, s.cin, s.cout)) return conv_wgrad_mfma_n(n, x, dz, dw, part, s, st, defer);
  for (int k = 0; k < n; ++k) {
    const hipError_t e = conv_wgrad(dt, x[k], dz[k], dw[k], part[k], s, st, nullptr, defer[k]);
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

bool dw_rows_ok(int dt, int nb, int H, int W, int C, const void* a, const void* b,
                const void* c) {
  return dw3_rows_ok(dt, nb, H, W, C, a, b, c);
}

hipError_t dw_forward_n(int n, const void* const* x, const void* w, const float* b,
                        void* const* y, int nb, int H, int W, int C, int relu, hipStream_t st) {
  if (n < 1 || n > kMaxGroup) return hipErrorInvalidValue;
  const long P = (long)nb * H * W;
  if (P == 0) return hipSuccess;
  DwIo io;
  for (int k = 0; k < kMaxGroup; ++k) {   // unused entries repeat the first
    io.x[k] = (const bf16_t*)x[k < n ? k : 0];
    io.y[k] = (bf16_t*)y[k < n ? k : 0];
  }
  const dim3 g((unsigned)cdiv((long)W * (C / 8), 256), (unsigned)(nb * cdiv(H, kDwRows)), n);
  ProfScope ps("dw3_rows_fwd", n * 18.0 * P * C, n * 4.0 * P * C, st);
  TGP_LAUNCH(ps, (dw3_rows_k<kDwRows, false>), g, dim3(256), 0, st, io, (const bf16_t*)w, b, H,
             W, C, relu);
  return launch_status();
}

hipError_t dw_dgrad_n(int n, const void* const* dz, const void* w, void* const* dx, int nb,
                      int H, int W, int C, hipStream_t st) {
  if (n < 1 || n > kMaxGroup) return hipErrorInvalidValue;
  const long P = (long)nb * H * W;
  if (P == 0) return hipSuccess;
  DwIo io;
  for (int k = 0; k < kMaxGroup; ++k) {
    io.x[k] = (const bf16_t*)dz[k < n ? k : 0];
    io.y[k] = (bf16_t*)dx[k < n ? k : 0];
  }
  const dim3 g((unsigned)cdiv((long)W * (C / 8), 256), (unsigned)(nb * cdiv(H, kDwRows)), n);
  ProfScope ps("dw3_rows_dgrad", n * 18.0 * P * C, n * 4.0 * P * C, st);
  TGP_LAUNCH(ps, (dw3_rows_k<kDwRows, true>), g, dim3(256), 0, st, io, (const bf16_t*)w,
             (const float*)nullptr, H, W, C, 0);
  return launch_status();
}

bool dw_dgrad_mask_ok(int nb, int H, int W, int C) {
  return C % 8 == 0 && 256 % (C / 8) == 0 && (long)W * (C / 8) % 256 == 0 &&
         (long)nb * cdiv(H, kDwRows) <= 65535 && 2.0 * nb * H * W * C < 2147483648.0;
}

int dw_dgrad_mask_rows(int nb, int H, int W, int C) {
  return (int)((long)W * (C / 8) / 256 * nb * cdiv(H, kDwRows));
}

hipError_t dw_dgrad_mask_n(int n, const void* const* dz, const void* w, void* const* dx,
                           const void* const* y, float* const* part, int nb, int H, int W, int C,
                           hipStream_t st) {
  if (n < 1 || n > kMaxGroup || !dw_dgrad_mask_ok(nb, H, W, C)) return hipErrorInvalidValue;
  const long P = (long)nb * H * W;
  if (P == 0) return hipSuccess;
  DwIo io;
  for (int k = 0; k < kMaxGroup; ++k) {
    const int q = k < n ? k : 0;
    io.x[k] = (const bf16_t*)dz[q];
    io.y[k] = (bf16_t*)dx[q];
    io.m[k] = (const bf16_t*)y[q];
    io.part[k] = part[q];
    if (!io.x[k] || !io.y[k] || !io.m[k] || !io.part[k]) return hipErrorInvalidValue;
  }
  const dim3 g((unsigned)((long)W * (C / 8) / 256), (unsigned)(nb * cdiv(H, kDwRows)), n);
  ProfScope ps("dw3_rows_dgrad_mask", n * 18.0 * P * C, n * 6.0 * P * C, st);
  TGP_LAUNCH(ps, (dw3_rows_k<kDwRows, true, true>), g, dim3(256), 0, st, io, (const bf16_t*)w,
             (const float*)nullptr, H, W, C, 0);
  return launch_status();
}

hipError_t dw_wgrad_n(int n, const void* const* x, const void* const* dz, float* const* dw,
                      float* const* part, int nb, int H, int W, int C, hipStream_t st,
                      ReduceJob* const* defer) {
  if (n < 1 || n > kMaxGroup) return hipErrorInvalidValue;
  const long P = (long)nb * H * W;
  const long E = (long)C * 9;
  if (P == 0) return hipSuccess;
  const int S = dw3_wgrad_blocks(nb, H, W, C);
  DwWgIo io;
  for (int k = 0; k < kMaxGroup; ++k) {
    io.x[k] = (const bf16_t*)x[k < n ? k : 0];
    io.dz[k] = (const bf16_t*)dz[k < n ? k : 0];
    io.part[k] = part[k < n ? k : 0];
  }
  const dim3 g((unsigned)cdiv((long)W * (C / 8), 256), (unsigned)(nb * cdiv(H, kDwWgradRows)), n);
  {
    ProfScope ps("dw3_wgrad_rows", n * 18.0 * P * C, n * (4.0 * P * C + 4.0 * S * E), st);
    TGP_LAUNCH(ps, (dw3_wgrad_rows_k<kDwWgradRows>), g, dim3(256), 0, st, io, H, W, C);
  }
  hipError_t e = launch_status();
  if (defer) {   // left to the caller's accumulation, in the same order
    for (int k = 0; k < n; ++k) *defer[k] = ReduceJob{part[k], dw[k], E, S};
    return e;
  }
  // the sums, two per reduction launch
  for (int k = 0; k < n && e == hipSuccess; k += 2) {
    if (k + 1 < n) {
      const ReduceJob second{part[k + 1], dw[k + 1], E, S};
      e = splitk_reduce_launch(part[k], dw[k], E, S, st, &second);
    } else {
      e = splitk_reduce_launch(part[k], dw[k], E, S, st);
    }
  }
  return e;
}

hipError_t dw_forward(int dt, const void* x, const void* w, const float* b, void* y, int nb,
                      int H, int W, int C, int relu, hipStream_t st) {
  long P = (long)nb * H * W;
  if (dw3_rows_ok(dt, nb, H, W, C, x, w, y))
    return dw_forward_n(1, &x, w, b, &y, nb, H, W, C, relu, st);
  dim3 g(cdiv(P * C, 256));
  ProfScope ps("dw_forward", 18.0 * P * C, (dt == 0 ? 4.0 : 8.0) * P * C, st);
  if (dt == 0)
    TGP_LAUNCH(ps, dw_fwd<bf16_t>, g, dim3(256), 0, st, (const bf16_t*)x, (const bf16_t*)w,
                       b, (bf16_t*)y, P, H, W, C, relu);
  else
    TGP_LAUNCH(ps, dw_fwd<float>, g, dim3(256), 0, st, (const float*)x, (const float*)w, b,
                       (float*)y, P, H, W, C, relu);
  return launch_status();
}

hipError_t dw_dgrad(int dt, const void* dz, const void* w, void* dx, int nb, int H, int W,
                    int C, hipStream_t st) {
  long P = (long)nb * H * W;
  if (dw3_rows_ok(dt, nb, H, W, C, dz, w, dx))
    return dw_dgrad_n(1, &dz, w, &dx, nb, H, W, C, st);
  dim3 g(cdiv(P * C, 256));
  ProfScope ps("dw_dgrad", 18.0 * P * C, (dt == 0 ? 4.0 : 8.0) * P * C, st);
  if (dt == 0)
    TGP_LAUNCH(ps, dw_dgrad_k<bf16_t>, g, dim3(256), 0, st, (const bf16_t*)dz,
                       (const bf16_t*)w, (bf16_t*)dx, P, H, W, C);
  else
    TGP_LAUNCH(ps, dw_dgrad_k<float>, g, dim3(256), 0, st, (const float*)dz,
                       (const float*)w, (float*)dx, P, H, W, C);
  return launch_status();
}

size_t dw_wgrad_partial_floats(int nb, int H, int W, int C) {
  long P = (long)nb * H * W;
  const size_t direct = (size_t)direct_wgrad_splits(P) * C * 9;
  const size_t rows = (C % 8 == 0 && C > 0 && 256 % (C / 8) == 0)
                          ? (size_t)dw3_wgrad_blocks(nb, H, W, C) * C * 9
                          : 0;
  return direct > rows ? direct : rows;
}

hipError_t dw_wgrad(int dt, const void* x, const void* dz, float* dw, float* partial, int nb,
                    int H, int W, int C, hipStream_t st) {
  long P = (long)nb * H * W;
  long E = (long)C * 9;
  if (dw3_rows_ok(dt, nb, H, W, C, x, dz, partial) && P > 0)
    return dw_wgrad_n(1, &x, &dz, &dw, &partial, nb, H, W, C, st);
  long pps = direct_wgrad_pps(P);
  int S = direct_wgrad_splits(P);
  dim3 g(cdiv(E, 256), S);
  {
  ProfScope ps("dw_wgrad", 18.0 * P * C, (dt == 0 ? 4.0 : 8.0) * P * C + 4.0 * S * E, st);
  if (dt == 0)
    TGP_LAUNCH(ps, dw_wgrad_k<bf16_t>, g, dim3(256), 0, st, (const bf16_t*)x,
                       (const bf16_t*)dz, partial, P, H, W, C, pps);
  else
    TGP_LAUNCH(ps, dw_wgrad_k<float>, g, dim3(256), 0, st, (const float*)x,
                       (const float*)dz, partial, P, H, W, C, pps);
  }
  hipError_t e = launch_status();
  if (e != hipSuccess) return e;
  return splitk_reduce_launch(partial, dw, E, S, st);
}

hipError_t relu_backward(int dt, const void* dy, const void* dskip, const void* y, void* dz,
                         int relu, long n, hipStream_t st) {
  int N = dt == 0 ? 8 : 4;
  int vec = al16(dy) && al16(dz) && (!dskip || al16(dskip)) && (!relu || al16(y)) ? 1 : 0;
  dim3 g(cdiv(n, 256L * N));
  ProfScope ps("relu_backward", 0.0, (dt == 0 ? 2.0 : 4.0) * n * (3 + (dskip ? 1 : 0) - (relu ? 0 : 1)), st);
  if (dt == 0)
    TGP_LAUNCH(ps, relu_bwd_k<bf16_t>, g, dim3(256), 0, st, (const bf16_t*)dy,
                       (const bf16_t*)dskip, (const bf16_t*)y, (bf16_t*)dz, relu, n, vec);
  else
    TGP_LAUNCH(ps, relu_bwd_k<float>, g, dim3(256), 0, st, (const float*)dy,
                       (const float*)dskip, (const float*)y, (float*)dz, relu, n, vec);
  return launch_status();
}

static long colsum_rows(long P) { return P < 1024 ? (P < 1 ? 1 : P) : 1024; }
size_t colsum_partial_floats(long P, int C) {
  return (size_t)cdiv(P, colsum_rows(P)) * C;
}

// Rows per block of the fused ReLU-backward / bias kernel: about 1024 blocks
// (a multiple of the block's row lanes), so deep layers with few pixels and
// many channels still fill the chip.
static long relu_bias_rows(long P, int C, int N) {
  int nl = 256 / (C / N);
  long r = (P + 1023) / 1024;
  r = (r + nl - 1) / nl * nl;
  return r < nl ? nl : r;
}
bool relu_bias_fusable(int dt, int C, const void* dy, const void* dskip, const void* y,
                       const void* dz) {
  int N = dt == 0 ? 8 : 4;
  if (C % N) return false;
  int CP = C / N;
  return CP <= 256 && 256 % CP == 0 && al16(dy) && al16(dz) && (!dskip || al16(dskip)) &&
         al16(y);
}
size_t relu_bias_partial_floats(int dt, long P, int C) {
  const int N = dt == 0 ? 8 : 4;
  if (C % N || C / N > 256 || 256 % (C / N)) return 0;   // not fusable
  // blocks over P pixels, or over the P / 4 windows of the pooled variant
  const long b1 = cdiv(P, relu_bias_rows(P, C, N));
  const long b2 = cdiv(P / 4, relu_bias_rows(P / 4, C, N));
  return (size_t)(b1 > b2 ? b1 : b2) * C;
}
bool pool_relu_bias_fusable(int dt, int C, int H, int W, const void* dp, const void* dskip,
                            const void* y, const void* dz) {
  return H % 2 == 0 && W % 2 == 0 && H >= 2 && W >= 2 && relu_bias_fusable(dt, C, dp, dskip, y, dz);
}

template <typename T>
static RbPtrs<T> rb_ptrs(const RbArgs& a) {
  return RbPtrs<T>{(const T*)a.dy, (const T*)a.dskip, (const T*)a.y, (T*)a.dz, a.partial};
}
// The group's pointer sets; unused entries repeat the first.
template <typename T>
static RbGroup<T> rb_group(int n, const RbArgs* a) {
  RbGroup<T> g;
  for (int k = 0; k < kMaxGroup; ++k) {
    const RbPtrs<T> p = rb_ptrs<T>(a[k < n ? k : 0]);
    g.dy[k] = p.dy;
    g.ds[k] = p.ds;
    g.y[k] = p.y;
    g.dz[k] = p.dz;
    g.part[k] = p.part;
  }
  return g;
}
// n within 1 .. kMaxGroup, all with or all without a skip gradient.
static bool rb_group_ok(int n, const RbArgs* a) {
  if (n < 1 || n > kMaxGroup) return false;
  for (int k = 1; k < n; ++k)
    if ((a[k].dskip == nullptr) != (a[0].dskip == nullptr)) return false;
  return true;
}

// The bias sums of n launched micro-batches: left pending (defer) or reduced.
static hipError_t rb_finish(int n, const RbArgs* a, long C, int nblk, hipStream_t st) {
  for (int k = 0; k < n; ++k) {
    if (a[k].defer) {
      *a[k].defer = ReduceJob{a[k].partial, a[k].db, C, nblk};
    } else {
      const hipError_t e = splitk_reduce_launch(a[k].partial, a[k].db, C, nblk, st);
      if (e != hipSuccess) return e;
    }
  }
  return hipSuccess;
}

hipError_t relu_backward_bias_n(int dt, int n, const RbArgs* a, int relu, long P, int C,
                                hipStream_t st) {
  if (!rb_group_ok(n, a)) return hipErrorInvalidValue;
  long rows = relu_bias_rows(P, C, dt == 0 ? 8 : 4);
  int nb = cdiv(P, rows);
  {
    ProfScope ps("relu_backward_bias", 0.0,
                 n * ((dt == 0 ? 2.0 : 4.0) * P * C * (3 + (a[0].dskip ? 1 : 0) - (relu ? 0 : 1)) +
                      4.0 * nb * C),
                 st);
    if (dt == 0)
      TGP_LAUNCH(ps, relu_bwd_bias_k<bf16_t>, dim3(nb, n), dim3(256), 0, st,
                 rb_group<bf16_t>(n, a), relu, P, C, rows);
    else
      TGP_LAUNCH(ps, relu_bwd_bias_k<float>, dim3(nb, n), dim3(256), 0, st,
                 rb_group<float>(n, a), relu, P, C, rows);
  }
  hipError_t e = launch_status();
  if (e != hipSuccess) return e;
  return rb_finish(n, a, C, nb, st);
}

hipError_t relu_backward_bias(int dt, const void* dy, const void* dskip, const void* y, void* dz,
                              int relu, float* db, float* partial, long P, int C,
                              hipStream_t st, ReduceJob* defer) {
  const RbArgs a{dy, dskip, y, dz, db, partial, defer};
  return relu_backward_bias_n(dt, 1, &a, relu, P, C, st);
}

hipError_t pool_relu_backward_bias_n(int dt, int n, const RbArgs* a, int relu, int nb, int H,
                                     int W, int C, hipStream_t st) {
  if (!rb_group_ok(n, a)) return hipErrorInvalidValue;
  for (int k = 0; k < n; ++k)
    if (!pool_relu_bias_fusable(dt, C, H, W, a[k].dy, a[k].dskip, a[k].y, a[k].dz))
      return hipErrorInvalidValue;
  const long P2 = (long)nb * (H / 2) * (W / 2);
  const long rows = relu_bias_rows(P2, C, dt == 0 ? 8 : 4);
  const int nbk = cdiv(P2, rows);
  {
    const double esz = dt == 0 ? 2.0 : 4.0;
    ProfScope ps("pool_relu_backward_bias", 0.0,
                 n * (esz * 4.0 * P2 * C * (2 + (a[0].dskip ? 1 : 0)) + esz * P2 * C +
                      4.0 * nbk * C),
                 st);
    if (dt == 0)
      TGP_LAUNCH(ps, pool_relu_bwd_bias_k<bf16_t>, dim3(nbk, n), dim3(256), 0, st,
                 rb_group<bf16_t>(n, a), relu, nb, H, W, C, rows);
    else
      TGP_LAUNCH(ps, pool_relu_bwd_bias_k<float>, dim3(nbk, n), dim3(256), 0, st,
                 rb_group<float>(n, a), relu, nb, H, W, C, rows);
  }
  hipError_t e = launch_status();
  if (e != hipSuccess) return e;
  return rb_finish(n, a, C, nbk, st);
}

hipError_t pool_relu_backward_bias(int dt, const void* dp, const void* dskip, const void* y,
                                   void* dz, int relu, float* db, float* partial, int nb, int H,
                                   int W, int C, hipStream_t st, ReduceJob* defer) {
  const RbArgs a{dp, dskip, y, dz, db, partial, defer};
  return pool_relu_backward_bias_n(dt, 1, &a, relu, nb, H, W, C, st);
}

hipError_t bias_grad(int dt, const void* dz, float* db, float* partial, long P, int C,
                     hipStream_t st) {
  long rows = colsum_rows(P);
  int nb = cdiv(P, rows);
  dim3 g(cdiv(C, 64), nb);
  {
  ProfScope ps("bias_colsum", 0.0, (dt == 0 ? 2.0 : 4.0) * P * C + 4.0 * nb * C, st);
  if (dt == 0)
    TGP_LAUNCH(ps, colsum_k<bf16_t>, g, dim3(256), 0, st, (const bf16_t*)dz, partial, P, C, rows);
  else
    TGP_LAUNCH(ps, colsum_k<float>, g, dim3(256), 0, st, (const float*)dz, partial, P, C, rows);
  }
  hipError_t e = launch_status();
  if (e != hipSuccess) return e;
  return splitk_reduce_launch(partial, db, C, nb, st);
}

template <typename T>
static PoolGroup<T> pool_group(int n, const void* const* x, void* const* y) {
  PoolGroup<T> g;
  for (int k = 0; k < kMaxGroup; ++k) {   // unused entries repeat the first
    g.x[k] = (const T*)x[k < n ? k : 0];
    g.y[k] = (T*)y[k < n ? k : 0];
  }
  return g;
}

hipError_t maxpool_forward_n(int dt, int n, const void* const* x, void* const* y, int nb, int H,
                             int W, int C, hipStream_t st) {
  if (n < 1 || n > kMaxGroup) return hipErrorInvalidValue;
  for (int k = 0; k < n; ++k)
    if (!x[k] || !y[k]) return hipErrorInvalidValue;
  int N = dt == 0 ? 8 : 4;
  long total = (long)nb * (H / 2) * (W / 2) * (C / N);
  dim3 g(cdiv(total, 256), n);
  ProfScope ps("maxpool_forward", 0.0, n * (dt == 0 ? 2.0 : 4.0) * nb * H * W * C * 1.25, st);
  if (dt == 0)
    TGP_LAUNCH(ps, maxpool_fwd_k<bf16_t>, g, dim3(256), 0, st, pool_group<bf16_t>(n, x, y), nb, H,
               W, C);
  else
    TGP_LAUNCH(ps, maxpool_fwd_k<float>, g, dim3(256), 0, st, pool_group<float>(n, x, y), nb, H,
               W, C);
  return launch_status();
}

hipError_t maxpool_forward(int dt, const void* x, void* y, int nb, int H, int W, int C,
                           hipStream_t st) {
  return maxpool_forward_n(dt, 1, &x, &y, nb, H, W, C, st);
}

hipError_t maxpool_backward(int dt, const void* x, const void* dy, void* dx, int nb, int H,
                            int W, int C, hipStream_t st) {
  int N = dt == 0 ? 8 : 4;
  long total = (long)nb * (H / 2) * (W / 2) * (C / N);
  dim3 g(cdiv(total, 256));
  ProfScope ps("maxpool_backward", 0.0, (dt == 0 ? 2.0 : 4.0) * nb * H * W * C * 2.25, st);
  if (dt == 0)
    TGP_LAUNCH(ps, maxpool_bwd_k<bf16_t>, g, dim3(256), 0, st, (const bf16_t*)x,
                       (const bf16_t*)dy, (bf16_t*)dx, nb, H, W, C);
  else
    TGP_LAUNCH(ps, maxpool_bwd_k<float>, g, dim3(256), 0, st, (const float*)x,
                       (const float*)dy, (float*)dx, nb, H, W, C);
  return launch_status();
}

hipError_t upcat_forward(int dt, const void* prev, const void* skip, void* out, int nb, int H,
                         int W, int C1, int C2, hipStream_t st) {
  int N = dt == 0 ? 8 : 4;
  long total = (long)nb * H * W * ((C1 + C2) / N);
  dim3 g(cdiv(total, 256));
  ProfScope ps("upcat_forward", 0.0, (dt == 0 ? 2.0 : 4.0) * nb * H * W * (0.25 * C1 + C2 + C1 + C2), st);
  if (dt == 0)
    TGP_LAUNCH(ps, upcat_fwd_k<bf16_t>, g, dim3(256), 0, st, (const bf16_t*)prev,
                       (const bf16_t*)skip, (bf16_t*)out, nb, H, W, C1, C2);
  else
    TGP_LAUNCH(ps, upcat_fwd_k<float>, g, dim3(256), 0, st, (const float*)prev,
                       (const float*)skip, (float*)out, nb, H, W, C1, C2);
  return launch_status();
}

hipError_t upcat_backward(int dt, const void* dcat, void* dprev, void* dskip, int nb, int H,
                          int W, int C1, int C2, hipStream_t st) {
  int N = dt == 0 ? 8 : 4;
  long t1 = (long)nb * (H / 2) * (W / 2) * (C1 / N);
  long P = (long)nb * H * W;
  ProfScope ps("upcat_backward", 0.0, (dt == 0 ? 2.0 : 4.0) * P * (C1 + 0.25 * C1 + 2.0 * C2), st);
  if (dt == 0) {
    TGP_LAUNCH(ps, upcat_bwd_prev_k<bf16_t>, dim3(cdiv(t1, 256)), dim3(256), 0, st,
                       (const bf16_t*)dcat, (bf16_t*)dprev, nb, H, W, C1, C2);
    TGP_LAUNCH(ps, upcat_bwd_skip_k<bf16_t>, dim3(cdiv(P * (C2 / N), 256)), dim3(256), 0, st,
                       (const bf16_t*)dcat, (bf16_t*)dskip, P, C1, C2);
  } else {
    TGP_LAUNCH(ps, upcat_bwd_prev_k<float>, dim3(cdiv(t1, 256)), dim3(256), 0, st,
                       (const float*)dcat, (float*)dprev, nb, H, W, C1, C2);
    TGP_LAUNCH(ps, upcat_bwd_skip_k<float>, dim3(cdiv(P * (C2 / N), 256)), dim3(256), 0, st,
                       (const float*)dcat, (float*)dskip, P, C1, C2);
  }
  return launch_status();
}

static long mse_per_block(long n) { return n < 4096 ? 4096 : 16384; }
size_t mse_partial_floats(long n) { return (size_t)cdiv(n, mse_per_block(n)); }

hipError_t mse_forward_backward(int dt, const void* y, const void* t, void* dy,
                                float* loss_part, float* partial, long n, float inv_numel,
                                hipStream_t st) {
  long pb = mse_per_block(n);
  int nb = cdiv(n, pb);
  {
  ProfScope ps("mse", 3.0 * n, (dt == 0 ? 6.0 : 12.0) * n, st);
  if (dt == 0)
    TGP_LAUNCH(ps, mse_k<bf16_t>, dim3(nb), dim3(256), 0, st, (const bf16_t*)y,
                       (const bf16_t*)t, (bf16_t*)dy, partial, n, inv_numel, pb);
  else
    TGP_LAUNCH(ps, mse_k<float>, dim3(nb), dim3(256), 0, st, (const float*)y,
                       (const float*)t, (float*)dy, partial, n, inv_numel, pb);
  }
  hipError_t e = launch_status();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(serial_sum_k, dim3(1), dim3(64), 0, st, (const float*)partial, nb, 1.0f,
                     loss_part);
  return launch_status();
}

hipError_t loss_finalize(const float* parts, int m, float inv_numel, float* loss,
                         hipStream_t st) {
  hipLaunchKernelGGL(serial_sum_k, dim3(1), dim3(64), 0, st, parts, m, inv_numel, loss);
  return launch_status();
}

hipError_t grad_accumulate_batch(AccBatch b, int overwrite, hipStream_t st) {
  if (b.count < 0 || b.count > kMaxAcc || b.ng < 1 || b.ng > kMaxGroup) return hipErrorInvalidValue;
  long blocks = 0;
  double bytes = 0;
  int used = 0;
  for (int k = 0; k < b.count; ++k) {
    if (b.n[k] <= 0 || b.S[k] < 1) continue;
    b.acc[used] = b.acc[k]; b.g[used] = b.g[k]; b.gstride[used] = b.gstride[k];
    b.n[used] = b.n[k]; b.S[used] = b.S[k];
    b.blk0[used] = (int)blocks;
    const int C4 = acc_c4(b.S[k]);
    blocks += b.n[k] % 4 ? cdiv(b.n[k], 1024L) : cdiv(b.n[k], 4L * C4);
    bytes += 4.0 * b.n[k] * ((double)b.S[k] * b.ng + (overwrite ? 1 : 2));
    ++used;
  }
  b.count = used;
  if (used == 0) return hipSuccess;
  if (blocks >= (1L << 31)) return hipErrorInvalidValue;
  ProfScope ps("reduce_accumulate", 0.0, bytes, st);
  const unsigned grid = (unsigned)(blocks < 512 ? blocks : 512);   // two blocks per CU
  if (b.ng == 1)
    TGP_LAUNCH(ps, reduce_accumulate_k<1>, dim3(grid), dim3(1024), 0, st, b, overwrite,
               (int)blocks);
  else
    TGP_LAUNCH(ps, reduce_accumulate_k<0>, dim3(grid), dim3(1024), 0, st, b, overwrite,
               (int)blocks);
  return launch_status();
}

hipError_t grad_accumulate(float* acc, const float* g, long n, int overwrite, hipStream_t st) {
  ProfScope ps("grad_accumulate", (double)n, (overwrite ? 8.0 : 12.0) * n, st);
  TGP_LAUNCH(ps, accumulate_k, dim3(cdiv(n, 1024)), dim3(256), 0, st, acc, g, n, overwrite);
  return launch_status();
}

}  // namespace tgpk
