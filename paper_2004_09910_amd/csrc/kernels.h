// Internal launcher interface between the host runtime and the HIP kernels.
// Every launcher enqueues on `st` and returns the launch status.  dt selects
// the storage type of activations and weights: 0 = bfloat16, 1 = float32.
#pragma once
#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace tgpk {

// Micro-batches of one layer that one launch may cover (the same shape and
// weights, separate tensors).
constexpr int kMaxGroup = 16;

// One convolution at one micro-batch: nb samples of H x W, NHWC.
struct ConvShape {
  int nb, H, W, cin, cout, taps;  // taps = 9 (3x3, pad 1) or 1 (1x1)
  long pixels() const { return (long)nb * H * W; }
};

// y = act(conv(x, w) + b); w is KRSC [cout][taps][cin].  Deep shapes split
// the K loop; their fp32 partials go to `part` (conv_forward_partial_floats
// floats; part_cap is the space available).
size_t conv_forward_partial_floats(int dt, const ConvShape& s);
hipError_t conv_forward(int dt, const void* x, const void* w, const float* b, void* y,
                        const ConvShape& s, int relu, float* part, size_t part_cap,
                        hipStream_t st);
// 16x16x32-MFMA 3x3 convolution on row-aligned tiles (bf16; Cin % 32 == 0,
// Cout % 64 == 0, Cout <= 1024): whether it supports a shape, and the launch
// (y = act(conv(x, w) + b), or the data gradient when given the transformed
// weight and no bias).
bool conv_rowtile_ok(const ConvShape& s);
hipError_t conv_forward_rowtile(const void* x, const void* w, const float* b, void* y,
                                const ConvShape& s, int relu, hipStream_t st);
extern int g_rowtile_cfg;
// 32x32x16-MFMA 3x3 convolution on whole-row tiles with all nine taps per
// 16-channel stage (bf16; W in {24, 48, 96, 192}, Cin % 16 == 0, Cout % 64
// == 0): whether it supports a shape, and the launch over n (1 ..
// kMaxGroup) micro-batches x[k] -> y[k] (same contract as
// conv_forward_rowtile for each).
int conv_rows32_tiles(const ConvShape& s);
bool conv_rows32_ok(const ConvShape& s);
hipError_t conv_forward_rows32(int n, const void* const* x, const void* w, const float* b,
                               void* const* y, const ConvShape& s, int relu, hipStream_t st);
extern int g_rows32_cfg;
extern int g_rows32_ch;
extern int g_wgrad_ks;
extern int g_rowtile_mask;
extern thread_local int t_in_dgrad;
// Row-blocked 3x3 weight gradient on 32x32x16 MFMA with transpose LDS reads
// (bf16; W in {48, 96, 192}, Cin and Cout multiples of 64): whether it
// supports a shape, the fp32 partial-slice scratch it needs, and the launch
// (dw = sum over pixels, summed over its K ranges in a fixed order).
// out[e] = sum_{k < S} part[k E + e] in a fixed order that depends only on
// (E, S); `extra`, if given, is a second independent sum of the same kind run
// in the same launch (its order then also depends on the first sum's S).
struct ReduceJob {
  const float* part;
  float* out;
  long E;
  int S;
};
hipError_t splitk_reduce_launch(const float* part, float* out, long E, int S, hipStream_t st,
                               const ReduceJob* extra = nullptr);
bool wgrad_rows_ok(const ConvShape& s);
size_t wgrad_rows_partial_floats(const ConvShape& s);
hipError_t conv_wgrad_rows_launch(const void* x, const void* dz, float* dw, float* partial,
                                  const ConvShape& s, hipStream_t st,
                                  const ReduceJob* extra = nullptr, ReduceJob* defer = nullptr);
// n (1 .. kMaxGroup) micro-batches in one launch, each sum left pending in
// *defer[k].
hipError_t conv_wgrad_rows_launch_n(int n, const void* const* x, const void* const* dz,
                                    float* const* dw, float* const* partial, const ConvShape& s,
                                    hipStream_t st, ReduceJob* const* defer);

// Whether the data-gradient kernel for this shape reads the transformed
// weight wt = [cin][taps][cout] (taps rotated by 180 degrees).
bool conv_dgrad_uses_wt(int dt, const ConvShape& s);
// Builds those transformed weights, wt[ci][tap'][co] = w[co][taps-1-tap'][ci],
// for up to kMaxWt tensors in one launch (passed by value).
constexpr int kMaxWt = 32;
struct WtBatch {
  int count;
  const void* w[kMaxWt];
  void* wt[kMaxWt];
  int cout[kMaxWt], cin[kMaxWt], taps[kMaxWt];
  int blk0[kMaxWt];   // first block of each tensor (filled by the launcher)
};
hipError_t weight_transform_batch(int dt, WtBatch b, hipStream_t st);
// dx[p][ci] = sum_{co,tap} dz[p - off(tap)][co] w[co][tap][ci]
hipError_t conv_dgrad(int dt, const void* dz, const void* w, const void* wt, void* dx,
                      const ConvShape& s, float* part, size_t part_cap, hipStream_t st);
// Weight gradient of one micro-batch into dw (float32, KRSC), via split-K
// partials in `partial` (conv_wgrad_partial_floats floats) reduced in fixed
// split order.  `extra`, if given, is a pending sum (the bias gradient's)
// that runs in the same reduction launch.  With `defer` (and no `extra`)
// only the partials are written and *defer describes the sum still to run
// (S = 1 with part = dw when the kernel wrote the gradient itself).
size_t conv_wgrad_partial_floats(int dt, const ConvShape& s);
hipError_t conv_wgrad(int dt, const void* x, const void* dz, float* dw, float* partial,
                      const ConvShape& s, hipStream_t st, const ReduceJob* extra = nullptr,
                      ReduceJob* defer = nullptr);

// The same three operations for n (1 .. kMaxGroup) micro-batches of one
// layer (the same weights, separate tensors; array element k is micro-batch
// k's): one launch where the chosen kernel takes them all, else launches of
// two and one, with the same values as n single calls.  conv_wgrad_n always
// leaves every sum pending (*defer[k]).
hipError_t conv_forward_n(int dt, int n, const void* const* x, const void* w, const float* b,
                          void* const* y, const ConvShape& s, int relu, float* const* part,
                          size_t part_cap, hipStream_t st);
hipError_t conv_dgrad_n(int dt, int n, const void* const* dz, const void* w, const void* wt,
                        void* const* dx, const ConvShape& s, float* const* part,
                        size_t part_cap, hipStream_t st);
hipError_t conv_wgrad_n(int dt, int n, const void* const* x, const void* const* dz,
                        float* const* dw, float* const* part, const ConvShape& s, hipStream_t st,
                        ReduceJob* const* defer);

// Depthwise 3x3 (pad 1), w = [c][9].
hipError_t dw_forward(int dt, const void* x, const void* w, const float* b, void* y, int nb,
                      int H, int W, int C, int relu, hipStream_t st);
hipError_t dw_dgrad(int dt, const void* dz, const void* w, void* dx, int nb, int H, int W,
                    int C, hipStream_t st);
size_t dw_wgrad_partial_floats(int nb, int H, int W, int C);
// n (1 .. kMaxGroup) micro-batches per launch for the bf16 row-window
// depthwise kernels, where dw_rows_ok holds for each micro-batch's tensors
// (a, b) and the weights or partial buffer c.  dw_wgrad_n reduces each sum
// at once (two per reduction launch), or with `defer` leaves sum k pending
// in *defer[k].
bool dw_rows_ok(int dt, int nb, int H, int W, int C, const void* a, const void* b,
                const void* c);
hipError_t dw_forward_n(int n, const void* const* x, const void* w, const float* b,
                        void* const* y, int nb, int H, int W, int C, int relu, hipStream_t st);
hipError_t dw_dgrad_n(int n, const void* const* dz, const void* w, void* const* dx, int nb,
                      int H, int W, int C, hipStream_t st);
// dw_dgrad_n whose stored result is the ReLU backward of the layer below
// (dz = dx where its output y > 0, else 0) and whose blocks leave that
// layer's bias-gradient column sums in part[k] (dw_dgrad_mask_rows rows of
// C floats, summed later in a fixed order); where dw_dgrad_mask_ok holds.
bool dw_dgrad_mask_ok(int nb, int H, int W, int C);
int dw_dgrad_mask_rows(int nb, int H, int W, int C);
hipError_t dw_dgrad_mask_n(int n, const void* const* dz, const void* w, void* const* dx,
                           const void* const* y, float* const* part, int nb, int H, int W, int C,
                           hipStream_t st);
hipError_t dw_wgrad_n(int n, const void* const* x, const void* const* dz, float* const* dw,
                      float* const* part, int nb, int H, int W, int C, hipStream_t st,
                      ReduceJob* const* defer = nullptr);
hipError_t dw_wgrad(int dt, const void* x, const void* dz, float* dw, float* partial, int nb,
                    int H, int W, int C, hipStream_t st);

// dz = (dy [+ dskip]) * [y > 0] (mask only when relu), stored in dt.
hipError_t relu_backward(int dt, const void* dy, const void* dskip, const void* y, void* dz,
                         int relu, long n, hipStream_t st);
// db[c] = sum_p dz[p][c] over P rows, fixed-order two-stage reduction.
size_t colsum_partial_floats(long P, int C);
hipError_t bias_grad(int dt, const void* dz, float* db, float* partial, long P, int C,
                     hipStream_t st);

// 2x2/2 max-pool of x (nb x H x W x C) into y; backward routes dy to the first
// maximal element of each window (row-major).
// n (1 .. kMaxGroup) micro-batches x[k] -> y[k] in one launch.
hipError_t maxpool_forward_n(int dt, int n, const void* const* x, void* const* y, int nb, int H,
                             int W, int C, hipStream_t st);
hipError_t maxpool_forward(int dt, const void* x, void* y, int nb, int H, int W, int C,
                           hipStream_t st);
hipError_t maxpool_backward(int dt, const void* x, const void* dy, void* dx, int nb, int H,
                            int W, int C, hipStream_t st);

// out (nb x H x W x (C1+C2)) = [nearest 2x upsample of prev (H/2 x W/2 x C1), skip].
hipError_t upcat_forward(int dt, const void* prev, const void* skip, void* out, int nb, int H,
                         int W, int C1, int C2, hipStream_t st);
// dprev = sum of 2x2 blocks of dcat[..., :C1]; dskip = dcat[..., C1:].
hipError_t upcat_backward(int dt, const void* dcat, void* dprev, void* dskip, int nb, int H,
                          int W, int C1, int C2, hipStream_t st);

// Squared-error part of one micro-batch: *loss_part = sum (y-t)^2 and
// dy = 2 (y-t) * inv_numel, fixed-order reduction.
size_t mse_partial_floats(long n);
hipError_t mse_forward_backward(int dt, const void* y, const void* t, void* dy,
                                float* loss_part, float* partial, long n, float inv_numel,
                                hipStream_t st);
// *loss = (sum_{i<m} parts[i]) * inv_numel, in order.
hipError_t loss_finalize(const float* parts, int m, float inv_numel, float* loss,
                         hipStream_t st);

// acc = g (overwrite) or acc + g, float32.
hipError_t grad_accumulate(float* acc, const float* g, long n, int overwrite, hipStream_t st);

// acc_k = r_k (overwrite) or acc_k + r_k, r_k = sum_{s < S_k} g_k[s n_k ..]
// (the pending split-K sums of one micro-batch's gradients), for up to
// kMaxAcc tensors in one launch (passed by value).  Each r_k is summed in a
// fixed order that depends on (n_k, S_k) only; it is not always the order
// of splitk_reduce_launch, so a layer's sums are either always left to the
// accumulation or always reduced at once.  With ng > 1 the launch does ng
// such accumulations in a row, micro-batch q's slices at g_k + q gstride_k:
// acc_k (+)= r_k(0), then acc_k += r_k(1), .., the same values as ng
// launches (overwrite applies to the first).
constexpr int kMaxAcc = 64;
struct AccBatch {
  int count;
  int ng;              // micro-batches per entry, 1 .. kMaxGroup
  float* acc[kMaxAcc];
  const float* g[kMaxAcc];
  long gstride[kMaxAcc];   // floats from one micro-batch's slices to the next's
  long n[kMaxAcc];
  int S[kMaxAcc];
  int blk0[kMaxAcc];   // first block of each entry (filled by the launcher)
};
hipError_t grad_accumulate_batch(AccBatch b, int overwrite, hipStream_t st);

// relu_backward fused with the bias gradient's column sums (fixed-order
// two-stage reduction), for layers where relu_bias_fusable() holds.
bool relu_bias_fusable(int dt, int C, const void* dy, const void* dskip, const void* y,
                       const void* dz);
size_t relu_bias_partial_floats(int dt, long P, int C);
// With `defer`, the bias gradient's column sums are left in `partial` and
// *defer describes the sum still to run (the caller passes it to conv_wgrad).
// One micro-batch's tensors for the fused ReLU-backward / bias-sum kernels
// (dy is the pool gradient for the pooled variant).
struct RbArgs {
  const void* dy;
  const void* dskip;
  const void* y;
  void* dz;
  float* db;
  float* partial;
  ReduceJob* defer;
};
// n (1 .. kMaxGroup) micro-batches of the same shape in one launch; all
// with or all without a skip gradient.
hipError_t relu_backward_bias_n(int dt, int n, const RbArgs* a, int relu, long P, int C,
                                hipStream_t st);
hipError_t pool_relu_backward_bias_n(int dt, int n, const RbArgs* a, int relu, int nb, int H,
                                     int W, int C, hipStream_t st);
hipError_t relu_backward_bias(int dt, const void* dy, const void* dskip, const void* y, void* dz,
                              int relu, float* db, float* partial, long P, int C,
                              hipStream_t st, ReduceJob* defer = nullptr);
// The same for a layer whose output y (nb x H x W x C, H and W even) feeds a
// 2x2/2 max pool, taking the pool's gradient dp (nb x H/2 x W/2 x C): dy is
// dp routed to the first maximal element of each window of y (the pool's
// backward, maxpool_backward), formed on the fly.  Same dz and partial-sum
// contract (its partials fit relu_bias_partial_floats(dt, nb H W, C)).
bool pool_relu_bias_fusable(int dt, int C, int H, int W, const void* dp, const void* dskip,
                            const void* y, const void* dz);
hipError_t pool_relu_backward_bias(int dt, const void* dp, const void* dskip, const void* y,
                                   void* dz, int relu, float* db, float* partial, int nb, int H,
                                   int W, int C, hipStream_t st, ReduceJob* defer = nullptr);

}  // namespace tgpk
