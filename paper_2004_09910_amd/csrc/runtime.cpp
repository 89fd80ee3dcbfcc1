// Host runtime behind the tgp C ABI: network description, FLOP partitioner,
// workspace planner, per-task state machine, the stage tasks F_{i,j},
// F'_{i,j} + B_{i,j} and the gradient accumulation, and the clock-cycle
// scheduler that issues them (Algorithm 1 and its reverse).  It owns no
// device memory: every buffer is a slice of caller-owned memory.
#include <hip/hip_runtime.h>
#include <rocprofiler-sdk-roctx/roctx.h>

#include <algorithm>
#include <array>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <map>
#include <mutex>
#include <string>
#include <vector>

#include "kernels.h"
#include "tgp.h"

namespace {

thread_local std::string g_err;

tgp_status fail(tgp_status s, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_err = buf;
  return s;
}

inline size_t al256(size_t x) { return (x + 255) & ~size_t(255); }

// Kernels read and write caller tensors with 16-byte vector accesses along
// the innermost (channel) dimension where a row of it spans a multiple of
// 16 bytes.  A micro-batch slice of a tensor whose channel row is R bytes
// must start at a multiple of the largest power of two up to 16 dividing R;
// whole tensors (weights, biases, accumulators, the step's inputs and
// outputs) at a multiple of 16.
bool aligned_to(const void* p, size_t a) { return ((uintptr_t)p & (a - 1)) == 0; }
bool row_aligned(const void* p, long row_bytes) {
  size_t need = 16;
  while (need > 1 && row_bytes % (long)need) need >>= 1;
  return aligned_to(p, need);
}

// roctx range around one task (F, F', B, ACC, LOSS) or a whole step, for
// timelines under a tracing tool; a no-op cost without one.
struct Range {
  Range(const char* what, int i, int j) {
    char buf[48];
    if (j > 0) snprintf(buf, sizeof buf, "%s i=%d j=%d", what, i, j);
    else snprintf(buf, sizeof buf, "%s i=%d", what, i);
    roctxRangePushA(buf);
  }
  explicit Range(const char* what) { roctxRangePushA(what); }
  ~Range() { roctxRangePop(); }
  Range(const Range&) = delete;
  Range& operator=(const Range&) = delete;
};

enum CellState : uint8_t { IDLE = 0, FWD = 1, BWD = 2, ACC = 3 };

struct LayerRt {
  tgp_layer d;
  int H = 0, W = 0;            // output size == conv input size (after prologue)
  int inH = 0, inW = 0, inC = 0;  // pre-prologue input (previous output / net input)
  int taps = 9;
  long w_elems = 0;
  int part = 0;                // 0-based partition
  const void* w = nullptr;
  const float* b = nullptr;
  float* dw_acc = nullptr;
  float* db_acc = nullptr;
  bool bound = false;
  // per micro-batch byte sizes
  size_t out_bytes = 0, pro_bytes = 0;
  // workspace offsets
  size_t o_scr_out = 0, o_scr_pro = 0, o_gw = 0, o_gb = 0, o_wt = 0;
  // gradient-slot offsets of the weight gradient's split-K partial slices
  // and the bias gradient's column-sum partials (0 bytes when unused)
  size_t o_gpart = 0, o_gcol = 0, o_gcol_floats = 0;
  bool defer_w = false, defer_b = false;   // partials kept for the accumulation
  std::vector<size_t> o_sto_out, o_sto_pro;  // per stored set
  bool has_wt = false;
  // mask_below: this (depthwise) layer's data gradient is stored as the ReLU
  // backward of the layer below, with that layer's bias column sums
  bool mask_below = false;
};

}  // namespace

struct tgp_net {
  std::vector<LayerRt> L;
  int in_c = 0, H = 0, W = 0, dt = 0, esz = 2;
  int n = 0;
  std::vector<int> lo, hi;
  std::map<int, int> stash_layer;  // stash id -> layer
  // plan
  bool planned = false;
  int B = 0, m = 0, b = 0, mode = 0;
  size_t ws_need = 0;
  char* ws = nullptr;
  size_t ws_size = 0;
  int nsets = 0;
  std::map<int, size_t> o_stash, o_stash_grad;  // offsets for micro-batch 1
  size_t stash_stride = 0;                      // bytes per micro-batch of stash area
  size_t o_g0 = 0, o_g1 = 0, o_dinp = 0, o_dz = 0, o_part = 0, o_colpart = 0, o_msepart = 0,
         o_loss = 0, o_fpart = 0, fpart_floats = 0;
  std::vector<size_t> o_bnd, o_gbnd;  // per (i, j) pipeline boundaries, [i*n + j]
  size_t o_out = 0, o_dy = 0, out_bytes_mb = 0;
  // Transient buffers (activations of checkpointed passes, per-micro-batch
  // gradients, transformed weights, temporaries) exist once per lane;
  // micro-batch i uses lane (i - 1) % lanes.  Their offsets above are
  // relative to the lane's base o_lane + lane * lane_stride.
  int lanes = 1;
  size_t o_lane = 0, lane_stride = 0;
  // Per-micro-batch gradients g_i^j (o_gw / o_gb / o_gpart / o_gcol of each
  // layer, relative to a slot): one slot with one lane, one per micro-batch
  // with several, so that no lane waits for the accumulation of its previous
  // micro-batch.  B_{i,j} leaves each gradient as partial sums in the slot
  // (pend[(i-1) L + l][0 weight, 1 bias] describes them) and
  // tgp_grad_accumulate reduces them straight into the accumulators.
  int gslots = 1;
  size_t o_gslot = 0, gslot_stride = 0;
  std::vector<std::array<tgpk::ReduceJob, 2>> pend;
  // [lane * n + j - 1]: the lane's transformed weights of partition j were
  // not refreshed at its first backward of this step (a paired backward
  // reads only its first micro-batch's lane); refreshed before a later use
  std::vector<char> wt_stale;
  // Streams and events tgp_pipeline_step forks onto with several lanes (one
  // per lane plus one for the accumulations), created on first use on the
  // device current then; default priority.
  std::vector<hipStream_t> lane_streams;
  std::vector<hipEvent_t> lane_events;
  int lane_device = -1;
  ~tgp_net() {
    for (auto e : lane_events) (void)hipEventDestroy(e);
    for (auto st : lane_streams) (void)hipStreamDestroy(st);
  }
  // Per-layer timing plan (tgp_layer_times_plan): one-layer partitions,
  // m = 1, plus four activation buffers from o_lt on; the caller's
  // partition is kept aside until tgp_layer_times restores it.
  bool lt_planned = false;
  size_t o_lt = 0, lt_act = 0;
  int lt_saved_n = 0;
  std::vector<int> lt_saved_lo, lt_saved_hi;
  // state per (i, j): index (i-1)*n + (j-1)
  std::vector<uint8_t> st;
  std::vector<const void*> saved_x;
  std::vector<void*> saved_y;
  std::vector<uint8_t> saved_ckpt;
};

namespace {

long out_elems_mb(const tgp_net* N, const LayerRt& l) { return (long)N->b * l.H * l.W * l.d.cout; }

int64_t layer_flops(const LayerRt& l) {
  if (l.d.kind == TGP_DWCONV3X3) return 2LL * l.H * l.W * l.d.cout * 9;
  return 2LL * l.H * l.W * l.d.cout * l.d.cin * l.taps;
}

// Contiguous split of per-layer costs into n parts: the largest part cost is
// minimised exactly; among such splits the sum of squared part costs (how
// uneven the parts are) is minimised; remaining ties go to the earliest cut
// points.  O(n L^2) dynamic programmes, exact integer arithmetic.
bool balance_dp(const std::vector<int64_t>& c, int n, std::vector<int>& bal) {
  typedef unsigned __int128 u128;
  int L = (int)c.size();
  if (n < 1 || n > L) return false;
  std::vector<int64_t> pre(L + 1, 0);
  for (int i = 0; i < L; ++i) pre[i + 1] = pre[i] + c[i];
  const int64_t INF = INT64_MAX;
  // best[k][s]: smallest achievable max part cost splitting layers s..L-1 into k parts
  std::vector<std::vector<int64_t>> best(n + 1, std::vector<int64_t>(L + 1, INF));
  best[0][L] = 0;
  for (int k = 1; k <= n; ++k)
    for (int s = L - k; s >= 0; --s)
      for (int e = s + 1; e <= L - (k - 1); ++e) {
        if (best[k - 1][e] == INF) continue;
        int64_t v = std::max(best[k - 1][e], pre[e] - pre[s]);
        if (v < best[k][s]) best[k][s] = v;
      }
  const int64_t opt = best[n][0];
  // sq[k][s]: smallest sum of squared part costs splitting s..L-1 into k parts
  // with every part <= opt.
  const u128 UINF = ~(u128)0;
  std::vector<std::vector<u128>> sq(n + 1, std::vector<u128>(L + 1, UINF));
  sq[0][L] = 0;
  for (int k = 1; k <= n; ++k)
    for (int s = L - k; s >= 0; --s)
      for (int e = s + 1; e <= L - (k - 1); ++e) {
        int64_t part = pre[e] - pre[s];
        if (part > opt || sq[k - 1][e] == UINF) continue;
        u128 v = sq[k - 1][e] + (u128)part * (u128)part;
        if (v < sq[k][s]) sq[k][s] = v;
      }
  bal.assign(n, 0);
  int s = 0;
  for (int k = n; k >= 1; --k) {
    int chosen = -1;
    for (int e = s + 1; e <= L - (k - 1); ++e) {
      int64_t part = pre[e] - pre[s];
      if (part > opt || sq[k - 1][e] == UINF) continue;
      if (sq[k - 1][e] + (u128)part * (u128)part == sq[k][s]) { chosen = e; break; }
    }
    if (chosen < 0) return false;
    bal[n - k] = chosen - s;
    s = chosen;
  }
  return s == L;
}

int vecN(int dt) { return dt == TGP_BF16 ? 8 : 4; }

bool ckpt_of(int mode, int i, int m) {
  return mode == TGP_CKPT_ALWAYS || (mode == TGP_CKPT_EXCEPT_LAST && i < m);
}

int cell(const tgp_net* N, int i, int j) { return (i - 1) * N->n + (j - 1); }

hipStream_t S(void* s) { return (hipStream_t)s; }

#define HIPCHK(expr, name)                                                         \
  do {                                                                             \
    hipError_t e_ = (expr);                                                        \
    if (e_ != hipSuccess)                                                          \
      return fail(TGP_EHIP, "%s: %s", name, hipGetErrorString(e_));                \
  } while (0)

char* W_(tgp_net* N, size_t off) { return N->ws + off; }
// Gradient slot buffer at slot-relative offset off, for micro-batch i.
char* G_(tgp_net* N, int i, size_t off) {
  return N->ws + N->o_gslot + (size_t)((i - 1) % N->gslots) * N->gslot_stride + off;
}
// Transient buffer at lane-relative offset off, for micro-batch i.
char* T_(tgp_net* N, int i, size_t off) {
  return N->ws + N->o_lane + (size_t)((i - 1) % N->lanes) * N->lane_stride + off;
}

// ------------------------------------------------------------ per-layer device work

struct ActView {
  const void* in0;              // partition input
  std::vector<const void*> out; // per layer in partition
  std::vector<const void*> pro; // per layer in partition (nullptr if none)
};

size_t stash_off(const tgp_net* N, int i, int sid, bool grad) {
  auto& m = grad ? N->o_stash_grad : N->o_stash;
  return m.at(sid) + (size_t)(i - 1) * N->stash_stride;
}

constexpr int MG = tgpk::kMaxGroup;

// Forward over partition j for a group of cnt (1 .. MG) micro-batches
// iv[k], layer by layer; phase[k]: 0 = checkpointed forward, 1 = storing
// forward, 2 = recompute.  A group runs each convolution as one launch where
// the kernel takes all its tensors, else as launches of two and one (same
// values as one at a time).
tgp_status run_forward_g(tgp_net* N, int j, int cnt, const int* iv, const int* phase,
                         const void* const* x_in, void* const* y_out, hipStream_t st) {
  const int lo = N->lo[j - 1], hi = N->hi[j - 1];
  int set[MG];
  const void* src[MG];
  for (int k = 0; k < cnt; ++k) {
    set[k] = (phase[k] == 1) ? (N->mode == TGP_CKPT_NEVER ? iv[k] - 1 : 0) : -1;
    src[k] = x_in[k];
  }
  for (int l = lo; l < hi; ++l) {
    LayerRt& Lr = N->L[l];
    const tgp_layer& d = Lr.d;
    void* out[MG];
    const void* cin_ptr[MG];
    void* pro_ptr[MG];
    float* fpart[MG];
    for (int k = 0; k < cnt; ++k) {
      const int i = iv[k];
      if (phase[k] == 2) out[k] = T_(N, i, Lr.o_scr_out);
      else if (l == hi - 1) out[k] = y_out[k];
      else if (d.stash_id >= 0) out[k] = W_(N, stash_off(N, i, d.stash_id, false));
      else if (phase[k] == 1) out[k] = W_(N, Lr.o_sto_out[set[k]]);
      else out[k] = T_(N, i, Lr.o_scr_out);
      cin_ptr[k] = src[k];
      if (d.prologue != TGP_PRO_NONE) {
        void* pro = (phase[k] == 1) ? W_(N, Lr.o_sto_pro[set[k]]) : T_(N, i, Lr.o_scr_pro);
        if (d.prologue == TGP_PRO_UPCAT2) {
          const LayerRt& sl = N->L[N->stash_layer.at(d.pop_id)];
          HIPCHK(tgpk::upcat_forward(N->dt, src[k], W_(N, stash_off(N, i, d.pop_id, false)), pro,
                                     N->b, Lr.H, Lr.W, Lr.inC, sl.d.cout, st),
                 "upcat_forward");
        }
        cin_ptr[k] = pro;
        pro_ptr[k] = pro;
      }
      fpart[k] = (float*)T_(N, i, N->o_fpart);
    }
    if (d.prologue == TGP_PRO_MAXPOOL2)   // the group's pools in one launch
      HIPCHK(tgpk::maxpool_forward_n(N->dt, cnt, src, pro_ptr, N->b, Lr.inH, Lr.inW, Lr.inC, st),
             "maxpool_forward");
    if (d.kind == TGP_DWCONV3X3) {
      // the row-window depthwise kernel takes the whole group in one launch
      bool rows = cnt > 1;
      for (int k = 0; k < cnt; ++k)
        rows = rows && tgpk::dw_rows_ok(N->dt, N->b, Lr.H, Lr.W, d.cout, cin_ptr[k], out[k], Lr.w);
      if (rows) {
        HIPCHK(tgpk::dw_forward_n(cnt, cin_ptr, Lr.w, d.bias ? Lr.b : nullptr, out, N->b, Lr.H,
                                  Lr.W, d.cout, d.relu, st),
               "dw_forward");
      } else {
        for (int k = 0; k < cnt; ++k)
          HIPCHK(tgpk::dw_forward(N->dt, cin_ptr[k], Lr.w, d.bias ? Lr.b : nullptr, out[k], N->b,
                                  Lr.H, Lr.W, d.cout, d.relu, st),
                 "dw_forward");
      }
    } else {
      tgpk::ConvShape s{N->b, Lr.H, Lr.W, d.cin, d.cout, Lr.taps};
      if (cnt > 1)
        HIPCHK(tgpk::conv_forward_n(N->dt, cnt, cin_ptr, Lr.w, d.bias ? Lr.b : nullptr, out, s,
                                    d.relu, fpart, N->fpart_floats, st),
               "conv_forward_n");
      else
        HIPCHK(tgpk::conv_forward(N->dt, cin_ptr[0], Lr.w, d.bias ? Lr.b : nullptr, out[0], s,
                                  d.relu, (float*)T_(N, iv[0], N->o_fpart), N->fpart_floats, st),
               "conv_forward");
    }
    for (int k = 0; k < cnt; ++k) {
      // a stashed layer that ends the partition wrote the partition output;
      // its consumer reads the stash slot (a recompute leaves the slot as
      // the forward wrote it, bit for bit)
      if (phase[k] != 2 && l == hi - 1 && d.stash_id >= 0)
        HIPCHK(hipMemcpyAsync(W_(N, stash_off(N, iv[k], d.stash_id, false)), out[k], Lr.out_bytes,
                              hipMemcpyDeviceToDevice, st),
               "stash copy");
      src[k] = out[k];
    }
  }
  return TGP_OK;
}

tgp_status run_forward(tgp_net* N, int j, int i, int phase, const void* x_in, void* y_out,
                       hipStream_t st) {
  return run_forward_g(N, j, 1, &i, &phase, &x_in, &y_out, st);
}

// Pointers the backward of (i, j) reads: layer outputs and prologue outputs.
void activation_view(tgp_net* N, int j, int i, bool ckpt, ActView& v) {
  const int lo = N->lo[j - 1], hi = N->hi[j - 1];
  int c = cell(N, i, j);
  v.in0 = N->saved_x[c];
  v.out.assign(hi - lo, nullptr);
  v.pro.assign(hi - lo, nullptr);
  int set = N->mode == TGP_CKPT_NEVER ? i - 1 : 0;
  for (int l = lo; l < hi; ++l) {
    LayerRt& Lr = N->L[l];
    if (ckpt) {
      v.out[l - lo] = T_(N, i, Lr.o_scr_out);
      if (Lr.d.prologue != TGP_PRO_NONE) v.pro[l - lo] = T_(N, i, Lr.o_scr_pro);
    } else {
      if (l == hi - 1) v.out[l - lo] = N->saved_y[c];
      else if (Lr.d.stash_id >= 0) v.out[l - lo] = W_(N, stash_off(N, i, Lr.d.stash_id, false));
      else v.out[l - lo] = W_(N, Lr.o_sto_out[set]);
      if (Lr.d.prologue != TGP_PRO_NONE) v.pro[l - lo] = W_(N, Lr.o_sto_pro[set]);
    }
  }
}

// Per-micro-batch state of a backward pass.
struct BwdMb {
  int i = 0;
  ActView v;
  void *gcur = nullptr, *gnext = nullptr, *dz = nullptr, *dinp = nullptr;
  float *part = nullptr, *colpart = nullptr;
  const void* dy = nullptr;
  // the pool gradient of layer l + 1's max-pool prologue, when its backward
  // is left to layer l's ReLU backward (dy then names the buffer it would
  // have filled)
  const void* dy_pool = nullptr;
  // dy is already this layer's dz, and its bias column sums (dz_rows rows)
  // are in its column slot (layer l + 1's masked data gradient)
  bool dz_ready = false;
  int dz_rows = 0;
};

// F' (where checkpointed) and B for a group of cnt (1 .. MG) micro-batches
// iv[k] of partition j, layer by layer; a group runs the weight and data
// gradients of each convolution as one launch where the kernel takes all its
// tensors, else as launches of two and one (same values as one at a time).
// dx_in[k] are all null or all set.
tgp_status run_backward_g(tgp_net* N, int j, int cnt, const int* iv,
                          const void* const* dy_out, void* const* dx_in, hipStream_t st) {
  const int lo = N->lo[j - 1], hi = N->hi[j - 1];
  {
    int rc[MG], ph[MG], rcn = 0;
    const void* rx[MG];
    void* ry[MG] = {};
    for (int k = 0; k < MG; ++k) ph[k] = 2;
    for (int k = 0; k < cnt; ++k)
      if (N->saved_ckpt[cell(N, iv[k], j)]) {
        rc[rcn] = iv[k];
        rx[rcn] = N->saved_x[cell(N, iv[k], j)];
        ++rcn;
      }
    if (rcn) {
      Range rg("F'", rc[0], j);
      tgp_status r = run_forward_g(N, j, rcn, rc, ph, rx, ry, st);
      if (r != TGP_OK) return r;
    }
  }
  Range rg("B", iv[0], j);
  BwdMb M[MG];
  auto stale = [&](int i) -> char& {
    return N->wt_stale[(size_t)((i - 1) % N->lanes) * N->n + (j - 1)];
  };
  auto refresh_wt = [&](int i) -> tgp_status {
    // one launch for the partition's layers (several when more than kMaxWt)
    tgpk::WtBatch wb;
    wb.count = 0;
    for (int l = lo; l < hi; ++l) {
      LayerRt& Lr = N->L[l];
      if (!Lr.has_wt) continue;
      const int k = wb.count++;
      wb.w[k] = Lr.w;
      wb.wt[k] = T_(N, i, Lr.o_wt);
      wb.cout[k] = Lr.d.cout;
      wb.cin[k] = Lr.d.cin;
      wb.taps[k] = Lr.taps;
      if (wb.count == tgpk::kMaxWt || l == hi - 1) {
        HIPCHK(tgpk::weight_transform_batch(N->dt, wb, st), "weight_transform");
        wb.count = 0;
      }
    }
    if (wb.count > 0) HIPCHK(tgpk::weight_transform_batch(N->dt, wb, st), "weight_transform");
    stale(i) = 0;
    return TGP_OK;
  };
  for (int k = 0; k < cnt; ++k) {
    const int i = iv[k];
    if (i > N->m - N->lanes) {
      // first backward of partition j on this lane in this step: refresh the
      // lane's transformed weights used by the data-gradient kernels (a
      // group reads its first micro-batch's, so the other lanes are
      // refreshed when a later backward of this step reads them)
      if (k > 0) {
        stale(i) = 1;
      } else {
        tgp_status r = refresh_wt(i);
        if (r != TGP_OK) return r;
      }
    }
  }
  if (stale(iv[0])) {
    tgp_status r = refresh_wt(iv[0]);
    if (r != TGP_OK) return r;
  }
  for (int k = 0; k < cnt; ++k) {
    const int i = iv[k];
    BwdMb& B = M[k];
    B.i = i;
    activation_view(N, j, i, N->saved_ckpt[cell(N, i, j)], B.v);
    B.gcur = T_(N, i, N->o_g0);
    B.gnext = T_(N, i, N->o_g1);
    B.dz = T_(N, i, N->o_dz);
    B.dinp = T_(N, i, N->o_dinp);
    B.part = (float*)T_(N, i, N->o_part);          // weight partials reduced at once
    B.colpart = (float*)T_(N, i, N->o_colpart);    // bias partials reduced at once
    B.dy = dy_out[k];
  }
  for (int l = hi - 1; l >= lo; --l) {
    LayerRt& Lr = N->L[l];
    const tgp_layer& d = Lr.d;
    const void* src[MG];
    const void* cin_ptr[MG];
    const void* dzk[MG];   // the layer's dz: B.dz, or the incoming dy itself
    std::array<tgpk::ReduceJob, 2>* pjs[MG];
    const void* yk[MG];
    const void* dskipk[MG];
    float* gbk[MG];
    float* bpartk[MG];
    tgpk::ReduceJob* bdeferk[MG];
    const long nout = out_elems_mb(N, Lr);
    const long P = (long)N->b * Lr.H * Lr.W;
    for (int k = 0; k < cnt; ++k) {
      BwdMb& B = M[k];
      dzk[k] = B.dz;
      const int i = B.i;
      yk[k] = B.v.out[l - lo];
      src[k] = (l == lo) ? B.v.in0 : B.v.out[l - 1 - lo];  // pre-prologue input
      cin_ptr[k] = d.prologue != TGP_PRO_NONE ? B.v.pro[l - lo] : src[k];
      dskipk[k] = d.stash_id >= 0 ? W_(N, stash_off(N, i, d.stash_id, true)) : nullptr;
      // both gradients stay partial sums in the slot, reduced by the
      // accumulation (the bias's column sums only where relu_backward_bias
      // computes them; bias_grad reduces its own)
      std::array<tgpk::ReduceJob, 2>& pj = N->pend[(size_t)(i - 1) * N->L.size() + l];
      pjs[k] = &pj;
      gbk[k] = d.bias ? (float*)G_(N, i, Lr.o_gb) : nullptr;
      pj[1] = tgpk::ReduceJob{gbk[k], gbk[k], d.bias ? (long)d.cout : 0, 0};   // S = 0: not yet run
      // column partials: kept in the slot, or (too large to keep) reduced at once
      bpartk[k] = Lr.defer_b ? (float*)G_(N, i, Lr.o_gcol) : B.colpart;
      bdeferk[k] = Lr.defer_b ? &pj[1] : nullptr;
      if (B.dz_ready) {
        // layer l + 1's data gradient stored this layer's dz and its bias
        // column sums: no ReLU backward here
        dzk[k] = B.dy;
        pj[1] = tgpk::ReduceJob{bpartk[k], gbk[k], (long)d.cout, B.dz_rows};
        B.dz_ready = false;
      }
    }
    // The fused kernels take the whole group in one launch when every
    // micro-batch qualifies (they always do together: same shape and flags,
    // buffers of the same alignment).
    tgpk::RbArgs ra[MG];
    auto fill_ra = [&](const void* const* dyv) {
      for (int k = 0; k < cnt; ++k)
        ra[k] = tgpk::RbArgs{dyv[k], dskipk[k], yk[k], M[k].dz, gbk[k], bpartk[k], bdeferk[k]};
    };
    auto ran = [&](int k) {
      if (!bdeferk[k]) (*pjs[k])[1].S = 1;
    };
    bool all_pool = cnt > 0;
    for (int k = 0; k < cnt; ++k)
      all_pool = all_pool && M[k].dy_pool && d.bias && Lr.o_gcol_floats &&
                 tgpk::pool_relu_bias_fusable(N->dt, d.cout, Lr.H, Lr.W, M[k].dy_pool, dskipk[k],
                                              yk[k], M[k].dz);
    if (all_pool) {
      const void* dps[MG];
      for (int k = 0; k < cnt; ++k) dps[k] = M[k].dy_pool;
      fill_ra(dps);
      HIPCHK(tgpk::pool_relu_backward_bias_n(N->dt, cnt, ra, d.relu, N->b, Lr.H, Lr.W, d.cout, st),
             "pool_relu_backward_bias");
      for (int k = 0; k < cnt; ++k) {
        ran(k);
        M[k].dy_pool = nullptr;
      }
    }
    for (int k = 0; k < cnt; ++k) {
      BwdMb& B = M[k];
      if (B.dy_pool && d.bias && Lr.o_gcol_floats &&
          tgpk::pool_relu_bias_fusable(N->dt, d.cout, Lr.H, Lr.W, B.dy_pool, dskipk[k], yk[k],
                                       B.dz)) {
        HIPCHK(tgpk::pool_relu_backward_bias(N->dt, B.dy_pool, dskipk[k], yk[k], B.dz, d.relu,
                                             gbk[k], bpartk[k], N->b, Lr.H, Lr.W, d.cout, st,
                                             bdeferk[k]),
               "pool_relu_backward_bias");
        ran(k);
        B.dy_pool = nullptr;
      } else if (B.dy_pool) {
        HIPCHK(tgpk::maxpool_backward(N->dt, yk[k], B.dy_pool, (void*)B.dy, N->b, Lr.H, Lr.W,
                                      d.cout, st),
               "maxpool_backward");
        B.dy_pool = nullptr;
      }
    }
    bool all_rb = cnt > 0;
    for (int k = 0; k < cnt; ++k)
      all_rb = all_rb && (*pjs[k])[1].S == 0 && d.bias && Lr.o_gcol_floats &&
               tgpk::relu_bias_fusable(N->dt, d.cout, M[k].dy, dskipk[k], yk[k], M[k].dz);
    if (all_rb) {
      const void* dys[MG];
      for (int k = 0; k < cnt; ++k) dys[k] = M[k].dy;
      fill_ra(dys);
      HIPCHK(tgpk::relu_backward_bias_n(N->dt, cnt, ra, d.relu, P, d.cout, st),
             "relu_backward_bias");
      for (int k = 0; k < cnt; ++k) ran(k);
    }
    for (int k = 0; k < cnt; ++k) {
      BwdMb& B = M[k];
      std::array<tgpk::ReduceJob, 2>& pj = *pjs[k];
      if (pj[1].S == 0 && d.bias && Lr.o_gcol_floats &&
          tgpk::relu_bias_fusable(N->dt, d.cout, B.dy, dskipk[k], yk[k], B.dz)) {
        HIPCHK(tgpk::relu_backward_bias(N->dt, B.dy, dskipk[k], yk[k], B.dz, d.relu, gbk[k],
                                        bpartk[k], P, d.cout, st, bdeferk[k]),
               "relu_backward_bias");
        ran(k);
      } else if (pj[1].S == 0 && !d.relu && !d.bias && !dskipk[k]) {
        // no ReLU, bias or skip: dz is dy itself, read in place (the
        // buffer holding dy is not written again before the next layer)
        dzk[k] = B.dy;
        pj[1].S = 1;
      } else if (pj[1].S == 0) {
        HIPCHK(tgpk::relu_backward(N->dt, B.dy, dskipk[k], yk[k], B.dz, d.relu, nout, st),
               "relu_backward");
        if (d.bias)
          HIPCHK(tgpk::bias_grad(N->dt, B.dz, gbk[k], B.colpart, P, d.cout, st), "bias_grad");
        pj[1].S = 1;
      }
      float* gw = (float*)G_(N, B.i, Lr.o_gw);
      pj[0] = tgpk::ReduceJob{gw, gw, Lr.w_elems, 1};
    }
    // weight gradient
    tgpk::ConvShape s{N->b, Lr.H, Lr.W, d.cin, d.cout, Lr.taps};
    // one depthwise launch for the group, its sums left to the accumulation
    // when the layer keeps its partials in the slots
    bool dw_wrows = d.kind == TGP_DWCONV3X3;
    float* dw_parts[MG];
    for (int k = 0; k < cnt; ++k) {
      dw_parts[k] = d.kind == TGP_DWCONV3X3 && Lr.defer_w ? (float*)G_(N, M[k].i, Lr.o_gpart)
                                                          : M[k].part;
      dw_wrows = dw_wrows && tgpk::dw_rows_ok(N->dt, N->b, Lr.H, Lr.W, d.cout, cin_ptr[k], dzk[k],
                                              dw_parts[k]);
    }
    if (d.kind != TGP_DWCONV3X3 && cnt > 1 && Lr.defer_w) {
      float* gws[MG];
      float* gps[MG];
      tgpk::ReduceJob* dfs[MG];
      for (int k = 0; k < cnt; ++k) {
        gws[k] = (float*)G_(N, M[k].i, Lr.o_gw);
        gps[k] = (float*)G_(N, M[k].i, Lr.o_gpart);
        dfs[k] = &(*pjs[k])[0];
      }
      HIPCHK(tgpk::conv_wgrad_n(N->dt, cnt, cin_ptr, dzk, gws, gps, s, st, dfs), "conv_wgrad_n");
    } else if (dw_wrows && (cnt > 1 || Lr.defer_w)) {
      float* gws[MG];
      tgpk::ReduceJob* dfs[MG];
      for (int k = 0; k < cnt; ++k) {
        gws[k] = (float*)G_(N, M[k].i, Lr.o_gw);
        dfs[k] = &(*pjs[k])[0];
      }
      HIPCHK(tgpk::dw_wgrad_n(cnt, cin_ptr, dzk, gws, dw_parts, N->b, Lr.H, Lr.W, d.cout, st,
                              Lr.defer_w ? dfs : nullptr),
             "dw_wgrad");
    } else {
      for (int k = 0; k < cnt; ++k) {
        BwdMb& B = M[k];
        float* gw = (float*)G_(N, B.i, Lr.o_gw);
        if (d.kind == TGP_DWCONV3X3) {
          HIPCHK(tgpk::dw_wgrad(N->dt, cin_ptr[k], dzk[k], gw, B.part, N->b, Lr.H, Lr.W, d.cout,
                                st),
                 "dw_wgrad");
        } else {
          HIPCHK(tgpk::conv_wgrad(N->dt, cin_ptr[k], dzk[k], gw,
                                  Lr.defer_w ? (float*)G_(N, B.i, Lr.o_gpart) : B.part, s, st,
                                  nullptr, Lr.defer_w ? &(*pjs[k])[0] : nullptr),
                 "conv_wgrad");
        }
      }
    }
    if (l == lo && dx_in[0] == nullptr) break;
    // data gradient, into the gradient of the pre-prologue input
    void* dest_prev[MG];
    void* dgrad_out[MG];
    for (int k = 0; k < cnt; ++k) {
      dest_prev[k] = (l == lo) ? dx_in[k] : M[k].gnext;
      dgrad_out[k] = d.prologue == TGP_PRO_NONE ? dest_prev[k] : M[k].dinp;
    }
    bool dw_drows = d.kind == TGP_DWCONV3X3 && cnt > 1;
    for (int k = 0; k < cnt; ++k)
      dw_drows = dw_drows && tgpk::dw_rows_ok(N->dt, N->b, Lr.H, Lr.W, d.cout, dzk[k],
                                              dgrad_out[k], Lr.w);
    // the ReLU backward of layer l - 1 folded into this data gradient (planned
    // when it applies; the tensors' alignment is checked here)
    bool masked = Lr.mask_below && l > lo && d.prologue == TGP_PRO_NONE;
    const void* masks[MG];
    float* mparts[MG];
    for (int k = 0; k < cnt && masked; ++k) {
      masks[k] = M[k].v.out[l - 1 - lo];
      mparts[k] = (float*)G_(N, M[k].i, N->L[l - 1].o_gcol);
      masked = tgpk::dw_rows_ok(N->dt, N->b, Lr.H, Lr.W, d.cout, dzk[k], dgrad_out[k], Lr.w) &&
               tgpk::dw_rows_ok(N->dt, N->b, Lr.H, Lr.W, d.cout, masks[k], dgrad_out[k], Lr.w);
    }
    if (masked) {
      HIPCHK(tgpk::dw_dgrad_mask_n(cnt, dzk, Lr.w, dgrad_out, masks, mparts, N->b, Lr.H, Lr.W,
                                   d.cout, st),
             "dw_dgrad_mask");
      for (int k = 0; k < cnt; ++k) {
        M[k].dz_ready = true;
        M[k].dz_rows = tgpk::dw_dgrad_mask_rows(N->b, Lr.H, Lr.W, d.cout);
      }
    } else if (dw_drows) {
      HIPCHK(tgpk::dw_dgrad_n(cnt, dzk, Lr.w, dgrad_out, N->b, Lr.H, Lr.W, d.cout, st), "dw_dgrad");
    } else if (d.kind == TGP_DWCONV3X3) {
      for (int k = 0; k < cnt; ++k)
        HIPCHK(tgpk::dw_dgrad(N->dt, dzk[k], Lr.w, dgrad_out[k], N->b, Lr.H, Lr.W, d.cout, st),
               "dw_dgrad");
    } else if (cnt > 1) {
      // the lanes' transformed weights are equal copies; the first's serves all
      float* fps[MG];
      for (int k = 0; k < cnt; ++k) fps[k] = (float*)T_(N, M[k].i, N->o_fpart);
      HIPCHK(tgpk::conv_dgrad_n(N->dt, cnt, dzk, Lr.w,
                                Lr.has_wt ? T_(N, M[0].i, Lr.o_wt) : nullptr, dgrad_out, s, fps,
                                N->fpart_floats, st),
             "conv_dgrad_n");
    } else {
      HIPCHK(tgpk::conv_dgrad(N->dt, dzk[0], Lr.w, Lr.has_wt ? T_(N, M[0].i, Lr.o_wt) : nullptr,
                              dgrad_out[0], s, (float*)T_(N, M[0].i, N->o_fpart),
                              N->fpart_floats, st),
             "conv_dgrad");
    }
    for (int k = 0; k < cnt; ++k) {
      BwdMb& B = M[k];
      if (d.prologue == TGP_PRO_MAXPOOL2 && l > lo) {
        B.dy_pool = B.dinp;   // routed by layer l - 1's ReLU backward
      } else if (d.prologue == TGP_PRO_MAXPOOL2) {
        HIPCHK(tgpk::maxpool_backward(N->dt, src[k], B.dinp, dest_prev[k], N->b, Lr.inH, Lr.inW,
                                      Lr.inC, st),
               "maxpool_backward");
      } else if (d.prologue == TGP_PRO_UPCAT2) {
        const LayerRt& sl = N->L[N->stash_layer.at(d.pop_id)];
        HIPCHK(tgpk::upcat_backward(N->dt, B.dinp, dest_prev[k],
                                    W_(N, stash_off(N, B.i, d.pop_id, true)), N->b, Lr.H, Lr.W,
                                    Lr.inC, sl.d.cout, st),
               "upcat_backward");
      }
      B.dy = B.gnext;
      std::swap(B.gcur, B.gnext);
    }
  }
  return TGP_OK;
}

tgp_status run_backward(tgp_net* N, int j, int i, const void* dy_out, void* dx_in,
                        hipStream_t st) {
  return run_backward_g(N, j, 1, &i, &dy_out, &dx_in, st);
}

tgp_status run_accumulate(tgp_net* N, int j, int i, int overwrite, hipStream_t st) {
  Range rg("ACC", i, j);
  tgpk::AccBatch batch;
  batch.count = 0;
  batch.ng = 1;
  auto flush = [&]() -> tgp_status {
    if (batch.count == 0) return TGP_OK;
    HIPCHK(tgpk::grad_accumulate_batch(batch, overwrite, st), "grad_accumulate");
    batch.count = 0;
    return TGP_OK;
  };
  auto add = [&](float* acc, const tgpk::ReduceJob& job) -> tgp_status {
    if (batch.count == tgpk::kMaxAcc) {
      tgp_status r = flush();
      if (r != TGP_OK) return r;
    }
    batch.acc[batch.count] = acc;
    batch.g[batch.count] = job.part;
    batch.gstride[batch.count] = 0;
    batch.n[batch.count] = job.E;
    batch.S[batch.count] = job.S;
    ++batch.count;
    return TGP_OK;
  };
  for (int l = N->lo[j - 1]; l < N->hi[j - 1]; ++l) {
    LayerRt& Lr = N->L[l];
    const std::array<tgpk::ReduceJob, 2>& pj = N->pend[(size_t)(i - 1) * N->L.size() + l];
    tgp_status r = add(Lr.dw_acc, pj[0]);
    if (r == TGP_OK && Lr.d.bias) r = add(Lr.db_acc, pj[1]);
    if (r != TGP_OK) return r;
  }
  return flush();
}

// The accumulations of micro-batches i0, i0 - 1, .., i0 - cnt + 1 (in that
// order) for partition j, as one launch when every tensor's pending sums of
// the cnt micro-batches have one shape and lie at one stride from each
// other (the per-micro-batch gradient slots), else one launch per
// micro-batch.  The values are those of cnt run_accumulate calls.
tgp_status run_accumulate_g(tgp_net* N, int j, int i0, int cnt, int overwrite, hipStream_t st) {
  const size_t L = N->L.size();
  auto job = [&](int q, int l, int w) -> const tgpk::ReduceJob& {
    return N->pend[(size_t)(i0 - q - 1) * L + l][w];
  };
  tgpk::AccBatch batch;
  batch.count = 0;
  batch.ng = cnt;
  bool one = cnt > 1;
  std::vector<std::pair<float*, std::pair<int, int>>> ents;   // (acc, (layer, which))
  for (int l = N->lo[j - 1]; l < N->hi[j - 1] && one; ++l) {
    LayerRt& Lr = N->L[l];
    for (int w = 0; w < (Lr.d.bias ? 2 : 1) && one; ++w) {
      const tgpk::ReduceJob& j0 = job(0, l, w);
      const long stride = cnt > 1 ? (long)(job(1, l, w).part - j0.part) : 0;
      for (int q = 1; q < cnt && one; ++q) {
        const tgpk::ReduceJob& jq = job(q, l, w);
        one = jq.E == j0.E && jq.S == j0.S && jq.part - j0.part == (long)q * stride;
      }
      ents.push_back({w ? Lr.db_acc : Lr.dw_acc, {l, w}});
    }
  }
  if (!one || ents.size() > (size_t)tgpk::kMaxAcc) {
    for (int q = 0; q < cnt; ++q) {
      tgp_status r = run_accumulate(N, j, i0 - q, q == 0 ? overwrite : 0, st);
      if (r != TGP_OK) return r;
    }
    return TGP_OK;
  }
  Range rg("ACC", i0, j);
  for (auto& e : ents) {
    const tgpk::ReduceJob& j0 = job(0, e.second.first, e.second.second);
    const int k = batch.count++;
    batch.acc[k] = e.first;
    batch.g[k] = j0.part;
    batch.gstride[k] = (long)(job(1, e.second.first, e.second.second).part - j0.part);
    batch.n[k] = j0.E;
    batch.S[k] = j0.S;
  }
  HIPCHK(tgpk::grad_accumulate_batch(batch, overwrite, st), "grad_accumulate");
  return TGP_OK;
}

// B_{i,j} may run once B_{i+1,j} has: with one gradient slot per
// micro-batch its accumulation may come later (the slots are distinct),
// with a shared slot it must have run (B_{i,j} overwrites the slot).
bool follows_ok(const tgp_net* N, int i, int j) {
  const int s = N->st[cell(N, i + 1, j)];
  return s == ACC || (s == BWD && N->gslots >= N->m);
}

// Plan and workspace present, and the layers of partition j (all partitions
// for j = 0) bound.
tgp_status check_ready(const tgp_net* N, int j = 0) {
  if (!N) return fail(TGP_EINVAL, "net is NULL");
  if (!N->planned) return fail(TGP_ESTATE, "tgp_plan has not been called");
  if (!N->ws) return fail(TGP_ESTATE, "no workspace bound");
  int lo = 0, hi = (int)N->L.size();
  if (j >= 1 && j <= N->n) { lo = N->lo[j - 1]; hi = N->hi[j - 1]; }
  for (int l = lo; l < hi; ++l)
    if (!N->L[l].bound) return fail(TGP_ESTATE, "layer %d has no bound parameters", l);
  return TGP_OK;
}

// Alignment of the micro-batch slices a stage call gets: the partition's
// input (or its gradient) and output (or its gradient); either may be NULL.
tgp_status check_slices(const tgp_net* N, int j, const void* in, const void* out) {
  const LayerRt& first = N->L[N->lo[j - 1]];
  const LayerRt& last = N->L[N->hi[j - 1] - 1];
  if (in && !row_aligned(in, (long)first.inC * N->esz))
    return fail(TGP_EINVAL, "partition %d input pointer %p is not aligned to its %ld-byte rows",
                j, in, (long)first.inC * N->esz);
  if (out && !row_aligned(out, (long)last.d.cout * N->esz))
    return fail(TGP_EINVAL, "partition %d output pointer %p is not aligned to its %ld-byte rows",
                j, out, (long)last.d.cout * N->esz);
  return TGP_OK;
}

// ------------------------------------------------------------ schedule

struct Exec {
  virtual ~Exec() {}
  virtual tgp_status forward(int i, int j, bool ckpt) = 0;
  virtual tgp_status loss(int i) = 0;
  virtual tgp_status backward(int i, int j, bool recompute) = 0;
  virtual tgp_status accumulate(int i, int j, bool overwrite) = 0;
};

// Forward clocks k = 1..m+n-1 run every F_{i,j} with i + j - 1 = k, j
// ascending (Algorithm 1; tasks of one clock are independent).  The loss of
// micro-batch i is taken right after F_{i,n}.  Backward clocks run in the
// reverse order with j descending, which keeps B_{i,j+1} before B_{i,j} and
// B_{i+1,j} before B_{i,j} (Sec. 2.1); each B_{i,j} is preceded by its
// recompute when F_{i,j} was checkpointed and followed by the accumulation of
// g_i^j.
tgp_status run_schedule(int m, int n, int mode, Exec& ex) {
  for (int k = 1; k <= m + n - 1; ++k)
    for (int j = 1; j <= n; ++j) {
      int i = k - j + 1;
      if (i < 1 || i > m) continue;
      tgp_status r = ex.forward(i, j, ckpt_of(mode, i, m));
      if (r != TGP_OK) return r;
      if (j == n && (r = ex.loss(i)) != TGP_OK) return r;
    }
  for (int k = m + n - 1; k >= 1; --k)
    for (int j = n; j >= 1; --j) {
      int i = k - j + 1;
      if (i < 1 || i > m) continue;
      tgp_status r = ex.backward(i, j, ckpt_of(mode, i, m));
      if (r != TGP_OK) return r;
      if ((r = ex.accumulate(i, j, i == m)) != TGP_OK) return r;
    }
  return TGP_OK;
}

struct TraceExec : Exec {
  std::vector<int32_t> ops;
  void put(int op, int i, int j) { ops.push_back(op); ops.push_back(i); ops.push_back(j); }
  tgp_status forward(int i, int j, bool) override { put(TGP_OP_FORWARD, i, j); return TGP_OK; }
  tgp_status loss(int i) override { put(TGP_OP_LOSS, i, 0); return TGP_OK; }
  tgp_status backward(int i, int j, bool rc) override {
    if (rc) put(TGP_OP_RECOMPUTE, i, j);
    put(TGP_OP_BACKWARD, i, j);
    return TGP_OK;
  }
  tgp_status accumulate(int i, int j, bool) override { put(TGP_OP_ACCUMULATE, i, j); return TGP_OK; }
};

size_t slot_bytes_mb(const tgp_net* N, int l) {  // output of layer l for one micro-batch
  return al256((size_t)N->b * N->L[l].H * N->L[l].W * N->L[l].d.cout * N->esz);
}

struct GpuExec : Exec {
  tgp_net* N;
  const char* x;
  const char* target;
  float* loss_dev;
  char* y_out;
  hipStream_t st;
  size_t in_mb_bytes, out_mb_bytes;
  // With K > 1 lanes, micro-batch i's tasks run on lane[(i - 1) % K] and the
  // accumulations, in schedule order, on acc, which waits for each B_{i,j}
  // through its lane's event (every cross-stream edge points from a lane to
  // acc, never back).  K = 1: everything on st.
  int K = 1;
  hipStream_t lane[TGP_MAX_LANES] = {};
  hipEvent_t lane_ev[TGP_MAX_LANES] = {};
  hipStream_t acc = nullptr;
  hipStream_t on(int i) const { return K > 1 ? lane[(i - 1) % K] : st; }
  const void* bnd(int i, int j) {  // output of partition j for micro-batch i (j = 0: input)
    if (j == 0) return x + (size_t)(i - 1) * in_mb_bytes;
    if (j == N->n) return y_out ? (const void*)(y_out + (size_t)(i - 1) * out_mb_bytes)
                                : (const void*)W_(N, N->o_out + (size_t)(i - 1) * al256(out_mb_bytes));
    return W_(N, N->o_bnd[(i - 1) * N->n + j]);
  }
  void* gbnd(int i, int j) {  // gradient of the output of partition j
    if (j == N->n) return W_(N, N->o_dy + (size_t)(i - 1) * al256(out_mb_bytes));
    return W_(N, N->o_gbnd[(i - 1) * N->n + j]);
  }
  tgp_status forward(int i, int j, bool ckpt) override {
    return tgp_stage_forward(N, j, i, ckpt ? 1 : 0, bnd(i, j - 1), (void*)bnd(i, j), on(i));
  }
  tgp_status loss(int i) override {
    Range rg("LOSS", i, 0);
    const LayerRt& last = N->L.back();
    long n_mb = (long)N->b * last.H * last.W * last.d.cout;
    long numel = n_mb * N->m;
    HIPCHK(tgpk::mse_forward_backward(N->dt, bnd(i, N->n),
                                      target + (size_t)(i - 1) * out_mb_bytes, gbnd(i, N->n),
                                      (float*)W_(N, N->o_loss) + (i - 1),
                                      (float*)T_(N, i, N->o_msepart), n_mb, 1.0f / (float)numel,
                                      on(i)),
           "mse_forward_backward");
    return TGP_OK;
  }
  tgp_status backward(int i, int j, bool) override {
    tgp_status r = tgp_stage_backward_recompute(N, j, i, gbnd(i, j),
                                                j > 1 ? gbnd(i, j - 1) : nullptr, on(i));
    if (r != TGP_OK || K == 1) return r;
    const int k = (i - 1) % K;
    HIPCHK(hipEventRecord(lane_ev[k], lane[k]), "hipEventRecord");
    HIPCHK(hipStreamWaitEvent(acc, lane_ev[k], 0), "hipStreamWaitEvent");
    return TGP_OK;
  }
  // With a gradient slot per micro-batch (K > 1), the accumulations of
  // partition j are issued in groups of up to kAccGroup consecutive
  // micro-batches (i0 down to i0 - count + 1, the schedule's order), one
  // launch each: every g^j is read and written once per group, with the
  // values of one accumulation per micro-batch.
  static constexpr int kAccGroup = 8;
  std::vector<int> acc_top, acc_cnt;
  tgp_status accumulate(int i, int j, bool ow) override {
    if (K == 1 || N->gslots < N->m) return tgp_grad_accumulate(N, j, i, ow ? 1 : 0, K > 1 ? acc : st);
    if (acc_cnt.size() < (size_t)N->n + 1) {
      acc_top.assign(N->n + 1, 0);
      acc_cnt.assign(N->n + 1, 0);
    }
    if (acc_cnt[j] == 0) acc_top[j] = i;
    ++acc_cnt[j];
    if (acc_cnt[j] < kAccGroup && i > 1) return TGP_OK;
    const int top = acc_top[j], cnt = acc_cnt[j];
    acc_cnt[j] = 0;
    return tgp_grad_accumulate_n(N, j, top, cnt, top == N->m ? 1 : 0, acc);
  }
};

}  // namespace

// ============================================================ C ABI

namespace tgpk {
extern int g_fwd_variant;
extern int g_fwd_order;
extern int g_fwd_split;
extern int g_rowtile_mask;
extern int g_rows32_ch;
extern int g_wgrad_ks;
extern int g_wgrad_rows3;
}

extern "C" {

const char* tgp_last_error(void) { return g_err.c_str(); }

// Kernel-selection overrides for tests and measurement sweeps (the first
// two are declared in tgp.h; split and order are sweep-only).
int tgp_debug_set_fwd_variant(int v) {
  int old = tgpk::g_fwd_variant;
  tgpk::g_fwd_variant = v;
  return old;
}
int tgp_debug_set_fwd_split(int v) {
  int old = tgpk::g_fwd_split;
  tgpk::g_fwd_split = v;
  return old;
}
int tgp_debug_set_rowtile_mask(int v) {
  int old = tgpk::g_rowtile_mask;
  tgpk::g_rowtile_mask = v;
  tgpk::g_rows32_ch = (v >> 4 & 1) ? 2 : 0;
  tgpk::g_wgrad_ks = (v >> 5 & 1) ? 1 : 0;
  tgpk::g_wgrad_rows3 = (v >> 6 & 1) ? 0 : 1;
  return old;
}
int tgp_debug_set_fwd_order(int v) {
  int old = tgpk::g_fwd_order;
  tgpk::g_fwd_order = v;
  return old;
}

tgp_status tgp_net_create(const tgp_layer* layers, int n_layers, int in_c, int H, int W,
                          int dtype, tgp_net** out) {
  g_err.clear();
  if (!out) return fail(TGP_EINVAL, "out is NULL");
  *out = nullptr;
  if (!layers || n_layers < 1) return fail(TGP_EINVAL, "need at least one layer");
  if (in_c < 1 || H < 1 || W < 1) return fail(TGP_EINVAL, "bad input shape");
  if (dtype != TGP_BF16 && dtype != TGP_FP32) return fail(TGP_EINVAL, "bad dtype %d", dtype);
  tgp_net* N = new tgp_net;
  N->in_c = in_c; N->H = H; N->W = W; N->dt = dtype; N->esz = dtype == TGP_BF16 ? 2 : 4;
  int c = in_c, h = H, w = W;
  std::map<int, std::pair<int, std::pair<int, int>>> stashed;  // id -> (C, (H, W))
  const int V = vecN(dtype);
  for (int l = 0; l < n_layers; ++l) {
    LayerRt Lr;
    Lr.d = layers[l];
    const tgp_layer& d = Lr.d;
    auto bad = [&](tgp_status s, const char* why) {
      delete N;
      return fail(s, "layer %d: %s", l, why);
    };
    if (d.kind < 0 || d.kind > 2) return bad(TGP_EINVAL, "bad kind");
    if (d.cin < 1 || d.cout < 1) return bad(TGP_EINVAL, "bad channel count");
    if (d.prologue < 0 || d.prologue > 2) return bad(TGP_EINVAL, "bad prologue");
    if (d.stash_id < -1 || d.stash_id > 63 || d.pop_id < -1 || d.pop_id > 63)
      return bad(TGP_EINVAL, "skip id out of range");
    Lr.inH = h; Lr.inW = w; Lr.inC = c;
    int want = c;
    if (d.prologue == TGP_PRO_MAXPOOL2) {
      if (h % 2 || w % 2) return bad(TGP_EINVAL, "max-pool of an odd size");
      if (c % V) return bad(TGP_EUNSUPPORTED, "max-pool channels must be a multiple of 8 (bf16) / 4 (fp32)");
      h /= 2; w /= 2;
    } else if (d.prologue == TGP_PRO_UPCAT2) {
      auto it = stashed.find(d.pop_id);
      if (it == stashed.end()) return bad(TGP_EINVAL, "pops a skip no earlier layer stashed");
      h *= 2; w *= 2;
      if (it->second.second != std::make_pair(h, w)) return bad(TGP_EINVAL, "skip size mismatch");
      if (c % V || it->second.first % V)
        return bad(TGP_EUNSUPPORTED, "upsample-concat channels must be a multiple of 8 (bf16) / 4 (fp32)");
      want = c + it->second.first;
      stashed.erase(it);
    } else if (d.pop_id >= 0) {
      return bad(TGP_EINVAL, "pop_id set without an UPCAT2 prologue");
    }
    if (d.cin != want) return bad(TGP_EINVAL, "cin does not match the incoming channels");
    if (d.kind == TGP_DWCONV3X3 && d.cin != d.cout) return bad(TGP_EINVAL, "depthwise needs cin == cout");
    Lr.H = h; Lr.W = w;
    Lr.taps = d.kind == TGP_CONV1X1 ? 1 : 9;
    Lr.w_elems = d.kind == TGP_DWCONV3X3 ? (long)d.cout * 9 : (long)d.cout * d.cin * Lr.taps;
    c = d.cout;
    if (d.stash_id >= 0) {
      if (N->stash_layer.count(d.stash_id)) return bad(TGP_EINVAL, "stash id used twice");
      N->stash_layer[d.stash_id] = l;
      stashed[d.stash_id] = {c, {h, w}};
    }
    N->L.push_back(Lr);
  }
  N->n = 1;
  N->lo = {0};
  N->hi = {n_layers};
  *out = N;
  return TGP_OK;
}

void tgp_net_destroy(tgp_net* net) { delete net; }

tgp_status tgp_layer_flops(const tgp_net* N, int layer, int64_t* flops) {
  if (!N || !flops) return fail(TGP_EINVAL, "NULL argument");
  if (layer < 0 || layer >= (int)N->L.size()) return fail(TGP_EINVAL, "bad layer %d", layer);
  *flops = layer_flops(N->L[layer]);
  return TGP_OK;
}

tgp_status tgp_balance_minmax(const int64_t* cost, int L, int n, int* balance) {
  if (!cost || !balance || L < 1) return fail(TGP_EINVAL, "bad arguments");
  if (n < 1 || n > L) return fail(TGP_EINVAL, "n=%d must be in 1..%d", n, L);
  std::vector<int64_t> c(cost, cost + L);
  for (auto v : c)
    if (v < 0) return fail(TGP_EINVAL, "negative cost");
  std::vector<int> bal;
  if (!balance_dp(c, n, bal)) return fail(TGP_EINVAL, "no split");
  std::copy(bal.begin(), bal.end(), balance);
  return TGP_OK;
}

tgp_status tgp_set_partition(tgp_net* N, int n, const int* balance) {
  if (!N) return fail(TGP_EINVAL, "net is NULL");
  N->lt_planned = false;
  int L = (int)N->L.size();
  if (n < 1 || n > L) return fail(TGP_EINVAL, "n=%d must be in 1..%d", n, L);
  std::vector<int> bal;
  if (balance) {
    int sum = 0;
    for (int k = 0; k < n; ++k) {
      if (balance[k] < 1) return fail(TGP_EINVAL, "empty partition %d", k + 1);
      sum += balance[k];
    }
    if (sum != L) return fail(TGP_EINVAL, "balance sums to %d, need %d", sum, L);
    bal.assign(balance, balance + n);
  } else {
    std::vector<int64_t> c;
    for (auto& l : N->L) c.push_back(layer_flops(l));
    if (!balance_dp(c, n, bal)) return fail(TGP_EINVAL, "no split");
  }
  N->n = n;
  N->lo.assign(n, 0);
  N->hi.assign(n, 0);
  int s = 0;
  for (int k = 0; k < n; ++k) {
    N->lo[k] = s;
    s += bal[k];
    N->hi[k] = s;
    for (int l = N->lo[k]; l < N->hi[k]; ++l) N->L[l].part = k;
  }
  N->planned = false;
  N->ws = nullptr;
  return TGP_OK;
}

tgp_status tgp_get_partition(const tgp_net* N, int* n, int* balance) {
  if (!N || !n) return fail(TGP_EINVAL, "NULL argument");
  *n = N->n;
  if (balance)
    for (int k = 0; k < N->n; ++k) balance[k] = N->hi[k] - N->lo[k];
  return TGP_OK;
}

tgp_status tgp_bind_params(tgp_net* N, int layer, const void* w, const float* b, float* dw_acc,
                           float* db_acc) {
  if (!N) return fail(TGP_EINVAL, "net is NULL");
  if (layer < 0 || layer >= (int)N->L.size()) return fail(TGP_EINVAL, "bad layer %d", layer);
  LayerRt& Lr = N->L[layer];
  if (!w || !dw_acc) return fail(TGP_EINVAL, "layer %d: NULL weight or accumulator", layer);
  if (Lr.d.bias && (!b || !db_acc)) return fail(TGP_EINVAL, "layer %d: bias pointers missing", layer);
  if (!Lr.d.bias && (b || db_acc)) return fail(TGP_EINVAL, "layer %d has no bias", layer);
  if (!aligned_to(w, 16) || !aligned_to(dw_acc, 16) || (b && !aligned_to(b, 16)) ||
      (db_acc && !aligned_to(db_acc, 16)))
    return fail(TGP_EINVAL, "layer %d: weight, bias and accumulator pointers must be 16-byte "
                "aligned", layer);
  Lr.w = w; Lr.b = b; Lr.dw_acc = dw_acc; Lr.db_acc = db_acc; Lr.bound = true;
  return TGP_OK;
}

tgp_status tgp_set_lanes(tgp_net* N, int lanes) {
  if (!N) return fail(TGP_EINVAL, "net is NULL");
  if (lanes < 1 || lanes > TGP_MAX_LANES) return fail(TGP_EINVAL, "lanes=%d out of 1..%d", lanes, TGP_MAX_LANES);
  N->lanes = lanes;
  N->planned = false;
  N->ws = nullptr;
  return TGP_OK;
}

tgp_status tgp_plan(tgp_net* N, int B, int m, int mode, size_t* bytes) {
  if (!N || !bytes) return fail(TGP_EINVAL, "NULL argument");
  N->lt_planned = false;
  if (m < 1 || B < 1) return fail(TGP_EINVAL, "B and m must be positive");
  if (B % m) return fail(TGP_EINVAL, "B=%d is not divisible by m=%d", B, m);
  if (mode < 0 || mode > 2) return fail(TGP_EINVAL, "bad checkpoint mode %d", mode);
  N->B = B; N->m = m; N->b = B / m; N->mode = mode;
  const int n = N->n;
  for (auto& l : N->L)
    if ((long)N->b * l.H * l.W >= (1L << 31) / 4 || (long)N->b * l.inH * l.inW >= (1L << 31) / 4)
      return fail(TGP_EINVAL, "micro-batch too large for 32-bit pixel indices");
  size_t off = 0, loff = 0;
  auto take = [&](size_t bytes_) { size_t o = off; off += al256(bytes_); return o; };
  auto takeL = [&](size_t bytes_) { size_t o = loff; loff += al256(bytes_); return o; };
  size_t goff = 0;
  auto takeG = [&](size_t bytes_) { size_t o = goff; goff += al256(bytes_); return o; };
  // skips and their gradients, one slot per micro-batch
  N->o_stash.clear(); N->o_stash_grad.clear();
  size_t stride = 0;
  for (auto& kv : N->stash_layer) stride += slot_bytes_mb(N, kv.second);
  N->stash_stride = stride;
  size_t base = take(stride * m), acc = 0;
  for (auto& kv : N->stash_layer) { N->o_stash[kv.first] = base + acc; acc += slot_bytes_mb(N, kv.second); }
  base = take(stride * m); acc = 0;
  for (auto& kv : N->stash_layer) { N->o_stash_grad[kv.first] = base + acc; acc += slot_bytes_mb(N, kv.second); }
  // transient activations (checkpointed forward and recompute)
  size_t max_act = 0, max_pro = 0;
  for (size_t l = 0; l < N->L.size(); ++l) {
    LayerRt& Lr = N->L[l];
    Lr.out_bytes = (size_t)N->b * Lr.H * Lr.W * Lr.d.cout * N->esz;
    Lr.pro_bytes = Lr.d.prologue != TGP_PRO_NONE ? (size_t)N->b * Lr.H * Lr.W * Lr.d.cin * N->esz : 0;
    size_t in_bytes = (size_t)N->b * Lr.inH * Lr.inW * Lr.inC * N->esz;
    max_act = std::max({max_act, Lr.out_bytes, in_bytes});
    max_pro = std::max(max_pro, Lr.pro_bytes);
    Lr.o_scr_out = takeL(Lr.out_bytes);
    Lr.o_scr_pro = Lr.pro_bytes ? takeL(Lr.pro_bytes) : 0;
  }
  // stored activations of non-checkpointed micro-batches
  N->nsets = mode == TGP_CKPT_NEVER ? m : (mode == TGP_CKPT_EXCEPT_LAST ? 1 : 0);
  for (size_t l = 0; l < N->L.size(); ++l) {
    LayerRt& Lr = N->L[l];
    Lr.o_sto_out.assign(N->nsets, 0);
    Lr.o_sto_pro.assign(N->nsets, 0);
    bool last_of_part = (int)l == N->hi[Lr.part] - 1;
    for (int s = 0; s < N->nsets; ++s) {
      if (!last_of_part && Lr.d.stash_id < 0) Lr.o_sto_out[s] = take(Lr.out_bytes);
      if (Lr.pro_bytes) Lr.o_sto_pro[s] = take(Lr.pro_bytes);
    }
  }
  // per-micro-batch gradients g_i and transformed weights
  size_t max_part = 0, max_col = 0;
  for (auto& Lr : N->L) {
    Lr.o_gw = takeG(Lr.w_elems * 4);
    Lr.o_gb = Lr.d.bias ? takeG(Lr.d.cout * 4) : 0;
    tgpk::ConvShape s{N->b, Lr.H, Lr.W, Lr.d.cin, Lr.d.cout, Lr.taps};
    Lr.has_wt = Lr.d.kind != TGP_DWCONV3X3 && tgpk::conv_dgrad_uses_wt(N->dt, s);
    Lr.o_wt = Lr.has_wt ? takeL(Lr.w_elems * N->esz) : 0;
    // Split-K partials stay in the slot for the accumulation to sum when a
    // layer's are at most kDeferBytes per micro-batch; larger ones (deep,
    // wide layers) are reduced at once through a lane buffer, so the slots
    // do not grow with the sum of every layer's partials.
    constexpr size_t kDeferBytes = 32u << 20;
    const long P = (long)N->b * Lr.H * Lr.W;
    Lr.defer_w = false;
    Lr.o_gpart = 0;
    if (Lr.d.kind == TGP_DWCONV3X3) {
      // the row-window kernel's partials stay in the slot for the
      // accumulation (its sum order differs from the immediate reduction's,
      // so the choice is made here, for every call of the plan)
      const size_t pf = tgpk::dw_wgrad_partial_floats(N->b, Lr.H, Lr.W, Lr.d.cout);
      max_part = std::max(max_part, pf);
      Lr.defer_w = N->dt == TGP_BF16 && pf * 4 <= kDeferBytes;
      if (Lr.defer_w) Lr.o_gpart = takeG(std::max<size_t>(pf, 1) * 4);
    } else {
      const size_t pf = tgpk::conv_wgrad_partial_floats(N->dt, s);
      Lr.defer_w = pf * 4 <= kDeferBytes;
      if (Lr.defer_w) Lr.o_gpart = takeG(std::max<size_t>(pf, 1) * 4);
      else max_part = std::max(max_part, pf);
    }
    Lr.o_gcol_floats = Lr.d.bias ? tgpk::relu_bias_partial_floats(N->dt, P, Lr.d.cout) : 0;
    {
      // this layer's ReLU backward folded into the data gradient of a
      // depthwise layer above it in the partition (bf16, no prologue there,
      // no skip here); its column slot then holds that kernel's sums too
      const int li = (int)(&Lr - &N->L[0]);
      if (li + 1 < (int)N->L.size()) {
        LayerRt& U = N->L[li + 1];
        U.mask_below = N->dt == TGP_BF16 && U.part == Lr.part &&
                       U.d.kind == TGP_DWCONV3X3 && U.d.prologue == TGP_PRO_NONE &&
                       Lr.d.relu && Lr.d.bias && Lr.d.stash_id < 0 && Lr.o_gcol_floats &&
                       U.H == Lr.H && U.W == Lr.W && U.d.cin == Lr.d.cout &&
                       tgpk::dw_dgrad_mask_ok(N->b, U.H, U.W, U.d.cout);
        if (U.mask_below)
          Lr.o_gcol_floats = std::max<size_t>(
              Lr.o_gcol_floats,
              (size_t)tgpk::dw_dgrad_mask_rows(N->b, U.H, U.W, U.d.cout) * Lr.d.cout);
      }
    }
    Lr.defer_b = Lr.o_gcol_floats && Lr.o_gcol_floats * 4 <= kDeferBytes;
    {
      const size_t li = (size_t)(&Lr - &N->L[0]);
      if (li + 1 < N->L.size() && N->L[li + 1].mask_below && !Lr.defer_b)
        N->L[li + 1].mask_below = false;   // its sums need the slot
    }
    Lr.o_gcol = Lr.defer_b ? takeG(Lr.o_gcol_floats * 4) : 0;
    if (Lr.o_gcol_floats && !Lr.defer_b) max_col = std::max(max_col, Lr.o_gcol_floats);
    max_col = std::max(max_col, tgpk::colsum_partial_floats(P, Lr.d.cout));
  }
  N->o_g0 = takeL(max_act);
  N->o_g1 = takeL(max_act);
  N->o_dz = takeL(max_act);
  N->o_dinp = takeL(std::max<size_t>(max_pro, 16));
  N->o_part = takeL(std::max<size_t>(max_part, 1) * 4);
  size_t max_fpart = 0;   // split-K partials of forward / data-gradient convolutions
  for (auto& Lr : N->L) {
    if (Lr.d.kind == TGP_DWCONV3X3) continue;
    tgpk::ConvShape f{N->b, Lr.H, Lr.W, Lr.d.cin, Lr.d.cout, Lr.taps};
    tgpk::ConvShape d{N->b, Lr.H, Lr.W, Lr.d.cout, Lr.d.cin, Lr.taps};
    max_fpart = std::max({max_fpart, tgpk::conv_forward_partial_floats(N->dt, f),
                          tgpk::conv_forward_partial_floats(N->dt, d)});
  }
  N->fpart_floats = max_fpart;
  N->o_fpart = takeL(std::max<size_t>(max_fpart, 4) * 4);
  N->o_colpart = takeL(max_col * 4);
  const LayerRt& last = N->L.back();
  long out_mb = (long)N->b * last.H * last.W * last.d.cout;
  N->out_bytes_mb = out_mb * N->esz;
  N->o_msepart = takeL(tgpk::mse_partial_floats(out_mb) * 4);
  N->o_loss = take(m * 4);
  // pipeline boundaries
  N->o_bnd.assign((size_t)m * n + n, 0);
  N->o_gbnd.assign((size_t)m * n + n, 0);
  for (int i = 1; i <= m; ++i)
    for (int j = 1; j < n; ++j) {
      N->o_bnd[(i - 1) * n + j] = take(N->L[N->hi[j - 1] - 1].out_bytes);
      N->o_gbnd[(i - 1) * n + j] = take(N->L[N->hi[j - 1] - 1].out_bytes);
    }
  N->o_out = take(al256(N->out_bytes_mb) * m);
  N->o_dy = take(al256(N->out_bytes_mb) * m);
  N->lane_stride = al256(loff);
  N->o_lane = take(N->lane_stride * N->lanes);
  N->gslots = N->lanes > 1 ? m : 1;
  N->gslot_stride = al256(goff);
  N->o_gslot = take(N->gslot_stride * N->gslots);
  N->ws_need = off;
  N->planned = true;
  N->ws = nullptr;
  N->ws_size = 0;
  N->st.assign((size_t)m * n, IDLE);
  N->saved_x.assign((size_t)m * n, nullptr);
  N->saved_y.assign((size_t)m * n, nullptr);
  N->saved_ckpt.assign((size_t)m * n, 0);
  N->pend.assign((size_t)m * N->L.size(), std::array<tgpk::ReduceJob, 2>{});
  N->wt_stale.assign((size_t)N->lanes * N->n, 0);
  *bytes = off;
  return TGP_OK;
}

tgp_status tgp_bind_workspace(tgp_net* N, void* dev, size_t bytes) {
  if (!N) return fail(TGP_EINVAL, "net is NULL");
  if (!N->planned) return fail(TGP_ESTATE, "tgp_plan has not been called");
  if (!dev) return fail(TGP_EINVAL, "workspace is NULL");
  if ((uintptr_t)dev & 255) return fail(TGP_EINVAL, "workspace must be 256-byte aligned");
  if (bytes < N->ws_need)
    return fail(TGP_ENOSPACE, "workspace of %zu bytes, need %zu", bytes, N->ws_need);
  N->ws = (char*)dev;
  N->ws_size = bytes;
  return TGP_OK;
}

tgp_status tgp_stash_ptr(tgp_net* N, int i, int stash_id, int grad, void** p) {
  if (!N || !p) return fail(TGP_EINVAL, "NULL argument");
  if (!N->planned || !N->ws) return fail(TGP_ESTATE, "no plan or workspace");
  if (i < 1 || i > N->m) return fail(TGP_EINVAL, "micro-batch %d out of 1..%d", i, N->m);
  if (!N->stash_layer.count(stash_id)) return fail(TGP_EINVAL, "no skip %d", stash_id);
  *p = W_(N, stash_off(N, i, stash_id, grad != 0));
  return TGP_OK;
}

// ------------------------------------------------------------ time-based balance

tgp_status tgp_layer_times_plan(tgp_net* N, int b, int mode, size_t* bytes) {
  if (!N || !bytes) return fail(TGP_EINVAL, "NULL argument");
  if (b < 1) return fail(TGP_EINVAL, "b must be positive");
  const int L = (int)N->L.size();
  if (!N->lt_planned) {   // keep the caller's partition (not an earlier timing plan's)
    N->lt_saved_n = N->n;
    N->lt_saved_lo = N->lo;
    N->lt_saved_hi = N->hi;
  }
  const int saved_n = N->lt_saved_n;
  const std::vector<int> saved_lo = N->lt_saved_lo, saved_hi = N->lt_saved_hi;
  std::vector<int> ones(L, 1);
  tgp_status r = tgp_set_partition(N, L, ones.data());
  size_t off = 0;
  if (r == TGP_OK) r = tgp_plan(N, b, 1, mode, &off);
  N->lt_saved_n = saved_n;
  N->lt_saved_lo = saved_lo;
  N->lt_saved_hi = saved_hi;
  if (r != TGP_OK) return r;
  size_t act = 16;
  for (const auto& l : N->L)
    act = std::max({act, l.out_bytes, (size_t)b * l.inH * l.inW * l.inC * N->esz});
  N->o_lt = al256(off);
  N->lt_act = al256(act);
  N->ws_need = N->o_lt + 4 * N->lt_act;
  N->lt_planned = true;
  *bytes = N->ws_need;
  return TGP_OK;
}

// The caller's partition back, no plan.
static void lt_restore(tgp_net* N) {
  const int L = (int)N->L.size();
  N->n = N->lt_saved_n;
  N->lo = N->lt_saved_lo;
  N->hi = N->lt_saved_hi;
  for (int k = 0; k < N->n; ++k)
    for (int l = N->lo[k]; l < N->hi[k] && l < L; ++l) N->L[l].part = k;
  N->lt_planned = false;
  N->planned = false;
  N->ws = nullptr;
}

static tgp_status lt_run(tgp_net* N, int iters, float* us, hipStream_t st, hipEvent_t e0, hipEvent_t e1) {
  const int L = (int)N->L.size();
  HIPCHK(hipMemsetAsync(N->ws, 0, N->ws_need, st), "hipMemsetAsync");
  char* X = N->ws + N->o_lt;
  char* Y = X + N->lt_act;
  char* DY = Y + N->lt_act;
  char* DX = DY + N->lt_act;
  const int ckpt = ckpt_of(N->mode, 1, 1) ? 1 : 0;
  for (int l = 0; l < L; ++l) {
    const int j = l + 1;
    double total_ms = 0;
    for (int it = 0; it <= iters; ++it) {   // it = 0 warms up
      HIPCHK(hipEventRecord(e0, st), "hipEventRecord");
      tgp_status r = tgp_stage_forward(N, j, 1, ckpt, X, Y, st);
      if (r == TGP_OK) r = tgp_stage_backward_recompute(N, j, 1, DY, l == 0 ? nullptr : DX, st);
      if (r == TGP_OK) r = tgp_grad_accumulate(N, j, 1, 1, st);
      if (r != TGP_OK) return r;
      HIPCHK(hipEventRecord(e1, st), "hipEventRecord");
      HIPCHK(hipEventSynchronize(e1), "hipEventSynchronize");
      float ms = 0;
      HIPCHK(hipEventElapsedTime(&ms, e0, e1), "hipEventElapsedTime");
      if (it > 0) total_ms += ms;
    }
    us[l] = (float)(total_ms / iters * 1000.0);
  }
  return TGP_OK;
}

tgp_status tgp_layer_times(tgp_net* N, void* ws, size_t bytes, int iters, float* us,
                           void* stream) {
  if (!N || !us) return fail(TGP_EINVAL, "NULL argument");
  if (!N->lt_planned) return fail(TGP_ESTATE, "tgp_layer_times_plan has not been called");
  if (iters < 1) return fail(TGP_EINVAL, "iters must be positive");
  tgp_status r = tgp_bind_workspace(N, ws, bytes);
  if (r == TGP_OK) r = check_ready(N);
  if (r != TGP_OK) return r;   // plan and partition kept: the caller may bind and retry
  hipEvent_t e0 = nullptr, e1 = nullptr;
  if (hipEventCreate(&e0) != hipSuccess || hipEventCreate(&e1) != hipSuccess) {
    if (e0) (void)hipEventDestroy(e0);
    lt_restore(N);
    return fail(TGP_EHIP, "hipEventCreate failed");
  }
  r = lt_run(N, iters, us, S(stream), e0, e1);
  (void)hipEventDestroy(e0);
  (void)hipEventDestroy(e1);
  lt_restore(N);
  return r;
}

tgp_status tgp_balance_by_time(tgp_net* N, void* ws, size_t bytes, int iters, int n,
                               int* balance, float* us, void* stream) {
  if (!N || !balance) return fail(TGP_EINVAL, "NULL argument");
  const int L = (int)N->L.size();
  if (n < 1 || n > L) return fail(TGP_EINVAL, "n=%d must be in 1..%d", n, L);
  std::vector<float> t(L, 0.f);
  tgp_status r = tgp_layer_times(N, ws, bytes, iters, t.data(), stream);
  if (r != TGP_OK) return r;
  std::vector<int64_t> cost(L);
  for (int l = 0; l < L; ++l) cost[l] = (int64_t)std::llround((double)t[l] * 1000.0);   // ns
  std::vector<int> bal;
  if (!balance_dp(cost, n, bal)) return fail(TGP_EINVAL, "no split");
  r = tgp_set_partition(N, n, bal.data());
  if (r != TGP_OK) return r;
  std::copy(bal.begin(), bal.end(), balance);
  if (us) std::copy(t.begin(), t.end(), us);
  return TGP_OK;
}

tgp_status tgp_stage_forward(tgp_net* N, int j, int i, int checkpoint, const void* x_in,
                             void* y_out, void* stream) {
  tgp_status r = check_ready(N, j);
  if (r != TGP_OK) return r;
  if (j < 1 || j > N->n) return fail(TGP_EINVAL, "partition %d out of 1..%d", j, N->n);
  if (i < 1 || i > N->m) return fail(TGP_EINVAL, "micro-batch %d out of 1..%d", i, N->m);
  if (!x_in || !y_out) return fail(TGP_EINVAL, "NULL x_in or y_out");
  if ((r = check_slices(N, j, x_in, y_out)) != TGP_OK) return r;
  if ((checkpoint != 0) != ckpt_of(N->mode, i, N->m))
    return fail(TGP_EINVAL, "checkpoint=%d disagrees with the planned policy for i=%d", checkpoint, i);
  int c = cell(N, i, j);
  if (N->st[c] == FWD || N->st[c] == BWD)
    return fail(TGP_ESTATE, "F_{%d,%d} already ran in this step", i, j);
  Range rg("F", i, j);
  r = run_forward(N, j, i, checkpoint ? 0 : 1, x_in, y_out, S(stream));
  if (r != TGP_OK) return r;
  N->st[c] = FWD;
  N->saved_x[c] = x_in;
  N->saved_y[c] = y_out;
  N->saved_ckpt[c] = checkpoint ? 1 : 0;
  return TGP_OK;
}

tgp_status tgp_stage_backward_recompute(tgp_net* N, int j, int i, const void* dy_out,
                                        void* dx_in, void* stream) {
  tgp_status r = check_ready(N, j);
  if (r != TGP_OK) return r;
  if (j < 1 || j > N->n) return fail(TGP_EINVAL, "partition %d out of 1..%d", j, N->n);
  if (i < 1 || i > N->m) return fail(TGP_EINVAL, "micro-batch %d out of 1..%d", i, N->m);
  if (!dy_out) return fail(TGP_EINVAL, "NULL dy_out");
  if ((r = check_slices(N, j, dx_in, dy_out)) != TGP_OK) return r;
  int c = cell(N, i, j);
  if (N->st[c] != FWD) return fail(TGP_ESTATE, "B_{%d,%d} needs F_{%d,%d} first", i, j, i, j);
  if (i < N->m && !follows_ok(N, i, j))
    return fail(TGP_ESTATE, "B_{%d,%d} must follow B_{%d,%d}%s", i, j, i + 1, j,
                N->gslots < N->m ? " and its accumulation" : "");
  r = run_backward(N, j, i, dy_out, dx_in, S(stream));
  if (r != TGP_OK) return r;
  N->st[c] = BWD;
  return TGP_OK;
}

// F_{iv[k],j} for a group of cnt micro-batches on distinct lanes, in one
// pass of the partition's layers.
static tgp_status stage_forward_group(tgp_net* N, int j, int cnt, const int* iv, const int* ck,
                                      const void* const* xs, void* const* ys, void* stream) {
  tgp_status r = check_ready(N, j);
  if (r != TGP_OK) return r;
  if (j < 1 || j > N->n) return fail(TGP_EINVAL, "partition %d out of 1..%d", j, N->n);
  if (cnt < 1 || cnt > MG) return fail(TGP_EINVAL, "count %d out of 1..%d", cnt, MG);
  if (!ck || !xs || !ys) return fail(TGP_EINVAL, "NULL checkpoint, x_in or y_out array");
  for (int k = 0; k < cnt; ++k) {
    if (iv[k] < 1 || iv[k] > N->m) return fail(TGP_EINVAL, "micro-batch %d out of 1..%d", iv[k], N->m);
    if ((ck[k] != 0) != ckpt_of(N->mode, iv[k], N->m))
      return fail(TGP_EINVAL, "checkpoint=%d disagrees with the planned policy for i=%d", ck[k], iv[k]);
    const int c = cell(N, iv[k], j);
    if (N->st[c] == FWD || N->st[c] == BWD)
      return fail(TGP_ESTATE, "F_{%d,%d} already ran in this step", iv[k], j);
    for (int q = 0; q < k; ++q)
      if ((iv[q] - 1) % N->lanes == (iv[k] - 1) % N->lanes)
        return fail(TGP_EINVAL, "micro-batches %d and %d share a lane (lanes = %d)", iv[q], iv[k],
                    N->lanes);
    if (!xs[k] || !ys[k]) return fail(TGP_EINVAL, "NULL x_in or y_out");
    if ((r = check_slices(N, j, xs[k], ys[k])) != TGP_OK) return r;
  }
  Range rg("F", iv[0], j);
  int ph[MG];
  for (int k = 0; k < cnt; ++k) ph[k] = ck[k] ? 0 : 1;
  r = run_forward_g(N, j, cnt, iv, ph, xs, ys, S(stream));
  if (r != TGP_OK) return r;
  for (int k = 0; k < cnt; ++k) {
    const int c = cell(N, iv[k], j);
    N->st[c] = FWD;
    N->saved_x[c] = xs[k];
    N->saved_y[c] = ys[k];
    N->saved_ckpt[c] = ck[k] ? 1 : 0;
  }
  return TGP_OK;
}

tgp_status tgp_stage_forward2(tgp_net* N, int j, int i0, int i1, int checkpoint0,
                              int checkpoint1, const void* x0, const void* x1, void* y0,
                              void* y1, void* stream) {
  const int iv[2] = {i0, i1};
  const int ck[2] = {checkpoint0, checkpoint1};
  const void* xs[2] = {x0, x1};
  void* ys[2] = {y0, y1};
  return stage_forward_group(N, j, 2, iv, ck, xs, ys, stream);
}

tgp_status tgp_stage_forward_n(tgp_net* N, int j, int i0, int count, const int* checkpoint,
                               const void* const* x_in, void* const* y_out, void* stream) {
  if (count < 1 || count > MG) return fail(TGP_EINVAL, "count %d out of 1..%d", count, MG);
  int iv[MG];
  for (int k = 0; k < count; ++k) iv[k] = i0 + k;
  return stage_forward_group(N, j, count, iv, checkpoint, x_in, y_out, stream);
}

tgp_status tgp_stage_backward_recompute_n(tgp_net* N, int j, int i0, int count,
                                          const void* const* dy_out, void* const* dx_in,
                                          void* stream) {
  tgp_status r = check_ready(N, j);
  if (r != TGP_OK) return r;
  if (j < 1 || j > N->n) return fail(TGP_EINVAL, "partition %d out of 1..%d", j, N->n);
  if (count < 1 || count > MG) return fail(TGP_EINVAL, "count %d out of 1..%d", count, MG);
  if (i0 - count + 1 < 1 || i0 > N->m)
    return fail(TGP_EINVAL, "micro-batches %d down to %d out of 1..%d", i0, i0 - count + 1, N->m);
  if (count > 1 && (N->gslots < N->m || count > N->lanes))
    return fail(TGP_EINVAL, "%d backwards at once need %d or more lanes (lanes = %d)", count, count,
                N->lanes);
  if (!dy_out || !dx_in) return fail(TGP_EINVAL, "NULL dy_out or dx_in array");
  int iv[MG];
  for (int k = 0; k < count; ++k) {
    iv[k] = i0 - k;
    if (!dy_out[k]) return fail(TGP_EINVAL, "NULL dy_out");
    if ((dx_in[k] == nullptr) != (dx_in[0] == nullptr))
      return fail(TGP_EINVAL, "dx_in: all or none");
    if ((r = check_slices(N, j, dx_in[k], dy_out[k])) != TGP_OK) return r;
  }
  for (int k = 0; k < count; ++k)
    if (N->st[cell(N, iv[k], j)] != FWD)
      return fail(TGP_ESTATE, "B_{%d,%d} needs F_{%d,%d} first", iv[k], j, iv[k], j);
  if (i0 < N->m && !follows_ok(N, i0, j))
    return fail(TGP_ESTATE, "B_{%d,%d} must follow B_{%d,%d}%s", i0, j, i0 + 1, j,
                N->gslots < N->m ? " and its accumulation" : "");
  r = run_backward_g(N, j, count, iv, dy_out, dx_in, S(stream));
  if (r != TGP_OK) return r;
  for (int k = 0; k < count; ++k) N->st[cell(N, iv[k], j)] = BWD;
  return TGP_OK;
}

tgp_status tgp_stage_backward_recompute2(tgp_net* N, int j, int i0, int i1, const void* dy0,
                                         const void* dy1, void* dx0, void* dx1, void* stream) {
  if (i1 != i0 - 1) {
    tgp_status r = check_ready(N, j);
    if (r != TGP_OK) return r;
    return fail(TGP_EINVAL, "need i1 = i0 - 1 within 1..%d (got %d, %d)", N->m, i0, i1);
  }
  const void* dys[2] = {dy0, dy1};
  void* dxs[2] = {dx0, dx1};
  return tgp_stage_backward_recompute_n(N, j, i0, 2, dys, dxs, stream);
}

tgp_status tgp_grad_accumulate(tgp_net* N, int j, int i, int overwrite, void* stream) {
  tgp_status r = check_ready(N, j);
  if (r != TGP_OK) return r;
  if (j < 1 || j > N->n) return fail(TGP_EINVAL, "partition %d out of 1..%d", j, N->n);
  if (i < 1 || i > N->m) return fail(TGP_EINVAL, "micro-batch %d out of 1..%d", i, N->m);
  if ((overwrite != 0) != (i == N->m))
    return fail(TGP_EINVAL, "overwrite must be 1 exactly for i = m");
  int c = cell(N, i, j);
  if (N->st[c] != BWD) return fail(TGP_ESTATE, "accumulate (%d,%d) needs B_{%d,%d} first", i, j, i, j);
  if (i < N->m && N->st[cell(N, i + 1, j)] != ACC)
    return fail(TGP_ESTATE, "accumulate (%d,%d) must follow accumulate (%d,%d)", i, j, i + 1, j);
  r = run_accumulate(N, j, i, overwrite, S(stream));
  if (r != TGP_OK) return r;
  N->st[c] = ACC;
  return TGP_OK;
}

tgp_status tgp_grad_accumulate_n(tgp_net* N, int j, int i0, int count, int overwrite,
                                 void* stream) {
  tgp_status r = check_ready(N, j);
  if (r != TGP_OK) return r;
  if (j < 1 || j > N->n) return fail(TGP_EINVAL, "partition %d out of 1..%d", j, N->n);
  if (count < 1 || count > MG) return fail(TGP_EINVAL, "count %d out of 1..%d", count, MG);
  if (i0 - count + 1 < 1 || i0 > N->m)
    return fail(TGP_EINVAL, "micro-batches %d down to %d out of 1..%d", i0, i0 - count + 1, N->m);
  if ((overwrite != 0) != (i0 == N->m))
    return fail(TGP_EINVAL, "overwrite must be 1 exactly for i0 = m");
  for (int q = 0; q < count; ++q)
    if (N->st[cell(N, i0 - q, j)] != BWD)
      return fail(TGP_ESTATE, "accumulate (%d,%d) needs B_{%d,%d} first", i0 - q, j, i0 - q, j);
  if (i0 < N->m && N->st[cell(N, i0 + 1, j)] != ACC)
    return fail(TGP_ESTATE, "accumulate (%d,%d) must follow accumulate (%d,%d)", i0, j, i0 + 1, j);
  r = run_accumulate_g(N, j, i0, count, overwrite, S(stream));
  if (r != TGP_OK) return r;
  for (int q = 0; q < count; ++q) N->st[cell(N, i0 - q, j)] = ACC;
  return TGP_OK;
}

// Streams (count) and events (2 count) for tgp_pipeline_step's lanes, on the
// current device; recreated if the device changed.
static tgp_status lane_streams_ready(tgp_net* N, int count) {
  int dev = 0;
  HIPCHK(hipGetDevice(&dev), "hipGetDevice");
  if (N->lane_device != dev) {
    for (auto e : N->lane_events) (void)hipEventDestroy(e);
    for (auto st : N->lane_streams) (void)hipStreamDestroy(st);
    N->lane_events.clear();
    N->lane_streams.clear();
    N->lane_device = dev;
  }
  while ((int)N->lane_streams.size() < count) {
    hipStream_t st = nullptr;
    HIPCHK(hipStreamCreateWithFlags(&st, hipStreamNonBlocking), "hipStreamCreateWithFlags");
    N->lane_streams.push_back(st);
  }
  while ((int)N->lane_events.size() < 2 * count) {
    hipEvent_t e = nullptr;
    HIPCHK(hipEventCreateWithFlags(&e, hipEventDisableTiming), "hipEventCreateWithFlags");
    N->lane_events.push_back(e);
  }
  return TGP_OK;
}

tgp_status tgp_pipeline_step(tgp_net* N, const void* x, const void* target, int B, int m, int n,
                             int mode, float* loss_dev, void* y_out, void* stream) {
  tgp_status r = check_ready(N);
  if (r != TGP_OK) return r;
  if (!x || !target || !loss_dev) return fail(TGP_EINVAL, "NULL x, target or loss");
  if (!aligned_to(x, 16) || !aligned_to(target, 16) || (y_out && !aligned_to(y_out, 16)) ||
      !aligned_to(loss_dev, 4))
    return fail(TGP_EINVAL, "x, target and y_out must be 16-byte aligned, loss_dev 4-byte");
  if (B != N->B || m != N->m || mode != N->mode)
    return fail(TGP_EINVAL, "B/m/mode differ from tgp_plan (%d/%d/%d)", N->B, N->m, N->mode);
  if (n != N->n) return fail(TGP_EINVAL, "n=%d differs from the partition (%d)", n, N->n);
  for (int c = 0; c < m * n; ++c)
    if (N->st[c] == FWD || N->st[c] == BWD)
      return fail(TGP_ESTATE, "a stage step is in progress");
  Range rg("pipeline_step");
  GpuExec ex;
  ex.N = N;
  ex.x = (const char*)x;
  ex.target = (const char*)target;
  ex.loss_dev = loss_dev;
  ex.y_out = (char*)y_out;
  ex.st = S(stream);
  ex.in_mb_bytes = (size_t)N->b * N->H * N->W * N->in_c * N->esz;
  ex.out_mb_bytes = N->out_bytes_mb;
  ex.K = std::min(N->lanes, m);
  if (ex.K > 1) {
    // fork: lanes + the accumulation stream wait for the caller's stream
    r = lane_streams_ready(N, ex.K + 1);
    if (r != TGP_OK) return r;
    for (int k = 0; k < ex.K; ++k) {
      ex.lane[k] = N->lane_streams[k];
      ex.lane_ev[k] = N->lane_events[k];
    }
    ex.acc = N->lane_streams[ex.K];
    hipEvent_t fork = N->lane_events[ex.K];
    HIPCHK(hipEventRecord(fork, ex.st), "hipEventRecord");
    for (int k = 0; k <= ex.K; ++k)
      HIPCHK(hipStreamWaitEvent(N->lane_streams[k], fork, 0), "hipStreamWaitEvent");
  }
  r = run_schedule(m, n, mode, ex);
  if (r != TGP_OK) {
    // a task failed part way: the step is abandoned, so every task of it
    // returns to idle and the next step (or stage call) starts afresh
    const std::string msg = g_err;
    std::fill(N->st.begin(), N->st.end(), (uint8_t)IDLE);
    std::fill(N->wt_stale.begin(), N->wt_stale.end(), (char)0);
    g_err = msg;
  }
  if (ex.K > 1) {
    // join every lane, also after an error, so that no fork is left open in
    // a capture; the first failure is the one reported
    tgp_status rj = TGP_OK;
    for (int k = 0; k <= ex.K; ++k) {
      hipEvent_t e = N->lane_events[ex.K + 1 + k];
      hipError_t he = hipEventRecord(e, N->lane_streams[k]);
      if (he == hipSuccess) he = hipStreamWaitEvent(ex.st, e, 0);
      if (he != hipSuccess && rj == TGP_OK && r == TGP_OK)
        rj = fail(TGP_EHIP, "lane join: %s", hipGetErrorString(he));
    }
    if (r == TGP_OK) r = rj;
  }
  if (r != TGP_OK) return r;
  const LayerRt& last = N->L.back();
  long numel = (long)N->B * last.H * last.W * last.d.cout;
  HIPCHK(tgpk::loss_finalize((const float*)W_(N, N->o_loss), m, 1.0f / (float)numel, loss_dev,
                             S(stream)),
         "loss_finalize");
  return TGP_OK;
}

// ------------------------------------------------------------ static scratch
// The workspace of tgp_pipeline_step_static: a device array of
// TGP_STATIC_SCRATCH_BYTES that every device the library runs on holds from
// load to process end.  Host code never passes `scratch` itself to a kernel
// or a copy (in host code the name is a host-side stand-in, not a device
// address): it asks hipGetSymbolAddress for the array's address on each
// device once, keeps it per device and uses only that.
static __device__ __align__(256) unsigned char scratch[TGP_STATIC_SCRATCH_BYTES];

static std::mutex g_scratch_mu;
static void* g_scratch_dev[TGP_STATIC_MAX_DEVICES] = {};

// Device address of the current device's copy of `scratch`.
static tgp_status scratch_address(void** p) {
  int dev = 0;
  HIPCHK(hipGetDevice(&dev), "hipGetDevice");
  if (dev < 0 || dev >= TGP_STATIC_MAX_DEVICES)
    return fail(TGP_EUNSUPPORTED, "device %d beyond the %d the static scratch serves", dev,
                TGP_STATIC_MAX_DEVICES);
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_dev[dev]) {
    void* q = nullptr;
    HIPCHK(hipGetSymbolAddress(&q, HIP_SYMBOL(scratch)), "hipGetSymbolAddress(scratch)");
    if (!q || ((uintptr_t)q & 255))
      return fail(TGP_EHIP, "static scratch address %p is not 256-byte aligned", q);
    g_scratch_dev[dev] = q;
  }
  *p = g_scratch_dev[dev];
  return TGP_OK;
}

tgp_status tgp_pipeline_step_static(tgp_net* N, const void* x, const void* target, int B, int m,
                                    int n, int mode, float* loss_dev, void* y_out, void* stream) {
  if (!N) return fail(TGP_EINVAL, "net is NULL");
  if (!N->planned) return fail(TGP_ESTATE, "tgp_plan has not been called");
  if (N->ws_need > TGP_STATIC_SCRATCH_BYTES)
    return fail(TGP_ENOSPACE,
                "the plan needs a workspace of %zu bytes; the static scratch holds %zu",
                N->ws_need, (size_t)TGP_STATIC_SCRATCH_BYTES);
  if (N->lanes != 1)
    return fail(TGP_EINVAL, "the static-scratch step runs one lane (lanes = %d): call "
                "tgp_set_lanes(net, 1) before tgp_plan", N->lanes);
  void* p = nullptr;
  tgp_status r = scratch_address(&p);
  if (r != TGP_OK) return r;
  char* ws0 = N->ws;
  const size_t size0 = N->ws_size;
  N->ws = (char*)p;
  N->ws_size = TGP_STATIC_SCRATCH_BYTES;
  r = tgp_pipeline_step(N, x, target, B, m, n, mode, loss_dev, y_out, stream);
  N->ws = ws0;            // the bound workspace (if any) is the net's again
  N->ws_size = size0;
  return r;
}

tgp_status tgp_schedule_trace(int m, int n, int mode, int32_t* ops, int cap, int* count) {
  if (!count) return fail(TGP_EINVAL, "count is NULL");
  if (m < 1 || n < 1) return fail(TGP_EINVAL, "m and n must be positive");
  if (mode < 0 || mode > 2) return fail(TGP_EINVAL, "bad checkpoint mode %d", mode);
  TraceExec t;
  run_schedule(m, n, mode, t);
  *count = (int)(t.ops.size() / 3);
  if (*count > cap || (!ops && *count > 0)) return fail(TGP_EINVAL, "capacity %d < %d ops", cap, *count);
  std::copy(t.ops.begin(), t.ops.end(), ops);
  return TGP_OK;
}

}  // extern "C"
