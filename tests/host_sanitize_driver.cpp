// Host-side driver of the tgp C ABI for an AddressSanitizer / UBSan build of
// the runtime: every call here runs on the host only (network description,
// partitioner, planner, bindings, argument and state checks, schedule
// traces) and enqueues no device work, so it runs without a GPU.  Exits 0
// when every expectation holds; the sanitizers abort on their own findings.
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <random>
#include <vector>

#include "tgp.h"

static int failures = 0;
#define EXPECT(cond)                                                                  \
  do {                                                                                \
    if (!(cond)) {                                                                    \
      std::fprintf(stderr, "%s:%d: expectation failed: %s (%s)\n", __FILE__, __LINE__, #cond, \
                   tgp_last_error());                                                 \
      ++failures;                                                                     \
    }                                                                                 \
  } while (0)

static void* const FAKE = (void*)(uintptr_t)(1u << 20);   // never dereferenced

static tgp_layer conv(int cin, int cout, int pro = TGP_PRO_NONE, int stash = -1, int pop = -1,
                      int kind = TGP_CONV3X3, int relu = 1, int bias = 1) {
  tgp_layer l;
  l.kind = kind; l.cin = cin; l.cout = cout; l.relu = relu; l.bias = bias;
  l.prologue = pro; l.stash_id = stash; l.pop_id = pop;
  return l;
}

// U-Net of `levels` levels, base channels c at the first, input channels ic.
static std::vector<tgp_layer> unet(int levels, int c, int ic) {
  std::vector<tgp_layer> L;
  int prev = ic;
  for (int l = 0; l < levels; ++l) {
    const int C = c << l;
    L.push_back(conv(prev, C, l ? TGP_PRO_MAXPOOL2 : TGP_PRO_NONE));
    L.push_back(conv(C, C, TGP_PRO_NONE, l < levels - 1 ? l : -1));
    prev = C;
  }
  for (int l = levels - 2; l >= 0; --l) {
    const int C = c << l;
    L.push_back(conv(prev + C, C, TGP_PRO_UPCAT2, -1, l));
    L.push_back(conv(C, C));
    prev = C;
  }
  L.push_back(conv(prev, 1, TGP_PRO_NONE, -1, -1, TGP_CONV1X1, 0, 1));
  return L;
}

static void bind_all(tgp_net* N, int n_layers) {
  for (int l = 0; l < n_layers; ++l) EXPECT(tgp_bind_params(N, l, FAKE, (const float*)FAKE,
                                                            (float*)FAKE, (float*)FAKE) == TGP_OK);
}

int main() {
  // ---- network validation
  {
    tgp_net* N = nullptr;
    std::vector<tgp_layer> bad = {conv(4, 8)};
    EXPECT(tgp_net_create(bad.data(), 1, 8, 16, 16, TGP_BF16, &N) == TGP_EINVAL);
    std::vector<tgp_layer> pool = {conv(8, 8, TGP_PRO_MAXPOOL2)};
    EXPECT(tgp_net_create(pool.data(), 1, 8, 7, 16, TGP_BF16, &N) == TGP_EINVAL);
    std::vector<tgp_layer> popmiss = {conv(8, 8, TGP_PRO_UPCAT2, -1, 3)};
    EXPECT(tgp_net_create(popmiss.data(), 1, 8, 16, 16, TGP_BF16, &N) == TGP_EINVAL);
    EXPECT(tgp_net_create(bad.data(), 0, 8, 16, 16, TGP_BF16, &N) == TGP_EINVAL);
  }
  // ---- U-Nets of 2..6 levels: partitions, plans in every mode and lane count
  for (int levels = 2; levels <= 6; ++levels) {
    std::vector<tgp_layer> L = unet(levels, 64, 64);
    tgp_net* N = nullptr;
    const int hw = 8 << levels;
    EXPECT(tgp_net_create(L.data(), (int)L.size(), 64, hw, hw, TGP_BF16, &N) == TGP_OK);
    if (!N) continue;
    for (int l = 0; l < (int)L.size(); ++l) {
      int64_t f = 0;
      EXPECT(tgp_layer_flops(N, l, &f) == TGP_OK && f > 0);
    }
    EXPECT(tgp_layer_flops(N, (int)L.size(), nullptr) == TGP_EINVAL);
    bind_all(N, (int)L.size());
    for (int n = 1; n <= std::min<int>(8, (int)L.size()); ++n) {
      EXPECT(tgp_set_partition(N, n, nullptr) == TGP_OK);
      int got = 0;
      std::vector<int> bal(64);
      EXPECT(tgp_get_partition(N, &got, bal.data()) == TGP_OK && got == n);
      int sum = 0;
      for (int k = 0; k < got; ++k) sum += bal[k];
      EXPECT(sum == (int)L.size());
      for (int lanes = 1; lanes <= 3; ++lanes) {
        EXPECT(tgp_set_lanes(N, lanes) == TGP_OK);
        for (int mode = 0; mode < 3; ++mode)
          for (int m : {1, 2, 4, 8}) {
            size_t bytes = 0;
            EXPECT(tgp_plan(N, 8, m, mode, &bytes) == TGP_OK && bytes > 0);
            EXPECT(tgp_bind_workspace(N, FAKE, bytes - 1) == TGP_ENOSPACE);
            EXPECT(tgp_bind_workspace(N, (char*)FAKE + 16, bytes) == TGP_EINVAL);
            EXPECT(tgp_bind_workspace(N, FAKE, bytes) == TGP_OK);
            void* p = nullptr;
            EXPECT(tgp_stash_ptr(N, 1, 0, 0, &p) == TGP_OK && p);
            EXPECT(tgp_stash_ptr(N, m + 1, 0, 1, &p) == TGP_EINVAL);
            // state machine and argument checks (nothing is enqueued)
            EXPECT(tgp_stage_backward_recompute(N, 1, m, FAKE, nullptr, nullptr) == TGP_ESTATE);
            EXPECT(tgp_grad_accumulate(N, 1, m, 1, nullptr) == TGP_ESTATE);
            // the planned checkpoint decision for micro-batch 1; the calls
            // below all fail a host check, so none of them enqueues work
            const int ck = mode == TGP_CKPT_ALWAYS || (mode == TGP_CKPT_EXCEPT_LAST && m > 1);
            EXPECT(tgp_stage_forward(N, n + 1, 1, ck, FAKE, FAKE, nullptr) == TGP_EINVAL);
            EXPECT(tgp_stage_forward(N, 1, 1, !ck, FAKE, FAKE, nullptr) == TGP_EINVAL);
            EXPECT(tgp_stage_forward(N, 1, 1, ck, (char*)FAKE + 8, FAKE, nullptr) == TGP_EINVAL);
            EXPECT(tgp_pipeline_step(N, FAKE, FAKE, 16, m, n, mode, (float*)FAKE, nullptr,
                                     nullptr) == TGP_EINVAL);
            EXPECT(tgp_pipeline_step(N, FAKE, FAKE, 8, m, n, mode, (float*)((char*)FAKE + 2),
                                     nullptr, nullptr) == TGP_EINVAL);
            {   // group calls that fail a host check (count, order, lanes, state)
              const int ckv[4] = {ck, ck, ck, ck};
              const void* xs[4] = {FAKE, FAKE, FAKE, FAKE};
              void* ys[4] = {FAKE, FAKE, FAKE, FAKE};
              EXPECT(tgp_stage_forward_n(N, 1, 1, 0, ckv, xs, ys, nullptr) == TGP_EINVAL);
              EXPECT(tgp_stage_forward_n(N, 1, 1, 17, ckv, xs, ys, nullptr) == TGP_EINVAL);
              EXPECT(tgp_grad_accumulate_n(N, 1, m, 0, 1, nullptr) == TGP_EINVAL);
              EXPECT(tgp_grad_accumulate_n(N, 1, m, m + 1, 1, nullptr) == TGP_EINVAL);
              EXPECT(tgp_grad_accumulate_n(N, 1, m, 1, 0, nullptr) == TGP_EINVAL);
              EXPECT(tgp_grad_accumulate_n(N, 1, m, m, 1, nullptr) == TGP_ESTATE);
              EXPECT(tgp_stage_forward_n(N, 1, m, 2, ckv, xs, ys, nullptr) == TGP_EINVAL);
              EXPECT(tgp_stage_backward_recompute_n(N, 1, 1, 2, xs, ys, nullptr) == TGP_EINVAL);
              const tgp_status sb = tgp_stage_backward_recompute_n(N, 1, m, 1, xs, ys, nullptr);
              EXPECT(sb == TGP_ESTATE);
            }
            if (lanes > 1) {   // refused for its size or for its lanes
              const tgp_status st = tgp_pipeline_step_static(N, FAKE, FAKE, 8, m, n, mode,
                                                             (float*)FAKE, nullptr, nullptr);
              EXPECT(st == TGP_EINVAL || st == TGP_ENOSPACE);
            }
          }
      }
      EXPECT(tgp_set_lanes(N, 1) == TGP_OK);
    }
    // per-layer timing plan: host part only
    size_t bytes = 0;
    EXPECT(tgp_layer_times_plan(N, 2, TGP_CKPT_ALWAYS, &bytes) == TGP_OK && bytes > 0);
    EXPECT(tgp_layer_times(N, FAKE, 0, 1, nullptr, nullptr) != TGP_OK);
    tgp_net_destroy(N);
  }
  // ---- schedule traces for every (m, n, mode) up to 8
  for (int m = 1; m <= 8; ++m)
    for (int n = 1; n <= 8; ++n)
      for (int mode = 0; mode < 3; ++mode) {
        int count = 0;
        EXPECT(tgp_schedule_trace(m, n, mode, nullptr, 0, &count) == TGP_EINVAL || count == 0);
        std::vector<int32_t> ops(3 * (size_t)count);
        EXPECT(tgp_schedule_trace(m, n, mode, ops.data(), count, &count) == TGP_OK);
        int fwd = 0;
        for (int k = 0; k < count; ++k) fwd += ops[3 * k] == TGP_OP_FORWARD;
        EXPECT(fwd == m * n);
      }
  // ---- balance rule on random costs
  std::mt19937_64 rng(7);
  for (int trial = 0; trial < 200; ++trial) {
    const int L = 1 + (int)(rng() % 40), n = 1 + (int)(rng() % L);
    std::vector<int64_t> cost(L);
    for (auto& c : cost) c = (int64_t)(rng() % 1000000);
    std::vector<int> bal(n);
    EXPECT(tgp_balance_minmax(cost.data(), L, n, bal.data()) == TGP_OK);
    int sum = 0;
    for (int b : bal) { EXPECT(b >= 1); sum += b; }
    EXPECT(sum == L);
  }
  std::vector<int> bal(4);
  EXPECT(tgp_balance_minmax(nullptr, 3, 4, bal.data()) == TGP_EINVAL);
  if (failures) std::fprintf(stderr, "%d expectation(s) failed\n", failures);
  else std::printf("host driver: ok\n");
  return failures ? 1 : 0;
}
