// Host-side exercise of the library's scheduler (schedule.cpp) and of the
// oracle's C loops (oracle.c), built by tests/test_sanitize.py with
// AddressSanitizer and UndefinedBehaviorSanitizer: every descriptor of a
// grid is resolved, laid out and planned over its first steps and near the
// step-counter limit; the plans' invariants are checked; and the oracle's
// convolution and pooling run on small random inputs.  Any out-of-bounds
// access, overflow or other undefined behaviour aborts the program.
#include <cstdint>
#include <cstdio>
#include <cstdlib>
#include <random>
#include <vector>

#include "../../paper_2204_03418_amd/csrc/schedule.hpp"

extern "C" {
void ora_conv(const double* x, const uint8_t* tvalid, int64_t B, int64_t Cin, int64_t T,
              int64_t H, int64_t W, const double* wt, int64_t Cout, int64_t G, int64_t kT,
              int64_t kH, int64_t kW, const double* bias, int64_t sT, int64_t sH, int64_t sW,
              int64_t pH, int64_t pW, int64_t dT, int64_t dH, int64_t dW, double* y);
void ora_pool(int32_t kind, const double* x, const uint8_t* tvalid, int64_t B, int64_t C,
              int64_t T, int64_t H, int64_t W, int64_t kT, int64_t kH, int64_t kW, int64_t sT,
              int64_t sH, int64_t sW, int64_t pH, int64_t pW, int64_t dT, int64_t dH,
              int64_t dW, int32_t count_include_pad, double* y);
int64_t ora_out_len(int64_t L, int64_t k, int64_t s, int64_t p, int64_t d);
}

using namespace coinf;

static int failures = 0;
#define CHECK(c)                                                         \
  do {                                                                   \
    if (!(c)) {                                                          \
      std::fprintf(stderr, "check failed: %s (line %d)\n", #c, __LINE__); \
      ++failures;                                                        \
    }                                                                    \
  } while (0)

static void check_conv_plans(const ConvGeom& g) {
  const ConvLayout L = conv_layout(g);
  CHECK(L.total > 0 && L.ring_slot_elems > 0);
  std::vector<int64_t> firsts = {0, 1, 2, int64_t(g.f) + 3, kMaxSteps - 4 * g.f - 8};
  for (int64_t n0 : firsts) {
    for (int64_t n = n0; n < n0 + 3 * g.f + 6 && n < kMaxSteps; ++n) {
      for (int upd = 0; upd < 2; ++upd) {
        co_step_plan p;
        conv_plan(g, n, upd != 0, &p);
        CHECK(p.n_taps == g.kT);
        CHECK(p.emit == ((n >= g.d && (n - g.d) % g.sT == 0) ? 1 : 0));
        int emits = 0;
        for (int j = 0; j < p.n_taps; ++j) {
          const int a = p.action[j];
          CHECK(a >= CO_TAP_NONE && a <= CO_TAP_EMIT_FRESH);
          if (a == CO_TAP_NONE) continue;
          CHECK(p.slot[j] >= -1 && p.slot[j] < g.R);
          CHECK(p.target[j] >= 0);
          if (a == CO_TAP_EMIT || a == CO_TAP_EMIT_FRESH) {
            ++emits;
            CHECK(p.target[j] == p.out_index);
          }
        }
        CHECK(emits == p.emit);
      }
      const int64_t k = conv_emissions(g, n, 7);
      CHECK(k >= 0 && k <= 7);
    }
  }
  ConvGeom c = g;
  (void)conv_hash(c);
  if (g.algo == CO_ALGO_GEMM) {
    GemmConfig gc;
    CHECK(gemm_config(g, g.cfg, &gc));
  }
  GemmStepsConfig sc;
  (void)gemm_steps_config(g, &sc);
  (void)reg_pick(g);
  (void)packed_weight_bytes(g);
}

static void check_pool_plans(const PoolGeom& g) {
  const PoolLayout L = pool_layout(g);
  CHECK(L.total > 0);
  for (int64_t n0 : {int64_t(0), int64_t(g.f) + 1, kMaxSteps - 4 * g.f - 8}) {
    for (int64_t n = n0; n < n0 + 3 * g.f + 6 && n < kMaxSteps; ++n) {
      co_pool_plan p;
      pool_plan(g, n, &p);
      CHECK(p.write_slot >= 0 && p.write_slot < g.R);
      for (int j = 0; j < p.n_taps; ++j) CHECK(p.src[j] >= -2 && p.src[j] < g.R);
      CHECK(pool_emissions(g, n, 5) <= 5);
    }
  }
}

static void run_oracle(std::mt19937& rng) {
  std::normal_distribution<double> nd;
  for (int k = 1; k <= 3; ++k)
    for (int s = 1; s <= 2; ++s)
      for (int p = 0; p <= 1; ++p) {
        const int64_t B = 2, Cin = 4, Cout = 6, G = 2, T = 5, H = 4, W = 3;
        const int64_t To = ora_out_len(T, k, s, 0, 1), Ho = ora_out_len(H, k, 1, p, 1),
                      Wo = ora_out_len(W, k, 1, p, 1);
        if (To < 1 || Ho < 1 || Wo < 1) continue;
        std::vector<double> x(B * Cin * T * H * W), w(Cout * (Cin / G) * k * k * k), b(Cout);
        for (auto& v : x) v = nd(rng);
        for (auto& v : w) v = nd(rng);
        for (auto& v : b) v = nd(rng);
        std::vector<uint8_t> tv(T, 1);
        tv[0] = 0;
        std::vector<double> y(B * Cout * To * Ho * Wo);
        ora_conv(x.data(), tv.data(), B, Cin, T, H, W, w.data(), Cout, G, k, k, k, b.data(), s, 1,
                 1, p, p, 1, 1, 1, y.data());
        std::vector<double> z(B * Cin * To * Ho * Wo);
        for (int kind = 0; kind < 2; ++kind)
          ora_pool(kind, x.data(), tv.data(), B, Cin, T, H, W, k, k, k, s, 1, 1, p, p, 1, 1, 1,
                   1, z.data());
      }
}

int main() {
  int convs = 0, pools = 0;
  for (int sd = 0; sd <= 2; ++sd)
    for (int k : {1, 2, 3, 5, 9})
      for (int s : {1, 2, 3})
        for (int dil : {1, 2})
          for (int p : {0, 1, 2, 4})
            for (int groups : {1, 4})
              for (int dtype : {CO_F32, CO_BF16})
                for (int batch : {1, 3}) {
                  co_conv_desc d{};
                  d.spatial_dims = sd;
                  d.batch = batch;
                  d.in_channels = 8;
                  d.out_channels = groups == 4 ? 8 : 24;
                  d.groups = groups;
                  d.in_size[0] = sd >= 1 ? 9 : 1;
                  d.in_size[1] = sd >= 2 ? 6 : 1;
                  for (int a = 0; a < 3; ++a) {
                    const bool used = a <= sd;
                    d.kernel[a] = used ? (a == 0 ? k : 3) : 1;
                    d.stride[a] = a == 0 ? s : 1;
                    d.padding[a] = a == 0 ? p : (used ? 1 : 0);
                    d.dilation[a] = a == 0 ? dil : 1;
                  }
                  d.has_bias = 1;
                  d.dtype = dtype;
                  d.algo = CO_ALGO_AUTO;
                  ConvGeom g;
                  if (conv_geom(&d, &g) == CO_OK) {
                    ++convs;
                    check_conv_plans(g);
                  }
                  co_pool_desc pd{};
                  pd.kind = (k + s) % 2 ? CO_POOL_MAX : CO_POOL_AVG;
                  pd.spatial_dims = sd;
                  pd.batch = batch;
                  pd.channels = 8;
                  pd.in_size[0] = d.in_size[0];
                  pd.in_size[1] = d.in_size[1];
                  for (int a = 0; a < 3; ++a) {
                    pd.kernel[a] = d.kernel[a];
                    pd.stride[a] = d.stride[a];
                    pd.padding[a] = a == 0 ? p : 0;
                    pd.dilation[a] = pd.kind == CO_POOL_MAX ? d.dilation[a] : 1;
                  }
                  pd.count_include_pad = 1;
                  pd.dtype = dtype;
                  PoolGeom pg;
                  if (pool_geom(&pd, &pg) == CO_OK) {
                    ++pools;
                    check_pool_plans(pg);
                  }
                }
  std::mt19937 rng(12345);
  run_oracle(rng);
  std::printf("resolved %d convolution and %d pool descriptors; %d failed checks\n", convs, pools,
              failures);
  return failures == 0 ? 0 : 1;
}
