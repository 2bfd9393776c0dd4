/*
 * Oracle for the continual convolution / pooling step library.
 *
 * TEST INFRASTRUCTURE ONLY.  This file is a plain, slow, obviously correct
 * CPU implementation of ordinary (non-continual) convolution and pooling,
 * accumulated in double precision.  Only the test suite, the smoke check and
 * the CPU-baseline leg of the benchmark may load it.  It shares no code,
 * header, table or helper with the HIP library, and the HIP library never
 * loads it.
 *
 * Temporal padding is NOT a parameter here: the caller materialises every
 * temporal position of the window it wants reduced (padding frames included)
 * and marks each one valid (a real frame) or not (a padded frame) in `tvalid`.
 * For convolution an invalid frame is a zero frame, which is exactly zero
 * padding; for pooling an invalid frame is a pad (ignored by max, counted as 0
 * by average, and counted in the divisor only when count_include_pad is set).
 * Spatial padding is ordinary symmetric zero padding per frame.
 *
 * Layouts (Assumption 1 of the paper, section 3.1): input (B, C, T, H, W),
 * weight (C_out, C_in/groups, kT, kH, kW) as in PyTorch (Principle 1),
 * output (B, C_out, To, Ho, Wo).  Conv1d/2d are the H = W = 1 / W = 1 cases.
 */
#include <math.h>
#include <omp.h>
#include <stddef.h>
#include <stdint.h>

/* Thread count of the OpenMP loops below (the benchmark's CPU baseline times
 * the oracle at the host's full thread count and at one thread). */
void ora_set_threads(int32_t n) { omp_set_num_threads(n > 0 ? n : 1); }
int32_t ora_max_threads(void) { return omp_get_max_threads(); }

/* L_out = floor((L + 2p - d(k-1) - 1)/s) + 1, or 0 when the window does not fit. */
static int64_t out_len(int64_t L, int64_t k, int64_t s, int64_t p, int64_t d) {
  int64_t span = L + 2 * p - d * (k - 1) - 1;
  if (span < 0) return 0;
  return span / s + 1;
}

int64_t ora_out_len(int64_t L, int64_t k, int64_t s, int64_t p, int64_t d) {
  return out_len(L, k, s, p, d);
}

/*
 * Regular N-d cross-correlation, the definition PyTorch's ConvNd.forward uses
 * (Principle 1: a continual module's forward is identical to the nn module's):
 *
 *   y[b,o,t,i,j] = bias[o] + sum_{c<Cg} sum_{a<kT} sum_{u<kH} sum_{w<kW}
 *                  W[o,c,a,u,w] * X[b, g(o)*Cg + c, t*sT + a*dT,
 *                                   i*sH + u*dH - pH, j*sW + w*dW - pW]
 *
 * with g(o) = o / (C_out/groups), X zero outside the frame and zero on
 * temporal positions whose tvalid flag is 0.  No temporal padding is added.
 */
void ora_conv(const double* x, const uint8_t* tvalid,
              int64_t B, int64_t Cin, int64_t T, int64_t H, int64_t W,
              const double* wt, int64_t Cout, int64_t G,
              int64_t kT, int64_t kH, int64_t kW,
              const double* bias,
              int64_t sT, int64_t sH, int64_t sW,
              int64_t pH, int64_t pW,
              int64_t dT, int64_t dH, int64_t dW,
              double* y) {
  const int64_t Cg = Cin / G;
  const int64_t Og = Cout / G;
  const int64_t To = out_len(T, kT, sT, 0, dT);
  const int64_t Ho = out_len(H, kH, sH, pH, dH);
  const int64_t Wo = out_len(W, kW, sW, pW, dW);
  int64_t bo;
#pragma omp parallel for schedule(dynamic)
  for (bo = 0; bo < B * Cout; ++bo) {
    const int64_t b = bo / Cout, o = bo % Cout;
    const int64_t g = o / Og;
    for (int64_t t = 0; t < To; ++t)
      for (int64_t i = 0; i < Ho; ++i)
        for (int64_t j = 0; j < Wo; ++j) {
          double acc = bias ? bias[o] : 0.0;
          for (int64_t c = 0; c < Cg; ++c)
            for (int64_t a = 0; a < kT; ++a) {
              const int64_t ti = t * sT + a * dT;
              if (!tvalid[ti]) continue; /* zero frame */
              for (int64_t u = 0; u < kH; ++u) {
                const int64_t hi = i * sH + u * dH - pH;
                if (hi < 0 || hi >= H) continue;
                for (int64_t w = 0; w < kW; ++w) {
                  const int64_t wi = j * sW + w * dW - pW;
                  if (wi < 0 || wi >= W) continue;
                  const double wv = wt[(((o * Cg + c) * kT + a) * kH + u) * kW + w];
                  const double xv = x[((((b * Cin) + g * Cg + c) * T + ti) * H + hi) * W + wi];
                  acc += wv * xv;
                }
              }
            }
          y[(((b * Cout + o) * To + t) * Ho + i) * Wo + j] = acc;
        }
  }
}

/*
 * Regular N-d pooling, the definition of PyTorch's AvgPoolNd / MaxPoolNd
 * forward (Principle 1).  kind 0 = average, 1 = maximum.
 *   average: sum over the window's valid positions (pads add 0) divided by
 *            kT*kH*kW when count_include_pad, else by the number of valid
 *            positions in the window;
 *   maximum: maximum over the window's valid positions (pads are -inf).
 * Positions are valid when the temporal frame is flagged valid and the
 * spatial index lies inside the frame.
 */
void ora_pool(int32_t kind, const double* x, const uint8_t* tvalid,
              int64_t B, int64_t C, int64_t T, int64_t H, int64_t W,
              int64_t kT, int64_t kH, int64_t kW,
              int64_t sT, int64_t sH, int64_t sW,
              int64_t pH, int64_t pW,
              int64_t dT, int64_t dH, int64_t dW,
              int32_t count_include_pad,
              double* y) {
  const int64_t To = out_len(T, kT, sT, 0, dT);
  const int64_t Ho = out_len(H, kH, sH, pH, dH);
  const int64_t Wo = out_len(W, kW, sW, pW, dW);
  int64_t bc;
#pragma omp parallel for schedule(dynamic)
  for (bc = 0; bc < B * C; ++bc) {
    for (int64_t t = 0; t < To; ++t)
      for (int64_t i = 0; i < Ho; ++i)
        for (int64_t j = 0; j < Wo; ++j) {
          double sum = 0.0, mx = -INFINITY;
          int64_t count = 0;
          for (int64_t a = 0; a < kT; ++a) {
            const int64_t ti = t * sT + a * dT;
            if (!tvalid[ti]) continue;
            for (int64_t u = 0; u < kH; ++u) {
              const int64_t hi = i * sH + u * dH - pH;
              if (hi < 0 || hi >= H) continue;
              for (int64_t w = 0; w < kW; ++w) {
                const int64_t wi = j * sW + w * dW - pW;
                if (wi < 0 || wi >= W) continue;
                const double v = x[((bc * T + ti) * H + hi) * W + wi];
                sum += v;
                if (v > mx) mx = v;
                ++count;
              }
            }
          }
          double out;
          if (kind == 1) {
            out = mx;
          } else {
            const int64_t div = count_include_pad ? kT * kH * kW : count;
            out = div > 0 ? sum / (double)div : 0.0;
          }
          y[((bc * To + t) * Ho + i) * Wo + j] = out;
        }
  }
}
