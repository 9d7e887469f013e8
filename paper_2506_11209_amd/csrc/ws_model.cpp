// Performance model of the warp-specialised GEMM (paper, Section 2) and its
// execution simulator (Section 3.1), behind the C ABI of ws_model.h.
//
// The simulator walks the K-iterations of one workgroup in order and keeps
// the state of the three resources the model has: the DMA warp(s) (free from
// some time on), the MATH warp, and the ring of `stages` buffer slots (slot
// j mod stages is released when MATH of K-iteration j has finished).  A
// load starts when its DMA warp is free and its slot has been released; MATH
// of K-iteration j starts when MATH of j - 1 is done and both tiles of j have
// landed.  This is the max-plus system of Eq. 1-3 evaluated forward.
#include <math.h>
#include <stdint.h>

#include <vector>

#include "ws_model.h"

namespace {

struct Options {
  bool two_dma = false, persistent = false, finish_math = false;
};

Options read_options(const ws_model_options* o) {
  Options r;
  if (o) {
    r.two_dma = o->two_dma != 0;
    r.persistent = o->persistent != 0;
    r.finish_math = o->finish_math != 0;
  }
  return r;
}

// Simulate n K-iterations (tiles of `iters` K-iterations back to back when
// persistent).  Writes event times when the arrays are given; returns
// S_m of the last K-iteration and the summed MATH waiting time.
struct SimOut {
  double last_sm = 0.0;
  double wait = 0.0;
};

SimOut simulate(int64_t n, int32_t iters, int32_t stages, double t_math, double t_la, double t_lb,
                double t_epi, const Options& opt, double* s_a, double* s_b, double* s_m) {
  std::vector<double> release((size_t)stages, 0.0);  // slot release times (valid once used)
  double dma_free = 0.0;          // one DMA warp: free to start the next A load
  double a_free = 0.0, b_free = 0.0;  // two DMA warps
  double math_free = 0.0;         // MATH done with the previous K-iteration (and epilogue)
  SimOut out;
  for (int64_t j = 0; j < n; ++j) {
    const size_t slot = (size_t)(j % stages);
    const bool reused = j >= stages;  // slot must first be released by K-iteration j - stages
    const double rel = release[slot];
    double sa, sb, ready;
    if (!opt.two_dma) {
      sa = (j == 0) ? 0.0 : dma_free;
      if (reused && rel > sa) sa = rel;
      sb = sa + t_la;
      if (reused && rel > sb) sb = rel;
      dma_free = sb + t_lb;
      ready = dma_free;
    } else {
      sa = (j == 0) ? 0.0 : a_free;
      sb = (j == 0) ? 0.0 : b_free;
      if (reused) {
        if (rel > sa) sa = rel;
        if (rel > sb) sb = rel;
      }
      a_free = sa + t_la;
      b_free = sb + t_lb;
      ready = a_free > b_free ? a_free : b_free;
    }
    double sm = ready;
    if (j > 0 && math_free > sm) sm = math_free;
    out.wait += (j == 0) ? sm : sm - math_free;
    math_free = sm + t_math;
    release[slot] = math_free;
    if (opt.persistent && (j + 1) % iters == 0) math_free += t_epi;  // epilogue of the tile
    if (s_a) s_a[j] = sa;
    if (s_b) s_b[j] = sb;
    if (s_m) s_m[j] = sm;
    out.last_sm = sm;
  }
  return out;
}

bool positive(double x) { return x > 0.0 && isfinite(x); }

ws_status predict_core(int64_t M, int64_t N, int64_t K, int32_t tile_m, int32_t tile_n,
                       int32_t tile_k, int32_t stages, int32_t slots, double t_math, double t_la,
                       double t_lb, const ws_model_params* p, const ws_model_options* o,
                       ws_model_result* out) {
  const Options opt = read_options(o);
  const int64_t tiles = ((M + tile_m - 1) / tile_m) * ((N + tile_n - 1) / tile_n);
  const int64_t W = (tiles + slots - 1) / slots;
  const int64_t S = (K + tile_k - 1) / tile_k;
  if (W > INT32_MAX || S > INT32_MAX || W * S > (int64_t)1 << 31) return WS_ERR_INVALID_ARG;
  const double tail = p->t_epilogue + (opt.finish_math ? t_math : 0.0);
  ws_model_result r{};
  r.t_math = t_math;
  r.t_load_a = t_la;
  r.t_load_b = t_lb;
  r.rounds = (int32_t)W;
  r.iters = (int32_t)S;
  if (opt.persistent) {
    const SimOut s = simulate(W * S, (int32_t)S, stages, t_math, t_la, t_lb, p->t_epilogue, opt,
                              nullptr, nullptr, nullptr);
    r.total_us = s.last_sm + tail + p->t_init;
    r.round_us = (r.total_us - p->t_init) / (double)W;
    r.wait_us = s.wait;
  } else {
    const SimOut s =
        simulate(S, (int32_t)S, stages, t_math, t_la, t_lb, p->t_epilogue, opt, nullptr, nullptr, nullptr);
    r.round_us = s.last_sm + tail;
    r.total_us = r.round_us * (double)W + p->t_init;
    r.wait_us = (double)W * s.wait;
  }
  *out = r;
  return WS_OK;
}

bool sizes_ok(int64_t M, int64_t N, int64_t K, int32_t tile_m, int32_t tile_n, int32_t tile_k,
              int32_t stages, int32_t slots) {
  return M > 0 && N > 0 && K > 0 && tile_m > 0 && tile_n > 0 && tile_k > 0 && stages > 0 && slots > 0;
}

}  // namespace

extern "C" ws_status ws_model_predict(int64_t M, int64_t N, int64_t K, int32_t tile_m, int32_t tile_n,
                                      int32_t tile_k, int32_t stages, int32_t slots,
                                      const ws_model_params* p, const ws_model_options* o,
                                      ws_model_result* out) {
  if (!p || !out || !sizes_ok(M, N, K, tile_m, tile_n, tile_k, stages, slots)) return WS_ERR_INVALID_ARG;
  if (!positive(p->compute_throughput) || !positive(p->load_throughput)) return WS_ERR_INVALID_ARG;
  const double t_math =
      (double)((int64_t)tile_m * tile_n * tile_k) / p->compute_throughput + p->compute_latency;
  const double t_la = (double)((int64_t)tile_m * tile_k) / p->load_throughput + p->load_latency;
  const double t_lb = (double)((int64_t)tile_k * tile_n) / p->load_throughput + p->load_latency;
  return predict_core(M, N, K, tile_m, tile_n, tile_k, stages, slots, t_math, t_la, t_lb, p, o, out);
}

extern "C" ws_status ws_model_predict_costs(int64_t M, int64_t N, int64_t K, int32_t tile_m,
                                            int32_t tile_n, int32_t tile_k, int32_t stages,
                                            int32_t slots, double t_math, double t_load_a,
                                            double t_load_b, const ws_model_params* p,
                                            const ws_model_options* o, ws_model_result* out) {
  if (!p || !out || !sizes_ok(M, N, K, tile_m, tile_n, tile_k, stages, slots)) return WS_ERR_INVALID_ARG;
  if (!isfinite(t_math) || !isfinite(t_load_a) || !isfinite(t_load_b)) return WS_ERR_INVALID_ARG;
  return predict_core(M, N, K, tile_m, tile_n, tile_k, stages, slots, t_math, t_load_a, t_load_b, p, o,
                      out);
}

extern "C" ws_status ws_model_events(int32_t iters, int32_t rounds, int32_t stages, double t_math,
                                     double t_load_a, double t_load_b, double t_epilogue,
                                     const ws_model_options* o, double* s_a, double* s_b, double* s_m) {
  if (iters <= 0 || stages <= 0) return WS_ERR_INVALID_ARG;
  const Options opt = read_options(o);
  if (opt.persistent && rounds <= 0) return WS_ERR_INVALID_ARG;
  const int64_t n = opt.persistent ? (int64_t)rounds * iters : (int64_t)iters;
  simulate(n, iters, stages, t_math, t_load_a, t_load_b, t_epilogue, opt, s_a, s_b, s_m);
  return WS_OK;
}
