/*
 * ws_model.h -- C ABI of the performance model of the warp-specialised GEMM
 * (paper "A Performance Model for Warp Specialization Kernels", Section 2,
 * "Performance Model", and Section 3.1, "Execution Simulation").
 *
 * The model predicts the kernel time from the tiling tuple, the ring depth
 * and five calibrated machine parameters (Section 4.2):
 *     T_MATH   = T_M T_N T_K / compute_throughput + compute_latency
 *     T_LOAD-A = T_M T_K / load_throughput + load_latency
 *     T_LOAD-B = T_K T_N / load_throughput + load_latency
 * and the event recurrences of Section 2.2 (Eq. 1-3): S_a(i), S_b(i), S_m(i)
 * are the start times of the A load, the B load and the MATH of K-iteration i
 * (the paper's "stage") in one workgroup.  Overall time (Section 2.2):
 *     (S_m(S) + T_EPILOGUE) W + T_INIT,
 * with S = ceil(K / T_K) K-iterations and W = ceil(tiles / slots) rounds.
 *
 * Where the paper leaves the model open, the options select a reading:
 *   two_dma      0: one DMA warp loads A and then B (Eq. 1-3 as printed);
 *                1: two DMA warps, one per input tile, each chaining its own
 *                   loads; MATH waits for both tiles.
 *   persistent   0: the pipeline restarts every round (Section 2.1);
 *                1: one pipeline runs through all W rounds back to back, and
 *                   the epilogue of a tile delays the next tile's first MATH
 *                   (the persistent grid of the GPU kernel).
 *   finish_math  1: the round also waits for the last T_MATH (the prose says
 *                   a round ends when the last MATH finishes; the formula
 *                   stops at S_m(S) + T_EPILOGUE).
 * For i <= stages the buffer-release term S_m(i - stages) + T_MATH does not
 * exist and drops out of the max.
 *
 * Units: times in microseconds, throughputs in elements (loads) or
 * multiply-accumulates (MATH) per microsecond per workgroup.  Host-only,
 * no GPU needed; thread-safe.  Errors: WS_ERR_INVALID_ARG for NULL pointers,
 * non-positive sizes or throughputs.
 */
#ifndef WS_MODEL_H
#define WS_MODEL_H

#include <stdint.h>

#include "ws_gemm.h"

#ifdef __cplusplus
extern "C" {
#endif

typedef struct {
  double t_init;             /* launch overhead T_INIT */
  double t_epilogue;         /* one output-tile store T_EPILOGUE */
  double compute_throughput; /* multiply-accumulates per us, one workgroup */
  double compute_latency;    /* MATH startup latency */
  double load_throughput;    /* elements per us, one workgroup */
  double load_latency;       /* DMA startup latency */
} ws_model_params;

typedef struct {
  int32_t two_dma;     /* 0 or 1, see above */
  int32_t persistent;  /* 0 or 1 */
  int32_t finish_math; /* 0 or 1 */
} ws_model_options;

typedef struct {
  double total_us;   /* predicted kernel time */
  double round_us;   /* per-round time: S_m(S) + T_EPILOGUE (+ T_MATH); persistent: (total - T_INIT) / W */
  double t_math;     /* T_MATH of one K-iteration */
  double t_load_a;   /* T_LOAD-A */
  double t_load_b;   /* T_LOAD-B */
  double wait_us;    /* MATH waiting time summed over the K-iterations of all rounds
                        (Section 3.2, second objective) */
  int32_t rounds;    /* W */
  int32_t iters;     /* S */
} ws_model_result;

/* Predict the time of C = A B (M x K by K x N) with tile (tile_m, tile_n,
 * tile_k), a ring of `stages` K-iterations and `slots` workgroups running at
 * once (the paper's number of SMs).  opts may be NULL (all zero). */
ws_status ws_model_predict(int64_t M, int64_t N, int64_t K, int32_t tile_m, int32_t tile_n,
                           int32_t tile_k, int32_t stages, int32_t slots,
                           const ws_model_params* params, const ws_model_options* opts,
                           ws_model_result* out);

/* The same prediction from explicit per-K-iteration costs (T_MATH, T_LOAD-A,
 * T_LOAD-B measured for this configuration instead of the linear cost
 * model); params->t_init and params->t_epilogue are used, the throughputs
 * and latencies are ignored. */
ws_status ws_model_predict_costs(int64_t M, int64_t N, int64_t K, int32_t tile_m, int32_t tile_n,
                                 int32_t tile_k, int32_t stages, int32_t slots, double t_math,
                                 double t_load_a, double t_load_b, const ws_model_params* params,
                                 const ws_model_options* opts, ws_model_result* out);

/* Event times of one workgroup.  Writes n = iters (per-round schedule) or
 * n = rounds x iters (persistent) entries to each caller-owned array;
 * entry j holds the paper's index j + 1.  Any of s_a, s_b, s_m may be NULL. */
ws_status ws_model_events(int32_t iters, int32_t rounds, int32_t stages, double t_math,
                          double t_load_a, double t_load_b, double t_epilogue,
                          const ws_model_options* opts, double* s_a, double* s_b, double* s_m);

#ifdef __cplusplus
}
#endif

#endif /* WS_MODEL_H */
