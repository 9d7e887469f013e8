/*
 * ws_gemm.h -- C ABI of the warp-specialised tiled GEMM for AMD MI355X (gfx950).
 *
 * Operation (paper "A Performance Model for Warp Specialization Kernels",
 * Background, "General Matrix Multiplication"):
 *     C = A B,   A is M x K,  B is K x N,  C is M x N,
 * with the tiling tuple (T_M, T_N, T_K) of the same section: A is cut into
 * T_M x T_K tiles, B into T_K x T_N tiles, C into T_M x T_N tiles.
 *
 * Each output tile is computed by one workgroup in which producer (DMA)
 * wavefronts stream the A and B tiles of every K-iteration into a circular
 * buffer in LDS and consumer (MATH) wavefronts pop them, multiply-accumulate
 * and store the tile (Background, "The Warp Specialized GeMM Kernel in
 * CUTLASS", and Algorithm 1).  The consumer waves of a workgroup act as the
 * paper's MATH warp and its producer waves as its DMA warp(s).  Both
 * arrangements of that section exist (`split`):
 *   split 1  one DMA warp per MATH warp: every producer wave loads its share
 *            of the A tile and then of the B tile;
 *   split 2  two DMA warps per MATH warp: half of the producer waves load
 *            the A tile, the other half the B tile, concurrently.
 * Wave counts (consumer_waves, producer_waves, split):
 *   (1, 1, 1), (1, 2, 2), (4, 4, 1), (4, 8, 2), (4, 4, 2),
 *   (8, 4, 1), (8, 4, 2)  [eight consumer waves: 256 x 256 tiles only],
 *   and producer_waves = 0: the synchronous (not specialised) kernel.
 * `stages` is the circular buffer's capacity in K-iterations (the buffer of
 * Section 2.2 holding at most a fixed number of tiles).
 *
 * Data layout: A, B and C are dense and row-major (leading dimensions K, N
 * and N).  A and B hold IEEE binary16 (WS_F16) or bfloat16 (WS_BF16)
 * elements; C is binary32 unless an epilogue says otherwise.  Products are
 * accumulated in binary32.
 *
 * Epilogue: the paper's operation is C = A B.  ws_gemm_set_epilogue extends
 * it with the BLAS form C <- alpha (A B) + beta C and a 16-bit output type;
 * those handles run the general kernel variant (below).
 *
 * Shapes: the paper's model assumes the tiles divide the problem (T_M | M,
 * T_N | N, T_K | K).  Other shapes are accepted when K and N are multiples of
 * 8 (rows of 16 bytes): the grid covers ceil(M/T_M) x ceil(N/T_N) tiles, the
 * last K-iteration is partial, loads past the matrices read zeros and the
 * epilogue stores only inside C.  They run the general variant of the
 * kernel, which always uses the register-staged producers.
 *
 * Empty problems: M, N or K may be 0.  The configuration is still
 * validated; no GEMM kernel is launched (plan grid 0).  With M or N = 0 a
 * run does nothing; with K = 0 it writes C <- beta C (zeros for the default
 * epilogue: the product of an empty sum).  Pointers the run does not use
 * may be NULL: all three when M or N = 0, A and B when K = 0.
 *
 * Ownership: A, B and C are device pointers owned by the caller.  A handle
 * owns its host-side plan and a small device word for the wait watchdog.
 *
 * Errors: every function returns a ws_status; nothing throws or aborts across
 * this boundary.  Launches are asynchronous: a fault inside the kernel shows
 * up at the caller's next synchronisation of the stream.
 */
#ifndef WS_GEMM_H
#define WS_GEMM_H

#include <stdint.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

#define WS_GEMM_ABI_VERSION 7

typedef struct ws_gemm_handle* ws_gemm_t; /* opaque handle */

typedef enum { WS_F16 = 0, WS_BF16 = 1 } ws_dtype;

typedef enum {
  WS_OK = 0,
  WS_ERR_INVALID_ARG = 1,   /* NULL pointer, negative or oversized dimension, bad field */
  WS_ERR_UNSUPPORTED = 2,   /* valid request with no compiled kernel or wave arrangement */
  WS_ERR_LDS_OVERFLOW = 3,  /* stages x (A tile + B tile) does not fit in 160 KiB of LDS */
  WS_ERR_HIP = 4,           /* a HIP runtime call failed */
  WS_ERR_TIMEOUT = 5,       /* a producer/consumer wait exceeded its poll limit */
  WS_ERR_NOT_DIVISIBLE = 6  /* a ragged shape (tiles do not divide M, N or K) with K or N not a
                               multiple of 8, or with producer_waves = 0 */
} ws_status;

/* How producer waves move a tile from global memory into its LDS slot. */
typedef enum {
  WS_LOAD_REGISTERS = 0, /* buffer_load_dwordx4 into VGPRs several K-iterations ahead, then
                            ds_write_b128 once the slot is free (more bytes in flight) */
  WS_LOAD_DMA = 1        /* buffer_load_dwordx4 with the lds bit, straight into the slot once it
                            is free */
} ws_load_path;

typedef struct {
  int32_t tile_m, tile_n, tile_k; /* (T_M, T_N, T_K): powers of two, 32..256 (tile_k 32..128) */
  int32_t producer_waves;         /* DMA wavefronts per workgroup (see the list above) */
  int32_t consumer_waves;         /* MATH wavefronts per workgroup: 1, 4 (one per SIMD) or 8 (two) */
  int32_t stages;                 /* circular-buffer slots, 2..8 */
  int32_t dtype;                  /* ws_dtype of A and B */
  int32_t load_path;              /* ws_load_path of the producers */
  int32_t split;                  /* DMA warps per MATH warp, 1 or 2; 0 derives it from the wave
                                     counts: 2 when producer_waves == 2 consumer_waves, else 1 */
} ws_gemm_config;

typedef struct {
  int32_t grid;      /* persistent workgroups launched; 0 for an empty problem (M, N or K = 0) */
  int32_t block;     /* threads per workgroup: 64 x (producer_waves + consumer_waves) */
  int32_t lds_bytes; /* LDS per workgroup: 256 + stages x 2 x (T_M T_K + T_K T_N) */
  int32_t tiles_m, tiles_n, tiles; /* output tiles per dimension and in total (Section 2.1) */
  int32_t rounds;    /* dispatch rounds W = ceil(tiles / grid) (Section 2.1, "Wave") */
  int32_t iters;     /* K-iterations per tile S = K / T_K (Section 2.1, "Stage") */
  int32_t split;     /* 1 for one DMA warp per MATH warp, 2 for two */
  int32_t group_m;   /* tile rows per raster group */
  int32_t xcd_remap; /* 1 when workgroups are remapped so one XCD takes neighbouring tiles */
  int32_t ragged;    /* 1 when a tile does not divide its dimension */
  int32_t general;   /* 1 when the general kernel variant runs (ragged shapes, or a handle
                        with a non-default epilogue) */
} ws_gemm_plan_info;

/* Output element type of C. */
typedef enum { WS_OUT_F32 = 0, WS_OUT_BF16 = 1, WS_OUT_F16 = 2 } ws_out_dtype;

/* Epilogue of a handle: C <- alpha (A B) + beta C, computed in binary32 as
 * fma(beta, C, alpha * acc) and rounded once to out_dtype (round to nearest
 * even; out of range gives infinity).  With beta == 0, C is not read (NaN in
 * C does not propagate).  Default {1, 0, WS_OUT_F32}: the paper's C = A B. */
typedef struct {
  float alpha;
  float beta;
  int32_t out_dtype; /* ws_out_dtype; C's element type in ws_gemm_run */
} ws_gemm_epilogue;

typedef struct {
  int32_t spin_limit;     /* polls before a wait gives up (0: library default) */
  int32_t producer_delay; /* extra ~8k-cycle sleeps per K-iteration in every producer */
  int32_t consumer_delay; /* extra ~8k-cycle sleeps per K-iteration in every consumer */
} ws_gemm_debug;

/* ABI version of the loaded library (WS_GEMM_ABI_VERSION). */
int32_t ws_gemm_abi_version(void);

/* Static text for a status code (never NULL). */
const char* ws_gemm_status_str(ws_status s);

/* The HIP call and error text behind the last WS_ERR_HIP returned on this
 * thread ("" if none).  Static per-thread storage; never NULL. */
const char* ws_gemm_last_error(void);

/* Validate a configuration and derive its launch without touching a GPU.
 * num_cus: compute units to plan for; wgs_per_cu: resident workgroups per CU
 * (<= 0 derives it from LDS use, wave count and the registers the compiled
 * kernel allocates, recorded at build time).  The grid uses u <= wgs_per_cu
 * workgroups per CU, the u that minimises rounds x u (the largest on a tie),
 * so that no partly filled last round runs at the shared CUs' pace.
 * Fills *out on WS_OK. */
ws_status ws_gemm_plan(int64_t M, int64_t N, int64_t K, const ws_gemm_config* cfg,
                       int32_t num_cus, int32_t wgs_per_cu, ws_gemm_plan_info* out);

/* Output tile (tile_m_idx, tile_n_idx) that workgroup `wg` computes in
 * dispatch round `round` under plan `info` (as filled by ws_gemm_plan or
 * ws_gemm_query).  Returns WS_ERR_INVALID_ARG when that workgroup has no tile
 * in that round.  Host-only; describes the kernel's persistent tile loop. */
ws_status ws_gemm_schedule(const ws_gemm_plan_info* info, int32_t wg, int32_t round,
                           int32_t* tile_m_idx, int32_t* tile_n_idx);

/* Validate, pick the compiled kernel for cfg, query the current device and
 * allocate the handle.  The handle is bound to the device current at this
 * call; later runs must use a stream of that device. */
ws_status ws_gemm_create(int64_t M, int64_t N, int64_t K, const ws_gemm_config* cfg,
                         ws_gemm_t* out);

/* Enqueue C = A B (or the handle's epilogue) on `stream` (0 = the null
 * stream).  A (M x K) and B (K x N) must be 16-byte aligned device pointers,
 * C (M x N, element type of the epilogue's out_dtype) aligned to its element
 * size; pointers an empty problem does not use may be NULL.  Does not
 * synchronise.
 * Every element of C is written; nothing outside it. */
ws_status ws_gemm_run(ws_gemm_t h, const void* A, const void* B, void* C, hipStream_t stream);

/* Synchronise `stream`, then report and clear the watchdog word:
 * WS_ERR_TIMEOUT if any wait of a previous run on this handle gave up. */
ws_status ws_gemm_sync_status(ws_gemm_t h, hipStream_t stream);

/* Average shader clock of the runs since the last call (a measurement hook
 * for reporting a launch's fraction of peak against the clock it ran at).
 * Every GEMM launch of the handle has workgroup 0's first wave read the
 * shader-clock counter (s_memtime) and the 100 MHz reference counter
 * (s_memrealtime) at its start and its end and add the differences to two
 * device accumulators.  This call synchronises `stream`, returns the sums
 * and the number of launches they cover, and clears them.  The clock in MHz
 * is 100 * shader_cycles / ref_ticks.  Every kernel of the handle takes
 * part (GEMM, its general and traced twins, the calibration kernels) except
 * the empty calibration kernel and the K = 0 epilogue kernel. */
ws_status ws_gemm_clock(ws_gemm_t h, hipStream_t stream, uint64_t* shader_cycles,
                        uint64_t* ref_ticks, int64_t* launches);

/* The plan a handle launches with. */
ws_status ws_gemm_query(ws_gemm_t h, ws_gemm_plan_info* out);

/* Epilogue of later runs (NULL restores the default).  A non-default
 * epilogue switches the handle to the general kernel variant, with its own
 * launch (see ws_gemm_query).  WS_ERR_INVALID_ARG for a non-finite alpha or
 * beta or an unknown out_dtype; WS_ERR_UNSUPPORTED for a non-default
 * epilogue on a calibration handle, on a handle of the synchronous kernel
 * (producer_waves = 0), or while tracing is on (ws_gemm_set_trace refuses a
 * handle with a non-default epilogue likewise). */
ws_status ws_gemm_set_epilogue(ws_gemm_t h, const ws_gemm_epilogue* epi);

/* Test hooks: poll limit and injected producer/consumer delays for later
 * runs (NULL restores the defaults).  Delays force the buffer-full and
 * buffer-empty waits of Section 2.2; a tiny poll limit forces a timeout. */
ws_status ws_gemm_set_debug(ws_gemm_t h, const ws_gemm_debug* dbg);

/* Event trace of later runs (Section 2.2's events S_a, S_b, S_m, measured).
 * `buffer` is caller-owned device memory of at least wgs * iters * 8 * 4
 * bytes; workgroups 0 .. wgs-1 (wgs <= plan grid) each write iters records
 * of 8 uint32 shader-clock stamps (low 32 bits) per K-iteration q they
 * process, in order:
 *   0 A-tile issue start  1 B-tile issue start  2 A landed  3 B landed
 *   4 consumer sees slot full  5 consumer MFMA start  6 slot released
 *   7 epilogue end (last K-iteration of a tile; otherwise left untouched).
 * Records beyond the iterations a workgroup runs are left untouched.
 * NULL buffer turns tracing off.  Tracing costs a few instructions per
 * K-iteration in the traced workgroups. */
ws_status ws_gemm_set_trace(ws_gemm_t h, void* buffer, int64_t bytes, int32_t wgs, int32_t iters);

/* Calibration kernels of the performance model (paper, Section 4.2, "Measure
 * the Kernel Launch Time", "Measure the Epilogue Time", "Estimate the
 * Throughput and Startup Latency of the DMA and MATH Warps").  Each is the
 * GEMM kernel of cfg with one role reduced, launched with the GEMM's own
 * plan (grid, block, LDS ring), so it measures that kernel's costs:
 *   WS_CALIB_EMPTY     an empty kernel with the same launch (T_INIT);
 *   WS_CALIB_LOAD_A    producers load only the A tiles of every K-iteration
 *                      into the ring; consumers free each slot unread;
 *   WS_CALIB_LOAD_B    the same with only the B tiles;
 *   WS_CALIB_MATH      producers free slots without loading; consumers read
 *                      and multiply whatever the slots hold (no C stores);
 *   WS_CALIB_EPILOGUE  consumers store one zero tile per output tile, with
 *                      no K loop (T_EPILOGUE); the producers exit;
 *   WS_CALIB_LOAD_AB   producers load both tiles as in the GEMM; consumers
 *                      free each slot unread (the producers' own rate).
 * Run with ws_gemm_run (A, B, C as for the GEMM).  C is only written by
 * WS_CALIB_EPILOGUE (zeros); the other kinds leave it untouched.  Tracing is
 * not available on these handles.  WS_ERR_UNSUPPORTED when no calibration
 * variant of cfg was compiled, and for shapes the tiles do not divide or
 * empty problems (no GEMM launch to calibrate). */
typedef enum {
  WS_CALIB_NONE = -1, /* the GEMM itself (ws_gemm_create) */
  WS_CALIB_EMPTY = 0,
  WS_CALIB_LOAD_A = 1,
  WS_CALIB_LOAD_B = 2,
  WS_CALIB_MATH = 3,
  WS_CALIB_EPILOGUE = 4,
  WS_CALIB_LOAD_AB = 5
} ws_calib_kind;

ws_status ws_gemm_create_calibration(int64_t M, int64_t N, int64_t K, const ws_gemm_config* cfg,
                                     int32_t kind, ws_gemm_t* out);

/* C = A B in one call that allocates nothing, for callers that cannot
 * allocate device or host memory while they run: code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc.  It
 * validates and plans (M, N, K, cfg) as ws_gemm_create does, picks the same
 * kernel and launch (the general variant for shapes the tiles do not
 * divide; default epilogue, fp32 C) and enqueues it on `stream`, with no
 * handle, no hipMalloc / hipFree and no other allocating call.
 *
 * Scratch: the kernels' only device memory beyond A, B and C is the wait
 * watchdog's word.  Here it lives in a static 256-byte array of the library,
 * one copy per GPU (looked up on the first call on each device, with that
 * device current, and held until the process ends).  The kernels write it
 * only when a wait gives up; this entry point does not report that (use
 * ws_gemm_create / ws_gemm_run / ws_gemm_sync_status for the watchdog): such
 * a run exits early and leaves C incomplete.  The scratch need is fixed, so
 * no problem size is refused for it; sizes are limited as for
 * ws_gemm_create.  Calls that overlap on one GPU share that GPU's word.
 *
 * Arguments as for ws_gemm_create and ws_gemm_run (A, B 16-byte aligned
 * device pointers, C 4-byte aligned; those an empty problem does not use
 * may be NULL); `stream` 0 means the current device's null stream.
 * Asynchronous: returns once the launch is enqueued.  Errors as for those
 * two calls. */
ws_status ws_gemm_run_noalloc(int64_t M, int64_t N, int64_t K, const ws_gemm_config* cfg,
                              const void* A, const void* B, float* C, hipStream_t stream);

/* Free the handle; NULL is a no-op.  Must not race with runs using it. */
ws_status ws_gemm_destroy(ws_gemm_t h);

#ifdef __cplusplus
}
#endif

#endif /* WS_GEMM_H */
