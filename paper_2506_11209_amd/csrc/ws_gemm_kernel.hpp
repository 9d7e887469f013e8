// Warp-specialised tiled GEMM kernel for gfx950 (MI355X).
//
// C (M x N, fp32) = A (M x K) * B (K x N), A and B fp16 or bf16, all row-major.
// The kernel follows the producer/consumer structure of the GeMM-WS kernel the
// paper models (Section 1.3, Algorithm 1): inside each workgroup, producer
// ("DMA") wavefronts move A and B tiles from global memory into a circular
// buffer of `stages` slots in LDS, and consumer ("MATH") wavefronts take the
// tiles out, run the contraction on the matrix cores and write the output
// tile (the epilogue).  The two sides synchronise through wait/signal
// counters, one pair per slot (Section 1.3: the buffer blocks producers when
// full and consumers when empty).
//
// gfx950 mapping
//  * Roles are chosen per wavefront from the wave index, so no wave diverges
//    (Section 1.2).  Waves [0, NC) are consumers, waves [NC, NC + NP) are
//    producers.  With NC = 4 the consumers sit one per SIMD and tile the
//    output block 2 x 2.
//  * Producers use global_load_lds_dwordx4: 64 lanes x 16 bytes go straight
//    from memory into 1 KiB of LDS without passing through VGPRs.  The LDS
//    placement of every 16-byte chunk is chosen through the global address
//    each lane fetches.
//  * 1:1 split (NP == NC): every producer loads a share of the A tile and then
//    a share of the B tile, in that order (one DMA warp loading both tiles).
//    2:1 split (NP == 2 NC): the first half of the producers loads A, the
//    second half loads B, concurrently (two DMA warps, one tile each).
//  * Consumers read operands with ds_read_b128 (A, K-contiguous) and
//    ds_read_b64_tr_b16 (B, N-contiguous, transposed by the read) and
//    accumulate with v_mfma_f32_32x32x16_{bf16,f16} in fp32.
//  * The grid is persistent: at most one workgroup per CU slot, each walking
//    output tiles in dispatch rounds (Section 2.1, "Wave").  The tile order
//    places the tiles that run at the same time on one XCD next to each
//    other so that they share A row panels and B column panels in that XCD's
//    L2.
//
// LDS layout (dynamic shared memory)
//   [0, 256)            counters: full[8], empty[8], abort
//   [256 + s * STAGE)   slot s: A tile (TM x TK) then B tile (TK x TN)
// A tile: row-major, each row split in 16-byte chunks (8 elements); chunk c of
//   row r is stored at position c ^ swz_a(r).
// B tile: 4 x 16 element blocks of 128 bytes; block (kq, nq) holds rows
//   4 kq .. 4 kq + 3 and columns 16 nq .. 16 nq + 15, row-major inside the
//   block; blocks are ordered kq-major.  One 16-lane transposed read takes one
//   whole block.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "ws_gemm_plan.hpp"

namespace wsg {

typedef __attribute__((ext_vector_type(8))) __bf16 bf16x8_t;
typedef __attribute__((ext_vector_type(8))) _Float16 f16x8_t;
typedef __attribute__((ext_vector_type(4))) short i16x4_t;
typedef __attribute__((ext_vector_type(8))) short i16x8_t;
typedef __attribute__((ext_vector_type(16))) float f32x16_t;

#define WSG_LDS __attribute__((address_space(3)))

constexpr int kHeaderBytes = 256;
constexpr int kMaxStages = 8;

struct KernelArgs {
  const uint16_t* A;
  const uint16_t* B;
  float* C;
  int32_t M, N, K;
  int32_t tiles_m, tiles_n, num_tiles;
  int32_t iters;       // S = K / TK
  int32_t stages;      // ring slots P
  int32_t group_m;     // tile rows per raster group
  int32_t xcd_remap;   // 1: remap workgroup ids so one XCD gets consecutive tiles
  int32_t spin_limit;  // bounded waits: give up after this many polls
  int32_t producer_delay;  // debug: s_sleep bursts per K-iteration in producers
  int32_t consumer_delay;  // debug: s_sleep bursts per K-iteration in consumers
  int32_t* err;            // set to 1 when a bounded wait gives up
};

// XOR swizzle of the 16-byte chunks of A-tile row r.  It depends on r & 31
// only, so rows 32 apart share it and the consumer can fold whole 32-row
// blocks into instruction offsets.  Rows 0..15 read by one ds_read_b128 fall
// on distinct 16-byte bank groups (for both 128- and 256-byte bank rows).
template <int TK>
__host__ __device__ constexpr int swz_a(int r) {
  if constexpr (TK == 32) return ((r >> 1) ^ (r >> 3)) & 3;
  else if constexpr (TK == 64) return (r ^ ((r >> 3) & 1)) & 7;
  else return r & 15;
}

template <int TK>
constexpr bool swz_a_period32() {
  for (int r = 0; r < 256; ++r)
    if (swz_a<TK>(r) != swz_a<TK>(r & 31) || swz_a<TK>(r) < 0 || swz_a<TK>(r) >= TK / 8)
      return false;
  return true;
}
static_assert(swz_a_period32<32>() && swz_a_period32<64>() && swz_a_period32<128>(),
              "A swizzle must repeat every 32 rows and stay inside the row");

__device__ __forceinline__ uint32_t lds_peek(WSG_LDS uint32_t* p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
}

// Compiler-only fence: no memory access moves across it.
__device__ __forceinline__ void compiler_fence() { asm volatile("" ::: "memory"); }

template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(N >= 0 && N <= 63, "vmcnt range");
#if defined(__HIP_DEVICE_COMPILE__)
  asm volatile("s_waitcnt vmcnt(%0)" ::"n"(N) : "memory");
#endif
}

// signal(): add one to an LDS counter from lane 0 only, after every earlier
// LDS access of this wave has completed.  Done in one asm block with the exec
// mask narrowed to lane 0, so the surrounding code stays branch-free.
__device__ __forceinline__ void lds_signal(WSG_LDS uint32_t* p) {
#if defined(__HIP_DEVICE_COMPILE__)
  const uint32_t addr = (uint32_t)(uintptr_t)p;
  const uint32_t one = 1u;
  uint64_t saved;
  asm volatile(
      "s_waitcnt lgkmcnt(0)\n\t"
      "s_mov_b64 %0, exec\n\t"
      "s_mov_b64 exec, 1\n\t"
      "ds_add_u32 %1, %2\n\t"
      "s_mov_b64 exec, %0"
      : "=&s"(saved)
      : "v"(addr), "v"(one)
      : "memory");
#endif
}

// Blocking read of an LDS counter, issued from asm so that the compiler does
// not order it behind outstanding LDS-DMA loads (it cannot prove the counter
// and the DMA destination are disjoint).  Result is wave-uniform.
__device__ __forceinline__ uint32_t lds_read_now(WSG_LDS uint32_t* p) {
#if defined(__HIP_DEVICE_COMPILE__)
  const uint32_t addr = (uint32_t)(uintptr_t)p;
  uint32_t v;
  asm volatile(
      "ds_read_b32 %0, %1\n\t"
      "s_waitcnt lgkmcnt(0)"
      : "=v"(v)
      : "v"(addr)
      : "memory");
  return __builtin_amdgcn_readfirstlane(v);
#else
  return *p;
#endif
}

// wait(): poll *ctr until it reaches target (wrap-safe).  Returns false when
// the workgroup aborted or this wait exceeded the poll limit (it then raises
// the abort flag and the global error word, so every wave drains quickly).
// The result is wave-uniform.
__device__ __forceinline__ bool wait_counter(WSG_LDS uint32_t* ctr, uint32_t target,
                                             WSG_LDS uint32_t* abort_flag, int spin_limit,
                                             int32_t* err) {
  int spins = 0;
  bool ok = true;
  while (true) {
    const uint32_t v = lds_read_now(ctr);
    if ((int32_t)(v - target) >= 0) break;
    if (lds_read_now(abort_flag)) {
      ok = false;
      break;
    }
    if (++spins > spin_limit) {
      if ((threadIdx.x & 63) == 0) {
        __hip_atomic_store(abort_flag, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
        __hip_atomic_fetch_or(err, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      }
      ok = false;
      break;
    }
    __builtin_amdgcn_s_sleep(1);
  }
  compiler_fence();
  return __builtin_amdgcn_readfirstlane((int)ok) != 0;
}

__device__ __forceinline__ void debug_delay(int n) {
  for (int i = 0; i < n; ++i) __builtin_amdgcn_s_sleep(127);
}

template <bool BF16>
__device__ __forceinline__ f32x16_t mfma32x32x16(const i16x8_t& a, const i16x8_t& b,
                                                 const f32x16_t& c) {
  if constexpr (BF16)
    return __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8_t, a),
                                                   __builtin_bit_cast(bf16x8_t, b), c, 0, 0, 0);
  else
    return __builtin_amdgcn_mfma_f32_32x32x16_f16(__builtin_bit_cast(f16x8_t, a),
                                                  __builtin_bit_cast(f16x8_t, b), c, 0, 0, 0);
}

template <int TM, int TN, int TK, int NC, int SPLIT, bool BF16>
struct Cfg {
  static constexpr int NP = NC * SPLIT;              // producer waves
  static constexpr int NW = NC + NP;                 // waves per workgroup
  static constexpr int WGM = (NC == 4) ? 2 : 1;      // consumer grid rows
  static constexpr int WGN = (NC == 4) ? 2 : 1;      // consumer grid cols
  static constexpr int WM = TM / WGM;                // wave tile rows
  static constexpr int WN = TN / WGN;                // wave tile cols
  static constexpr int BM = WM / 32;                 // 32x32 blocks per wave (rows)
  static constexpr int BN = WN / 32;
  static constexpr int KS = TK / 16;                 // MFMA k-steps per K-iteration
  static constexpr int A_BYTES = TM * TK * 2;
  static constexpr int B_BYTES = TK * TN * 2;
  static constexpr int STAGE = A_BYTES + B_BYTES;
  static constexpr int A_INSTR = A_BYTES / 1024;     // 1 KiB DMA instructions per A tile
  static constexpr int B_INSTR = B_BYTES / 1024;
  static constexpr int CA = TK / 8;                  // 16-byte chunks per A row
  static constexpr int NQ = TN / 16;                 // B blocks per block-row
  static_assert(NC == 1 || NC == 4, "consumer waves must be 1 or 4");
  static_assert(SPLIT == 1 || SPLIT == 2, "split must be 1:1 or 2:1");
  static_assert(WM % 32 == 0 && WN % 32 == 0, "wave tile must be a multiple of 32x32");
  static_assert(TK == 32 || TK == 64 || TK == 128, "TK must be 32, 64 or 128");
  static_assert(A_BYTES % 1024 == 0 && B_BYTES % 1024 == 0, "tiles must be whole KiB");
};

// ---------------------------------------------------------------------------
// Per-workgroup tile sequence (identical in both roles).
// ---------------------------------------------------------------------------
__device__ __forceinline__ int first_slot(const KernelArgs& args) {
  const int G = gridDim.x;
  return args.xcd_remap ? xcd_slot(blockIdx.x, G) : (int)blockIdx.x;
}

// ---------------------------------------------------------------------------
// Producer (DMA warp).  Waits for a free slot, streams its share of the A
// and/or B tile of one K-iteration into that slot, and signals the slot full
// once the data has landed.  The data of K-iteration q is awaited only after
// the loads of q + 1 are issued, so two K-iterations are in flight per wave.
// ---------------------------------------------------------------------------
template <int TM, int TN, int TK, int NC, int SPLIT, bool BF16, bool DO_A, bool DO_B>
__device__ __forceinline__ void producer_loop(const KernelArgs& args, WSG_LDS char* smem,
                                              int a_rank, int b_rank, int lane) {
  using G = Cfg<TM, TN, TK, NC, SPLIT, BF16>;
  constexpr int A_GROUP = (SPLIT == 1) ? G::NP : G::NP / 2;  // waves sharing the A tile
  constexpr int B_GROUP = (SPLIT == 1) ? G::NP : G::NP / 2;
  constexpr int A_PER = DO_A ? G::A_INSTR / A_GROUP : 0;     // DMA instructions per wave
  constexpr int B_PER = DO_B ? G::B_INSTR / B_GROUP : 0;
  constexpr int LOADS = A_PER + B_PER;
  static_assert(G::A_INSTR % A_GROUP == 0 && G::B_INSTR % B_GROUP == 0, "even DMA split");
  static_assert(LOADS > 0 && LOADS <= 63, "vmcnt range");

  WSG_LDS uint32_t* full = (WSG_LDS uint32_t*)smem;
  WSG_LDS uint32_t* empty = full + kMaxStages;
  WSG_LDS uint32_t* abort_flag = full + 2 * kMaxStages;
  const int K = args.K, N = args.N;

  // Element offset, inside the tile, of the 16-byte chunk this lane fetches for
  // each of its DMA instructions (the LDS side is fixed: lane l writes bytes
  // 16 l .. 16 l + 15 of the instruction's KiB).
  uint32_t a_goff[A_PER > 0 ? A_PER : 1];  // bytes
  uint32_t b_goff[B_PER > 0 ? B_PER : 1];
#pragma unroll
  for (int n = 0; n < A_PER; ++n) {
    const int q = (a_rank + n * A_GROUP) * 64 + lane;  // chunk index in the LDS tile
    const int r = q / G::CA, p = q % G::CA;
    a_goff[n] = (uint32_t)(r * K + 8 * (p ^ swz_a<TK>(r))) * 2u;
  }
#pragma unroll
  for (int n = 0; n < B_PER; ++n) {
    const int q = (b_rank + n * B_GROUP) * 64 + lane;
    const int blk = q >> 3, w = q & 7;
    const int kq = blk / G::NQ, nq = blk % G::NQ;
    b_goff[n] = (uint32_t)((kq * 4 + (w >> 1)) * N + nq * 16 + (w & 1) * 8) * 2u;
  }

  const int Gd = gridDim.x;
  const uint32_t P = (uint32_t)args.stages;
  uint32_t q = 0;
  bool pending = false;
  uint32_t pending_slot = 0;
  for (int v = first_slot(args); v < args.num_tiles; v += Gd) {
    int ti, tj;
    tile_coords(v, args.tiles_m, args.tiles_n, args.group_m, &ti, &tj);
    const uint16_t* a_tile = args.A + (int64_t)ti * TM * K;
    const uint16_t* b_tile = args.B + (int64_t)tj * TN;
    for (int kk = 0; kk < args.iters; ++kk, ++q) {
      const uint32_t slot = q % P;
      const uint32_t use = q / P;
      if (use > 0) {
        // wait(): the slot is free once every consumer wave released use - 1.
        const uint32_t need = use * NC;
        if ((int32_t)(lds_read_now(&empty[slot]) - need) < 0) {
          if (pending) {  // publish the previous K-iteration before blocking
            wait_vmcnt<0>();
            lds_signal(&full[pending_slot]);
            pending = false;
          }
          if (!wait_counter(&empty[slot], need, abort_flag, args.spin_limit, args.err)) {
            wait_vmcnt<0>();  // no DMA into LDS may outlive the wave
            return;
          }
        }
      }
      if (args.producer_delay) debug_delay(args.producer_delay);
      compiler_fence();
      WSG_LDS char* a_dst = smem + kHeaderBytes + slot * G::STAGE;
      WSG_LDS char* b_dst = a_dst + G::A_BYTES;
      if constexpr (DO_A) {
        const char* src = (const char*)(a_tile + kk * TK);
#pragma unroll
        for (int n = 0; n < A_PER; ++n)
          __builtin_amdgcn_global_load_lds((const void*)(src + a_goff[n]),
                                           (WSG_LDS void*)(a_dst + (a_rank + n * A_GROUP) * 1024),
                                           16, 0, 0);
      }
      if constexpr (DO_B) {
        const char* src = (const char*)(b_tile + (int64_t)kk * TK * N);
#pragma unroll
        for (int n = 0; n < B_PER; ++n)
          __builtin_amdgcn_global_load_lds((const void*)(src + b_goff[n]),
                                           (WSG_LDS void*)(b_dst + (b_rank + n * B_GROUP) * 1024),
                                           16, 0, 0);
      }
      if (pending) {  // signal(): K-iteration q - 1 has landed
        wait_vmcnt<LOADS>();
        lds_signal(&full[pending_slot]);
      }
      pending = true;
      pending_slot = slot;
    }
  }
  if (pending) {
    wait_vmcnt<0>();
    lds_signal(&full[pending_slot]);
  }
}

template <int TM, int TN, int TK, int NC, int SPLIT, bool BF16>
__device__ __forceinline__ void producer(const KernelArgs& args, WSG_LDS char* smem, int pw,
                                         int lane) {
  using G = Cfg<TM, TN, TK, NC, SPLIT, BF16>;
  if constexpr (SPLIT == 1) {
    producer_loop<TM, TN, TK, NC, SPLIT, BF16, true, true>(args, smem, pw, pw, lane);
  } else {
    if (pw < G::NP / 2)
      producer_loop<TM, TN, TK, NC, SPLIT, BF16, true, false>(args, smem, pw, 0, lane);
    else
      producer_loop<TM, TN, TK, NC, SPLIT, BF16, false, true>(args, smem, 0, pw - G::NP / 2, lane);
  }
}

// ---------------------------------------------------------------------------
// Consumer (MATH wave).  Software-pipelined over MFMA k-steps: operands of
// step s + 1 are read from LDS while the MFMAs of step s run.  The slot of a
// K-iteration is released as soon as its last operands are in registers, and
// the next slot's counter is peeked one k-step early so the wait costs no
// latency when the producers are ahead.
// ---------------------------------------------------------------------------
template <int TM, int TN, int TK, int NC, int SPLIT, bool BF16>
struct ConsumerOps {
  using G = Cfg<TM, TN, TK, NC, SPLIT, BF16>;
  static constexpr int kReads = G::BM + 2 * G::BN;  // LDS reads per k-step
  static constexpr int kMfma = G::BM * G::BN;       // MFMAs per k-step
  // A operand of block mb at k-step s: 16 bytes at a_off[s] + mb * 32 rows.
  // B operand of block nb at k-step s: two transposed 8-byte reads.
  static __device__ __forceinline__ void load(i16x8_t (&fa)[G::BM], i16x8_t (&fb)[G::BN],
                                              WSG_LDS char* a_src, WSG_LDS char* b_src,
                                              uint32_t a_off, uint32_t b_off, int s) {
#pragma unroll
    for (int mb = 0; mb < G::BM; ++mb)
      fa[mb] = *(WSG_LDS i16x8_t*)(a_src + a_off + mb * 32 * TK * 2);
#pragma unroll
    for (int nb = 0; nb < G::BN; ++nb) {
      WSG_LDS char* p = b_src + b_off + ((4 * s) * G::NQ + 2 * nb) * 128;
      const i16x4_t lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((WSG_LDS i16x4_t*)p);
      const i16x4_t hi =
          __builtin_amdgcn_ds_read_tr16_b64_v4i16((WSG_LDS i16x4_t*)(p + G::NQ * 128));
      fb[nb] = __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7);
    }
  }
  static __device__ __forceinline__ void mma(f32x16_t (&acc)[G::BM][G::BN],
                                             const i16x8_t (&fa)[G::BM],
                                             const i16x8_t (&fb)[G::BN]) {
#pragma unroll
    for (int mb = 0; mb < G::BM; ++mb)
#pragma unroll
      for (int nb = 0; nb < G::BN; ++nb)
        acc[mb][nb] = mfma32x32x16<BF16>(fa[mb], fb[nb], acc[mb][nb]);
  }
};

template <int TM, int TN, int TK, int NC, int SPLIT, bool BF16>
__device__ __forceinline__ void consumer(const KernelArgs& args, WSG_LDS char* smem, int cw,
                                         int lane) {
  using G = Cfg<TM, TN, TK, NC, SPLIT, BF16>;
  using Ops = ConsumerOps<TM, TN, TK, NC, SPLIT, BF16>;
  static_assert(G::KS % 2 == 0, "k-steps per K-iteration must be even");
  WSG_LDS uint32_t* full = (WSG_LDS uint32_t*)smem;
  WSG_LDS uint32_t* empty = full + kMaxStages;
  WSG_LDS uint32_t* abort_flag = full + 2 * kMaxStages;

  const int wm = cw / G::WGN, wn = cw % G::WGN;
  // A: lane reads row wm*WM + mb*32 + lane%32, chunk 2s + lane/32 (swizzled;
  // the swizzle depends on row & 15, hence only on the lane).
  uint32_t a_off[G::KS];
  {
    const int r = wm * G::WM + (lane & 31);
#pragma unroll
    for (int s = 0; s < G::KS; ++s)
      a_off[s] = (uint32_t)(r * TK * 2 + (((2 * s + (lane >> 5)) ^ swz_a<TK>(r)) << 4));
  }
  // B: 16-lane group g reads block (kq = 4s + 2(g>>1) + h, nq = (wn*WN + 32 nb)/16 + (g&1)),
  // lane j of the group at byte 8j of the block.
  const int grp = lane >> 4;
  const uint32_t b_off =
      (uint32_t)(((2 * (grp >> 1)) * G::NQ + (wn * G::WN) / 16 + (grp & 1)) * 128 + 8 * (lane & 15));

  const int Gd = gridDim.x;
  const int g0 = first_slot(args);
  if (g0 >= args.num_tiles) return;
  const int my_tiles = (args.num_tiles - g0 + Gd - 1) / Gd;
  const uint32_t S = (uint32_t)args.iters;
  const uint32_t total = (uint32_t)my_tiles * S;
  const uint32_t P = (uint32_t)args.stages;
  const int N = args.N;

  int v = g0;
  int ti, tj;
  tile_coords(v, args.tiles_m, args.tiles_n, args.group_m, &ti, &tj);

  f32x16_t acc[G::BM][G::BN];
#pragma unroll
  for (int mb = 0; mb < G::BM; ++mb)
#pragma unroll
    for (int nb = 0; nb < G::BN; ++nb) acc[mb][nb] = f32x16_t{};

  i16x8_t fa[2][G::BM];
  i16x8_t fb[2][G::BN];

  // Prologue: wait for K-iteration 0 and read its first k-step.
  if (!wait_counter(&full[0], (uint32_t)G::NP, abort_flag, args.spin_limit, args.err)) return;
  Ops::load(fa[0], fb[0], smem + kHeaderBytes, smem + kHeaderBytes + G::A_BYTES, a_off[0], b_off,
            0);

  uint32_t q = 0, kk = 0;
  while (true) {
    const uint32_t slot = q % P;
    WSG_LDS char* a_src = smem + kHeaderBytes + slot * G::STAGE;
    WSG_LDS char* b_src = a_src + G::A_BYTES;
    const bool has_next = (q + 1) < total;
    const uint32_t nslot = (q + 1) % P;
    const uint32_t ntarget = ((q + 1) / P + 1) * (uint32_t)G::NP;
    uint32_t peek = 0;
    if (args.consumer_delay) debug_delay(args.consumer_delay);

    // k-steps 0 .. KS-2: read step s+1, multiply step s.  The scheduling
    // barriers keep each step's MFMAs ahead of the next step's reads.
#pragma unroll
    for (int s = 0; s + 1 < G::KS; ++s) {
      Ops::load(fa[(s + 1) & 1], fb[(s + 1) & 1], a_src, b_src, a_off[s + 1], b_off, s + 1);
      if (s + 2 == G::KS) peek = lds_peek(&full[nslot]);
      Ops::mma(acc, fa[s & 1], fb[s & 1]);
      // issue order inside the step: all LDS reads, then the MFMAs
      if (s + 2 == G::KS)
        __builtin_amdgcn_sched_group_barrier(0x100, Ops::kReads + 1, 0);
      else
        __builtin_amdgcn_sched_group_barrier(0x100, Ops::kReads, 0);
      __builtin_amdgcn_sched_group_barrier(0x008, Ops::kMfma, 0);
      __builtin_amdgcn_sched_barrier(0);
    }
    // signal(): every operand of this K-iteration is in registers.
    lds_signal(&empty[slot]);
    if (has_next) {
      // wait(): the peek was issued one k-step ago; poll only if it was early.
      if ((int32_t)(__builtin_amdgcn_readfirstlane(peek) - ntarget) < 0) {
        if (!wait_counter(&full[nslot], ntarget, abort_flag, args.spin_limit, args.err)) return;
      }
      compiler_fence();
      WSG_LDS char* na = smem + kHeaderBytes + nslot * G::STAGE;
      Ops::load(fa[0], fb[0], na, na + G::A_BYTES, a_off[0], b_off, 0);
    }
    Ops::mma(acc, fa[1], fb[1]);
    __builtin_amdgcn_sched_barrier(0);
    ++q;
    if (++kk == S) {
      // Epilogue: fp32 tile to C.  acc[mb][nb][e] is row 8(e/4) + 4(lane/32) + e%4,
      // column lane%32 of the 32x32 block.  The row pitch is made opaque here
      // so the address arithmetic stays in this block instead of being
      // hoisted (and spilled) out of the K loop.
      uint32_t ldc = (uint32_t)N * 4u;
      asm volatile("" : "+s"(ldc));
      char* cbase = (char*)args.C +
                    (((int64_t)ti * TM + wm * G::WM) * (int64_t)N + (int64_t)tj * TN + wn * G::WN) * 4;
      const uint32_t lane_off = (uint32_t)(4 * (lane >> 5)) * ldc + (uint32_t)(lane & 31) * 4u;
#pragma unroll
      for (int mb = 0; mb < G::BM; ++mb)
#pragma unroll
        for (int e = 0; e < 16; ++e) {
          char* rowp = cbase + (uint32_t)(mb * 32 + 8 * (e >> 2) + (e & 3)) * ldc;
#pragma unroll
          for (int nb = 0; nb < G::BN; ++nb)
            *(float*)(rowp + lane_off + nb * 128) = acc[mb][nb][e];
        }
      if (!has_next) break;
      kk = 0;
      v += Gd;
      tile_coords(v, args.tiles_m, args.tiles_n, args.group_m, &ti, &tj);
#pragma unroll
      for (int mb = 0; mb < G::BM; ++mb)
#pragma unroll
        for (int nb = 0; nb < G::BN; ++nb) acc[mb][nb] = f32x16_t{};
      __builtin_amdgcn_sched_barrier(0);
    }
  }
}

template <int TM, int TN, int TK, int NC, int SPLIT, bool BF16>
__global__ void __launch_bounds__((NC + NC * SPLIT) * 64) ws_gemm_kernel(KernelArgs args) {
  using G = Cfg<TM, TN, TK, NC, SPLIT, BF16>;
  extern __shared__ __attribute__((aligned(1024))) char smem_generic[];
  WSG_LDS char* smem = (WSG_LDS char*)smem_generic;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (threadIdx.x < 2 * kMaxStages + 1) ((WSG_LDS uint32_t*)smem)[threadIdx.x] = 0u;
  __syncthreads();
  if (wave < NC)
    consumer<TM, TN, TK, NC, SPLIT, BF16>(args, smem, wave, lane);
  else
    producer<TM, TN, TK, NC, SPLIT, BF16>(args, smem, wave - NC, lane);
}

}  // namespace wsg
