// Warp-specialised tiled GEMM kernel for gfx950 (MI355X).
//
// C (M x N, fp32) = A (M x K) * B (K x N), A and B fp16 or bf16, all row-major
// (the general variant below also stores alpha A B + beta C as fp32, bf16 or
// fp16, and handles partial edge tiles).
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
//    output block 2 x 2; with NC = 8 (256 x 256 tiles, four producer waves)
//    two per SIMD, 2 x 4.
//  * Producers move a tile in 16-byte chunks, 1 KiB per wave instruction,
//    either staged through VGPRs several K-iterations ahead
//    (buffer_load_dwordx4, then ds_write_b128 once the slot is free; the
//    default) or with buffer_load_dwordx4 ... lds straight into the slot.  The
//    LDS placement of every chunk is fixed by the lane; the layout below is
//    produced by choosing which global chunk each lane fetches.
//  * 1:1 split (NP == NC): every producer loads a share of the A tile and then
//    a share of the B tile, in that order (one DMA warp loading both tiles).
//    2:1 split (NP == 2 NC): the first half of the producers loads A, the
//    second half loads B, concurrently (two DMA warps, one tile each).
//  * Consumers read operands with ds_read_b128 (A, K-contiguous) and
//    ds_read_b64_tr_b16 (B, N-contiguous, transposed by the read) and
//    accumulate with v_mfma_f32_32x32x16_{bf16,f16} in fp32.  In the plain
//    kernels the K loop of a tile is a generated asm block (ws_deep_loop.inc,
//    configurations listed in gen_deep_loop.py): with two consumer waves per
//    SIMD (eight consumer waves, or four at 128 x 128 x 32 with two
//    workgroups per CU) the register-lean roll loop (consumer_roll, also in
//    the event-traced twin), with one the deep-prefetch loop that keeps the
//    reads of the next three k-steps in flight behind the MFMAs
//    (consumer_deep: 1:1 tiles of 64x128 and up at TK = 64 and 128x256x32,
//    2:1 tiles up to 128x128).  The other shapes, the general variant, the
//    traced twins of the deep-prefetch kernels and the 2:1 kernels of the
//    largest four-consumer tiles run compiler-scheduled consumers.
//  * The grid is persistent: at most one workgroup per CU slot, each walking
//    output tiles in dispatch rounds (Section 2.1, "Wave").  The tile order
//    places the tiles that run at the same time on one XCD next to each
//    other so that they share A row panels and B column panels in that XCD's
//    L2.
//  * Variants of one template: the plain GEMM, its event-traced twin, the
//    calibration kernels of the performance model (KernelMode), and the
//    general variant (GENERAL: partial tiles and the alpha / beta epilogue).
//    Slot and counter arithmetic is in ws_ring.hpp.
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

#include "ws_ring.hpp"

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
  void* C;             // fp32, or the general variant's output type
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
  uint32_t* trace;         // event trace (null: off), [trace_wgs][trace_iters][kTraceEvents]
  int32_t trace_wgs;       // workgroups 0 .. trace_wgs-1 are traced
  int32_t trace_iters;     // K-iterations recorded per workgroup
  int32_t load_path;       // producer load path: 0 register-staged, 1 LDS-DMA
  // General variant only: C <- alpha * (A B) + beta * C, C of type out_dtype.
  float alpha, beta;
  int32_t out_dtype;       // OutType
  // Launch clock (null: off): workgroup 0's first wave adds the shader-clock
  // cycles and the 100 MHz reference ticks it spans to clock[0] and clock[1],
  // and 1 to clock[2]; their ratio is the average shader clock of the launch.
  unsigned long long* clock;
};

// Output element type of the general variant's epilogue.
enum OutType { kOutF32 = 0, kOutBF16 = 1, kOutF16 = 2 };

// Event trace: one record of kTraceEvents 32-bit shader-clock stamps per
// K-iteration q of a traced workgroup (the paper's event analysis, Section
// 2.2: S_a(i), S_b(i), S_m(i)).
//   0  producer starts issuing the A tile of q            (S_a)
//   1  producer starts issuing the B tile of q            (S_b)
//   2  the A tile of q has landed in LDS (signal)
//   3  the B tile of q has landed in LDS (signal)
//   4  consumer wave 0 observes slot q full
//   5  consumer wave 0 starts the MFMAs of q              (S_m)
//   6  consumer wave 0 releases slot q
//   7  consumer wave 0 finished the epilogue (last K-iteration of a tile), else 0
constexpr int kTraceEvents = 8;
// LDS header words holding the producer stamps of each slot (indices 24..55).
constexpr int kStampIssueA = 24, kStampIssueB = 32, kStampLandA = 40, kStampLandB = 48;

// Launch clock (KernelArgs::clock), taken by one wave at the start and the
// end of the kernel.  Both counters are read with scalar loads that are
// waited for at once, so nothing of theirs is in flight afterwards.
struct LaunchClock {
  uint64_t c0 = 0, r0 = 0;
  bool on = false;
  __device__ __forceinline__ void start(const KernelArgs& args, int wave) {
    on = args.clock != nullptr && blockIdx.x == 0 && wave == 0;  // wave-uniform
    if (on) {
      c0 = __builtin_amdgcn_s_memtime();
      r0 = __builtin_amdgcn_s_memrealtime();
      asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
    }
  }
  __device__ __forceinline__ void stop(const KernelArgs& args, int lane) {
    if (on) {
      const uint64_t c1 = __builtin_amdgcn_s_memtime();
      const uint64_t r1 = __builtin_amdgcn_s_memrealtime();
      asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
      if (lane == 0) {
        atomicAdd(&args.clock[0], (unsigned long long)(c1 - c0));
        atomicAdd(&args.clock[1], (unsigned long long)(r1 - r0));
        atomicAdd(&args.clock[2], 1ull);
      }
    }
  }
};

// Low 32 bits of the shader-clock counter (s_memtime).
__device__ __forceinline__ uint32_t cycles32() {
  return (uint32_t)__builtin_amdgcn_s_memtime();
}

// XOR swizzle of the 16-byte chunks of A-tile row r.  It depends on r & 31
// only, so rows 32 apart share it and the consumer can fold whole 32-row
// blocks into instruction offsets.  The operand read (lane l: row l & 31,
// chunk l / 32, or that chunk XOR 2 for the next k-step) is free of LDS bank
// conflicts with these choices, as measured with SQ_LDS_BANK_CONFLICT on
// gfx950 at every block and slot base the kernels use; at TK = 32,
// ((r >> 1) ^ (r >> 3)) & 3 and (r >> 1) & 3 cost four conflict cycles per
// read and no swizzle twelve.
template <int TK>
__host__ __device__ constexpr int swz_a(int r) {
  if constexpr (TK == 32) return (r ^ (r >> 2)) & 3;
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

// True when rows r and r + step of an A tile use the same swizzle for every r.
template <int TK>
constexpr bool swz_a_step_invariant(int step) {
  for (int r = 0; r < 64; ++r)
    if (swz_a<TK>(r + step) != swz_a<TK>(r)) return false;
  return true;
}

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
// YOUNGER: how many of this wave's most recent LDS operations may still be
// outstanding (LDS operations of a wave complete in order, so every older
// one has completed).  Scalar-memory loads share the counter and complete
// out of order, but one in flight only makes the wait stricter: the count
// bounds LDS and scalar operations together, so when it is at most YOUNGER
// at most YOUNGER LDS operations are outstanding, and those are the youngest.
template <int YOUNGER = 0>
__device__ __forceinline__ void lds_signal(WSG_LDS uint32_t* p) {
  static_assert(YOUNGER >= 0 && YOUNGER <= 15, "lgkmcnt range");
#if defined(__HIP_DEVICE_COMPILE__)
  const uint32_t addr = (uint32_t)(uintptr_t)p;
  const uint32_t one = 1u;
  uint64_t saved;
  asm volatile(
      "s_waitcnt lgkmcnt(%3)\n\t"
      "s_mov_b64 %0, exec\n\t"
      "s_mov_b64 exec, 1\n\t"
      "ds_add_u32 %1, %2\n\t"
      "s_mov_b64 exec, %0"
      : "=&s"(saved)
      : "v"(addr), "v"(one), "n"(YOUNGER)
      : "memory");
#endif
}

// signal() of the counter at p, together with a read of the counter at
// `peek`: the read goes out before the wait that the signal needs anyway (for
// the wave's own LDS writes), so it costs no LDS round trip of its own.
// Returns the value read (wave-uniform); the counters are monotonic, so a
// value that already satisfies a later wait stays valid.
__device__ __forceinline__ uint32_t lds_signal_peek(WSG_LDS uint32_t* p, WSG_LDS uint32_t* peek) {
#if defined(__HIP_DEVICE_COMPILE__)
  const uint32_t addr = (uint32_t)(uintptr_t)p;
  const uint32_t paddr = (uint32_t)(uintptr_t)peek;
  const uint32_t one = 1u;
  uint64_t saved;
  uint32_t v;
  asm volatile(
      "ds_read_b32 %1, %3\n\t"
      "s_waitcnt lgkmcnt(0)\n\t"
      "s_mov_b64 %0, exec\n\t"
      "s_mov_b64 exec, 1\n\t"
      "ds_add_u32 %2, %4\n\t"
      "s_mov_b64 exec, %0"
      : "=&s"(saved), "=&v"(v)
      : "v"(addr), "v"(paddr), "v"(one)
      : "memory");
  return __builtin_amdgcn_readfirstlane(v);
#else
  *p += 1;
  return *peek;
#endif
}

// signal() when `enable` (wave-uniform) is non-zero, as one asm block, so
// the caller's control flow gets no join.
template <int YOUNGER = 0>
__device__ __forceinline__ void lds_signal_if(WSG_LDS uint32_t* p, uint32_t enable) {
  static_assert(YOUNGER >= 0 && YOUNGER <= 15, "lgkmcnt range");
#if defined(__HIP_DEVICE_COMPILE__)
  const uint32_t addr = (uint32_t)(uintptr_t)p;
  const uint32_t one = 1u;
  uint64_t saved;
  asm volatile(
      "s_cmp_eq_u32 %4, 0\n\t"
      "s_cbranch_scc1 1f\n\t"
      "s_waitcnt lgkmcnt(%3)\n\t"
      "s_mov_b64 %0, exec\n\t"
      "s_mov_b64 exec, 1\n\t"
      "ds_add_u32 %1, %2\n\t"
      "s_mov_b64 exec, %0\n"
      "1:"
      : "=&s"(saved)
      : "v"(addr), "v"(one), "n"(YOUNGER), "s"(__builtin_amdgcn_readfirstlane(enable))
      : "memory", "scc");
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

// Store a wave-uniform value to an LDS word from lane 0 (asm, so the producer's
// vmcnt accounting and the compiler's LDS ordering are untouched).
__device__ __forceinline__ void lds_stamp(WSG_LDS uint32_t* p, uint32_t value) {
#if defined(__HIP_DEVICE_COMPILE__)
  const uint32_t addr = (uint32_t)(uintptr_t)p;
  uint64_t saved;
  asm volatile(
      "s_mov_b64 %0, exec\n\t"
      "s_mov_b64 exec, 1\n\t"
      "ds_write_b32 %1, %2\n\t"
      "s_mov_b64 exec, %0"
      : "=&s"(saved)
      : "v"(addr), "v"(value)
      : "memory");
#endif
}

// wait(): poll *ctr until it reaches target (wrap-safe).  Returns true when
// it did; false when the workgroup aborted or this wait exceeded the poll
// limit (it then raises the workgroup abort flag and the device error word,
// so every wave drains quickly).  The result is wave-uniform.  The poll loop
// itself issues no vector-memory instruction, so it does not disturb the
// compiler's accounting of outstanding loads around it.
__device__ __forceinline__ void report_timeout(WSG_LDS uint32_t* abort_flag, int32_t* err) {
  if ((threadIdx.x & 63) == 0) {
    __hip_atomic_store(abort_flag, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
    __hip_atomic_fetch_or(err, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  }
}

__device__ __forceinline__ bool wait_counter(WSG_LDS uint32_t* ctr, uint32_t target,
                                             WSG_LDS uint32_t* abort_flag, int spin_limit,
                                             int32_t* err) {
  int spins = 0;
  int status = 0;  // 0 reached, 1 aborted elsewhere, 2 timed out here
  while (true) {
    const uint32_t v = lds_read_now(ctr);
    if ((int32_t)(v - target) >= 0) break;
    if (lds_read_now(abort_flag)) {
      status = 1;
      break;
    }
    if (++spins > spin_limit) {
      status = 2;
      break;
    }
    __builtin_amdgcn_s_sleep(1);
  }
  compiler_fence();
  status = __builtin_amdgcn_readfirstlane(status);
  if (status == 2) report_timeout(abort_flag, err);
  return status == 0;
}

// The same wait as one asm block, so that it adds no join to the caller's
// control flow (the consumer's K loop stays a single basic block and its
// operand registers are not shuffled around a join).  `seen` is a value of
// *ctr read earlier: when it already satisfies the target, nothing is read.
// Returns 0 when the counter reached the target, 1 when the workgroup abort
// flag is up, 2 after `limit` polls; wave-uniform.
__device__ __forceinline__ uint32_t wait_until(uint32_t seen, WSG_LDS uint32_t* ctr,
                                               WSG_LDS uint32_t* abort_flag, uint32_t target,
                                               int32_t limit, uint32_t enable = 1) {
#if defined(__HIP_DEVICE_COMPILE__)
  const uint32_t ca = (uint32_t)(uintptr_t)ctr, aa = (uint32_t)(uintptr_t)abort_flag;
  uint32_t st, spins, v0, v1;
  asm volatile(
      "s_mov_b32 %[st], 0\n\t"
      "s_cmp_eq_u32 %[en], 0\n\t"
      "s_cbranch_scc1 2f\n\t"
      "v_readfirstlane_b32 %[st], %[seen]\n\t"
      "s_sub_u32 %[st], %[st], %[target]\n\t"
      "s_cmp_ge_i32 %[st], 0\n\t"
      "s_mov_b32 %[st], 0\n\t"
      "s_cbranch_scc1 2f\n\t"
      "s_mov_b32 %[spins], 0\n"
      "1:\n\t"
      "ds_read_b32 %[v0], %[ca]\n\t"
      "ds_read_b32 %[v1], %[aa]\n\t"
      "s_waitcnt lgkmcnt(0)\n\t"
      "v_readfirstlane_b32 %[st], %[v0]\n\t"
      "s_sub_u32 %[st], %[st], %[target]\n\t"
      "s_cmp_ge_i32 %[st], 0\n\t"
      "s_mov_b32 %[st], 0\n\t"
      "s_cbranch_scc1 2f\n\t"
      "v_readfirstlane_b32 %[st], %[v1]\n\t"
      "s_cmp_lg_u32 %[st], 0\n\t"
      "s_mov_b32 %[st], 1\n\t"
      "s_cbranch_scc1 2f\n\t"
      "s_add_u32 %[spins], %[spins], 1\n\t"
      "s_cmp_gt_i32 %[spins], %[limit]\n\t"
      "s_mov_b32 %[st], 2\n\t"
      "s_cbranch_scc1 2f\n\t"
      "s_sleep 1\n\t"
      "s_branch 1b\n"
      "2:"
      : [st] "=&s"(st), [spins] "=&s"(spins), [v0] "=&v"(v0), [v1] "=&v"(v1)
      : [seen] "v"(seen), [target] "s"(__builtin_amdgcn_readfirstlane(target)), [ca] "v"(ca),
        [aa] "v"(aa), [limit] "s"(limit), [en] "s"(__builtin_amdgcn_readfirstlane(enable))
      : "memory", "scc");
  return st;
#else
  if (!enable) return 0u;
  return (int32_t)(*ctr - target) >= 0 ? 0u : (*abort_flag ? 1u : 2u);
#endif
}

// Test hook: n bursts of ~8k-cycle sleeps (n wave-uniform; 0 in production),
// as one asm block so that the caller's loop gets no join.
__device__ __forceinline__ void debug_delay(int n) {
#if defined(__HIP_DEVICE_COMPILE__)
  uint32_t left;
  asm volatile(
      "s_mov_b32 %0, %1\n\t"
      "s_cmp_le_i32 %0, 0\n\t"
      "s_cbranch_scc1 2f\n"
      "1:\n\t"
      "s_sleep 127\n\t"
      "s_sub_u32 %0, %0, 1\n\t"
      "s_cmp_lg_u32 %0, 0\n\t"
      "s_cbranch_scc1 1b\n"
      "2:"
      : "=&s"(left)
      : "s"(__builtin_amdgcn_readfirstlane(n))
      : "scc");
#else
  (void)n;
#endif
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

template <int TM, int TN, int TK, int NC, int NPW, int SPLIT, bool BF16>
struct Cfg {
  static constexpr int NP = NPW;                     // producer waves
  static constexpr int NW = NC + NP;                 // waves per workgroup
  static constexpr int WGM = (NC >= 4) ? 2 : 1;      // consumer grid rows
  static constexpr int WGN = (NC == 8) ? 4 : (NC == 4) ? 2 : 1;  // consumer grid cols
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
  static_assert(NC == 1 || NC == 4 || NC == 8, "consumer waves must be 1, 4 or 8");
  static_assert(SPLIT == 1 || SPLIT == 2, "split must be 1:1 or 2:1");
  // producer waves: one group of NC (1:1) or two of NC (2:1); with NC = 4 also
  // two groups of 2 (2:1 at eight waves); with NC = 8 one group of 4 (1:1) or
  // two of 2 (2:1), twelve waves in all.
  static_assert((NP == NC * SPLIT && NC != 8) || (NC == 4 && NP == 4) || (NC == 8 && NP == 4),
                "unsupported producer / consumer arrangement");
  static_assert(SPLIT == 1 || NP % 2 == 0, "two producer groups need an even number of waves");
  static_assert(WM % 32 == 0 && WN % 32 == 0, "wave tile must be a multiple of 32x32");
  static_assert(TK == 32 || TK == 64 || TK == 128, "TK must be 32, 64 or 128");
  static_assert(A_BYTES % 1024 == 0 && B_BYTES % 1024 == 0, "tiles must be whole KiB");
};

// What a kernel instance runs.  kModeGemm is the GEMM; the others are the
// calibration kernels of the paper's evaluation (Section 4.2), built from the
// same code so that they measure this kernel's own costs:
//   kModeLoadA / kModeLoadB  the producers load only the A (B) tiles of every
//                            K-iteration; the consumers take each slot and
//                            release it without reading it; C is not written.
//   kModeMath                the producers release slots without loading; the
//                            consumers read and multiply whatever the slots
//                            hold; C is not written.
//   kModeEpilogue            no K loop: the consumers store one zero tile per
//                            output tile, the producers exit.
//   kModeLoadAB              the producers load both tiles as in the GEMM; the
//                            consumers release every slot unread.
enum KernelMode {
  kModeGemm = 0, kModeLoadA = 1, kModeLoadB = 2, kModeMath = 3, kModeEpilogue = 4, kModeLoadAB = 5
};

typedef __attribute__((ext_vector_type(4))) int i32x4_t;

// Producer loads and the epilogue's stores go through a raw buffer resource
// over a tile panel: the base sits in SGPRs and each lane adds a 32-bit byte
// offset (panel offsets stay below 2^31, checked by the plan), so an access
// needs no 64-bit address arithmetic on the vector ALU of a SIMD whose other
// waves issue MFMAs.  Word 3 of the descriptor: data format
// 32 bits (field at bits 15-18 = 4), every other field zero (no swizzle, no
// index stride); the record count is the largest, so no offset is clipped.
constexpr int kRawBufferWord3 = 0x00020000;
__device__ __forceinline__ __amdgpu_buffer_rsrc_t panel_rsrc(const void* base) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, -1, kRawBufferWord3);
}
// Cache-policy operand of the raw buffer builtins that marks an access
// non-temporal (the `nt` bit).
constexpr int kBufferNonTemporal = 2;
__device__ __forceinline__ i32x4_t panel_load16(__amdgpu_buffer_rsrc_t r, uint32_t byte_off) {
  return __builtin_bit_cast(i32x4_t, __builtin_amdgcn_raw_buffer_load_b128(r, (int)byte_off, 0, 0));
}
// The general variant's producers read through resources whose record count
// ends at the end of the matrix (at most 2^31 bytes: the plan keeps panel
// offsets under 2^31).  A chunk outside A or B lies past the record count or
// is read from offset kOutsidePanel = 2^31; the range check of a raw buffer
// load returns zeros for it without touching memory.
constexpr uint32_t kOutsidePanel = 0x80000000u;
// Record count: the bytes from the panel base to the end of the matrix, at
// most 2^31; a row-major panel's rows past the matrix's last row read as
// zeros.
__device__ __forceinline__ __amdgpu_buffer_rsrc_t panel_rsrc_to_end(const void* base, int64_t bytes_left) {
  const uint32_t n = bytes_left < (int64_t)kOutsidePanel ? (uint32_t)bytes_left : kOutsidePanel;
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, (int)n, kRawBufferWord3);
}
// 16 bytes per lane straight into LDS: lane l's bytes land at dst + 16 l.
__device__ __forceinline__ void panel_load16_lds(__amdgpu_buffer_rsrc_t r, WSG_LDS void* dst, uint32_t byte_off) {
  __builtin_amdgcn_raw_ptr_buffer_load_lds(r, dst, 16, byte_off, 0, 0, 0);
}
// Epilogue: the fp32 tile of consumer wave (wm, wn) to C.  acc[mb][nb][e] is
// row 8(e/4) + 4(lane/32) + e%4, column lane%32 of the 32x32 block.  The row
// pitch is made opaque so that the address arithmetic stays here instead of
// being hoisted (and spilled) out of the caller's K loop.
//
// GENERAL: elements outside C (partial edge tiles) are not stored, and the
// epilogue is the BLAS one, C <- alpha * (A B) + beta * C, rounded once to
// the output type (round to nearest even); beta == 0 does not read C.
template <typename T>
__device__ __forceinline__ float load_out(const T* p) {
  return (float)*p;
}
// One specialisation per output type T, READ_C (beta != 0) and MASK (the
// wave tile crosses an edge of C).  The old C of EG consecutive k-step rows
// is loaded before any of them is stored, so those loads overlap.
template <int TM, int TN, int WM, int WN, int BM, int BN, int EG, typename T, bool READ_C, bool MASK>
__device__ __forceinline__ void store_tile_general(const KernelArgs& args,
                                                   const f32x16_t (&acc)[BM][BN], int ti, int tj,
                                                   int wm, int wn, int lane) {
  static_assert(16 % EG == 0, "row groups split the 16 accumulator rows");
  constexpr uint32_t ES = sizeof(T);
  const float alpha = args.alpha, beta = args.beta;
  uint32_t ldc = (uint32_t)args.N * ES;
  asm volatile("" : "+s"(ldc));
  // Lane-derived offsets are computed here, not hoisted into the caller's
  // prologue and kept (or spilled) across its K loop.
  asm volatile("" : "+v"(lane));
  const int r0 = ti * TM + wm * WM, c0 = tj * TN + wn * WN;
  char* cbase = (char*)args.C + ((int64_t)r0 * args.N + c0) * ES;
  const uint32_t lane_off = (uint32_t)(4 * (lane >> 5)) * ldc + (uint32_t)(lane & 31) * ES;
  // rows / columns of C left from this lane's first element
  const int rows_left = args.M - r0 - 4 * (lane >> 5);
  const int cols_left = args.N - c0 - (lane & 31);
#pragma unroll
  for (int mb = 0; mb < BM; ++mb)
#pragma unroll
    for (int e0 = 0; e0 < 16; e0 += EG) {
      float old[EG][BN];
      if constexpr (READ_C) {
#pragma unroll
        for (int i = 0; i < EG; ++i) {
          const int e = e0 + i, dr = mb * 32 + 8 * (e >> 2) + (e & 3);
#pragma unroll
          for (int nb = 0; nb < BN; ++nb) {
            old[i][nb] = 0.0f;
            if (!MASK || (dr < rows_left && nb * 32 < cols_left))
              old[i][nb] = load_out((const T*)(cbase + (uint32_t)dr * ldc + lane_off + nb * 32 * ES));
          }
        }
      }
#pragma unroll
      for (int i = 0; i < EG; ++i) {
        const int e = e0 + i, dr = mb * 32 + 8 * (e >> 2) + (e & 3);
#pragma unroll
        for (int nb = 0; nb < BN; ++nb) {
          if (!MASK || (dr < rows_left && nb * 32 < cols_left)) {
            float v = alpha * acc[mb][nb][e];
            if constexpr (READ_C) v = __builtin_fmaf(beta, old[i][nb], v);
            *(T*)(cbase + (uint32_t)dr * ldc + lane_off + nb * 32 * ES) = (T)v;
          }
        }
      }
    }
}

template <int TM, int TN, int WM, int WN, int BM, int BN, int EG, typename T>
__device__ __forceinline__ void store_tile_general_t(const KernelArgs& args,
                                                     const f32x16_t (&acc)[BM][BN], int ti, int tj,
                                                     int wm, int wn, int lane) {
  const bool read_c = args.beta != 0.0f;
  const bool mask = ti * TM + wm * WM + WM > args.M || tj * TN + wn * WN + WN > args.N;
  if (read_c) {
    if (mask)
      store_tile_general<TM, TN, WM, WN, BM, BN, EG, T, true, true>(args, acc, ti, tj, wm, wn, lane);
    else
      store_tile_general<TM, TN, WM, WN, BM, BN, EG, T, true, false>(args, acc, ti, tj, wm, wn, lane);
  } else {
    if (mask)
      store_tile_general<TM, TN, WM, WN, BM, BN, EG, T, false, true>(args, acc, ti, tj, wm, wn, lane);
    else
      store_tile_general<TM, TN, WM, WN, BM, BN, EG, T, false, false>(args, acc, ti, tj, wm, wn, lane);
  }
}

// EG: k-step rows whose old C values are loaded together by the general
// epilogue (fewer when registers are tight).
template <int TM, int TN, int WM, int WN, int BM, int BN, bool GENERAL = false, int EG = 16>
__device__ __forceinline__ void store_tile(const KernelArgs& args, const f32x16_t (&acc)[BM][BN],
                                           int ti, int tj, int wm, int wn, int lane) {
  if constexpr (GENERAL) {
    const int od = __builtin_amdgcn_readfirstlane(args.out_dtype);
    if (od == kOutBF16)
      store_tile_general_t<TM, TN, WM, WN, BM, BN, EG, __bf16>(args, acc, ti, tj, wm, wn, lane);
    else if (od == kOutF16)
      store_tile_general_t<TM, TN, WM, WN, BM, BN, EG, _Float16>(args, acc, ti, tj, wm, wn, lane);
    else
      store_tile_general_t<TM, TN, WM, WN, BM, BN, EG, float>(args, acc, ti, tj, wm, wn, lane);
  } else {
    uint32_t ldc = (uint32_t)args.N * 4u;
    asm volatile("" : "+s"(ldc));
    const char* cbase = (const char*)args.C +
                        (((int64_t)ti * TM + wm * WM) * (int64_t)args.N + (int64_t)tj * TN + wn * WN) * 4;
    // the wave tile's rows lie below T_M * N * 4 < 2^31 bytes from cbase
    const __amdgpu_buffer_rsrc_t crs = panel_rsrc(cbase);
    const uint32_t lane_off = (uint32_t)(4 * (lane >> 5)) * ldc + (uint32_t)(lane & 31) * 4u;
#pragma unroll
    for (int mb = 0; mb < BM; ++mb)
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        const uint32_t row_off = (uint32_t)(mb * 32 + 8 * (e >> 2) + (e & 3)) * ldc;  // wave-uniform
#pragma unroll
        for (int nb = 0; nb < BN; ++nb) {  // non-temporal: C is not read again here, the panels are
          // copy the element out first: a bit cast of a vector element lvalue reads element 0
          const float v = acc[mb][nb][e];
          __builtin_amdgcn_raw_buffer_store_b32(__builtin_bit_cast(uint32_t, v), crs, (int)(lane_off + nb * 128),
                                                (int)row_off, kBufferNonTemporal);
        }
      }
  }
}

// ---------------------------------------------------------------------------
// Per-workgroup tile sequence (identical in both roles).
// ---------------------------------------------------------------------------
__device__ __forceinline__ int first_slot(const KernelArgs& args) {
  const int G = gridDim.x;
  return args.xcd_remap ? xcd_slot(blockIdx.x, G) : (int)blockIdx.x;
}

// Events of one kind that a producer wave stores into its workgroup's trace
// record, batched: lane k of `vals` holds the event of K-iteration base + k
// (events arrive for consecutive K-iterations), and 64 of them go out in one
// store.  A store sits in the same vector-memory counter as the loads the
// wave waits for before it writes a slot, so one store per K-iteration would
// hold every slot back behind its write acknowledgement.
struct StampBatch {
  uint32_t vals = 0;
  uint32_t base = 0, n = 0;
};
// Adds the event of K-iteration iq; true when the batch is full.
__device__ __forceinline__ bool stamp_put(StampBatch& b, uint32_t iq, uint32_t value, int lane) {
  if (b.n == 0) b.base = iq;
  b.vals = ((uint32_t)lane == b.n) ? value : b.vals;
  return ++b.n == 64;
}
__device__ __forceinline__ void stamp_store(const StampBatch& b, __amdgpu_buffer_rsrc_t rec, int ev,
                                            uint32_t limit, int lane) {
  const uint32_t iq = b.base + (uint32_t)lane;
  if ((uint32_t)lane < b.n && iq < limit)
    __builtin_amdgcn_raw_buffer_store_b32(b.vals, rec, (int)((iq * kTraceEvents + (uint32_t)ev) * 4u), 0, 0);
}

// Events 0-3 of a producer wave (issue of its A / B loads of K-iteration q,
// their landing in the slot); A and B share one clock reading each.  With
// DIRECT (the eight-consumer arrangement, whose consumer does not copy stamps
// out of the LDS header) they go straight into the workgroup's trace record,
// batched; otherwise into the LDS header for consumer wave 0 to copy.
template <bool DIRECT>
struct ProducerStamps {
  // Bit 0: this wave stamps the A events, bit 1: the B events.  Kept as a
  // scalar integer, not as bools (those would be materialised as lane masks
  // through vector instructions).
  uint32_t who;
  int lane;
  uint32_t limit;
  __amdgpu_buffer_rsrc_t rec;
  StampBatch iss, land;
  __device__ ProducerStamps(const KernelArgs& args, bool stamps_a, bool stamps_b, int lane_)
      : who(__builtin_amdgcn_readfirstlane((stamps_a ? 1u : 0u) | (stamps_b ? 2u : 0u))), lane(lane_),
        limit(DIRECT ? (uint32_t)args.trace_iters : 0u),
        rec(panel_rsrc(DIRECT ? args.trace + (size_t)blockIdx.x * args.trace_iters * kTraceEvents : nullptr)) {}
  __device__ void flush(StampBatch& b, int ev_a, int ev_b) {
    if (who & 1u) stamp_store(b, rec, ev_a, limit, lane);
    if (who & 2u) stamp_store(b, rec, ev_b, limit, lane);
    b.n = 0;
  }
  __device__ void put(StampBatch& b, int ev_a, int ev_b, uint32_t q, uint32_t t, WSG_LDS uint32_t* hdr_a,
                      WSG_LDS uint32_t* hdr_b) {
    if constexpr (DIRECT) {
      if (who != 0u && stamp_put(b, q, t, lane)) flush(b, ev_a, ev_b);
    } else {
      if (who & 1u) lds_stamp(hdr_a, t);
      if (who & 2u) lds_stamp(hdr_b, t);
    }
  }
  __device__ void issued(uint32_t q, uint32_t t, WSG_LDS uint32_t* hdr_a, WSG_LDS uint32_t* hdr_b) {
    put(iss, 0, 1, q, t, hdr_a, hdr_b);
  }
  __device__ void landed(uint32_t q, uint32_t t, WSG_LDS uint32_t* hdr_a, WSG_LDS uint32_t* hdr_b) {
    put(land, 2, 3, q, t, hdr_a, hdr_b);
  }
  __device__ void finish() {
    if constexpr (DIRECT) {
      flush(iss, 0, 1);
      flush(land, 2, 3);
    }
  }
};

// A traced kernel runs its producer loop's traced instance only in the
// workgroups that record events; the others run the plain instance.
__device__ __forceinline__ bool traced_workgroup(const KernelArgs& args) {
  return args.trace != nullptr && (int)blockIdx.x < args.trace_wgs;
}

// ---------------------------------------------------------------------------
// Producer (DMA warp).  Waits for a free slot, streams its share of the A
// and/or B tile of one K-iteration into that slot, and signals the slot full
// once the data has landed.  Up to `lag` + 1 K-iterations are in flight per
// wave: iteration q is signalled once iteration q + lag has been issued.
// Before blocking on a slot that is still in use, every pending iteration is
// published (oldest first), so a consumer never waits on data that landed.
// ---------------------------------------------------------------------------

// Block until at most n of this wave's most recent K-iterations (LOADS DMA
// instructions each) are still in flight.
template <int LOADS>
__device__ __forceinline__ void wait_landed(uint32_t n) {
  switch (n) {
    case 0: wait_vmcnt<0>(); break;
    case 1: wait_vmcnt<(LOADS * 1 <= 63 ? LOADS * 1 : 0)>(); break;
    case 2: wait_vmcnt<(LOADS * 2 <= 63 ? LOADS * 2 : 0)>(); break;
    case 3: wait_vmcnt<(LOADS * 3 <= 63 ? LOADS * 3 : 0)>(); break;
    case 4: wait_vmcnt<(LOADS * 4 <= 63 ? LOADS * 4 : 0)>(); break;
    case 5: wait_vmcnt<(LOADS * 5 <= 63 ? LOADS * 5 : 0)>(); break;
    default: wait_vmcnt<(LOADS * 6 <= 63 ? LOADS * 6 : 0)>(); break;
  }
}

template <int TM, int TN, int TK, int NC, int NPW, int SPLIT, bool BF16, bool TRACE, bool DO_A, bool DO_B>
__device__ __forceinline__ void producer_loop(const KernelArgs& args, WSG_LDS char* smem,
                                              int a_rank, int b_rank, int lane) {
  using G = Cfg<TM, TN, TK, NC, NPW, SPLIT, BF16>;
  constexpr int A_GROUP = (SPLIT == 1) ? G::NP : G::NP / 2;  // waves sharing the A tile
  constexpr int B_GROUP = (SPLIT == 1) ? G::NP : G::NP / 2;
  constexpr int A_PER = DO_A ? G::A_INSTR / A_GROUP : 0;     // DMA instructions per wave
  constexpr int B_PER = DO_B ? G::B_INSTR / B_GROUP : 0;
  constexpr int LOADS = A_PER + B_PER;
  constexpr int MAX_LAG = (63 / LOADS) < 6 ? (63 / LOADS) : 6;
  static_assert(G::A_INSTR % A_GROUP == 0 && G::B_INSTR % B_GROUP == 0, "even DMA split");
  static_assert(LOADS > 0 && MAX_LAG >= 1, "vmcnt range");

  WSG_LDS uint32_t* full = (WSG_LDS uint32_t*)smem;
  WSG_LDS uint32_t* empty = full + kMaxStages;
  WSG_LDS uint32_t* abort_flag = full + 2 * kMaxStages;
  const int K = args.K, N = args.N;

  // Byte offset, inside the tile, of the 16-byte chunk this lane fetches for
  // each of its DMA instructions (the LDS side is fixed: lane l writes bytes
  // 16 l .. 16 l + 15 of the instruction's KiB).
  uint32_t a_goff[A_PER > 0 ? A_PER : 1];
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

  // TRACE: this instance runs only in workgroups that record events.
  constexpr bool tracing = TRACE;
  ProducerStamps<TRACE && NC == 8> stamps(args, DO_A && a_rank == 0, DO_B && b_rank == 0, lane);
  // signal(): data of the slot has landed; stamp its landing time first when tracing.
  auto publish = [&](uint32_t pq) {
    const uint32_t pslot = ring_slot(pq, (uint32_t)args.stages);
    if constexpr (tracing) stamps.landed(pq, cycles32(), &full[kStampLandA + pslot], &full[kStampLandB + pslot]);
    lds_signal(&full[pslot]);
  };
  const int Gd = gridDim.x;
  const uint32_t P = (uint32_t)args.stages;
  uint32_t lag = P > 3 ? P - 2 : 1;
  if (lag > (uint32_t)MAX_LAG) lag = MAX_LAG;
  uint32_t q = 0;      // next K-iteration to issue
  uint32_t q_sig = 0;  // next K-iteration to signal
  for (int v = first_slot(args); v < args.num_tiles; v += Gd) {
    int ti, tj;
    tile_coords(v, args.tiles_m, args.tiles_n, args.group_m, &ti, &tj);
    const uint16_t* a_tile = args.A + (int64_t)ti * TM * K;
    const uint16_t* b_tile = args.B + (int64_t)tj * TN;
    for (int kk = 0; kk < args.iters; ++kk, ++q) {
      const uint32_t slot = ring_slot(q, P);
      if (ring_use(q, P) > 0) {
        // wait(): the slot is free once every consumer wave released its previous use.
        const uint32_t need = ring_empty_target(q, P, NC);
        if ((int32_t)(lds_read_now(&empty[slot]) - need) < 0) {
          while (q_sig < q) {  // publish pending iterations first, oldest first
            wait_landed<LOADS>(q - q_sig - 1);
            publish(q_sig);
            ++q_sig;
          }
          if (!wait_counter(&empty[slot], need, abort_flag, args.spin_limit, args.err)) {
            wait_vmcnt<0>();  // no DMA into LDS may outlive the wave
            return;
          }
        }
      }
      debug_delay(args.producer_delay);
      compiler_fence();
      if constexpr (tracing) stamps.issued(q, cycles32(), &full[kStampIssueA + slot], &full[kStampIssueB + slot]);
      WSG_LDS char* a_dst = smem + kHeaderBytes + slot * G::STAGE;
      WSG_LDS char* b_dst = a_dst + G::A_BYTES;
      if constexpr (DO_A) {
        const __amdgpu_buffer_rsrc_t src = panel_rsrc(a_tile + kk * TK);
#pragma unroll
        for (int n = 0; n < A_PER; ++n)
          panel_load16_lds(src, (WSG_LDS void*)(a_dst + (a_rank + n * A_GROUP) * 1024), a_goff[n]);
      }
      if constexpr (DO_B) {
        const __amdgpu_buffer_rsrc_t src = panel_rsrc(b_tile + (int64_t)kk * TK * N);
#pragma unroll
        for (int n = 0; n < B_PER; ++n)
          panel_load16_lds(src, (WSG_LDS void*)(b_dst + (b_rank + n * B_GROUP) * 1024), b_goff[n]);
      }
      // signal(): iteration q - lag has landed once at most `lag` newer ones are in flight.
      if (q + 1 - q_sig > lag) {
        wait_landed<LOADS>(lag);
        publish(q_sig);
        ++q_sig;
      }
    }
  }
  while (q_sig < q) {
    wait_landed<LOADS>(q - q_sig - 1);
    publish(q_sig);
    ++q_sig;
  }
  stamps.finish();
}

// ---------------------------------------------------------------------------
// Register-staged producer (DMA warp).  The wave loads its share of the tiles
// of K-iteration q + L into VGPRs (buffer_load_dwordx4) while K-iteration q
// waits in registers for its slot; once the slot is free it writes q with
// ds_write_b128 and signals.  Bytes in flight per wave are L iterations'
// worth, independent of the LDS ring depth: producer waves get the kernel's
// full VGPR allocation (sized for the consumers) and would otherwise leave
// it idle.  The LDS layout is the one the LDS-DMA producer writes.
// ---------------------------------------------------------------------------
template <int TM, int TN, int TK, int NC, int NPW, int SPLIT, bool BF16, bool TRACE, bool DO_A, bool DO_B,
          bool GENERAL>
__device__ __forceinline__ void producer_loop_reg(const KernelArgs& args, WSG_LDS char* smem,
                                                  int a_rank, int b_rank, int lane) {
  using G = Cfg<TM, TN, TK, NC, NPW, SPLIT, BF16>;
  constexpr int A_GROUP = (SPLIT == 1) ? G::NP : G::NP / 2;
  constexpr int B_GROUP = (SPLIT == 1) ? G::NP : G::NP / 2;
  constexpr int A_PER = DO_A ? G::A_INSTR / A_GROUP : 0;
  constexpr int B_PER = DO_B ? G::B_INSTR / B_GROUP : 0;
  constexpr int LOADS = A_PER + B_PER;
  // VGPRs for staged tiles: what the consumers' allocation leaves (256 a wave
  // with eight waves, 168 with twelve; the 128 x 128 x 32 kernel held to 128
  // registers stages its cap of six K-iterations in 96)
  constexpr int STAGE_VGPRS = (G::NW <= 8) ? 152 : (NC == 8 ? 128 : 96);
  constexpr int L0 = STAGE_VGPRS / (4 * LOADS);
  constexpr int L1 = (63 / LOADS) < L0 ? (63 / LOADS) : L0;
  constexpr int L = L1 < 1 ? 1 : (L1 > 6 ? 6 : L1);  // K-iterations staged in VGPRs
  static_assert(G::A_INSTR % A_GROUP == 0 && G::B_INSTR % B_GROUP == 0, "even split");

  WSG_LDS uint32_t* full = (WSG_LDS uint32_t*)smem;
  WSG_LDS uint32_t* empty = full + kMaxStages;
  WSG_LDS uint32_t* abort_flag = full + 2 * kMaxStages;
  const int K = args.K, N = args.N;

  uint32_t goff[LOADS];  // byte offset of this lane's 16-byte chunk in the A / B tile
#pragma unroll
  for (int n = 0; n < A_PER; ++n) {
    const int q = (a_rank + n * A_GROUP) * 64 + lane;
    const int r = q / G::CA, p = q % G::CA;
    goff[n] = (uint32_t)(r * K + 8 * (p ^ swz_a<TK>(r))) * 2u;
  }
#pragma unroll
  for (int n = 0; n < B_PER; ++n) {
    const int q = (b_rank + n * B_GROUP) * 64 + lane;
    const int blk = q >> 3, w = q & 7;
    const int kq = blk / G::NQ, nq = blk % G::NQ;
    goff[A_PER + n] = (uint32_t)((kq * 4 + (w >> 1)) * N + nq * 16 + (w & 1) * 8) * 2u;
  }
  // The general variant needs registers for its edge tests: where a wave's
  // successive A (B) instructions lie a whole number of swizzle periods
  // (block rows) apart, it keeps only the first instruction's offset and
  // adds the (wave-uniform) step between instructions.
  constexpr int A_STEP = (64 / G::CA) * A_GROUP;  // A rows from one of a wave's instructions to the next
  constexpr bool kStrided = GENERAL && swz_a_step_invariant<TK>(A_STEP) && (8 * B_GROUP) % G::NQ == 0;
  constexpr int B_STEP = (8 * B_GROUP) / G::NQ;   // B block rows (4 K rows each) between instructions
  const uint32_t a_step = (uint32_t)A_STEP * (uint32_t)K * 2u;      // bytes, wave-uniform
  const uint32_t b_step = (uint32_t)(B_STEP * 4) * (uint32_t)N * 2u;
  // kStrided: the lane's K chunk of A and column chunk of B (the same for
  // all of its instructions)
  int a_kc0 = 0, b_nc0 = 0;
  if constexpr (kStrided) {
    const int qa = a_rank * 64 + lane;
    a_kc0 = 8 * ((qa % G::CA) ^ swz_a<TK>(qa / G::CA));
    const int qb = b_rank * 64 + lane;
    b_nc0 = ((qb >> 3) % G::NQ) * 16 + (qb & 1) * 8;
  }
  const uint32_t lane16 = (uint32_t)lane * 16u;

  // TRACE: this instance runs only in workgroups that record events.
  constexpr bool tracing = TRACE;
  ProducerStamps<TRACE && NC == 8> stamps(args, DO_A && a_rank == 0, DO_B && b_rank == 0, lane);
  const int Gd = gridDim.x;
  const int g0 = first_slot(args);
  const int my_tiles = (args.num_tiles - g0 + Gd - 1) / Gd;
  const uint32_t S = (uint32_t)args.iters;
  const uint32_t total = (uint32_t)my_tiles * S;
  const uint32_t P = (uint32_t)args.stages;

  // Issue cursor: the next K-iteration whose loads go out.
  int v_i = g0, ti_i = 0, tj_i = 0;
  uint32_t kk_i = 0, q_iss = 0;
  tile_coords(v_i, args.tiles_m, args.tiles_n, args.group_m, &ti_i, &tj_i);

  i32x4_t stage[L][LOADS];
  // Traced: one clock reading per K-iteration, taken once K-iteration q is in
  // its slot, stands for the landing of q and the issue of q + L (the loads
  // go out right after q's signal).
  uint32_t t_issue[L], t_now = 0;
  // Loads go out unconditionally (past the last K-iteration they re-read the
  // last valid tile and are never written to LDS), so every path through the
  // loop has the same number of loads in flight and the compiler's vmcnt
  // waits before each ds_write allow exactly L - 1 newer iterations.
  auto issue = [&](int u) {
    if constexpr (tracing) t_issue[u] = t_now;
    const char* a_src = (const char*)(args.A + (int64_t)ti_i * TM * K + kk_i * TK);
    const char* b_src = (const char*)(args.B + (int64_t)kk_i * TK * N + (int64_t)tj_i * TN);
    // GENERAL: rows, columns and K left from this K-iteration's tile origin
    // (wave-uniform; the origin is always inside A and B)
    int rows_left = 0, cols_left = 0, k_left = 0;
    if constexpr (GENERAL) {
      rows_left = args.M - ti_i * TM;
      cols_left = N - tj_i * TN;
      k_left = K - (int)kk_i * TK;
    }
    // GENERAL: the record counts end at the last row of A (the last K row
    // of B); offsets stay 16-byte multiples, so no chunk straddles the end
    const __amdgpu_buffer_rsrc_t ra =
        GENERAL ? panel_rsrc_to_end(a_src, ((int64_t)rows_left * K - (int64_t)kk_i * TK) * 2)
                : panel_rsrc(a_src);
    const __amdgpu_buffer_rsrc_t rb =
        GENERAL ? panel_rsrc_to_end(b_src, ((int64_t)k_left * N - (int64_t)tj_i * TN) * 2)
                : panel_rsrc(b_src);
    if (GENERAL) {
      // K and N are multiples of 8, so a 16-byte chunk is wholly inside or
      // wholly outside A / B.  Rows of A past M and K rows of B past K lie
      // beyond the record counts, and a chunk past K in A (past N in B)
      // loads from kOutsidePanel; the range check returns zeros for both, so
      // partial tiles and the tail of the last K-iteration contribute
      // nothing.  The test runs on every K-iteration, interior ones included: a branch
      // between an interior and an edge form of these loads gives the
      // compiler's wait-count analysis a path with fewer loads in flight,
      // and it then waits for all of them before each slot write.
      if constexpr (kStrided) {
        // From the lane's first chunks and the steps.  A lane whose K chunk
        // of A (column chunk of B) is past K (N) starts at kOutsidePanel,
        // and every chunk offset from there stays below 2^32
        // (a step times the chunk index is below 2^31).  The opaque copies
        // keep the compiler from hoisting one offset per chunk out of the
        // loop (they would not fit in the registers left).
        uint32_t ab = goff[0], bb = goff[A_PER];
        asm volatile("" : "+v"(ab), "+v"(bb));
        ab = a_kc0 < k_left ? ab : kOutsidePanel;
        bb = b_nc0 < cols_left ? bb : kOutsidePanel;
#pragma unroll
        for (int n = 0; n < A_PER; ++n) stage[u][n] = panel_load16(ra, ab + (uint32_t)n * a_step);
#pragma unroll
        for (int n = 0; n < B_PER; ++n) stage[u][A_PER + n] = panel_load16(rb, bb + (uint32_t)n * b_step);
      } else {
#pragma unroll
        for (int n = 0; n < A_PER; ++n) {
          const int q = (a_rank + n * A_GROUP) * 64 + lane;
          const int kc = 8 * ((q % G::CA) ^ swz_a<TK>(q / G::CA));
          stage[u][n] = panel_load16(ra, kc < k_left ? goff[n] : kOutsidePanel);
        }
#pragma unroll
        for (int n = 0; n < B_PER; ++n) {
          const int q = (b_rank + n * B_GROUP) * 64 + lane;
          const int nc8 = ((q >> 3) % G::NQ) * 16 + (q & 1) * 8;
          stage[u][A_PER + n] = panel_load16(rb, nc8 < cols_left ? goff[A_PER + n] : kOutsidePanel);
        }
      }
    } else {
#pragma unroll
      for (int n = 0; n < A_PER; ++n) stage[u][n] = panel_load16(ra, goff[n]);
#pragma unroll
      for (int n = 0; n < B_PER; ++n) stage[u][A_PER + n] = panel_load16(rb, goff[A_PER + n]);
    }
    if (q_iss + 1 < total) {
      ++q_iss;
      if (++kk_i == S) {
        kk_i = 0;
        v_i += Gd;
        tile_coords(v_i, args.tiles_m, args.tiles_n, args.group_m, &ti_i, &tj_i);
      }
    }
  };

  if constexpr (tracing) t_now = cycles32();
#pragma unroll
  for (int u = 0; u < L; ++u) issue(u);

  // Slot of the next K-iteration to write, the empty[] value its use needs
  // (0 for a slot's first use), and the value of that counter read with the
  // previous signal: when the consumers are ahead it already satisfies the
  // wait, and the wave skips an LDS round trip.
  uint32_t w_slot = 0, w_need = 0, seen = 0;
  for (uint32_t q0 = 0; q0 < total; q0 += L) {
#pragma unroll
    for (int u = 0; u < L; ++u) {
      const uint32_t q = q0 + u;
      if (q < total) {
      const uint32_t slot = w_slot;
      // No early exit when the wait fails (workgroup aborted, or this wait
      // timed out and raised the abort): the wave runs its remaining
      // K-iterations without waiting (every later wait sees the abort flag
      // at once) and leaves at the loop's end.  A return from inside the
      // loop would join the loop header in the compiler's control flow, and
      // its wait-count analysis would then drain every load in flight at the
      // first register stage of each pass through the stages.
      if ((int32_t)(seen - w_need) < 0)
        (void)wait_counter(&empty[slot], w_need, abort_flag, args.spin_limit, args.err);
      debug_delay(args.producer_delay);
      compiler_fence();
      WSG_LDS char* base = smem + kHeaderBytes + slot * G::STAGE + lane16;
#pragma unroll
      for (int n = 0; n < A_PER; ++n)
        *(WSG_LDS i32x4_t*)(base + (a_rank + n * A_GROUP) * 1024) = stage[u][n];
#pragma unroll
      for (int n = 0; n < B_PER; ++n)
        *(WSG_LDS i32x4_t*)(base + G::A_BYTES + (b_rank + n * B_GROUP) * 1024) = stage[u][A_PER + n];
      if constexpr (tracing) {
        t_now = cycles32();
        stamps.issued(q, t_issue[u], &full[kStampIssueA + slot], &full[kStampIssueB + slot]);
        stamps.landed(q, t_now, &full[kStampLandA + slot], &full[kStampLandB + slot]);
      }
      if (++w_slot == P) {
        w_slot = 0;
        w_need += NC;
      }
      // waits for the LDS writes, signals, and reads the next slot's empty[]
      seen = lds_signal_peek(&full[slot], &empty[w_slot]);
      }
      issue(u);  // refill this register stage with K-iteration q + L
    }
  }
  stamps.finish();
  wait_vmcnt<0>();
}

// Producer that loads nothing: waits for each slot to be free and signals it
// full (the calibration MATH kernel, and the idle half of a two-DMA split in
// the load calibration kernels).
template <int NC>
__device__ __forceinline__ void producer_signal_only(const KernelArgs& args, WSG_LDS char* smem) {
  WSG_LDS uint32_t* full = (WSG_LDS uint32_t*)smem;
  WSG_LDS uint32_t* empty = full + kMaxStages;
  WSG_LDS uint32_t* abort_flag = full + 2 * kMaxStages;
  const int Gd = gridDim.x;
  const int g0 = first_slot(args);
  const int my_tiles = g0 < args.num_tiles ? (args.num_tiles - g0 + Gd - 1) / Gd : 0;
  const uint32_t total = (uint32_t)my_tiles * (uint32_t)args.iters;
  const uint32_t P = (uint32_t)args.stages;
  for (uint32_t q = 0; q < total; ++q) {
    const uint32_t slot = ring_slot(q, P);
    if (ring_use(q, P) > 0 &&
        !wait_counter(&empty[slot], ring_empty_target(q, P, NC), abort_flag, args.spin_limit, args.err))
      return;
    lds_signal(&full[slot]);
  }
}

// One producer wave's loop on the configured load path; STAMP: it records
// trace events.
template <int TM, int TN, int TK, int NC, int NPW, int SPLIT, bool BF16, bool STAMP, bool DO_A, bool DO_B,
          bool GENERAL>
__device__ __forceinline__ void producer_run(const KernelArgs& args, WSG_LDS char* smem, int a_rank, int b_rank,
                                             int lane) {
  if constexpr (GENERAL) {  // partial tiles possible: always register-staged
    producer_loop_reg<TM, TN, TK, NC, NPW, SPLIT, BF16, STAMP, DO_A, DO_B, true>(args, smem, a_rank, b_rank,
                                                                            lane);
  } else if (args.load_path == 1) {  // wave-uniform: 0 = register-staged, 1 = LDS-DMA
    producer_loop<TM, TN, TK, NC, NPW, SPLIT, BF16, STAMP, DO_A, DO_B>(args, smem, a_rank, b_rank, lane);
  } else {
    producer_loop_reg<TM, TN, TK, NC, NPW, SPLIT, BF16, STAMP, DO_A, DO_B, false>(args, smem, a_rank, b_rank,
                                                                             lane);
  }
}

template <int TM, int TN, int TK, int NC, int NPW, int SPLIT, bool BF16, bool TRACE, bool DO_A, bool DO_B,
          bool GENERAL>
__device__ __forceinline__ void producer_share(const KernelArgs& args, WSG_LDS char* smem, int a_rank,
                                               int b_rank, int lane) {
  if constexpr (!DO_A && !DO_B) {
    producer_signal_only<NC>(args, smem);
  } else if (TRACE && traced_workgroup(args)) {
    producer_run<TM, TN, TK, NC, NPW, SPLIT, BF16, TRACE, DO_A, DO_B, GENERAL>(args, smem, a_rank, b_rank, lane);
  } else {
    producer_run<TM, TN, TK, NC, NPW, SPLIT, BF16, false, DO_A, DO_B, GENERAL>(args, smem, a_rank, b_rank, lane);
  }
}

template <int TM, int TN, int TK, int NC, int NPW, int SPLIT, bool BF16, bool TRACE, int MODE, bool GENERAL>
__device__ __forceinline__ void producer(const KernelArgs& args, WSG_LDS char* smem, int pw,
                                         int lane) {
  using G = Cfg<TM, TN, TK, NC, NPW, SPLIT, BF16>;
  constexpr bool LA = MODE == kModeGemm || MODE == kModeLoadA || MODE == kModeLoadAB;  // A loaded
  constexpr bool LB = MODE == kModeGemm || MODE == kModeLoadB || MODE == kModeLoadAB;  // B loaded
  if constexpr (MODE == kModeEpilogue) {
    return;
  } else if constexpr (SPLIT == 1) {
    producer_share<TM, TN, TK, NC, NPW, SPLIT, BF16, TRACE, LA, LB, GENERAL>(args, smem, pw, pw, lane);
  } else {
    if (pw < G::NP / 2)
      producer_share<TM, TN, TK, NC, NPW, SPLIT, BF16, TRACE, LA, false, GENERAL>(args, smem, pw, 0, lane);
    else
      producer_share<TM, TN, TK, NC, NPW, SPLIT, BF16, TRACE, false, LB, GENERAL>(args, smem, 0,
                                                                           pw - G::NP / 2, lane);
  }
}

// ---------------------------------------------------------------------------
// Consumer (MATH wave).  One K-iteration is KS MFMA k-steps of 16.  Inside a
// k-step the MFMAs run M-major: every column block nb of row block mb, then
// the next row block.  Operands for k-step s + 1 are read while k-step s
// multiplies:
//   * the B fragments of k-step s + 1 go to the other of two buffers at the
//     start of k-step s;
//   * A fragment mb is single-buffered and refilled right after its row of
//     MFMAs, (BM - 1) * BN MFMAs before its next use.
// The last k-step of a K-iteration reads k-step 0 of the next slot: the slot's
// full[] counter was peeked one k-step earlier, so the wait costs nothing
// when the producers are ahead.  The slot is released (empty[] signal) right
// after that k-step's reads are issued, once the older reads have completed.
// ---------------------------------------------------------------------------
template <int TM, int TN, int TK, int NC, int NPW, int SPLIT, bool BF16>
struct ConsumerOps {
  using G = Cfg<TM, TN, TK, NC, NPW, SPLIT, BF16>;
  static constexpr int kReads = G::BM + 2 * G::BN;  // LDS reads per k-step
  // A operand of row block mb: 16 bytes per lane at a_src + a_off + mb * 32 rows.
  static __device__ __forceinline__ void load_a(i16x8_t& fa, WSG_LDS char* a_src, uint32_t a_off,
                                                int mb) {
    fa = *(WSG_LDS i16x8_t*)(a_src + a_off + mb * 32 * TK * 2);
  }
  // B operand of column block nb at k-step s: two transposed 8-byte reads.
  static __device__ __forceinline__ void load_b(i16x8_t& fb, WSG_LDS char* b_src, uint32_t b_off,
                                                int s, int nb) {
    WSG_LDS char* p = b_src + b_off + ((4 * s) * G::NQ + 2 * nb) * 128;
    const i16x4_t lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((WSG_LDS i16x4_t*)p);
    const i16x4_t hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((WSG_LDS i16x4_t*)(p + G::NQ * 128));
    fb = __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7);
  }
};

template <int TM, int TN, int TK, int NC, int NPW, int SPLIT, bool BF16, bool TRACE, int MODE, bool GENERAL>
__device__ __forceinline__ void consumer(const KernelArgs& args, WSG_LDS char* smem, int cw,
                                         int lane) {
  using G = Cfg<TM, TN, TK, NC, NPW, SPLIT, BF16>;
  using Ops = ConsumerOps<TM, TN, TK, NC, NPW, SPLIT, BF16>;
  static_assert(G::KS >= 2, "a K-iteration holds at least two k-steps");
  WSG_LDS uint32_t* full = (WSG_LDS uint32_t*)smem;
  WSG_LDS uint32_t* empty = full + kMaxStages;
  WSG_LDS uint32_t* abort_flag = full + 2 * kMaxStages;

  const int wm = cw / G::WGN, wn = cw % G::WGN;
  // A: lane reads row wm*WM + mb*32 + lane%32, chunk 2s + lane/32 (swizzled;
  // the swizzle repeats every 32 rows, so it depends only on the lane).
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

  int v = g0;
  int ti, tj;
  tile_coords(v, args.tiles_m, args.tiles_n, args.group_m, &ti, &tj);

  f32x16_t acc[G::BM][G::BN];
#pragma unroll
  for (int mb = 0; mb < G::BM; ++mb)
#pragma unroll
    for (int nb = 0; nb < G::BN; ++nb) acc[mb][nb] = f32x16_t{};
  i16x8_t fa[G::BM];
  i16x8_t fb[2][G::BN];

  // Event trace (consumer wave 0 of traced workgroups writes the records).
  const bool tracing = TRACE && args.trace != nullptr && cw == 0 && (int)blockIdx.x < args.trace_wgs;
  uint32_t* trec = tracing ? args.trace + (size_t)blockIdx.x * args.trace_iters * kTraceEvents : nullptr;
  auto record = [&](uint32_t iq, int ev, uint32_t value) {
    if (tracing && iq < (uint32_t)args.trace_iters && lane == 0) trec[iq * kTraceEvents + ev] = value;
  };
  // Slot `ps` of K-iteration iq is full: copy the producer stamps, stamp "ready".
  auto record_ready = [&](uint32_t iq, uint32_t ps) {
    if (tracing) {
      const uint32_t t = cycles32();
      record(iq, 0, lds_read_now(&full[kStampIssueA + ps]));
      record(iq, 1, lds_read_now(&full[kStampIssueB + ps]));
      record(iq, 2, lds_read_now(&full[kStampLandA + ps]));
      record(iq, 3, lds_read_now(&full[kStampLandB + ps]));
      record(iq, 4, t);
    }
  };

  // Prologue: wait for K-iteration 0 and read k-step 0.
  if (!wait_counter(&full[ring_slot(0, P)], ring_full_target(0, P, G::NP), abort_flag,
                    args.spin_limit, args.err))
    return;
  record_ready(0, 0);
#pragma unroll
  for (int mb = 0; mb < G::BM; ++mb) Ops::load_a(fa[mb], smem + kHeaderBytes, a_off[0], mb);
#pragma unroll
  for (int nb = 0; nb < G::BN; ++nb)
    Ops::load_b(fb[0][nb], smem + kHeaderBytes + G::A_BYTES, b_off, 0, nb);

  uint32_t q = 0, kk = 0;
  while (true) {
    const uint32_t slot = ring_slot(q, P);
    WSG_LDS char* a_src = smem + kHeaderBytes + slot * G::STAGE;
    WSG_LDS char* b_src = a_src + G::A_BYTES;
    const bool has_next = (q + 1) < total;
    // After the last K-iteration the next-slot reads re-read this slot (and
    // are never used), so every path issues the same LDS operations.
    const uint32_t nslot = has_next ? ring_slot(q + 1, P) : slot;
    const uint32_t ntarget = has_next ? ring_full_target(q + 1, P, G::NP) : 0u;
    WSG_LDS char* na_src = smem + kHeaderBytes + nslot * G::STAGE;
    WSG_LDS char* nb_src = na_src + G::A_BYTES;
    uint32_t peek = 0;
    debug_delay(args.consumer_delay);
    if (tracing) record(q, 5, cycles32());
#pragma unroll
    for (int s = 0; s < G::KS; ++s) {
      const int cur = s & 1, nxt = cur ^ 1;
      const bool last = (s == G::KS - 1);
      if (s == G::KS - 2) {
        peek = lds_peek(&full[nslot]);  // before this k-step's reads
        __builtin_amdgcn_sched_barrier(0);
      }
      if (last) {
        const uint32_t st = wait_until(peek, &full[nslot], abort_flag, ntarget, args.spin_limit);
        if (st != 0) {
          if (st == 2) report_timeout(abort_flag, args.err);
          return;
        }
        compiler_fence();
        if (tracing && has_next) record_ready(q + 1, nslot);
      }
      WSG_LDS char* ra = last ? na_src : a_src;
      WSG_LDS char* rb = last ? nb_src : b_src;
      const int ts = last ? 0 : s + 1;
#pragma unroll
      for (int nb = 0; nb < G::BN; ++nb) Ops::load_b(fb[nxt][nb], rb, b_off, ts, nb);
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int mb = 0; mb < G::BM; ++mb) {
#pragma unroll
        for (int nb = 0; nb < G::BN; ++nb)
          acc[mb][nb] = mfma32x32x16<BF16>(fa[mb], fb[cur][nb], acc[mb][nb]);
        Ops::load_a(fa[mb], ra, a_off[ts], mb);
        __builtin_amdgcn_sched_barrier(0);
      }
      if (last) {
        // Every read of this slot is older than the kReads just issued.
        lds_signal<Ops::kReads>(&empty[slot]);
        if (tracing) record(q, 6, cycles32());
      }
    }
    ++q;
    if (++kk == S) {
      // The calibration MATH kernel keeps its products (the store below is
      // never taken: M > 0) without writing C.
      if (MODE != kModeMath || args.M < 0)
        store_tile<TM, TN, G::WM, G::WN, G::BM, G::BN, GENERAL, (G::NW > 8 ? 1 : (G::BN > 2 ? 32 / G::BN : 16))>(args, acc, ti, tj, wm, wn, lane);
      if (tracing) record(q - 1, 7, cycles32());
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

// ---------------------------------------------------------------------------
// Deep-prefetch consumer: the operands of k-step t are read during k-step
// t - 3, so three k-steps of LDS reads stay in flight behind the MFMAs.  The K
// loop of a tile is one generated asm block (DeepLoop, ws_deep_loop.inc,
// written by gen_deep_loop.py): its fragment registers are fixed and every
// wait on an LDS read is placed by hand.  A wave's LDS operations complete in
// order, so a wait names how many younger LDS operations may still be
// outstanding; waits cap at 15, the counter's range (a wait for fewer only
// waits longer).
//
// Per k-step t of a tile (KS k-steps per K-iteration, T = S KS in all):
//   * wait for the reads of k-step t;
//   * if k-step t + 3 exists and starts a new K-iteration, check that
//     K-iteration's slot is full (its counter was peeked when the read stream
//     entered the previous slot; poll, draining every read, only when it is
//     short) and peek at the next slot's counter; issue the reads of k-step
//     t + 3, one ahead of each MFMA of k-step t;
//   * when t + 2 ends a K-iteration, release that K-iteration's slot (its last
//     reads went out two k-steps earlier).
// The loop body is four k-steps, so a tile needs S KS divisible by 4
// (DeepLoop::kIterQuantum); TK = 32 tiles with an odd S take the
// compiler-scheduled consumer.  The tile's last four k-steps read nothing
// ahead and drain; the epilogue follows, and the next tile starts with a
// prologue (the reads of its first three k-steps).
// ---------------------------------------------------------------------------
#include "ws_deep_loop.inc"

template <int TM, int TN, int TK, int NC, int NPW, int SPLIT, bool BF16, int MODE, bool GENERAL>
__device__ __forceinline__ void consumer_deep(const KernelArgs& args, WSG_LDS char* smem, int cw,
                                              int lane) {
  using G = Cfg<TM, TN, TK, NC, NPW, SPLIT, BF16>;
  using Loop = DeepLoop<TM, TN, TK, NC, NPW, BF16>;
  static_assert(Loop::kAvailable && (G::KS == 4 || G::KS == 2), "deep consumer configuration");
  constexpr int BM = G::BM, BN = G::BN;
  WSG_LDS uint32_t* full = (WSG_LDS uint32_t*)smem;
  WSG_LDS uint32_t* empty = full + kMaxStages;
  WSG_LDS uint32_t* abort_flag = full + 2 * kMaxStages;

  const int wm = cw / G::WGN, wn = cw % G::WGN;
  // A operand of k-step s: row r, 16-byte chunk (2 s + lane / 32) ^ swz(r).
  // Slots start on 128-byte boundaries, so the address for k-step s is the
  // k-step 0 address with bits 5 and 6 XORed by 32 s.
  const int r = wm * G::WM + (lane & 31);
  const uint32_t a_off0 = (uint32_t)(r * TK * 2 + (((lane >> 5) ^ swz_a<TK>(r)) << 4));
  // B operand: the k-step's 4 x 16 blocks, as in ConsumerOps::load_b, past the A tile.
  const int grp = lane >> 4;
  const uint32_t b_off = (uint32_t)(G::A_BYTES +
                                    ((2 * (grp >> 1)) * G::NQ + (wn * G::WN) / 16 + (grp & 1)) * 128 +
                                    8 * (lane & 15));
  static_assert(kHeaderBytes % 128 == 0 && G::STAGE % 128 == 0, "slots on 128-byte boundaries");

  const uint32_t S = (uint32_t)args.iters;
  if (S % (uint32_t)Loop::kIterQuantum != 0) {
    consumer<TM, TN, TK, NC, NPW, SPLIT, BF16, false, MODE, GENERAL>(args, smem, cw, lane);
    return;
  }
  const int Gd = gridDim.x;
  const int g0 = first_slot(args);
  if (g0 >= args.num_tiles) return;
  const int my_tiles = (args.num_tiles - g0 + Gd - 1) / Gd;
  const uint32_t P = (uint32_t)args.stages;
  const uint32_t ring = (uint32_t)(uintptr_t)(smem + kHeaderBytes);
  const uint32_t fullb = (uint32_t)(uintptr_t)full;
  const uint32_t emptyb = (uint32_t)(uintptr_t)empty;
  const uint32_t abortb = (uint32_t)(uintptr_t)abort_flag;

  int v = g0, ti, tj;
  tile_coords(v, args.tiles_m, args.tiles_n, args.group_m, &ti, &tj);
  f32x16_t acc[BM][BN];
  uint32_t slot = 0, ftarget = (uint32_t)G::NP;  // K-iteration 0: ring_slot 0, ring_full_target NP
  for (int t = 0; t < my_tiles; ++t) {
#pragma unroll
    for (int mb = 0; mb < BM; ++mb)
#pragma unroll
      for (int nb = 0; nb < BN; ++nb) acc[mb][nb] = f32x16_t{};
    if (!wait_counter(&full[slot], ftarget, abort_flag, args.spin_limit, args.err)) return;
    const uint32_t st = Loop::tile(acc, a_off0, b_off, slot, ftarget, P, S, ring, fullb, emptyb, abortb,
                                   args.spin_limit, args.consumer_delay);
    if (st != 0) {
      if (st == 2) report_timeout(abort_flag, args.err);
      return;
    }
    // The calibration MATH kernel keeps its products (the store below is
    // never taken: M > 0) without writing C.
    if (MODE != kModeMath || args.M < 0)
      store_tile<TM, TN, G::WM, G::WN, BM, BN, GENERAL, (BN > 2 ? 32 / BN : 16)>(args, acc, ti, tj, wm, wn,
                                                                                  lane);
    v += Gd;
    tile_coords(v, args.tiles_m, args.tiles_n, args.group_m, &ti, &tj);
  }
}

// ---------------------------------------------------------------------------
// Consumer with two consumer waves per SIMD: the eight-consumer arrangement
// (2 x 4 grid of 128 x 64 wave tiles next to four producer waves) and the
// four-consumer 128 x 128 x 32 kernel held to 128 registers a wave (2 x 2
// grid of 64 x 64 wave tiles, two workgroups per CU).  The K loop of a tile is
// the generated RollLoop block (ws_deep_loop.inc).  Its fragments are
// single-buffered and refilled right after their last MFMA of the k-step; the
// other consumer wave of the SIMD covers the read latency.
// ---------------------------------------------------------------------------
template <int TM, int TN, int TK, int NC, int NPW, int SPLIT, bool BF16, bool TRACE, int MODE, bool GENERAL>
__device__ __forceinline__ void consumer_roll(const KernelArgs& args, WSG_LDS char* smem, int cw,
                                              int lane) {
  using G = Cfg<TM, TN, TK, NC, NPW, SPLIT, BF16>;
  using Loop = RollLoop<TM, TN, TK, NC, NPW, BF16>;
  static_assert(Loop::kAvailable, "roll consumer configuration");
  constexpr int BM = G::BM, BN = G::BN;
  WSG_LDS uint32_t* full = (WSG_LDS uint32_t*)smem;
  WSG_LDS uint32_t* empty = full + kMaxStages;
  WSG_LDS uint32_t* abort_flag = full + 2 * kMaxStages;

  const int wm = cw / G::WGN, wn = cw % G::WGN;
  // A operand of k-step 0: row r, 16-byte chunk (lane / 32) ^ swz(r); the
  // block moves it to k-step s by XORing 32 s into the byte offset.
  const int r = wm * G::WM + (lane & 31);
  const uint32_t a_off0 = (uint32_t)(r * TK * 2 + (((lane >> 5) ^ swz_a<TK>(r)) << 4));
  const int grp = lane >> 4;
  const uint32_t b_off = (uint32_t)(G::A_BYTES +
                                    ((2 * (grp >> 1)) * G::NQ + (wn * G::WN) / 16 + (grp & 1)) * 128 +
                                    8 * (lane & 15));
  static_assert(kHeaderBytes % 128 == 0 && G::STAGE % 128 == 0, "slots on 128-byte boundaries");

  const int Gd = gridDim.x;
  const int g0 = first_slot(args);
  if (g0 >= args.num_tiles) return;
  const int my_tiles = (args.num_tiles - g0 + Gd - 1) / Gd;
  const uint32_t P = (uint32_t)args.stages;
  const uint32_t S = (uint32_t)args.iters;
  const uint32_t ring = (uint32_t)(uintptr_t)(smem + kHeaderBytes);
  const uint32_t fullb = (uint32_t)(uintptr_t)full;
  const uint32_t emptyb = (uint32_t)(uintptr_t)empty;
  const uint32_t abortb = (uint32_t)(uintptr_t)abort_flag;

  // Event trace: consumer wave 0 of the traced workgroups runs the block's
  // traced twin, which stores events 4-6 of every K-iteration; the first
  // K-iteration's event 4 and each tile's event 7 are stored here.
  const bool tracing = TRACE && args.trace != nullptr && cw == 0 && (int)blockIdx.x < args.trace_wgs;
  uint32_t* trec = tracing ? args.trace + (size_t)blockIdx.x * args.trace_iters * kTraceEvents : nullptr;
  auto record = [&](uint32_t iq, int ev, uint32_t value) {
    if (tracing && iq < (uint32_t)args.trace_iters && lane == 0) trec[iq * kTraceEvents + ev] = value;
  };

  int v = g0, ti, tj;
  tile_coords(v, args.tiles_m, args.tiles_n, args.group_m, &ti, &tj);
  f32x16_t acc[BM][BN];
  uint32_t slot = 0, ftarget = (uint32_t)G::NP;  // K-iteration 0: ring_slot 0, ring_full_target NP
  for (int t = 0; t < my_tiles; ++t) {
#pragma unroll
    for (int mb = 0; mb < BM; ++mb)
#pragma unroll
      for (int nb = 0; nb < BN; ++nb) acc[mb][nb] = f32x16_t{};
    if (!wait_counter(&full[slot], ftarget, abort_flag, args.spin_limit, args.err)) return;
    const uint32_t q0 = (uint32_t)t * S;  // the tile's first K-iteration in this workgroup's sequence
    if (tracing) record(q0, 4, cycles32());  // the tile's first slot seen full
    const uint32_t base = ring + slot * (uint32_t)G::STAGE;
    uint32_t st;
    if (tracing)
      st = Loop::tile_traced(acc, base + a_off0, base + b_off, slot, ftarget, P, S, ring, fullb, emptyb,
                             abortb, args.spin_limit, args.consumer_delay, trec, q0,
                             (uint32_t)args.trace_iters);
    else
      st = Loop::tile(acc, base + a_off0, base + b_off, slot, ftarget, P, S, ring, fullb, emptyb, abortb,
                      args.spin_limit, args.consumer_delay);
    if (st != 0) {
      if (st == 2) report_timeout(abort_flag, args.err);
      return;
    }
    // The calibration MATH kernel keeps its products (the store below is
    // never taken: M > 0) without writing C.
    if (MODE != kModeMath || args.M < 0)
      store_tile<TM, TN, G::WM, G::WN, BM, BN, GENERAL, 1>(args, acc, ti, tj, wm, wn, lane);
    if (tracing) record(q0 + S - 1, 7, cycles32());
    v += Gd;
    tile_coords(v, args.tiles_m, args.tiles_n, args.group_m, &ti, &tj);
  }
}

// ---------------------------------------------------------------------------
// Register-lean consumer for three waves per SIMD (two producers per consumer
// with the largest wave tiles): every operand fragment is single-buffered and
// refilled right after its last MFMA of the k-step, and the loop body is one
// k-step, so each fragment has a single load site and keeps its registers.
// Waits and releases are branch-free asm blocks enabled on the last k-step
// of a K-iteration.  Same synchronisation as consumer().
// ---------------------------------------------------------------------------
template <int TM, int TN, int TK, int NC, int NPW, int SPLIT, bool BF16, bool TRACE, int MODE, bool GENERAL>
__device__ __forceinline__ void consumer_rolling(const KernelArgs& args, WSG_LDS char* smem, int cw,
                                                 int lane) {
  using G = Cfg<TM, TN, TK, NC, NPW, SPLIT, BF16>;
  using Ops = ConsumerOps<TM, TN, TK, NC, NPW, SPLIT, BF16>;
  WSG_LDS uint32_t* full = (WSG_LDS uint32_t*)smem;
  WSG_LDS uint32_t* empty = full + kMaxStages;
  WSG_LDS uint32_t* abort_flag = full + 2 * kMaxStages;

  const int wm = cw / G::WGN, wn = cw % G::WGN;
  // A operand of k-step s: a_off0 ^ (32 s).  The chunk of k-step s is
  // (2 s + lane / 32) ^ swz, and XOR acts bit by bit, so only bits 5.. of the
  // in-row byte offset change with s.
  const int r = wm * G::WM + (lane & 31);
  const uint32_t a_off0 = (uint32_t)(r * TK * 2 + (((lane >> 5) ^ swz_a<TK>(r)) << 4));
  const int grp = lane >> 4;
  const uint32_t b_off =
      (uint32_t)(((2 * (grp >> 1)) * G::NQ + (wn * G::WN) / 16 + (grp & 1)) * 128 + 8 * (lane & 15));
  const uint32_t ring = (uint32_t)(uintptr_t)smem + kHeaderBytes;

  const int Gd = gridDim.x;
  const int g0 = first_slot(args);
  if (g0 >= args.num_tiles) return;
  const int my_tiles = (args.num_tiles - g0 + Gd - 1) / Gd;
  const uint32_t S = (uint32_t)args.iters;
  const uint32_t total = (uint32_t)my_tiles * S;
  const uint32_t P = (uint32_t)args.stages;

  int v = g0;
  int ti, tj;
  tile_coords(v, args.tiles_m, args.tiles_n, args.group_m, &ti, &tj);

  f32x16_t acc[G::BM][G::BN];
#pragma unroll
  for (int mb = 0; mb < G::BM; ++mb)
#pragma unroll
    for (int nb = 0; nb < G::BN; ++nb) acc[mb][nb] = f32x16_t{};
  i16x8_t fa[G::BM];
  i16x8_t fb[G::BN];

  const bool tracing = TRACE && args.trace != nullptr && cw == 0 && (int)blockIdx.x < args.trace_wgs;
  uint32_t* trec = tracing ? args.trace + (size_t)blockIdx.x * args.trace_iters * kTraceEvents : nullptr;
  auto record = [&](uint32_t iq, int ev, uint32_t value) {
    if (tracing && iq < (uint32_t)args.trace_iters && lane == 0) trec[iq * kTraceEvents + ev] = value;
  };
  auto record_ready = [&](uint32_t iq, uint32_t ps) {
    if (tracing) {
      const uint32_t t = cycles32();
      record(iq, 0, lds_read_now(&full[kStampIssueA + ps]));
      record(iq, 1, lds_read_now(&full[kStampIssueB + ps]));
      record(iq, 2, lds_read_now(&full[kStampLandA + ps]));
      record(iq, 3, lds_read_now(&full[kStampLandB + ps]));
      record(iq, 4, t);
    }
  };

  if (!wait_counter(&full[ring_slot(0, P)], ring_full_target(0, P, G::NP), abort_flag,
                    args.spin_limit, args.err))
    return;
  record_ready(0, 0);
  // full[] of the slot the next wait is for, read one k-step before that
  // wait.  Read here before the first operand loads, so that on every path
  // into the loop a whole k-step of loads is younger than it and the wait
  // for it does not drain them.
  uint32_t peek = lds_peek(&full[ring_slot(1, P)]);
  __builtin_amdgcn_sched_barrier(0);
#pragma unroll
  for (int mb = 0; mb < G::BM; ++mb) Ops::load_a(fa[mb], smem + kHeaderBytes, a_off0, mb);
#pragma unroll
  for (int nb = 0; nb < G::BN; ++nb)
    Ops::load_b(fb[nb], smem + kHeaderBytes + G::A_BYTES, b_off, 0, nb);

  uint32_t q = 0, kk = 0, s = 0;
  // (nslot, ntarget): slot and full[] target of K-iteration q + 1.
  uint32_t slot = 0, nslot = ring_slot(1, P);
  uint32_t ntarget = ring_full_target(1, P, G::NP);
  while (true) {
    const uint32_t last = (s == (uint32_t)G::KS - 1) ? 1u : 0u;
    const bool has_next = (q + 1) < total;
    const uint32_t do_wait = (last && has_next) ? 1u : 0u;
    debug_delay(s == 0 ? args.consumer_delay : 0);
    if (tracing && s == 0) record(q, 5, cycles32());
    const uint32_t st = wait_until(peek, &full[nslot], abort_flag, ntarget, args.spin_limit, do_wait);
    if (st != 0) {
      if (st == 2) report_timeout(abort_flag, args.err);
      return;
    }
    compiler_fence();
    if (tracing && do_wait) record_ready(q + 1, nslot);
    {
      const uint32_t pslot = last ? ((nslot + 1 == P) ? 0u : nslot + 1) : nslot;
      peek = lds_peek(&full[pslot]);
      __builtin_amdgcn_sched_barrier(0);
    }
    // Source of the next k-step: k-step s + 1 of this slot, or k-step 0 of
    // the next slot (this slot again after the last K-iteration; never used).
    const uint32_t ts = last ? 0u : s + 1;
    const uint32_t src = ring + (do_wait ? nslot : slot) * (uint32_t)G::STAGE;
    WSG_LDS char* ra = (WSG_LDS char*)(uintptr_t)(src);
    WSG_LDS char* rb = (WSG_LDS char*)(uintptr_t)(src + G::A_BYTES + ts * (uint32_t)(4 * G::NQ * 128));
    const uint32_t a_off = a_off0 ^ (32u * ts);
#pragma unroll
    for (int nb = 0; nb < G::BN; ++nb) {
#pragma unroll
      for (int mb = 0; mb < G::BM; ++mb) {
        acc[mb][nb] = mfma32x32x16<BF16>(fa[mb], fb[nb], acc[mb][nb]);
        if (nb == G::BN - 1) Ops::load_a(fa[mb], ra, a_off, mb);
        __builtin_amdgcn_sched_barrier(0);
      }
      Ops::load_b(fb[nb], rb, b_off, 0, nb);
      __builtin_amdgcn_sched_barrier(0);
    }
    // Every read of this slot is older than the kReads just issued.
    lds_signal_if<Ops::kReads>(&empty[slot], last);
    if (!last) {
      ++s;
      continue;
    }
    if (tracing) record(q, 6, cycles32());
    s = 0;
    slot = nslot;
    ring_advance(nslot, ntarget, P, G::NP);
    ++q;
    if (++kk == S) {
      // The calibration MATH kernel keeps its products (the store below is
      // never taken: M > 0) without writing C.
      if (MODE != kModeMath || args.M < 0)
        store_tile<TM, TN, G::WM, G::WN, G::BM, G::BN, GENERAL, 1>(args, acc, ti, tj, wm, wn, lane);
      if (tracing) record(q - 1, 7, cycles32());
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

// Calibration consumers.  Release-only: take every slot in order and free it
// without reading it (load calibration).  Epilogue-only: store a zero tile
// for every output tile of the workgroup, with no K loop.
template <int NP, int NC>
__device__ __forceinline__ void consumer_release_only(const KernelArgs& args, WSG_LDS char* smem) {
  WSG_LDS uint32_t* full = (WSG_LDS uint32_t*)smem;
  WSG_LDS uint32_t* empty = full + kMaxStages;
  WSG_LDS uint32_t* abort_flag = full + 2 * kMaxStages;
  const int Gd = gridDim.x;
  const int g0 = first_slot(args);
  const int my_tiles = g0 < args.num_tiles ? (args.num_tiles - g0 + Gd - 1) / Gd : 0;
  const uint32_t total = (uint32_t)my_tiles * (uint32_t)args.iters;
  const uint32_t P = (uint32_t)args.stages;
  for (uint32_t q = 0; q < total; ++q) {
    const uint32_t slot = ring_slot(q, P);
    if (!wait_counter(&full[slot], ring_full_target(q, P, NP), abort_flag, args.spin_limit, args.err))
      return;
    lds_signal(&empty[slot]);
  }
}

template <int TM, int TN, int TK, int NC, int NPW, int SPLIT, bool BF16>
__device__ __forceinline__ void consumer_epilogue_only(const KernelArgs& args, int cw, int lane) {
  using G = Cfg<TM, TN, TK, NC, NPW, SPLIT, BF16>;
  const int wm = cw / G::WGN, wn = cw % G::WGN;
  f32x16_t acc[G::BM][G::BN];
#pragma unroll
  for (int mb = 0; mb < G::BM; ++mb)
#pragma unroll
    for (int nb = 0; nb < G::BN; ++nb) acc[mb][nb] = f32x16_t{};
  for (int v = first_slot(args); v < args.num_tiles; v += (int)gridDim.x) {
    int ti, tj;
    tile_coords(v, args.tiles_m, args.tiles_n, args.group_m, &ti, &tj);
    store_tile<TM, TN, G::WM, G::WN, G::BM, G::BN>(args, acc, ti, tj, wm, wn, lane);
  }
}

// The epilogue of a product with K = 0 (nothing to multiply): C <- beta C
// over n elements of type T; zeros when beta == 0 (C is then not read).
template <typename T>
__global__ void __launch_bounds__(256) ws_scale_kernel(void* C, int64_t n, float beta) {
  T* c = (T*)C;
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += stride)
    c[i] = beta == 0.0f ? (T)0.0f : (T)(beta * load_out(c + i));
}

// Calibration of the launch itself (T_INIT): an empty kernel launched with
// the GEMM's grid, block and LDS size.  A template so that every translation
// unit including this header may instantiate it.
template <int UNUSED = 0>
__global__ void __launch_bounds__(1024) ws_empty_kernel(KernelArgs) {}

// Waves per SIMD a kernel's register allocation must leave room for: the
// four-consumer roll loop holds its kernel to 128 registers a wave so that two
// workgroups of eight waves share a CU; every other kernel is sized for one
// workgroup (what the compiler assumes without the bound).
template <int TM, int TN, int TK, int NC, int NPW, bool BF16, bool GENERAL>
constexpr int kernel_waves_per_simd() {
  return (NC == 4 && !GENERAL && RollLoop<TM, TN, TK, NC, NPW, BF16>::kAvailable) ? 4 : (NC + NPW + 3) / 4;
}

template <int TM, int TN, int TK, int NC, int NPW, int SPLIT, bool BF16, bool TRACE, int MODE, bool GENERAL>
__global__ void __launch_bounds__((NC + NPW) * 64, (kernel_waves_per_simd<TM, TN, TK, NC, NPW, BF16, GENERAL>()))
    ws_gemm_kernel(KernelArgs args) {
  using G = Cfg<TM, TN, TK, NC, NPW, SPLIT, BF16>;
  extern __shared__ __attribute__((aligned(1024))) char smem_generic[];
  WSG_LDS char* smem = (WSG_LDS char*)smem_generic;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  LaunchClock clk;
  clk.start(args, wave);
  if (threadIdx.x < 2 * kMaxStages + 1) ((WSG_LDS uint32_t*)smem)[threadIdx.x] = 0u;
  __syncthreads();
  if (wave < NC) {
    if constexpr (MODE == kModeLoadA || MODE == kModeLoadB || MODE == kModeLoadAB) {
      consumer_release_only<G::NP, NC>(args, smem);
    } else if constexpr (MODE == kModeEpilogue) {
      consumer_epilogue_only<TM, TN, TK, NC, NPW, SPLIT, BF16>(args, wave, lane);
    } else if constexpr ((!GENERAL || NC == 8) && (MODE == kModeGemm || MODE == kModeMath) &&
                         RollLoop<TM, TN, TK, NC, NPW, BF16>::kAvailable) {
      // Two consumer waves per SIMD (eight consumer waves, or four with two
      // workgroups per CU): the generated register-lean K loop (and its
      // event-traced twin).  The general variant of the eight-consumer
      // arrangement runs it too: its producers zero-fill what lies outside A
      // and B, so the K loop is the plain one, and only the epilogue differs.
      consumer_roll<TM, TN, TK, NC, NPW, SPLIT, BF16, TRACE, MODE, GENERAL>(args, smem, wave, lane);
    } else if constexpr (G::NW > 8 && G::BM * G::BN >= 8) {
      // Three waves per SIMD leave 168 VGPRs: the largest wave tiles then
      // take the single-buffered consumer.
      consumer_rolling<TM, TN, TK, NC, NPW, SPLIT, BF16, TRACE, MODE, GENERAL>(args, smem, wave, lane);
    } else if constexpr (!TRACE && (MODE == kModeGemm || MODE == kModeMath) &&
                         DeepLoop<TM, TN, TK, NC, NPW, BF16>::kAvailable) {
      // One producer group with the largest tiles (DeepLoop lists them): the
      // hand-scheduled deep-prefetch K loop, in the general variant too (its
      // producers zero-fill what lies outside A and B).
      consumer_deep<TM, TN, TK, NC, NPW, SPLIT, BF16, MODE, GENERAL>(args, smem, wave, lane);
    } else {
      consumer<TM, TN, TK, NC, NPW, SPLIT, BF16, TRACE, MODE, GENERAL>(args, smem, wave, lane);
    }
  } else {
    producer<TM, TN, TK, NC, NPW, SPLIT, BF16, TRACE, MODE, GENERAL>(args, smem, wave - NC, lane);
  }
  clk.stop(args, lane);
}

}  // namespace wsg
