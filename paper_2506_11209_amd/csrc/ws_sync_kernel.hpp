// Synchronous (not warp-specialised) tiled GEMM: the baseline of the paper's
// Section 2.1, "Stage" -- a kernel whose K-iterations load their A and B tiles
// and then multiply them, with no overlap between the two (ring depth 1); and
// the conventional double-buffered variant (ring depth 2: the tiles of
// K-iteration q + 1 are requested before q is multiplied).  Every wave both
// loads and computes; there is no role split and no semaphore, only
// workgroup barriers.
//
// Same tiling, LDS layout, operand reads, MFMA and epilogue as the
// warp-specialised kernel (ws_gemm_kernel.hpp), so the two differ only in the
// organisation of the work.  Loads go straight into LDS (buffer_load_dwordx4
// with the lds bit, through the same tile-panel buffer resources).
#pragma once

#include "ws_gemm_kernel.hpp"

namespace wsg {

template <int TM, int TN, int TK, int NC>
struct SyncCfg {
  static constexpr int WGM = (NC == 4) ? 2 : 1;
  static constexpr int WGN = (NC == 4) ? 2 : 1;
  static constexpr int WM = TM / WGM, WN = TN / WGN;
  static constexpr int BM = WM / 32, BN = WN / 32;
  static constexpr int KS = TK / 16;
  static constexpr int A_BYTES = TM * TK * 2, B_BYTES = TK * TN * 2;
  static constexpr int STAGE = A_BYTES + B_BYTES;
  static constexpr int A_PER = A_BYTES / 1024 / NC;  // DMA instructions per wave per K-iteration
  static constexpr int B_PER = B_BYTES / 1024 / NC;
  static constexpr int CA = TK / 8;
  static constexpr int NQ = TN / 16;
  static_assert(NC == 1 || NC == 4, "1 or 4 waves");
  static_assert(WM % 32 == 0 && WN % 32 == 0, "wave tile must be a multiple of 32x32");
  static_assert(A_BYTES % (1024 * NC) == 0 && B_BYTES % (1024 * NC) == 0, "even DMA split");
};

template <int TM, int TN, int TK, int NC, bool BF16>
__global__ void __launch_bounds__(NC * 64) ws_sync_kernel(KernelArgs args) {
  using G = SyncCfg<TM, TN, TK, NC>;
  extern __shared__ __attribute__((aligned(1024))) char smem_generic[];
  WSG_LDS char* ring = (WSG_LDS char*)smem_generic + kHeaderBytes;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  const int K = args.K, N = args.N;
  const int P = args.stages;  // 1: synchronous; 2: double-buffered
  LaunchClock clk;
  clk.start(args, wave);

  // This wave's share of every tile, as in the producers of the specialised
  // kernel: chunk (wave + n * NC) * 64 + lane of the LDS tile.
  uint32_t a_goff[G::A_PER], b_goff[G::B_PER];
#pragma unroll
  for (int n = 0; n < G::A_PER; ++n) {
    const int q = (wave + n * NC) * 64 + lane;
    const int r = q / G::CA, p = q % G::CA;
    a_goff[n] = (uint32_t)(r * K + 8 * (p ^ swz_a<TK>(r))) * 2u;
  }
#pragma unroll
  for (int n = 0; n < G::B_PER; ++n) {
    const int q = (wave + n * NC) * 64 + lane;
    const int blk = q >> 3, w = q & 7;
    const int kq = blk / G::NQ, nq = blk % G::NQ;
    b_goff[n] = (uint32_t)((kq * 4 + (w >> 1)) * N + nq * 16 + (w & 1) * 8) * 2u;
  }
  auto issue = [&](int ti, int tj, int kk, int slot) {
    const __amdgpu_buffer_rsrc_t a_src = panel_rsrc(args.A + (int64_t)ti * TM * K + kk * TK);
    const __amdgpu_buffer_rsrc_t b_src = panel_rsrc(args.B + (int64_t)kk * TK * N + (int64_t)tj * TN);
    WSG_LDS char* dst = ring + slot * G::STAGE;
#pragma unroll
    for (int n = 0; n < G::A_PER; ++n)
      panel_load16_lds(a_src, (WSG_LDS void*)(dst + (wave + n * NC) * 1024), a_goff[n]);
#pragma unroll
    for (int n = 0; n < G::B_PER; ++n)
      panel_load16_lds(b_src, (WSG_LDS void*)(dst + G::A_BYTES + (wave + n * NC) * 1024), b_goff[n]);
  };

  // Operand offsets (same layout and reads as the specialised consumers).
  const int wm = wave / G::WGN, wn = wave % G::WGN;
  uint32_t a_off[G::KS];
  {
    const int r = wm * G::WM + (lane & 31);
#pragma unroll
    for (int s = 0; s < G::KS; ++s)
      a_off[s] = (uint32_t)(r * TK * 2 + (((2 * s + (lane >> 5)) ^ swz_a<TK>(r)) << 4));
  }
  const int grp = lane >> 4;
  const uint32_t b_off =
      (uint32_t)(((2 * (grp >> 1)) * G::NQ + (wn * G::WN) / 16 + (grp & 1)) * 128 + 8 * (lane & 15));

  f32x16_t acc[G::BM][G::BN];
  i16x8_t fa[2][G::BM], fb[2][G::BN];
  auto read = [&](WSG_LDS char* slot_base, int s, int buf) {
#pragma unroll
    for (int mb = 0; mb < G::BM; ++mb)
      fa[buf][mb] = *(WSG_LDS i16x8_t*)(slot_base + a_off[s] + mb * 32 * TK * 2);
#pragma unroll
    for (int nb = 0; nb < G::BN; ++nb) {
      WSG_LDS char* p = slot_base + G::A_BYTES + b_off + ((4 * s) * G::NQ + 2 * nb) * 128;
      const i16x4_t lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((WSG_LDS i16x4_t*)p);
      const i16x4_t hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((WSG_LDS i16x4_t*)(p + G::NQ * 128));
      fb[buf][nb] = __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7);
    }
  };

  const int Gd = gridDim.x;
  const int g0 = first_slot(args);
  const int S = args.iters;
  // Next K-iteration to request (double-buffered variant): tile index and k.
  int nv = g0, nkk = 0;
  int nti = 0, ntj = 0;
  if (nv < args.num_tiles) tile_coords(nv, args.tiles_m, args.tiles_n, args.group_m, &nti, &ntj);
  uint32_t q = 0;
  if (P == 2 && nv < args.num_tiles) {
    issue(nti, ntj, 0, 0);
    nkk = 1;
    if (nkk == S) {
      nkk = 0;
      nv += Gd;
      if (nv < args.num_tiles) tile_coords(nv, args.tiles_m, args.tiles_n, args.group_m, &nti, &ntj);
    }
  }
  for (int v = g0; v < args.num_tiles; v += Gd) {
    int ti, tj;
    tile_coords(v, args.tiles_m, args.tiles_n, args.group_m, &ti, &tj);
#pragma unroll
    for (int mb = 0; mb < G::BM; ++mb)
#pragma unroll
      for (int nb = 0; nb < G::BN; ++nb) acc[mb][nb] = f32x16_t{};
    for (int kk = 0; kk < S; ++kk, ++q) {
      const int slot = (P == 2) ? (int)(q & 1) : 0;
      if (P == 1) issue(ti, tj, kk, 0);  // load, then wait: no overlap
      wait_vmcnt<0>();      // this wave's tiles of K-iteration q have landed
      __syncthreads();      // ... and every wave's; the other slot is no longer read
      if (P == 2 && nv < args.num_tiles) {  // request K-iteration q + 1 into the other slot
        issue(nti, ntj, nkk, slot ^ 1);
        if (++nkk == S) {
          nkk = 0;
          nv += Gd;
          if (nv < args.num_tiles) tile_coords(nv, args.tiles_m, args.tiles_n, args.group_m, &nti, &ntj);
        }
      }
      WSG_LDS char* base = ring + slot * G::STAGE;
      read(base, 0, 0);
#pragma unroll
      for (int s = 0; s < G::KS; ++s) {
        if (s + 1 < G::KS) read(base, s + 1, (s + 1) & 1);
#pragma unroll
        for (int mb = 0; mb < G::BM; ++mb)
#pragma unroll
          for (int nb = 0; nb < G::BN; ++nb)
            acc[mb][nb] = mfma32x32x16<BF16>(fa[s & 1][mb], fb[s & 1][nb], acc[mb][nb]);
      }
      if (P == 1) __syncthreads();  // every wave has read the slot before it is refilled
    }
    store_tile<TM, TN, G::WM, G::WN, G::BM, G::BN>(args, acc, ti, tj, wm, wn, lane);
  }
  wait_vmcnt<0>();  // no load into LDS outlives the workgroup
  clk.stop(args, lane);
}

}  // namespace wsg
