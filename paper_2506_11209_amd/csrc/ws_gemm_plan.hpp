// Launch planning for the warp-specialised GEMM (host) and the tile raster
// shared by host and device.
//
// Terms (paper, Section 2.1):
//   output tiles  = (M / TM) * (N / TN)
//   dispatch rounds W = ceil(tiles / workgroups)   ("waves" in the paper)
//   K-iterations  S = K / TK                       ("stages" in the paper)
// The paper assumes TM | M, TN | N and TK | K so that every round and every
// K-iteration has the same cost; other shapes are planned with ceil() and run
// the ragged kernel variant.
#pragma once

#include <stdint.h>

#if defined(__HIPCC__)
#define WSG_HD __host__ __device__
#else
#define WSG_HD
#endif

namespace wsg {

// Raster: schedule index v -> output tile (ti, tj).  Tiles are taken in
// groups of group_m tile rows; inside a group, consecutive v walk down the
// rows first, then across the columns.  A run of consecutive v therefore
// covers a compact group_m x (run / group_m) block of output tiles.
WSG_HD inline void tile_coords(int v, int tiles_m, int tiles_n, int group_m, int* ti, int* tj) {
  const int per_group = group_m * tiles_n;
  const int grp = v / per_group;
  const int first = grp * group_m;
  const int rows = (tiles_m - first < group_m) ? (tiles_m - first) : group_m;
  const int rem = v - grp * per_group;
  *ti = first + rem % rows;
  *tj = rem / rows;
}

// Workgroup id -> schedule slot.  Workgroup g runs on XCD g % 8; the remap
// gives XCD x the consecutive slots [x * G/8, (x+1) * G/8), so tiles that run
// concurrently on one XCD are neighbours in the raster.  Requires G % 8 == 0.
WSG_HD inline int xcd_slot(int g, int G) { return (g & 7) * (G >> 3) + (g >> 3); }

struct PlanIn {
  int64_t M, N, K;
  int32_t tile_m, tile_n, tile_k;
  int32_t producer_waves, consumer_waves, stages, dtype, load_path;
  int32_t split;       // DMA warps per MATH warp (1 or 2); 0: derived from the wave counts
  int32_t num_cus;     // compute units on the device
  int32_t wgs_per_cu;  // resident workgroups per CU (<= 0: derive from LDS, waves and registers)
  int32_t vgprs, agprs;  // registers per wave of the kernel (0: unknown, not a limit)
};

struct PlanOut {
  int32_t grid, block, lds_bytes;
  int32_t tiles_m, tiles_n, tiles, rounds, iters;
  int32_t split, group_m, xcd_remap;
  int32_t ragged;  // 1 when a tile does not divide its dimension (edge tiles are partial)
};

enum PlanStatus {
  kPlanOk = 0,
  kPlanInvalid = 1,
  kPlanNotDivisible = 6,
  kPlanUnsupported = 2,
  kPlanLdsOverflow = 3,
};

constexpr int kLdsLimit = 163840;   // bytes of LDS per workgroup on gfx950
constexpr int kPlanHeaderBytes = 256;
constexpr int kPlanMaxStages = 8;
constexpr int kMaxWavesPerCu = 32;
constexpr int kMaxWgsPerCu = 16;
constexpr int kMaxWavesPerSimd = 8;
constexpr int kRegsPerSimdLane = 512;  // unified VGPR + AGPR file per lane of a SIMD

// Waves of one kernel that fit on a SIMD by registers: arch VGPRs rounded to
// the accumulator offset granule (4), AGPRs after them, the total allocated
// in granules of 8.
inline int waves_per_simd_by_regs(int vgprs, int agprs) {
  if (vgprs <= 0 && agprs <= 0) return kMaxWavesPerSimd;
  int total = ((vgprs + 3) / 4) * 4 + agprs;
  total = ((total + 7) / 8) * 8;
  const int w = kRegsPerSimdLane / total;
  return w < kMaxWavesPerSimd ? w : kMaxWavesPerSimd;
}

// DMA warps per MATH warp of a wave arrangement (consumer waves nc, producer
// waves np, requested split; 0 requests the one the wave counts imply), or
// -1 when no kernel has that arrangement.  0 for the synchronous kernel.
inline int arrangement_split(int nc, int np, int split) {
  if (np == 0) return (nc == 1 || nc == 4) && split == 0 ? 0 : -1;
  if (split == 0) split = (np == 2 * nc) ? 2 : 1;
  if (nc == 1) return (np == split) ? split : -1;
  if (nc == 4) return (np == 4 || (np == 8 && split == 2)) ? split : -1;
  if (nc == 8) return np == 4 ? split : -1;
  return -1;
}

inline bool is_pow2_in(int x, int lo, int hi) {
  return x >= lo && x <= hi && (x & (x - 1)) == 0;
}

// Pure host computation: validates a configuration and derives the launch.
inline int plan_launch(const PlanIn& in, PlanOut* out) {
  if (!out) return kPlanInvalid;
  *out = PlanOut{};
  if (in.M < 0 || in.N < 0 || in.K < 0) return kPlanInvalid;
  if (in.M > (1 << 30) || in.N > (1 << 30) || in.K > (1 << 30)) return kPlanInvalid;
  if (in.dtype != 0 && in.dtype != 1) return kPlanInvalid;
  if (in.load_path != 0 && in.load_path != 1) return kPlanInvalid;
  if (!is_pow2_in(in.tile_m, 32, 256) || !is_pow2_in(in.tile_n, 32, 256) ||
      !is_pow2_in(in.tile_k, 32, 128))
    return kPlanInvalid;
  const int nc = in.consumer_waves, np = in.producer_waves;
  if (in.split < 0 || in.split > 2) return kPlanInvalid;
  if (nc != 1 && nc != 4 && nc != 8) return kPlanUnsupported;
  // np == 0: the synchronous kernel (every wave loads and computes), ring
  // depth 1 (no overlap) or 2 (double-buffered).
  const int split = arrangement_split(nc, np, in.split);
  if (split < 0) return kPlanUnsupported;
  const int wm = in.tile_m / (nc >= 4 ? 2 : 1), wn = in.tile_n / (nc == 8 ? 4 : nc == 4 ? 2 : 1);
  // Wave tiles hold their fp32 accumulators in registers: up to 128 x 64 when
  // producer waves share the SIMDs, up to 128 x 128 when they do not.
  if (wm < 32 || wn < 32 || wm * wn > (np == 0 ? 128 * 128 : 128 * 64)) return kPlanUnsupported;
  if (np == 0 ? (in.stages < 1 || in.stages > 2) : (in.stages < 2 || in.stages > kPlanMaxStages))
    return kPlanInvalid;
  const int64_t stage = 2ll * (in.tile_m * in.tile_k + in.tile_k * in.tile_n);
  const int64_t lds = kPlanHeaderBytes + in.stages * stage;
  if (lds > kLdsLimit) return kPlanLdsOverflow;
  if (in.num_cus <= 0) return kPlanInvalid;
  // An empty problem (M, N or K = 0) launches no GEMM kernel: grid 0.  With
  // K = 0 and M N > 0, running it still writes C (the epilogue of a zero
  // product).
  if (in.M == 0 || in.N == 0 || in.K == 0) {
    out->block = 64 * (nc + np);
    out->lds_bytes = (int32_t)lds;
    out->tiles_m = (int32_t)((in.M + in.tile_m - 1) / in.tile_m);
    out->tiles_n = (int32_t)((in.N + in.tile_n - 1) / in.tile_n);
    out->iters = (int32_t)((in.K + in.tile_k - 1) / in.tile_k);
    out->split = split;
    out->group_m = 1;
    return kPlanOk;
  }
  // The paper's model assumes whole tiles.  Other shapes run the general
  // kernel variant (partial edge tiles, a partial last K-iteration), which
  // needs 16-byte rows of A and B (K and N multiples of 8) and producer waves.
  const bool ragged = (in.M % in.tile_m) || (in.N % in.tile_n) || (in.K % in.tile_k);
  if (ragged && (in.K % 8 || in.N % 8 || np == 0)) return kPlanNotDivisible;
  // byte offsets inside one tile panel (A, B and the C epilogue) are 32-bit
  if ((int64_t)in.tile_m * in.K * 2 >= (1ll << 31) || (int64_t)in.tile_k * in.N * 2 >= (1ll << 31) ||
      (int64_t)in.tile_m * in.N * 4 >= (1ll << 31))
    return kPlanInvalid;

  const int64_t tm = (in.M + in.tile_m - 1) / in.tile_m, tn = (in.N + in.tile_n - 1) / in.tile_n;
  if (tm * tn >= (1ll << 31)) return kPlanInvalid;
  const int tiles = (int)(tm * tn);
  const int waves = nc + np;
  int occ = in.wgs_per_cu;
  if (occ <= 0) {
    occ = (int)(kLdsLimit / lds);
    if (kMaxWavesPerCu / waves < occ) occ = kMaxWavesPerCu / waves;
    // the 4 SIMDs of a CU offer 4 x (waves per SIMD) wave slots, which the
    // waves of resident workgroups share
    const int by_regs = 4 * waves_per_simd_by_regs(in.vgprs, in.agprs) / waves;
    if (by_regs < occ) occ = by_regs;
    if (kMaxWgsPerCu < occ) occ = kMaxWgsPerCu;
  }
  if (occ < 1) occ = 1;
  // Of the occ workgroups a CU can hold, use the count u that minimises
  // rounds x u (workgroups sharing a CU progress about u times slower), the
  // largest on a tie: a last round that only part of the slots take costs a
  // whole round of the shared CUs (4096 tiles on 256 CUs: five resident
  // workgroups would need four rounds of five, four need four rounds of four).
  int use = 1;
  int64_t best = -1;
  for (int u = 1; u <= occ; ++u) {
    const int64_t slots_u = (int64_t)in.num_cus * u;
    const int64_t cost = ((tiles + slots_u - 1) / slots_u) * u;
    if (best < 0 || cost <= best) {
      best = cost;
      use = u;
    }
  }
  int64_t slots = (int64_t)in.num_cus * use;
  const int grid = (int)(tiles < slots ? tiles : slots);
  const int xcd_remap = (grid % 8 == 0) ? 1 : 0;  // the remap needs whole XCD groups

  // group_m: choose the tile-row group that minimises the A + B panel width a
  // single XCD touches per round.
  const int per_xcd = xcd_remap ? grid / 8 : grid;
  int best_gm = 1;
  int64_t best_cost = -1;
  for (int gm = 1; gm <= tm; gm *= 2) {
    const int64_t rows = gm;
    int64_t cols = (per_xcd + rows - 1) / rows;
    if (cols > tn) cols = tn;
    const int64_t cost = rows * in.tile_m + cols * in.tile_n;
    if (best_cost < 0 || cost < best_cost) {
      best_cost = cost;
      best_gm = gm;
    }
  }

  out->grid = grid;
  out->block = 64 * waves;
  out->lds_bytes = (int32_t)lds;
  out->tiles_m = (int32_t)tm;
  out->tiles_n = (int32_t)tn;
  out->tiles = tiles;
  out->rounds = (tiles + grid - 1) / grid;
  out->iters = (int32_t)((in.K + in.tile_k - 1) / in.tile_k);
  out->split = split;  // 0 for the synchronous kernel
  out->group_m = best_gm;
  out->xcd_remap = xcd_remap;
  out->ragged = ragged ? 1 : 0;
  return kPlanOk;
}

// Output tile computed by workgroup g in dispatch round r of a plan
// (returns false when that workgroup has no tile in that round).
inline bool scheduled_tile(const PlanOut& p, int g, int r, int* ti, int* tj) {
  if (g < 0 || g >= p.grid || r < 0) return false;
  const int slot = p.xcd_remap ? xcd_slot(g, p.grid) : g;
  const int64_t v = (int64_t)r * p.grid + slot;
  if (v >= p.tiles) return false;
  tile_coords((int)v, p.tiles_m, p.tiles_n, p.group_m, ti, tj);
  return true;
}

}  // namespace wsg
