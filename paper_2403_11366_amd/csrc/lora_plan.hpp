// Launch plans: the one place that decides which kernel instantiations a
// call runs, with which grid and over which output columns.  The launchers
// in lora_fwd.hip, lora_bwd.hip and lora_merge.hip execute these plans, and
// lora_linear_plan() in the C ABI reports them (host only, no GPU needed), so
// tools and tests see exactly what a call will launch.
#pragma once

#include <stdint.h>
#include <stdio.h>

#include <type_traits>

#include "lora_launch.hpp"

namespace lora {

enum KernelId : int {
  K_UPASS = 0,     // lora_u_kernel<RP, TPW, KEEP>: U = X A^T on its own (rank > 16, and under dropout)
  K_FWD = 1,       // lora_fwd_kernel<BM, BN, WM, WN, RP, GRP, UPRE, KFULL, DMA>
  K_FWD_KS = 2,    // lora_fwd_ks_kernel<GRP, KFULL, DMA, UPRE>
  K_DU = 3,        // lora_bwd_du_dma_kernel<RP, TPW> (r a multiple of 8), else lora_bwd_du_kernel<RP, TPW>
  K_TOKRED = 4,    // lora_tokred_dma_kernel<RP>, or lora_tokred_kernel<RP, true> with a keep mask
  K_DX = 5,        // lora_bwd_dx_kernel<BM, BN, WM, WN, RP, DROP, GRP, FULL>
  K_DXF = 6,       // lora_bwd_dxf_kernel<FULL, FASTB>
  K_FINALIZE = 7,  // lora_finalize_kernel
  K_MERGE = 8,     // lora_merge_kernel<RP, 64>
  K_MASK = 9,      // lora_keep_mask_kernel: the dropout keep mask from the counter-based generator
};

// One kernel launch.  Fields a kernel does not use stay zero / false.
struct Launch {
  KernelId id;
  int bm, bn, wm, wn;          // GEMM output tile and wave layout
  int rp;                      // padded rank the instantiation is built for
  int tpw;                     // tokens per workgroup (U pass, dU)
  bool drop, grp, upre, full, dma, fastb;   // template switches (see KernelId)
  int64_t col_begin, col_end;  // GEMM output columns [col_begin, col_end)
  int tiles_m, tiles_n;        // GEMM tile grid (the grid is their product)
  int64_t grid;                // workgroups
  int block;                   // threads per workgroup
  bool finalize;               // dX: the workgroups' tails finalize dA and dB
  int member;                  // grouped calls: the projection a per-member launch serves
  int part;                    // token reductions: 0 dB and dA, 1 dB only, 2 a group's stacked dA
};

constexpr int kMaxLaunches = 4 + 2 * kMaxGroup;

struct Plan {
  int count = 0;
  Launch l[kMaxLaunches];
  void add(const Launch& x) {
    if (count < kMaxLaunches) l[count++] = x;
  }
};

inline Launch blank_launch(KernelId id) {
  Launch x{};
  x.id = id;
  return x;
}

// Forward instantiations exist for padded ranks 16, 32 and 64 (r = 33 .. 64
// all use 64); backward ones for 16, 32, 48 and 64.
inline int fwd_rank(int64_t r) { return r <= 16 ? 16 : (r <= 32 ? 32 : 64); }

inline void tile_dims(GemmTile t, int& bm, int& bn, int& wm, int& wn) {
  switch (t) {
    case TILE_256x256: bm = 256; bn = 256; wm = 2; wn = 4; break;
    case TILE_128x256: bm = 128; bn = 256; wm = 2; wn = 4; break;
    default: bm = 128; bn = 128; wm = 2; wn = 2; break;
  }
}

inline Launch gemm_launch(KernelId id, GemmTile t, int64_t M, int64_t col_begin, int64_t col_end, int tiles_n) {
  Launch x = blank_launch(id);
  tile_dims(t, x.bm, x.bn, x.wm, x.wn);
  x.col_begin = col_begin;
  x.col_end = col_end;
  x.tiles_m = (int)((M + x.bm - 1) / x.bm);
  x.tiles_n = tiles_n >= 0 ? tiles_n : (int)((col_end - col_begin + x.bn - 1) / x.bn);
  x.grid = (int64_t)x.tiles_m * x.tiles_n;
  x.block = 64 * x.wm * x.wn;
  return x;
}

// Forward GEMM launch(es) for output columns [cb, ce) with tile t.  `first`:
// the launch whose range starts at column 0 (it writes U, or the U pass runs
// before it).  U comes from the U pass for single projections of rank above
// 16, on the 256 x 256 tile (where recomputing rank 16 in every tile costs
// more than the pass: 7B up_proj forward 387 -> 371 us), and under dropout
// (drop: the pass applies the keep mask, and the GEMM then runs exactly as
// without dropout); otherwise the tile computes it.  For a group, tiles_n is
// the summed column tiles.
inline void plan_fwd_part(Plan& p, GemmTile t, int64_t m, int64_t k, int64_t r, int64_t cb, int64_t ce,
                          bool first, bool drop, bool grp, int tiles_n) {
  const bool kfull = k % 64 == 0;
  const bool upre = !grp && (drop || fwd_rank(r) >= 32 || t == TILE_256x256);
  if (upre && first) {
    Launch u = blank_launch(K_UPASS);
    u.rp = fwd_rank(r);
    u.drop = drop;
    // 32 tokens per workgroup (A read half as often) unless that leaves
    // compute units idle, then 16, then 8
    u.tpw = (m + 31) / 32 >= 256 ? 32 : ((m + 15) / 16 >= 256 ? 16 : 8);
    u.grid = (m + u.tpw - 1) / u.tpw;
    u.block = 256;
    p.add(u);
  }
  Launch x = gemm_launch(K_FWD, t, m, cb, ce, tiles_n);
  x.grp = grp;
  x.upre = upre;
  x.full = kfull;
  if (t == TILE_128x256 && r <= 16) {
    // k-split tile; single-round launches copy their stages straight into LDS
    x.id = K_FWD_KS;
    x.rp = 16;
    x.dma = kfull && !grp && x.grid <= 256;
    p.add(x);
    return;
  }
  x.rp = fwd_rank(r);
  x.dma = t == TILE_256x256 && kfull;
  p.add(x);
}

// lora_linear_fwd / lora_linear_fwd_dropout (the same tiles and column split;
// under dropout the U pass applies the mask).
inline Plan plan_fwd(int64_t m, int64_t n, int64_t k, int64_t r, bool drop) {
  Plan p;
  const GemmSplit s = plan_gemm_split(m, n);
  plan_fwd_part(p, s.t1, m, k, r, 0, s.n1, true, drop, false, -1);
  if (s.n1 < n) plan_fwd_part(p, s.t2, m, k, r, s.n1, n, false, drop, false, -1);
  return p;
}

// lora_linear_group_fwd: one launch over the output tiles of all members, the
// tile chosen for m x (sum of n).  A group of one is the single projection.
inline Plan plan_group_fwd(int count, const int64_t* n, int64_t m, int64_t k, int64_t r) {
  if (count == 1) return plan_fwd(m, n[0], k, r, false);
  int64_t ntot = 0;
  for (int g = 0; g < count; ++g) ntot += n[g];
  const GemmTile t = choose_gemm_tile(m, ntot);
  int bm, bn, wm, wn;
  tile_dims(t, bm, bn, wm, wn);
  int tiles_n = 0;
  for (int g = 0; g < count; ++g) tiles_n += (int)((n[g] + bn - 1) / bn);
  Plan p;
  plan_fwd_part(p, t, m, k, r, 0, 0, true, false, true, tiles_n);
  return p;
}

// dX GEMM launch over columns [cb, ce).  FULL (no bound checks on the n-stage
// loads) needs every n a multiple of 64 and whole column tiles; the 256-wide
// FULL tiles copy their stages straight into LDS.  The 256 x 256 tile runs
// only FULL: its register-staged variant keeps values in scratch beside the
// 128 accumulators, so without FULL the range takes the 128 x 256 tile.
inline void plan_dx_part(Plan& p, GemmTile t, int64_t m, int rp, int64_t cb, int64_t ce, bool n_whole, bool drop,
                         bool grp, bool finalize) {
  int bm, bn, wm, wn;
  tile_dims(t, bm, bn, wm, wn);
  bool full = n_whole && (ce - cb) % bn == 0;
  if (t == TILE_256x256 && !full) {
    t = TILE_128x256;
    tile_dims(t, bm, bn, wm, wn);
    full = n_whole && (ce - cb) % bn == 0;
  }
  Launch x = gemm_launch(K_DX, t, m, cb, ce, -1);
  x.rp = rp;
  x.drop = drop;
  x.grp = grp;
  x.full = full;
  x.dma = full && bn == 256;
  x.finalize = finalize;
  p.add(x);
}

inline Launch du_launch(const BwdLayout& L, int64_t r, int member) {
  Launch x = blank_launch(K_DU);
  x.rp = L.rp;
  x.fastb = r % 8 == 0;   // 16-byte pieces of B then lie inside one row: the direct-to-LDS kernel
  // the most tokens per workgroup (each reads all of B) that still leaves no
  // compute unit idle; 32 tokens from padded rank 32 on, where B is at least
  // as many bytes per workgroup as 16 tokens of dY
  x.tpw = L.mp / 16 < 256 ? 8 : (L.rp >= 32 && L.mp / 32 >= 256 ? 32 : 16);
  x.grid = L.mp / x.tpw;
  x.block = x.fastb ? 256 : 512;
  x.member = member;
  return x;
}

// Token reductions run four waves per workgroup.
inline int tokred_threads(int) { return 256; }

inline Launch tokred_launch(const BwdLayout& L, bool keep, int member, int part = 0) {
  Launch x = blank_launch(K_TOKRED);
  x.rp = L.rp;
  x.drop = keep;
  x.grid = (int64_t)L.plan_b.col_tiles * L.plan_b.splits + (part == 0 ? (int64_t)L.plan_a.col_tiles * L.plan_a.splits : 0);
  x.block = tokred_threads(x.rp);
  x.member = member;
  x.part = part;
  return x;
}

// lora_linear_bwd / lora_linear_bwd_dropout: dU, the token reductions, then
// the dX GEMM (its columns split between two launches as for the forward; the
// first one's tails finalize dA and dB).
inline Plan plan_bwd(int64_t m, int64_t n, int64_t k, int64_t r, bool drop) {
  const BwdLayout L = bwd_layout(m, n, k, r);
  Plan p;
  p.add(du_launch(L, r, 0));
  p.add(tokred_launch(L, drop, 0));
  const bool n_whole = n % 64 == 0;
  if (drop) {
    const GemmTile t = choose_gemm_tile(m, k) == TILE_128x128 ? TILE_128x128 : TILE_128x256;
    plan_dx_part(p, t, m, L.rp, 0, k, n_whole, true, false, true);
    return p;
  }
  const GemmSplit s = plan_gemm_split(m, k);
  plan_dx_part(p, s.t1, m, L.rp, 0, s.n1, n_whole, false, false, true);
  if (s.n1 < k) plan_dx_part(p, s.t2, m, L.rp, s.n1, k, n_whole, false, false, false);
  return p;
}

// lora_linear_group_bwd: per member dU and the token reductions, then one dX
// launch over the concatenated contraction (split like the single one).  For
// groups of three or more whose padded ranks add up to at most 64 the dA
// reductions of all members run as one (a stacked rank over one pass of X)
// after the members' dB reductions.
inline Plan plan_group_bwd(int count, const int64_t* n, int64_t m, int64_t k, int64_t r) {
  if (count == 1) return plan_bwd(m, n[0], k, r, false);
  const GroupBwdLayout G = group_bwd_layout(count, n, m, k, r);
  Plan p;
  bool n_whole = true;
  for (int g = 0; g < count; ++g) {
    p.add(du_launch(G.L[g], r, g));
    p.add(tokred_launch(G.L[g], false, g, G.stacked ? 1 : 0));
    n_whole = n_whole && n[g] % 64 == 0;
  }
  if (G.stacked) {
    Launch x = blank_launch(K_TOKRED);
    x.rp = G.rpt;
    x.grid = (int64_t)G.plan_a.col_tiles * G.plan_a.splits;
    x.block = tokred_threads(x.rp);
    x.member = -1;
    x.part = 2;
    p.add(x);
  }
  const int rp = G.L[0].rp;
  const GemmSplit s = plan_gemm_split(m, k);
  plan_dx_part(p, s.t1, m, rp, 0, s.n1, n_whole, false, true, true);
  if (s.n1 < k) plan_dx_part(p, s.t2, m, rp, s.n1, k, n_whole, false, true, false);
  return p;
}

// lora_linear_bwd_fused (r <= 16): the dX launch that also forms dU and the dB
// partials, the dA token reduction, the finalize.
inline Plan plan_bwd_fused(int64_t m, int64_t n, int64_t k, int64_t r) {
  const BwdFusedLayout L = bwd_fused_layout(m, n, k, r);
  Plan p;
  Launch x = gemm_launch(K_DXF, TILE_128x256, m, 0, k, -1);
  x.rp = 16;
  x.fastb = r % 8 == 0;
  x.full = x.fastb && n % 64 == 0 && k % 256 == 0;
  p.add(x);
  Launch t = blank_launch(K_TOKRED);
  t.rp = 16;
  t.grid = (int64_t)L.plan_a.col_tiles * L.plan_a.splits;
  t.block = tokred_threads(t.rp);
  p.add(t);
  Launch f = blank_launch(K_FINALIZE);
  const int64_t total = n * r + r * k;
  f.grid = (total + 255) / 256 < 2048 ? (total + 255) / 256 : 2048;
  f.block = 256;
  p.add(f);
  return p;
}

// lora_linear_merge: 64 x 128 tiles of W.
constexpr int kMergeRows = 64;
inline Plan plan_merge(int64_t n, int64_t k, int64_t r) {
  Plan p;
  Launch x = blank_launch(K_MERGE);
  x.rp = pad_rank(r);
  x.tiles_m = (int)((n + kMergeRows - 1) / kMergeRows);
  x.tiles_n = (int)((k + 127) / 128);
  x.grid = (int64_t)x.tiles_m * x.tiles_n;
  x.block = 256;
  p.add(x);
  return p;
}

// lora_dropout_keep_mask: kMaskBytesPerThread mask bytes (two per generator
// block) per thread.
constexpr int kMaskBytesPerThread = 4;
inline Plan plan_keep_mask(int64_t m, int64_t k) {
  Plan p;
  Launch x = blank_launch(K_MASK);
  x.grid = (m * (k / 8) + kMaskBytesPerThread * 256 - 1) / (kMaskBytesPerThread * 256);
  x.block = 256;
  p.add(x);
  return p;
}

// The instantiation's name as profilers print it (demangled, without the
// argument list).
inline void launch_name(const Launch& x, char* buf, size_t len) {
  auto b = [](bool v) { return v ? "true" : "false"; };
  switch (x.id) {
    case K_UPASS: snprintf(buf, len, "lora::lora_u_kernel<%d, %d, %s>", x.rp, x.tpw, b(x.drop)); break;
    case K_FWD:
      snprintf(buf, len, "lora::lora_fwd_kernel<%d, %d, %d, %d, %d, %s, %s, %s, %s>", x.bm, x.bn, x.wm, x.wn, x.rp,
               b(x.grp), b(x.upre), b(x.full), b(x.dma));
      break;
    case K_FWD_KS:
      snprintf(buf, len, "lora::lora_fwd_ks_kernel<%s, %s, %s, %s>", b(x.grp), b(x.full), b(x.dma), b(x.upre));
      break;
    case K_DU:
      snprintf(buf, len, x.fastb ? "lora::lora_bwd_du_dma_kernel<%d, %d>" : "lora::lora_bwd_du_kernel<%d, %d>", x.rp,
               x.tpw);
      break;
    case K_TOKRED:
      if (x.drop) snprintf(buf, len, "lora::lora_tokred_kernel<%d, true>", x.rp);
      else snprintf(buf, len, "lora::lora_tokred_dma_kernel<%d>", x.rp);
      break;
    case K_DX:
      snprintf(buf, len, "lora::lora_bwd_dx_kernel<%d, %d, %d, %d, %d, %s, %s, %s>", x.bm, x.bn, x.wm, x.wn, x.rp,
               b(x.drop), b(x.grp), b(x.full));
      break;
    case K_DXF: snprintf(buf, len, "lora::lora_bwd_dxf_kernel<%s, %s>", b(x.full), b(x.fastb)); break;
    case K_FINALIZE: snprintf(buf, len, "lora::lora_finalize_kernel"); break;
    case K_MERGE: snprintf(buf, len, "lora::lora_merge_kernel<%d, %d>", x.rp, kMergeRows); break;
    case K_MASK: snprintf(buf, len, "lora::lora_keep_mask_kernel"); break;
  }
}

// Runtime switches to compile-time constants for the launchers' dispatch.
template <typename F>
inline hipError_t with_bool(bool v, F&& f) {
  return v ? f(std::true_type{}) : f(std::false_type{});
}

template <int... Vs, typename F>
inline hipError_t with_int(int v, F&& f) {
  hipError_t e = hipErrorInvalidValue;
  (void)((v == Vs ? (e = f(std::integral_constant<int, Vs>{}), true) : false) || ...);
  return e;
}

// The GEMM tile of a launch as one code: 0 = 256x256, 1 = 128x256, 2 = 128x128.
inline int tile_code(const Launch& x) { return x.bm == 256 ? 0 : (x.bn == 256 ? 1 : 2); }

}  // namespace lora
