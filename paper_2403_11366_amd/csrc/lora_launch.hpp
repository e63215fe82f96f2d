// Internal interface between the C ABI (argument checks, workspace layout) and
// the kernel launchers.  Shapes here have already been validated.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace lora {

// Rank padded to the matrix-core granularity of 16 (r in 1..64 -> 16..64).
inline int pad_rank(int64_t r) { return (int)((r + 15) / 16) * 16; }

// Token count padded to the 64-token chunk of the split-K reductions.
inline int64_t pad_tokens(int64_t m) { return (m + 63) / 64 * 64; }

// Output tiles of the two large GEMMs (tokens x features): 256x256 and 128x256
// run 8 waves (two per SIMD) as 2 x 4 waves of 128 x 64 and 64 x 64;
// 128x128 runs 4 waves of 64 x 64.
enum GemmTile { TILE_256x256 = 0, TILE_128x256 = 1, TILE_128x128 = 2 };

// Pick the output tile of the two large GEMMs for an M x N output.  Every
// workgroup of these kernels fills one compute unit (LDS-limited), so the
// kernel runs in ceil(tiles / 256) rounds on 256 CUs; the estimate is rounds
// times the per-tile work divided by a relative per-tile efficiency (larger
// tiles read less LDS and L2 per flop).
inline GemmTile choose_gemm_tile(int64_t M, int64_t N) {
  struct C { GemmTile t; int bm, bn; double eff; };
  const C cands[3] = {{TILE_256x256, 256, 256, 1.0}, {TILE_128x256, 128, 256, 0.9},
                      {TILE_128x128, 128, 128, 0.75}};
  GemmTile best = TILE_256x256;
  double best_cost = 1e300;
  for (const C& c : cands) {
    const int64_t tiles = ((M + c.bm - 1) / c.bm) * ((N + c.bn - 1) / c.bn);
    const double rounds = (double)((tiles + 255) / 256);
    const double cost = rounds * c.bm * c.bn / c.eff;
    if (cost < best_cost) { best_cost = cost; best = c.t; }
  }
  return best;
}

// Column split of one large GEMM with an M x N output: columns [0, n1) with
// tile t1, then columns [n1, N) with tile t2 in a second launch.  Taken when
// the split, whose second part is at most one round of 256 workgroups, is
// estimated more than 5% faster than the single tiling (estimate: rounds x
// tile area / relative efficiency, 1.0, 0.9 and 0.72 for 256x256, 128x256
// and 128x128, measured at 4096 x 5120 x 5120 and 4096 x 13824 x 5120).
// Typical cases: 4096 x 5120, where 640 tiles of 128x256 take three rounds
// and 256 tiles of 256x256 plus 256 tiles of 128x128 take two; 4096 x 13824,
// where 1728 tiles of 128x256 take seven rounds and 768 tiles of 256x256 plus
// 192 of 128x256 take four (forward 607-616 -> 537 us).  Among equal
// estimates the largest n1 wins.
// n1 == N: no split.
struct GemmSplit { GemmTile t1, t2; int64_t n1; };
inline GemmSplit plan_gemm_split(int64_t M, int64_t N) {
  struct C { GemmTile t; int bm, bn; double eff; };
  const C cands[3] = {{TILE_256x256, 256, 256, 1.0}, {TILE_128x256, 128, 256, 0.9},
                      {TILE_128x128, 128, 128, 0.72}};
  auto tiles = [&](const C& c, int64_t n) { return ((M + c.bm - 1) / c.bm) * ((n + c.bn - 1) / c.bn); };
  auto cost = [&](const C& c, int64_t n) { return (double)((tiles(c, n) + 255) / 256) * c.bm * c.bn / c.eff; };
  const GemmTile t0 = choose_gemm_tile(M, N);
  GemmSplit best{t0, t0, N};
  double best_cost = 0.95 * cost(cands[(int)t0], N);
  bool found = false;
  for (const C& c1 : cands)
    for (int64_t n1 = c1.bn; n1 < N; n1 += c1.bn)
      for (const C& c2 : cands) {
        if (tiles(c2, N - n1) > 256) continue;
        const double c = cost(c1, n1) + cost(c2, N - n1);
        if (c < best_cost || (found && c == best_cost && n1 > best.n1)) {
          best_cost = c;
          best = GemmSplit{c1.t, c2.t, n1};
          found = true;
        }
      }
  return best;
}

// Split-K plan of a token reduction out[t][c] = sum_i P[t][i] Q[i][c] over
// `cols` columns: columns in tiles of kRedCols, tokens in `splits` ranges of
// `span` tokens (a multiple of 64).  Splits are capped so the fp32 partial
// sums stay at most 1/8 of the bytes of Q (1/16 at rank 64, where fewer,
// longer splits measured faster: 7B down_proj backward 875 vs 891 us).
constexpr int kRedCols = 128;
struct RedPlan { int64_t span; int splits; int col_tiles; };
inline RedPlan plan_reduction(int64_t m, int64_t cols, int rp) {
  const int64_t mp = pad_tokens(m);
  const int col_tiles = (int)((cols + kRedCols - 1) / kRedCols);
  int64_t s = (1024 + col_tiles - 1) / col_tiles;
  int64_t cap = m / ((rp >= 64 ? 32 : 16) * (int64_t)rp);
  if (cap < 1) cap = 1;
  if (s > cap) s = cap;
  if (s > mp / 64) s = mp / 64;
  if (s < 1) s = 1;
  int64_t span = (mp + s - 1) / s;
  span = (span + 63) / 64 * 64;
  const int splits = (int)((mp + span - 1) / span);
  return RedPlan{span, splits, col_tiles};
}

// Backward workspace, byte offsets of each region (256-byte aligned).
struct BwdLayout {
  size_t ut2;    // Ut2  [RP][mp]     bf16: U^T
  size_t du2;    // dU2  [mp][2RP]    bf16: dU as high part (cols 0..RP) and low part
  size_t dut2;   // dUt2 [RP][mp]     bf16: s dU^T
  size_t pb;     // partial dB^T [splits_b][RP][n] fp32
  size_t pa;     // partial dA   [splits_a][RP][k] fp32
  size_t total;
  RedPlan plan_b, plan_a;
  int rp;
  int64_t mp;
};

inline size_t align256(size_t x) { return (x + 255) / 256 * 256; }

inline BwdLayout bwd_layout(int64_t m, int64_t n, int64_t k, int64_t r) {
  BwdLayout L;
  L.rp = pad_rank(r);
  L.mp = pad_tokens(m);
  L.plan_b = plan_reduction(m, n, L.rp);
  L.plan_a = plan_reduction(m, k, L.rp);
  const size_t rp = (size_t)L.rp, mp = (size_t)L.mp;
  size_t off = 0;
  L.ut2 = off;  off = align256(off + rp * mp * 2);
  L.du2 = off;  off = align256(off + mp * 2 * rp * 2);
  L.dut2 = off; off = align256(off + rp * mp * 2);
  L.pb = off;   off = align256(off + (size_t)L.plan_b.splits * rp * (size_t)n * 4);
  L.pa = off;   off = align256(off + (size_t)L.plan_a.splits * rp * (size_t)k * 4);
  L.total = off;
  return L;
}

// Workspace of the fused backward (rank <= 16): dUt2 [16][mp] bf16 (s dU^T,
// written by the dX launch for the dA reduction), the dB^T
// partials of the dX launch [tiles_m][16][n] fp32 (one per 128-token tile
// row) and the dA partials of the token reduction [splits][16][k] fp32.
struct BwdFusedLayout {
  size_t dut2, pb, pa, total;
  RedPlan plan_a;
  int64_t mp;
  int tiles_m;
};

inline BwdFusedLayout bwd_fused_layout(int64_t m, int64_t n, int64_t k, int64_t r) {
  (void)r;
  BwdFusedLayout L;
  L.mp = pad_tokens(m);
  L.tiles_m = (int)((m + 127) / 128);
  L.plan_a = plan_reduction(m, k, 16);
  size_t off = 0;
  L.dut2 = off; off = align256(off + 16 * (size_t)L.mp * 2);
  L.pb = off;   off = align256(off + (size_t)L.tiles_m * 16 * (size_t)n * 4);
  L.pa = off;   off = align256(off + (size_t)L.plan_a.splits * 16 * (size_t)k * 4);
  L.total = off;
  return L;
}

struct FwdArgs {
  const uint16_t *X, *W, *A, *B;
  uint16_t* Y;
  float* U;
  int64_t m, n, k, r;
  float s;
  const uint8_t* keep = nullptr;   // dropout keep bits [m][k/8], or none
  float inv_keep = 1.0f;           // 1 / (1 - p)
  bool u_ready = false;            // U already in place (second launch of a column split)
};

struct BwdArgs {
  const uint16_t *dY, *X, *W, *A, *B;
  const float* U;
  uint16_t* dX;
  float *dA, *dB;
  char* ws;
  int64_t m, n, k, r;
  float s;
  const uint8_t* keep = nullptr;   // dropout keep bits [m][k/8], or none
  float inv_keep = 1.0f;           // 1 / (1 - p)
};

// Projections that share one input X (q, k, v of an attention block; gate and
// up of an MLP): at most kMaxGroup, one rank and alpha for the group.
constexpr int kMaxGroup = 8;

// Kernel argument (by value) of the grouped forward: per-projection pointers;
// the output tiles of all projections form one grid, projection g owning
// column tiles tile0[g] .. tile0[g+1]-1.
struct FwdGroup {
  const uint16_t* W[kMaxGroup];
  const uint16_t* A[kMaxGroup];
  const uint16_t* B[kMaxGroup];
  uint16_t* Y[kMaxGroup];
  float* U[kMaxGroup];
  int n[kMaxGroup];
  int tile0[kMaxGroup];
  int count;
};

struct GroupFwdArgs {
  const uint16_t* X;
  int count;
  int64_t n[kMaxGroup];
  const uint16_t *W[kMaxGroup], *A[kMaxGroup], *B[kMaxGroup];
  uint16_t* Y[kMaxGroup];
  float* U[kMaxGroup];
  int64_t m, k, r;
  float s;
};

struct GroupBwdArgs {
  const uint16_t* X;
  int count;
  int64_t n[kMaxGroup];
  const uint16_t *dY[kMaxGroup], *W[kMaxGroup], *A[kMaxGroup], *B[kMaxGroup];
  const float* U[kMaxGroup];
  uint16_t* dX;
  float *dA[kMaxGroup], *dB[kMaxGroup];
  char* ws;
  int64_t m, k, r;
  float s;
};

// Grouped backward workspace: one backward layout per projection, back to
// back; for groups of three or more whose padded ranks add up to at most 64
// (q, k, v at rank 16 or less), also a stacked dU^T of all members and the
// partials of one dA reduction over X for the whole group (13B q, k, v: 13.4
// us instead of three 6.4 us passes; for a pair such as gate, up the stacked
// pass measured no faster than two, 14.8 vs 12.8 us, so pairs keep theirs):
//   dut_stack [RPT][mp] bf16, RPT = count x RP: member g's rows at g RP ..
//   pa_stack  [splits][RPT][k] fp32 partial dA of all members
// (the members' own dUt2 and pa regions then stay unused).
struct GroupBwdLayout {
  BwdLayout L[kMaxGroup];
  size_t off[kMaxGroup];
  bool stacked;
  int rpt;
  size_t dut_stack, pa_stack;
  RedPlan plan_a;
  size_t total;
};

constexpr int kMaxStackedRank = 64;

inline GroupBwdLayout group_bwd_layout(int count, const int64_t* n, int64_t m, int64_t k, int64_t r) {
  GroupBwdLayout G{};
  size_t off = 0;
  for (int g = 0; g < count; ++g) {
    G.L[g] = bwd_layout(m, n[g], k, r);
    G.off[g] = off;
    off = align256(off + G.L[g].total);
  }
  G.rpt = count * pad_rank(r);
  G.stacked = count >= 3 && G.rpt <= kMaxStackedRank;
  if (G.stacked) {
    const size_t mp = (size_t)pad_tokens(m);
    G.plan_a = plan_reduction(m, k, G.rpt);
    G.dut_stack = off;
    off = align256(off + (size_t)G.rpt * mp * 2);
    G.pa_stack = off;
    off = align256(off + (size_t)G.plan_a.splits * G.rpt * (size_t)k * 4);
  }
  G.total = off;
  return G;
}

// Dropout keep mask drawn on the device (lora_mask.hip).
struct MaskArgs {
  uint64_t seed, offset;   // Philox key word 0 and the first counter
  uint32_t thr;            // keep iff the 16-bit draw is below thr (thr <= 2^16)
  uint8_t* keep;           // [m, k/8] packed bits
  int64_t m, k;
};

hipError_t launch_keep_mask(const MaskArgs& a, hipStream_t st);

struct MergeArgs {
  const uint16_t* W;       // [n, k]
  const uint16_t *A, *B;   // [r, k], [n, r]
  uint16_t* Wout;          // [n, k], may equal W
  int64_t n, k, r;
  float ss;                // sign * alpha / r
};

// Scratch of lora_linear_bwd_noalloc: a fixed device array per GPU holding
// the backward workspace (the largest Llama-2 projection shapes need 21 MiB).
constexpr size_t kNoAllocScratchBytes = size_t(32) << 20;

hipError_t launch_fwd(const FwdArgs& a, hipStream_t st);
hipError_t launch_bwd_noalloc(const BwdArgs& a, hipStream_t st);   // workspace: the library's scratch array
hipError_t launch_merge(const MergeArgs& a, hipStream_t st);
hipError_t launch_bwd(const BwdArgs& a, hipStream_t st);
hipError_t launch_bwd_fused(const BwdArgs& a, hipStream_t st);   // rank <= 16, no dropout
hipError_t launch_fwd_group(const GroupFwdArgs& a, hipStream_t st);
hipError_t launch_bwd_group(const GroupBwdArgs& a, hipStream_t st);

}  // namespace lora
