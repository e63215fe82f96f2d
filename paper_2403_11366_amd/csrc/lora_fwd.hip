// Forward of the LoRA-adapted linear layer (Eq. 1 of JORA, Section 3):
//   U = X A^T,   Y = X W^T + s U B^T,   s = alpha / r.
//
// Kernels (one launch per call; a U pass before it for rank > 16, on the
// 256 x 256 tile and under dropout, and a second GEMM launch when the columns
// are split between two tiles):
//   lora_fwd_ks_kernel  the 128 x 256 tile for rank <= 16 (the 7B q_proj
//                       shape): wave pairs split the k substeps of each
//                       stage, see its own comment.
//   lora_fwd_kernel     the other tiles (256 x 256, 128 x 256, 128 x 128)
//                       and grouped launches; described below.
//   lora_u_kernel       U = X A^T on its own (under dropout with the keep
//                       mask applied), followed by a GEMM tile without U
//                       columns.
// A launch covers the output columns from n_begin on (plan_gemm_split);
// the launch whose range starts at column 0 writes U.
//
// lora_fwd_kernel: each workgroup owns a BM x BN tile of Y (BM tokens x BN output
// features) and walks k in stages of 64.  Per stage it stages three
// k-contiguous tiles in LDS -- X[BM rows], W[BN rows] and the LoRA
// down-projection A padded to RP rows -- so each X tile is read once and
// feeds both the W columns and the r extra "U columns".  Global loads run two
// stages ahead in registers and are stored to the free LDS buffer piece by
// piece during the stage before their use (one barrier per stage).
//
// Matrix-core products use v_mfma_f32_32x32x16_bf16 and are formed transposed
// (W and A as the A operand, X as the B operand), so each lane's accumulator
// holds runs of 4 consecutive output features of one token.
//
// The U columns of a token fragment are accumulated by the waves that share
// it (each wave owns fixed fragments and k substeps, so the U products are
// branch-free).  After the k loop the epilogue parks U in LDS, writes it out
// (first tile column only), and adds s U B^T to the accumulators with a
// short matrix-core pass over t in which s U enters as a bf16 high part and
// a bf16 low part, then rounds Y to bf16 and stores it through a per-wave
// LDS block (store_block_32x64) so that stores write whole 128-byte rows.
#include <type_traits>

#include "lora_device.hpp"
#include "lora_launch.hpp"
#include "lora_plan.hpp"

namespace lora {

// With GRP the grid covers the output tiles of a group of projections that
// read the same X (FwdGroup): each workgroup first selects its projection's
// W, A, B, Y, U and n, then runs exactly the single-projection tile.
//
// With UPRE, U = X A^T has been computed by lora_u_kernel: the k loop stages
// no A rows and runs no U products, and the epilogue reads U back.
//
// KFULL (k a multiple of 64): the loads carry no k-bound checks, and below the
// 256 x 256 tile the stages run in pairs with compile-time LDS buffers.
//
// DMA (the 256 x 256 tile with KFULL): each stage is copied from
// global memory straight into the free LDS buffer at the top of the stage
// before it (one 16-byte chunk per lane per copy instruction, the swizzle
// applied to the global addresses), with no staging registers; the stage's
// closing barrier waits for those copies (copy_barrier).  With UPRE as well,
// the fragment reads are issued as inline assembly, two register sets deep
// (see the loop below).
template <int BM, int BN, int WM, int WN, int RP, bool GRP, bool UPRE, bool KFULL, bool DMA>
__global__ __launch_bounds__(64 * WM * WN) void lora_fwd_kernel(
    const u16* __restrict__ X, const u16* __restrict__ W, const u16* __restrict__ A,
    const u16* __restrict__ B, u16* __restrict__ Y,
    float* __restrict__ U, int m, int n, int k, int r, float s, int tiles_m, int tiles_n,
    int n_begin, FwdGroup grp) {
  constexpr int NW = WM * WN;
  constexpr int NT = 64 * NW;
  constexpr int WTI = BM / WM, WTJ = BN / WN;   // tokens, features per wave
  constexpr int FI = WTI / 32;                   // token fragments (B operand)
  constexpr int FJ = WTJ / 32;                   // feature fragments (A operand)
  // U work.  For RP = 16 (rank <= 16) U runs on v_mfma_f32_16x16x32_bf16: a
  // wave row's WTI tokens form WTI/16 groups of 16, GPW per wave, each over
  // the 32-wide halves of the stage (substeps 0-1 and 2-3).  For RP >= 32 it
  // runs on the 32x32x16 form: the FI token fragments of a wave row are shared
  // by its WN waves; with FI >= WN each wave owns FUW fragments, with FI < WN
  // NDUP waves share a fragment and split its k substeps (partial sums added in
  // the epilogue).
  constexpr bool U16 = RP == 16;
  constexpr int FT = U16 ? 1 : RP / 32;          // U row fragments (A operand)
  constexpr int FUW = U16 ? 1 : (FI >= WN ? FI / WN : 1);
  constexpr int NDUP = U16 ? 1 : (FI >= WN ? 1 : WN / FI);
  constexpr int GPW = U16 ? (WTI / 16) / WN : 1;
  constexpr int RPS = UPRE ? 0 : RP;             // A rows staged per stage
  constexpr int ROWS = BM + BN + RPS;            // 128-byte rows per 64-wide stage
  constexpr int STAGE = ROWS * 128;
  constexpr int CX = BM * 8, CW = BN * 8, CA = RPS * 8;  // 16-byte chunks per region
  constexpr int LX = (CX + NT - 1) / NT, LW = (CW + NT - 1) / NT, LA = UPRE ? 1 : (CA + NT - 1) / NT;
  static_assert(WTI % 32 == 0 && WTJ % 32 == 0 && (U16 || RP % 32 == 0), "32x32 fragments");
  static_assert(!U16 || ((WTI / 16) % WN == 0 && GPW >= 1), "U groups split evenly");
  static_assert(CX % 64 == 0 && CW % 64 == 0 && CA % 64 == 0, "regions end on wave boundaries");
  static_assert(U16 || (FI >= WN ? FI % WN == 0 : WN % FI == 0), "U fragments split evenly");
  static_assert(4 % NDUP == 0, "U substeps split evenly");
  static_assert(2 * STAGE <= 160 * 1024, "LDS budget");
  constexpr int RPU = RP + 4, RPB = RP + 8;     // padded row lengths of the epilogue's U and B copies
  constexpr int NUS = UPRE ? 1 : NDUP;           // U copies in the epilogue
  static_assert(NUS * BM * RPU * 4 + BN * RPB * 2 <= 2 * STAGE, "epilogue LDS reuse");

  __shared__ __attribute__((aligned(1024))) char smem[2 * STAGE];

  int tm, tn;
  tile_coords(tiles_m, tiles_n, 8, (int)blockIdx.x, tm, tn);
  if (GRP) {   // projection of this column tile (uniform; compile-time indices only)
    int sel = 0;
#pragma unroll
    for (int q = 1; q < kMaxGroup; ++q)
      if (q < grp.count && tn >= grp.tile0[q]) sel = q;
#pragma unroll
    for (int q = 0; q < kMaxGroup; ++q)
      if (q == sel) {
        W = grp.W[q]; A = grp.A[q]; B = grp.B[q]; Y = grp.Y[q]; U = grp.U[q];
        n = grp.n[q];
        tn -= grp.tile0[q];
      }
  }
  const int m0 = tm * BM, n0 = n_begin + tn * BN;
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = uniform(tid >> 6);
  const int wm = wave / WN, wn = wave % WN;
  const int g = lane >> 5, c32 = lane & 31;
  const int g16 = lane >> 4, c16 = lane & 15;
  const int udup = NDUP > 1 ? wn / FI : 0;       // which share of the U substeps

  const uint32_t rowbytes = (uint32_t)k * 2;
  const __amdgpu_buffer_rsrc_t rsX = make_rsrc(X + (size_t)m0 * k, (uint64_t)min(BM, m - m0) * rowbytes);
  const __amdgpu_buffer_rsrc_t rsW = make_rsrc(W + (size_t)n0 * k, (uint64_t)min(BN, n - n0) * rowbytes);
  const __amdgpu_buffer_rsrc_t rsA = make_rsrc(A, (uint64_t)r * rowbytes);

  // Register staging of one k-block of the three regions: thread chunk
  // q = tid + i NT of a region is row q/8, k-chunk q%8 (coalesced 128-byte
  // rows).  The block moves in four pieces, one per 16-wide substep of the
  // stage that stores it: 0 = X rows, 1 and 2 = the two halves of the W rows,
  // 3 = A rows.
  constexpr int LW1 = (LW + 1) / 2;
  int4v gx[LX], gw[LW], ga[LA];
  auto gload = [&](int kb, int piece) LORA_INLINE {
    const int k0 = kb * 64;
    if (piece == 0) {
#pragma unroll
      for (int i = 0; i < LX; ++i) {
        const int q = tid + i * NT;
        if (CX % NT != 0 && wave * 64 + i * NT >= CX) break;   // wave-uniform
        const int kk = k0 + 8 * (q & 7);
        gx[i] = buf_load16(rsX, (KFULL || kk < k) ? (uint32_t)(q >> 3) * rowbytes + (uint32_t)kk * 2 : kOOB);
      }
    } else if (piece <= 2) {
#pragma unroll
      for (int i = piece == 1 ? 0 : LW1; i < (piece == 1 ? LW1 : LW); ++i) {
        const int q = tid + i * NT;
        if (CW % NT != 0 && wave * 64 + i * NT >= CW) break;   // wave-uniform
        const int kk = k0 + 8 * (q & 7);
        gw[i] = buf_load16(rsW, (KFULL || kk < k) ? (uint32_t)(q >> 3) * rowbytes + (uint32_t)kk * 2 : kOOB);
      }
    } else if (!UPRE) {
#pragma unroll
      for (int i = 0; i < LA; ++i) {
        const int q = tid + i * NT;
        if (CA % NT != 0 && wave * 64 + i * NT >= CA) break;   // wave-uniform
        const int kk = k0 + 8 * (q & 7);
        ga[i] = buf_load16(rsA, (KFULL || kk < k) ? (uint32_t)(q >> 3) * rowbytes + (uint32_t)kk * 2 : kOOB);
      }
    }
  };
  auto swrite = [&](int buf, int piece) LORA_INLINE {
    char* sb = smem + buf * STAGE;
    if (piece == 0) {
#pragma unroll
      for (int i = 0; i < LX; ++i) {
        const int q = tid + i * NT;
        if (CX % NT != 0 && wave * 64 + i * NT >= CX) break;   // wave-uniform
        *reinterpret_cast<int4v*>(sb + kc_offset(q >> 3, q & 7)) = gx[i];
      }
    } else if (piece <= 2) {
#pragma unroll
      for (int i = piece == 1 ? 0 : LW1; i < (piece == 1 ? LW1 : LW); ++i) {
        const int q = tid + i * NT;
        if (CW % NT != 0 && wave * 64 + i * NT >= CW) break;   // wave-uniform
        *reinterpret_cast<int4v*>(sb + BM * 128 + kc_offset(q >> 3, q & 7)) = gw[i];
      }
    } else if (!UPRE) {
#pragma unroll
      for (int i = 0; i < LA; ++i) {
        const int q = tid + i * NT;
        if (CA % NT != 0 && wave * 64 + i * NT >= CA) break;   // wave-uniform
        *reinterpret_cast<int4v*>(sb + (BM + BN) * 128 + kc_offset(q >> 3, q & 7)) = ga[i];
      }
    }
  };

  floatx16 acc[FJ][FI];
  floatx16 uacc[FT][FUW];      // U on the 32x32x16 form (RP >= 32)
  floatx4 uacc16[GPW];         // U on the 16x16x32 form (RP = 16)
#pragma unroll
  for (int a = 0; a < GPW; ++a) uacc16[a] = floatx4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int a = 0; a < FJ; ++a)
#pragma unroll
    for (int b = 0; b < FI; ++b) acc[a][b] = floatx16{};
#pragma unroll
  for (int a = 0; a < FT; ++a)
#pragma unroll
    for (int b = 0; b < FUW; ++b) uacc[a][b] = floatx16{};
  int urow[FUW];
#pragma unroll
  for (int fu = 0; fu < FUW; ++fu) urow[fu] = wm * WTI + 32 * ((wn + WN * fu) % FI) + c32;
  int urow16[GPW];
#pragma unroll
  for (int gg = 0; gg < GPW; ++gg) urow16[gg] = wm * WTI + 16 * (wn * GPW + gg) + c16;

  // Fragments of the next 16-wide substep are read while the current one
  // multiplies (two register sets, p = substep parity).  The U products of a
  // shared token fragment run on substeps ks % NDUP == 0 only: there share
  // udup multiplies the k columns of substep ks + udup, so every wave executes
  // the same instruction stream.
  short8 fw[2][FJ], fx[2][FI], fa[2][FT], fxu[2][FUW];
  short8 fa16[2], fxu16[2][GPW];
  auto read_frags = [&](const char* sb, int ks, int p) LORA_INLINE {
    const char* Xs = sb;
    const char* Ws = sb + BM * 128;
    const char* As = sb + (BM + BN) * 128;
    const int ch = 2 * ks + g;
#pragma unroll
    for (int fj = 0; fj < FJ; ++fj) fw[p][fj] = kc_read(Ws, wn * WTJ + 32 * fj + c32, ch);
#pragma unroll
    for (int fi = 0; fi < FI; ++fi) fx[p][fi] = kc_read(Xs, wm * WTI + 32 * fi + c32, ch);
    if (UPRE) {
    } else if (U16) {
      if (ks % 2 == 0) {   // the 32-wide half starting at substep ks: chunks 2 ks + g16
        fa16[p] = kc_read(As, c16, 2 * ks + g16);
#pragma unroll
        for (int gg = 0; gg < GPW; ++gg) fxu16[p][gg] = kc_read(Xs, urow16[gg], 2 * ks + g16);
      }
    } else if (ks % NDUP == 0) {
      const int uch = ch + 2 * udup;
#pragma unroll
      for (int ft = 0; ft < FT; ++ft) fa[p][ft] = kc_read(As, 32 * ft + c32, uch);
#pragma unroll
      for (int fu = 0; fu < FUW; ++fu) fxu[p][fu] = kc_read(Xs, urow[fu], uch);
    }
  };
  auto multiply = [&](int p, int ks) LORA_INLINE {
#pragma unroll
    for (int fi = 0; fi < FI; ++fi)
#pragma unroll
      for (int fj = 0; fj < FJ; ++fj) acc[fj][fi] = mfma32x32x16(fw[p][fj], fx[p][fi], acc[fj][fi]);
    if (UPRE) {
    } else if (U16) {
      if (ks % 2 == 0) {
#pragma unroll
        for (int gg = 0; gg < GPW; ++gg) uacc16[gg] = mfma16x16x32(fa16[p], fxu16[p][gg], uacc16[gg]);
      }
    } else if (ks % NDUP == 0) {
#pragma unroll
      for (int fu = 0; fu < FUW; ++fu)
#pragma unroll
        for (int ft = 0; ft < FT; ++ft) uacc[ft][fu] = mfma32x32x16(fa[p][ft], fxu[p][fu], uacc[ft][fu]);
    }
  };

  // Pipeline.  At the top of stage kb the staging registers hold k-block
  // kb+1 (loaded one stage earlier); piece ks of it is stored to the free LDS
  // buffer at substep ks, and its registers are then reloaded with block kb+2.
  // With ROT the loop is rotated by one substep: the products of substep 3 of
  // stage kb-1 are issued after the barrier, while the first fragments of
  // stage kb are being read (their operands are zeroed for stage 0, adding
  // exact zeros).  The 256 x 256 tile has no registers to spare for it.  The k
  // loop is peeled so the steady state carries no conditionals.
  constexpr bool ROT = BM * BN < 256 * 256;
  if (ROT) {
#pragma unroll
    for (int j = 0; j < FJ; ++j) fw[1][j] = short8{};
#pragma unroll
    for (int j = 0; j < FI; ++j) fx[1][j] = short8{};
#pragma unroll
    for (int j = 0; j < FT; ++j) fa[1][j] = short8{};
#pragma unroll
    for (int j = 0; j < FUW; ++j) fxu[1][j] = short8{};
    fa16[1] = short8{};
#pragma unroll
    for (int j = 0; j < GPW; ++j) fxu16[1][j] = short8{};
  }
  // bufc: the stage's LDS buffer as a compile-time constant, or -1 for the
  // parity of kb at run time
  auto stage = [&](int kb, auto bufc, bool write_next, bool load_next) LORA_INLINE {
    constexpr int BUF = decltype(bufc)::value;
    const int cur = BUF >= 0 ? BUF : (kb & 1);
    const char* sb = smem + cur * STAGE;
    read_frags(sb, 0, 0);
    if (ROT) multiply(1, 3);
#pragma unroll
    for (int ks = 0; ks < 4; ++ks) {
      if (write_next) swrite(cur ^ 1, ks);
      if (load_next) gload(kb + 2, ks);
      if (ks < 3) read_frags(sb, ks + 1, (ks + 1) & 1);
      if (ks < 3 || !ROT) multiply(ks & 1, ks);
    }
    __syncthreads();
  };
  const int nkb = (k + 63) / 64;
  using B0 = std::integral_constant<int, 0>;
  using B1 = std::integral_constant<int, 1>;
  using BR = std::integral_constant<int, -1>;
  if constexpr (DMA) {
    static_assert(KFULL && !ROT, "copy pipeline shape");
    // Copy instruction j of a region covers its rows 8j .. 8j+7: lane l takes
    // position l % 8 of row 8j + l / 8, i.e. logical chunk (l % 8) ^ kc_swz(row).
    constexpr int JX = BM / 8, JW = BN / 8, JA = RPS / 8;
    static_assert(JX % NW == 0 && JW % NW == 0, "copies split evenly");
    const int dl_row = lane >> 3, dl_cp = lane & 7;
    auto voff = [&](int j) LORA_INLINE {
      const int row = 8 * j + dl_row;
      return (uint32_t)row * rowbytes + (uint32_t)((dl_cp ^ kc_swz(row)) << 4);
    };
    auto dload = [&](int kb, int buf) LORA_INLINE {
      const uint32_t k0b = (uint32_t)kb * 128;
      char* sb = smem + buf * STAGE;
#pragma unroll
      for (int i = 0; i < JX / NW; ++i) dma16(rsX, voff(wave + NW * i), k0b, sb + (wave + NW * i) * 1024);
#pragma unroll
      for (int i = 0; i < JW / NW; ++i)
        dma16(rsW, voff(wave + NW * i), k0b, sb + BM * 128 + (wave + NW * i) * 1024);
#pragma unroll
      for (int i = 0; i < (JA + NW - 1) / NW; ++i)
        if (wave + NW * i < JA) dma16(rsA, voff(wave + NW * i), k0b, sb + (BM + BN) * 128 + (wave + NW * i) * 1024);
    };
    dload(0, 0);
    copy_barrier<0>();
    if constexpr (UPRE) {
      // Fragment reads as inline assembly, two register sets deep: the reads
      // of substep ks+1 are issued before the products of substep ks, which
      // wait (s_waitcnt lgkmcnt) only for their own six reads.  (Left to
      // itself the compiler folds the two sets into one and waits for each
      // pair of reads right before its products.)  Chunk c of row p sits at
      // p*128 | ((c ^ kc_swz(p)) << 4); for the lane's chunk 2ks + g that is
      // base ^ (ks << 5) with base = p*128 | ((kc_swz(p) ^ g) << 4), and the
      // fragments of a wave are 32 rows (4096 bytes) apart with the same
      // swizzle, so one address register per operand and buffer suffices.
      static_assert(FJ == 2 && FI == 4, "reads per substep");
      const uint32_t sg = (uint32_t)((kc_swz(c32) ^ g) << 4);
      const uint32_t wb0 = lds_addr(smem + BM * 128 + (wn * WTJ + c32) * 128) | sg;
      const uint32_t xb0 = lds_addr(smem + (wm * WTI + c32) * 128) | sg;
      auto areads = [&](int buf, int ks, int p) LORA_INLINE {   // (ks, buf, p: constants after inlining)
        const uint32_t wb = wb0 + (uint32_t)buf * STAGE, xb = xb0 + (uint32_t)buf * STAGE;
        uint32_t ta, tb;
        asm volatile(
            "v_xor_b32 %[ta], %[kx], %[wb]\n\t"
            "v_xor_b32 %[tb], %[kx], %[xb]\n\t"
            "ds_read_b128 %[w0], %[ta]\n\t"
            "ds_read_b128 %[w1], %[ta] offset:4096\n\t"
            "ds_read_b128 %[x0], %[tb]\n\t"
            "ds_read_b128 %[x1], %[tb] offset:4096\n\t"
            "ds_read_b128 %[x2], %[tb] offset:8192\n\t"
            "ds_read_b128 %[x3], %[tb] offset:12288"
            : [w0] "=v"(fw[p][0]), [w1] "=v"(fw[p][1]), [x0] "=v"(fx[p][0]), [x1] "=v"(fx[p][1]),
              [x2] "=v"(fx[p][2]), [x3] "=v"(fx[p][3]), [ta] "=&v"(ta), [tb] "=&v"(tb)
            : [wb] "v"(wb), [xb] "v"(xb), [kx] "i"(ks << 5));
      };
      auto amult = [&](int p, bool last) LORA_INLINE {
        if (last)
          asm volatile("s_waitcnt lgkmcnt(0)"
                       : "+v"(fw[p][0]), "+v"(fw[p][1]), "+v"(fx[p][0]), "+v"(fx[p][1]), "+v"(fx[p][2]),
                         "+v"(fx[p][3]));
        else
          asm volatile("s_waitcnt lgkmcnt(6)"
                       : "+v"(fw[p][0]), "+v"(fw[p][1]), "+v"(fx[p][0]), "+v"(fx[p][1]), "+v"(fx[p][2]),
                         "+v"(fx[p][3]));
#pragma unroll
        for (int fi = 0; fi < FI; ++fi)
#pragma unroll
          for (int fj = 0; fj < FJ; ++fj) acc[fj][fi] = mfma32x32x16(fw[p][fj], fx[p][fi], acc[fj][fi]);
      };
      auto astage = [&](int kb, auto bufc, bool load_next) LORA_INLINE {
        constexpr int BUF = decltype(bufc)::value;
        if (load_next) dload(kb + 1, BUF ^ 1);   // read in stage kb-1, free since its barrier
        areads(BUF, 0, 0);
        areads(BUF, 1, 1);
        amult(0, false);
        areads(BUF, 2, 0);
        amult(1, false);
        areads(BUF, 3, 1);
        amult(0, false);
        amult(1, true);
        copy_barrier<0>();
      };
      int kb = 0;
      for (; kb + 2 < nkb; kb += 2) {
        astage(kb, B0{}, true);
        astage(kb + 1, B1{}, true);
      }
      if (kb < nkb) astage(kb, B0{}, kb + 1 < nkb);
      if (kb + 1 < nkb) astage(kb + 1, B1{}, false);
    } else {
      auto dstage = [&](int kb, auto bufc, bool load_next) LORA_INLINE {
        constexpr int BUF = decltype(bufc)::value;
        if (load_next) dload(kb + 1, BUF ^ 1);   // read in stage kb-1, free since its barrier
        const char* sb = smem + BUF * STAGE;
        read_frags(sb, 0, 0);
#pragma unroll
        for (int ks = 0; ks < 4; ++ks) {
          if (ks < 3) read_frags(sb, ks + 1, (ks + 1) & 1);
          multiply(ks & 1, ks);
        }
        copy_barrier<0>();
      };
      int kb = 0;
      for (; kb + 2 < nkb; kb += 2) {
        dstage(kb, B0{}, true);
        dstage(kb + 1, B1{}, true);
      }
      if (kb < nkb) dstage(kb, B0{}, kb + 1 < nkb);
      if (kb + 1 < nkb) dstage(kb + 1, B1{}, false);
    }
  } else {
#pragma unroll
    for (int pc = 0; pc < 4; ++pc) gload(0, pc);
#pragma unroll
    for (int pc = 0; pc < 4; ++pc) swrite(0, pc);
    __syncthreads();
    if (nkb > 1) {
#pragma unroll
      for (int pc = 0; pc < 4; ++pc) gload(1, pc);
    }
    int kb = 0;
    if constexpr (KFULL && BM * BN < 256 * 256) {
      for (; kb + 3 < nkb; kb += 2) {
        stage(kb, B0{}, true, true);
        stage(kb + 1, B1{}, true, true);
      }
    }
    for (; kb + 2 < nkb; ++kb) stage(kb, BR{}, true, true);
    if (kb + 1 < nkb) stage(kb++, BR{}, true, false);
    stage(kb, BR{}, false, false);
    if (ROT) multiply(1, 3);
  }

  // ---- epilogue ------------------------------------------------------------
  // LDS reuse: Us [NUS][BM][RPU] fp32 partial U (summed in fixed order below),
  // then Bs [BN][RPB] bf16 (B rows of this tile, zero beyond r and n).  The
  // rows are padded by 16 bytes so that the 16 lanes of a read group, which
  // read 16 consecutive rows, fall in different banks.  Rows n0 .. n0+jn-1 of
  // B are contiguous, so they are fetched as 16-byte chunks of 8 elements, all
  // issued before the first wait, and scattered into Bs.
  float* Us = reinterpret_cast<float*>(smem);
  u16* Bs = reinterpret_cast<u16*>(smem + NUS * BM * RPU * 4);
  constexpr int BCH = (BN * RP / 8 + NT - 1) / NT;   // chunks per thread (r <= RP)
  const int jn = min(BN, n - n0);
  const int nch = jn * r / 8;                       // exact: n and n0 are multiples of 8
  const __amdgpu_buffer_rsrc_t rsB = make_rsrc(B + (size_t)n0 * r, (uint64_t)nch * 16);
  int4v bv[BCH];
#pragma unroll
  for (int i = 0; i < BCH; ++i) {
    const int q = tid + i * NT;
    bv[i] = buf_load16(rsB, q < nch ? (uint32_t)q * 16 : kOOB);
  }
  if (UPRE) {   // U of the tile's tokens from the U pass (zero beyond r and m), all loads issued before the first use
    constexpr int UPT = BM * RP / NT;
    static_assert(BM * RP % NT == 0, "U values per thread");
    const __amdgpu_buffer_rsrc_t rsU = make_rsrc(U + (size_t)m0 * r, (uint64_t)min(BM, m - m0) * r * 4);
    float uv[UPT];
#pragma unroll
    for (int i = 0; i < UPT; ++i) {
      const int e = tid + i * NT, il = e / RP, t = e - il * RP;
      uv[i] = buf_load4f(rsU, t < r ? (uint32_t)(il * r + t) * 4 : kOOB);
    }
#pragma unroll
    for (int i = 0; i < UPT; ++i) {
      const int e = tid + i * NT, il = e / RP, t = e - il * RP;
      Us[il * RPU + t] = uv[i];
    }
  } else if (U16) {   // lane holds token column c16 of its group, U rows t = 4 g16 .. +3
#pragma unroll
    for (int gg = 0; gg < GPW; ++gg)
#pragma unroll
      for (int q = 0; q < 4; ++q) Us[urow16[gg] * RPU + 4 * g16 + q] = uacc16[gg][q];
  } else {
#pragma unroll
    for (int fu = 0; fu < FUW; ++fu) {
      const int il = urow[fu];
#pragma unroll
      for (int ft = 0; ft < FT; ++ft)
#pragma unroll
        for (int q = 0; q < 16; ++q) {
          const int t = 32 * ft + 8 * (q >> 2) + 4 * g + (q & 3);
          Us[(udup * BM + il) * RPU + t] = uacc[ft][fu][q];
        }
    }
  }
  for (int e = tid; e < BN * RPB / 8; e += NT) reinterpret_cast<int4v*>(Bs)[e] = int4v{0, 0, 0, 0};
  __syncthreads();
  {
    // element idx of the chunks is B row idx / r, column idx % r; the quotient
    // comes from a float product that stays at least 0.5/r away from an integer
    const float rinv = 1.0f / (float)r;
#pragma unroll
    for (int i = 0; i < BCH; ++i) {
      const int q = tid + i * NT;
      if (q < nch) {
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          const int idx = 8 * q + e;
          const int j = (int)(((float)idx + 0.5f) * rinv);
          const int t = idx - j * r;
          Bs[j * RPB + t] = (u16)((uint32_t)bv[i][e >> 1] >> (16 * (e & 1)));
        }
      }
    }
  }
  if (NDUP > 1 && !UPRE) {  // fold the partial U sums into copy 0 (fixed order)
    for (int e = tid; e < BM * RP; e += NT) {
      const int o = (e / RP) * RPU + e % RP;
      float v = Us[o];
#pragma unroll
      for (int d = 1; d < NDUP; ++d) v += Us[d * BM * RPU + o];
      Us[o] = v;
    }
  }
  __syncthreads();
  if (n0 == 0 && !UPRE) {   // U output: the first tile column writes it
    for (int e = tid; e < BM * RP; e += NT) {
      const int il = e / RP, t = e - il * RP;
      if (m0 + il < m && t < r) U[(size_t)(m0 + il) * r + t] = Us[il * RPU + t];
    }
  }

  // acc += s U B^T, formed as Y^T += B (sU)^T over t in blocks of 16, each
  // block once with the high and once with the low bf16 part of sU.
  const int tblocks = (r + 15) / 16;
  for (int tb = 0; tb < tblocks; ++tb) {
    const int t0 = 16 * tb + 8 * g;
    short8 bfr[FJ];
#pragma unroll
    for (int fj = 0; fj < FJ; ++fj) {
      const int jl = wn * WTJ + 32 * fj + c32;
      bfr[fj] = *reinterpret_cast<const short8*>(Bs + jl * RPB + t0);
    }
#pragma unroll
    for (int fi = 0; fi < FI; ++fi) {
      const int il = wm * WTI + 32 * fi + c32;
      const float* up = Us + il * RPU + t0;
      short8 uh, ul;
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const float v = s * up[e];
        const u16 hi = f32_to_bf16(v);
        uh[e] = (short)hi;
        ul[e] = (short)f32_to_bf16(v - bf16_to_f32(hi));
      }
#pragma unroll
      for (int fj = 0; fj < FJ; ++fj) {
        acc[fj][fi] = mfma32x32x16(bfr[fj], uh, acc[fj][fi]);
        acc[fj][fi] = mfma32x32x16(bfr[fj], ul, acc[fj][fi]);
      }
    }
  }

  // store Y: each wave's 32-token blocks of its 64 features through a
  // wave-private LDS region (free once every wave is past the reads above)
  static_assert(FJ == 2 && NW * kYsBytes <= 2 * STAGE, "output staging");
  __syncthreads();
  const int j0 = n0 + wn * WTJ;
#pragma unroll
  for (int fi = 0; fi < FI; ++fi) {
    const int i0 = m0 + wm * WTI + 32 * fi;
    store_block_32x64(acc[0][fi], acc[1][fi], smem + wave * kYsBytes, Y + (size_t)i0 * n + j0, (size_t)n, m - i0,
                      n - j0, lane);
  }
}

// ---------------------------------------------------------------------------
// U = X A^T on its own: for ranks above 16 (in the fused tile every output
// tile recomputes all RP U columns of its tokens, RP / BN more matrix-core
// work, a quarter at RP = 64 on the 256-wide tile; this pass computes them
// once), and under LoRA dropout (KEEP: U = (keep X) A^T / (1 - p), so the
// GEMM that follows needs no mask).  TPW (16 or 32) tokens per workgroup,
// four waves.  The k loop runs in stages of 64; wave w takes stages w, w + 4,
// ... and copies each of them (its TPW X rows and RP A rows, 128 bytes a row,
// eight whole row pieces per copy instruction with the swizzle of kc_offset
// applied to the global addresses; under KEEP also the stage's keep bits, 8
// bytes a token, 4 bytes a lane) from global memory straight into a private
// ring of NSW LDS stages, NSW - 1 stages ahead.  No barrier in the loop: the
// wave waits only for its own copies.  (Loads of 16 rows x 64 bytes per
// instruction straight into matrix-core operands kept the L1 busy
// translating addresses; a shared ring with a barrier per stage was bound by
// each stage's short compute chain.)  Each wave accumulates all RP x TPW of U
// over its stages (16x16x32 products; under KEEP each X fragment of 8 k is
// masked with its keep byte first); the four partial sums are added in wave
// order through LDS at the end (bit-identical from run to run) and written
// as fp32 U [m][r], scaled by inv_keep under KEEP.  With TPW = 8 (launches
// whose 16-token workgroups would leave compute units idle) a stage still
// holds 16 X rows for the 16-token products; rows 8..15 are zeroed once and
// never copied into, and only the first 8 tokens' U is written.
template <int RP, int TPW, bool KEEP>
__global__ __launch_bounds__(256) void lora_u_kernel(const u16* __restrict__ X, const u16* __restrict__ A,
                                                     const uint8_t* __restrict__ keep, float* __restrict__ U, int m,
                                                     int k, int r, float inv_keep) {
  constexpr int NWV = 4;
  constexpr int XR = TPW < 16 ? 16 : TPW;        // X rows of a stage (rows TPW .. XR-1 stay zero)
  constexpr int ROWS = XR + RP;                  // 128-byte rows per stage: X rows, then A rows
  constexpr int MOFF = ROWS * 128;               // keep bytes of the stage: [TPW][8]
  constexpr int STAGE = MOFF + (KEEP ? 256 : 0);
  constexpr int CPS = (TPW + RP) / 8;            // 1 KB copies per stage
  constexpr int CPW = CPS + (KEEP ? 1 : 0);      // copy instructions per stage (the wave's own)
  constexpr int NSW = (156 * 1024) / (NWV * STAGE) < 6 ? (156 * 1024) / (NWV * STAGE) : 6;   // ring stages per wave
  constexpr int FT = RP / 16, TG = XR / 16;
  constexpr int RED = NWV * FT * TG * 64 * 16;   // cross-wave sum: [NWV][FT][TG][64] float4
  constexpr int SMEM = NWV * NSW * STAGE > RED ? NWV * NSW * STAGE : RED;
  static_assert(TPW == 8 || TPW == 16 || TPW == 32, "tokens per workgroup");
  static_assert(NSW >= 3 && CPW * (NSW - 2) < 64, "copies in flight fit the wait counter");
  static_assert(FT * TG <= 8, "fragments per wave");
  __shared__ __attribute__((aligned(1024))) char smem[SMEM];
  const int i0 = blockIdx.x * TPW;
  const int tid = threadIdx.x, lane = tid & 63, wave = uniform(tid >> 6);
  const int g = lane >> 4, c16 = lane & 15;
  const uint32_t rowbytes = (uint32_t)k * 2;
  const int rows = uniform(max(0, min(TPW, m - i0)));
  const __amdgpu_buffer_rsrc_t rsX = make_rsrc(X + (size_t)i0 * k, (uint64_t)rows * rowbytes);
  const __amdgpu_buffer_rsrc_t rsA = make_rsrc(A, (uint64_t)r * rowbytes);
  const uint32_t kb8 = (uint32_t)k / 8;          // keep bytes per token (k % 64 == 0 with dropout)
  const __amdgpu_buffer_rsrc_t rsK =
      make_rsrc(KEEP ? (const void*)(keep + (size_t)i0 * kb8) : (const void*)X, KEEP ? (uint64_t)rows * kb8 : 0);
  char* ring = smem + wave * NSW * STAGE;

  // Copy c of a stage fills 8 rows: X rows 8c .. 8c+7 (8c < TPW), else A rows
  // 8c - TPW .. +7 at stage rows XR + 8c - TPW ..; this lane's row lane/8 of
  // the eight at physical chunk lane%8, which holds logical chunk
  // (lane%8) ^ kc_swz(stage row).  Rows past m or r, k past the end and stages
  // past the wave's last read zero.
  const int c8 = lane & 7, r8 = lane >> 3;
  const int nst = (k + 63) / 64;
  auto issue = [&](int j, int buf) LORA_INLINE {   // the wave's j-th stage
    const int st = wave + NWV * j;
    const int k0 = st * 64;
    const bool live = st < nst;
    char* sb = ring + buf * STAGE;
#pragma unroll
    for (int c = 0; c < CPS; ++c) {
      const bool isx = 8 * c < TPW;   // uniform
      const int row = 8 * c + r8;
      const int srow = isx ? row : row + (XR - TPW);   // stage row
      const int lc = c8 ^ kc_swz(srow);
      const int grow = isx ? row : row - TPW;
      const uint32_t off = live && k0 + 8 * lc < k ? (uint32_t)grow * rowbytes + (uint32_t)(k0 + 8 * lc) * 2 : kOOB;
      dma16(isx ? rsX : rsA, off, 0, sb + (isx ? c : c + (XR - TPW) / 8) * 1024);
    }
    if (KEEP)   // lane l: bytes 4 (l % 2) .. +3 of token l / 2's stage bits (lanes past TPW tokens: zero)
      dma4(rsK, live && (lane >> 1) < TPW ? (uint32_t)(lane >> 1) * kb8 + (uint32_t)k0 / 8 + 4 * (lane & 1) : kOOB,
           0, sb + MOFF);
  };
  floatx4 acc[FT][TG];
#pragma unroll
  for (int ft = 0; ft < FT; ++ft)
#pragma unroll
    for (int tg = 0; tg < TG; ++tg) acc[ft][tg] = floatx4{0.f, 0.f, 0.f, 0.f};
  auto compute = [&](int buf) LORA_INLINE {
    const char* sb = ring + buf * STAGE;
#pragma unroll
    for (int kk = 0; kk < 2; ++kk) {
      const int ch = 4 * kk + g;
      short8 xf[TG], af[FT];
#pragma unroll
      for (int tg = 0; tg < TG; ++tg) {
        xf[tg] = kc_read(sb, 16 * tg + c16, ch);
        if constexpr (KEEP) xf[tg] = keep_mask8(xf[tg], (uint32_t)(uint8_t)sb[MOFF + (16 * tg + c16) * 8 + ch]);
      }
#pragma unroll
      for (int ft = 0; ft < FT; ++ft) af[ft] = kc_read(sb, XR + 16 * ft + c16, ch);
#pragma unroll
      for (int ft = 0; ft < FT; ++ft)
#pragma unroll
        for (int tg = 0; tg < TG; ++tg) acc[ft][tg] = mfma16x16x32(af[ft], xf[tg], acc[ft][tg]);
    }
  };

  const int nsw = wave < nst ? (nst - wave + NWV - 1) / NWV : 0;   // this wave's stages
  if constexpr (TPW < 16) {   // the zero X rows TPW .. 15 of every ring stage (8 rows: 16 bytes a lane)
    static_assert(TPW == 8, "one 1 KB block of zero rows");
#pragma unroll
    for (int b = 0; b < NSW; ++b) *reinterpret_cast<int4v*>(ring + b * STAGE + TPW * 128 + lane * 16) = int4v{0, 0, 0, 0};
  }
#pragma unroll
  for (int j = 0; j < NSW - 1; ++j) issue(j, j);
  for (int j = 0; j < nsw; ++j) {
    wait_vmcnt<CPW * (NSW - 2)>();   // the wave's stage j has landed
    issue(j + NSW - 1, (j + NSW - 1) % NSW);   // into the buffer of stage j - 1, read already
    compute(j % NSW);
  }
  wait_vmcnt<0>();   // the trailing copies (zeros) land before the LDS is reused

  // Cross-wave sum in wave order; lane of (ft, tg): rank rows 16 ft + 4 g ..
  // +3 of token 16 tg + c16.
  floatx4* red = reinterpret_cast<floatx4*>(smem);
  __syncthreads();
#pragma unroll
  for (int ft = 0; ft < FT; ++ft)
#pragma unroll
    for (int tg = 0; tg < TG; ++tg) red[((wave * FT + ft) * TG + tg) * 64 + lane] = acc[ft][tg];
  __syncthreads();
  for (int e = wave; e < FT * TG; e += NWV) {
    const int ft = e / TG, tg = e - ft * TG;
    floatx4 v = red[((0 * FT + ft) * TG + tg) * 64 + lane];
#pragma unroll
    for (int w = 1; w < NWV; ++w) v += red[((w * FT + ft) * TG + tg) * 64 + lane];
    const int i = i0 + 16 * tg + c16;
    if (i < m && 16 * tg + c16 < TPW) {
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int t = 16 * ft + 4 * g + j;
        if (t < r) U[(size_t)i * r + t] = KEEP ? inv_keep * v[j] : v[j];
      }
    }
  }
}

// ---------------------------------------------------------------------------
// The 128 x 256 tile for rank <= 16 with the k substeps split between wave
// pairs.  Eight waves: wave (wk, wm, wn) multiplies the 64 tokens wm and the
// 128 features wn of the tile over substeps 2 wk and 2 wk + 1 of every 64-wide
// stage (the 32-wide k half wk).  Per stage a wave issues as many products as
// in the 2 x 4 layout of 64 x 64 wave tiles but reads 12 operand fragments
// instead of 16, and two waves still share each SIMD.  The U columns run on
// v_mfma_f32_16x16x32_bf16: wave (wk, wm, wn) owns the 16-token groups
// 2 wn, 2 wn + 1 of its token half, over its k half.
//
// After the k loop the two k-half partial sums of each output are added in
// fixed order through LDS: wave wk keeps feature fragments 2 wk, 2 wk + 1 and
// sends the other two to its partner, so each wave then holds a complete
// 64 x 64 block (features wn 128 + 64 wk ..) for the epilogue, which is the one
// of the 2 x 4 layout.  GRP selects the projection of a grouped launch as in
// lora_fwd_kernel.
//
// DMA (k a multiple of 64; used for launches of at most one round): the
// stages go from global memory straight into three LDS buffers (one 16-byte
// chunk per lane per copy instruction, the chunk swizzle applied to the
// global addresses), two stages ahead and without staging registers; each
// stage ends with a barrier that waits only for this wave's copies of the
// next stage (copy_barrier).
//
// UPRE (LoRA dropout: U from the masked U pass): the stages hold no A rows,
// the loop runs no U products, and the epilogue reads U back.
template <bool GRP, bool KFULL, bool DMA, bool UPRE>
__global__ __launch_bounds__(512) void lora_fwd_ks_kernel(
    const u16* __restrict__ X, const u16* __restrict__ W, const u16* __restrict__ A,
    const u16* __restrict__ B, u16* __restrict__ Y, float* __restrict__ U, int m, int n, int k, int r, float s,
    int tiles_m, int tiles_n, int n_begin, FwdGroup grp) {
  constexpr int BM = 128, BN = 256, NT = 512, RP = 16;
  constexpr int WTI = 64, WTJ = 128, FI = 2, FJ = 4;
  constexpr int GPW = 2;                          // 16-token U groups per wave
  constexpr int RPS = UPRE ? 0 : RP;              // A rows staged per stage
  constexpr int ROWS = BM + BN + RPS;
  constexpr int STAGE = ROWS * 128;
  constexpr int CX = BM * 8, CW = BN * 8, CA = RPS * 8;
  constexpr int LX = CX / NT, LW = CW / NT, LA = UPRE ? 1 : (CA + NT - 1) / NT;
  static_assert(!(UPRE && GRP), "U from the U pass only for single projections");
  constexpr int XCH = 8 * 16 * 1024;              // exchange: 8 waves x 32 fragments x 64 lanes x 4 B
  static_assert(!DMA || KFULL, "the copies carry no k-bound checks");
  constexpr int NBUF = DMA ? 3 : 2;                       // LDS stage buffers
  constexpr int BS_OFF = DMA ? NBUF * STAGE : XCH + 2 * BM * RP * 4;
  constexpr int EPI = (BS_OFF > XCH + 2 * BM * RP * 4 ? BS_OFF : XCH + 2 * BM * RP * 4) + BN * RP * 2;
  constexpr int SMEM = EPI > NBUF * STAGE ? EPI : NBUF * STAGE;
  __shared__ __attribute__((aligned(1024))) char smem[SMEM];

  int tm, tn;
  tile_coords(tiles_m, tiles_n, 8, (int)blockIdx.x, tm, tn);
  if (GRP) {
    int sel = 0;
#pragma unroll
    for (int q = 1; q < kMaxGroup; ++q)
      if (q < grp.count && tn >= grp.tile0[q]) sel = q;
#pragma unroll
    for (int q = 0; q < kMaxGroup; ++q)
      if (q == sel) {
        W = grp.W[q]; A = grp.A[q]; B = grp.B[q]; Y = grp.Y[q]; U = grp.U[q];
        n = grp.n[q];
        tn -= grp.tile0[q];
      }
  }
  const int m0 = tm * BM, n0 = n_begin + tn * BN;
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = uniform(tid >> 6);
  const int wk = wave >> 2, wm = (wave >> 1) & 1, wn = wave & 1;
  const int g = lane >> 5, c32 = lane & 31;
  const int g16 = lane >> 4, c16 = lane & 15;

  const uint32_t rowbytes = (uint32_t)k * 2;
  const __amdgpu_buffer_rsrc_t rsX = make_rsrc(X + (size_t)m0 * k, (uint64_t)min(BM, m - m0) * rowbytes);
  const __amdgpu_buffer_rsrc_t rsW = make_rsrc(W + (size_t)n0 * k, (uint64_t)min(BN, n - n0) * rowbytes);
  const __amdgpu_buffer_rsrc_t rsA = make_rsrc(A, (uint64_t)r * rowbytes);

  // Register staging of one k-block as in lora_fwd_kernel, stored in two
  // pieces (0 = X and A rows, 1 = W rows), one per substep of the stage.
  int4v gx[LX], gw[LW], ga[LA];
  auto gload = [&](int kb, int piece) LORA_INLINE {
    const int k0 = kb * 64;
    if (piece == 0) {
#pragma unroll
      for (int i = 0; i < LX; ++i) {
        const int q = tid + i * NT;
        const int kk = k0 + 8 * (q & 7);
        gx[i] = buf_load16(rsX, (KFULL || kk < k) ? (uint32_t)(q >> 3) * rowbytes + (uint32_t)kk * 2 : kOOB);
      }
#pragma unroll
      for (int i = 0; i < LA; ++i) {
        if (UPRE) break;
        const int q = tid + i * NT;
        if (CA % NT != 0 && wave * 64 + i * NT >= CA) break;
        const int kk = k0 + 8 * (q & 7);
        ga[i] = buf_load16(rsA, (KFULL || kk < k) ? (uint32_t)(q >> 3) * rowbytes + (uint32_t)kk * 2 : kOOB);
      }
    } else {
#pragma unroll
      for (int i = 0; i < LW; ++i) {
        const int q = tid + i * NT;
        const int kk = k0 + 8 * (q & 7);
        gw[i] = buf_load16(rsW, (KFULL || kk < k) ? (uint32_t)(q >> 3) * rowbytes + (uint32_t)kk * 2 : kOOB);
      }
    }
  };
  auto swrite = [&](int buf, int piece) LORA_INLINE {
    char* sb = smem + buf * STAGE;
    if (piece == 0) {
#pragma unroll
      for (int i = 0; i < LX; ++i) {
        const int q = tid + i * NT;
        *reinterpret_cast<int4v*>(sb + kc_offset(q >> 3, q & 7)) = gx[i];
      }
#pragma unroll
      for (int i = 0; i < LA; ++i) {
        if (UPRE) break;
        const int q = tid + i * NT;
        if (CA % NT != 0 && wave * 64 + i * NT >= CA) break;
        *reinterpret_cast<int4v*>(sb + (BM + BN) * 128 + kc_offset(q >> 3, q & 7)) = ga[i];
      }
    } else {
#pragma unroll
      for (int i = 0; i < LW; ++i) {
        const int q = tid + i * NT;
        *reinterpret_cast<int4v*>(sb + BM * 128 + kc_offset(q >> 3, q & 7)) = gw[i];
      }
    }
  };

  floatx16 acc[FJ][FI];
#pragma unroll
  for (int a = 0; a < FJ; ++a)
#pragma unroll
    for (int b = 0; b < FI; ++b) acc[a][b] = floatx16{};
  floatx4 uacc16[GPW];
#pragma unroll
  for (int a = 0; a < GPW; ++a) uacc16[a] = floatx4{0.f, 0.f, 0.f, 0.f};
  int urow16[GPW];
#pragma unroll
  for (int gg = 0; gg < GPW; ++gg) urow16[gg] = wm * WTI + 16 * (wn * GPW + gg) + c16;

  short8 fw[2][FJ], fx[2][FI], fa16, fxu16[GPW];
  // Fragments of the wave's substep j (0, 1), global substep 2 wk + j; the
  // U operands of the wave's 32-wide k half are read with substep 0.
  auto read_frags = [&](const char* sb, int j, int p) LORA_INLINE {
    const char* Xs = sb;
    const char* Ws = sb + BM * 128;
    const char* As = sb + (BM + BN) * 128;
    const int ch = 2 * (2 * wk + j) + g;
#pragma unroll
    for (int fj = 0; fj < FJ; ++fj) fw[p][fj] = kc_read(Ws, wn * WTJ + 32 * fj + c32, ch);
#pragma unroll
    for (int fi = 0; fi < FI; ++fi) fx[p][fi] = kc_read(Xs, wm * WTI + 32 * fi + c32, ch);
    if (!UPRE && j == 0) {   // the wave's 32-wide half: chunks 4 wk + g16
      fa16 = kc_read(As, c16, 4 * wk + g16);
#pragma unroll
      for (int gg = 0; gg < GPW; ++gg) fxu16[gg] = kc_read(Xs, urow16[gg], 4 * wk + g16);
    }
  };
  auto multiply = [&](int p, int j) LORA_INLINE {
#pragma unroll
    for (int fi = 0; fi < FI; ++fi)
#pragma unroll
      for (int fj = 0; fj < FJ; ++fj) acc[fj][fi] = mfma32x32x16(fw[p][fj], fx[p][fi], acc[fj][fi]);
    if (!UPRE && j == 0) {
#pragma unroll
      for (int gg = 0; gg < GPW; ++gg) uacc16[gg] = mfma16x16x32(fa16, fxu16[gg], uacc16[gg]);
    }
  };
  // Pipeline of lora_fwd_kernel with two substeps per wave and stage: at the
  // top of stage kb the registers hold block kb+1; each piece is stored to the
  // free buffer and reloaded with block kb+2; fragments of substep 1 are read
  // while substep 0 multiplies.
  auto stage = [&](int kb, auto bufc, bool write_next, bool load_next) LORA_INLINE {
    constexpr int BUF = decltype(bufc)::value;    // -1: the buffer of kb's parity at run time
    const int cur = BUF >= 0 ? BUF : (kb & 1);
    const char* sb = smem + cur * STAGE;
    read_frags(sb, 0, 0);
    if (write_next) swrite(cur ^ 1, 0);
    if (load_next) gload(kb + 2, 0);
    read_frags(sb, 1, 1);
    multiply(0, 0);
    if (write_next) swrite(cur ^ 1, 1);
    if (load_next) gload(kb + 2, 1);
    multiply(1, 1);
    __syncthreads();
  };
  using B0 = std::integral_constant<int, 0>;
  using B1 = std::integral_constant<int, 1>;
  using BR = std::integral_constant<int, -1>;
  u16* Bs = reinterpret_cast<u16*>(smem + BS_OFF);   // B rows for the epilogue, staged in the prologue
  if constexpr (DMA) {
  const int nkb = (k + 63) / 64;
  // Copies straight into LDS: instruction j of a tile covers its rows 8j ..
  // 8j + 7, lane l position l % 8 of row 8j + l / 8, which holds the row's
  // logical chunk (l % 8) ^ kc_swz(row) (the swizzle is applied on the global
  // side).  Per stage a wave issues 2 X, 4 W and (waves 0, 1) 1 A copies.
  const int dl_row = lane >> 3, dl_cp = lane & 7;
  auto voff = [&](int j) LORA_INLINE {
    const int row = 8 * j + dl_row;
    return (uint32_t)row * rowbytes + (uint32_t)((dl_cp ^ kc_swz(row)) << 4);
  };
  auto dload = [&](int kb, int buf) LORA_INLINE {
    const uint32_t k0b = (uint32_t)kb * 128;
    char* sb = smem + buf * STAGE;
#pragma unroll
    for (int i = 0; i < 2; ++i) dma16(rsX, voff(wave + 8 * i), k0b, sb + (wave + 8 * i) * 1024);
#pragma unroll
    for (int i = 0; i < 4; ++i) dma16(rsW, voff(wave + 8 * i), k0b, sb + BM * 128 + (wave + 8 * i) * 1024);
    if (!UPRE && wave < 2) dma16(rsA, voff(wave), k0b, sb + (BM + BN) * 128 + wave * 1024);
  };
  constexpr int NDMA_MIN = 6;   // fewest copies any wave issues per stage
  dload(0, 0);
  if (nkb > 1) dload(1, 1);
  // B rows of the tile for the epilogue, staged once beside the pipeline's
  // buffers: Bs [BN][RP] bf16, zero beyond r and n; thread tid fills entries
  // t0b .. t0b + 7 of row tid / (RP / 8).
  {
    static_assert(BN * RP / 8 == NT, "one chunk of Bs per thread");
    const int j = tid / (RP / 8), t0b = 8 * (tid % (RP / 8));
    int4v v = int4v{0, 0, 0, 0};
    if (j < min(BN, n - n0) && t0b < r) {
      const u16* brow = B + (size_t)(n0 + j) * r;
      if ((r & 7) == 0) {
        v = *reinterpret_cast<const int4v*>(brow + t0b);
      } else {
        uint32_t w[4];
#pragma unroll
        for (int x = 0; x < 4; ++x) {
          const uint32_t lo = t0b + 2 * x < r ? brow[t0b + 2 * x] : 0u;
          const uint32_t hi = t0b + 2 * x + 1 < r ? brow[t0b + 2 * x + 1] : 0u;
          w[x] = lo | (hi << 16);
        }
        v = int4v{(int)w[0], (int)w[1], (int)w[2], (int)w[3]};
      }
    }
    *reinterpret_cast<int4v*>(Bs + j * RP + t0b) = v;
  }
  copy_barrier<0>();   // every copy and load of the prologue has landed
  // Stage kb reads buffer kb % 3; at its top the copies of stage kb+2 go to
  // buffer (kb+2) % 3, which every wave finished reading in stage kb-1; at
  // its end each wave waits for its copies of stage kb+1 before the barrier.
  auto dstage = [&](int kb, auto bufc, bool load_next) LORA_INLINE {
    constexpr int BUF = decltype(bufc)::value;
    if (load_next) dload(kb + 2, (BUF + 2) % 3);
    const char* sb = smem + BUF * STAGE;
    read_frags(sb, 0, 0);
    read_frags(sb, 1, 1);
    multiply(0, 0);
    multiply(1, 1);
    if (load_next) copy_barrier<NDMA_MIN>();
    else copy_barrier<0>();
  };
  using D0 = std::integral_constant<int, 0>;
  using D1 = std::integral_constant<int, 1>;
  using D2 = std::integral_constant<int, 2>;
  int kb = 0;
  for (; kb + 5 < nkb; kb += 3) {
    dstage(kb, D0{}, true);
    dstage(kb + 1, D1{}, true);
    dstage(kb + 2, D2{}, true);
  }
  if (kb < nkb) dstage(kb, D0{}, kb + 2 < nkb);
  if (kb + 1 < nkb) dstage(kb + 1, D1{}, kb + 3 < nkb);
  if (kb + 2 < nkb) dstage(kb + 2, D2{}, kb + 4 < nkb);
  if (kb + 3 < nkb) dstage(kb + 3, D0{}, false);
  if (kb + 4 < nkb) dstage(kb + 4, D1{}, false);
  } else {
  const int nkb = (k + 63) / 64;
  gload(0, 0);
  gload(0, 1);
  // B rows of the tile for the epilogue, staged once beside the pipeline's
  // buffers: Bs [BN][RP] bf16, zero beyond r and n; thread tid fills entries
  // t0b .. t0b + 7 of row tid / (RP / 8).
  {
    static_assert(BN * RP / 8 == NT, "one chunk of Bs per thread");
    const int j = tid / (RP / 8), t0b = 8 * (tid % (RP / 8));
    int4v v = int4v{0, 0, 0, 0};
    if (j < min(BN, n - n0) && t0b < r) {
      const u16* brow = B + (size_t)(n0 + j) * r;
      if ((r & 7) == 0) {
        v = *reinterpret_cast<const int4v*>(brow + t0b);
      } else {
        uint32_t w[4];
#pragma unroll
        for (int x = 0; x < 4; ++x) {
          const uint32_t lo = t0b + 2 * x < r ? brow[t0b + 2 * x] : 0u;
          const uint32_t hi = t0b + 2 * x + 1 < r ? brow[t0b + 2 * x + 1] : 0u;
          w[x] = lo | (hi << 16);
        }
        v = int4v{(int)w[0], (int)w[1], (int)w[2], (int)w[3]};
      }
    }
    *reinterpret_cast<int4v*>(Bs + j * RP + t0b) = v;
  }
  swrite(0, 0);
  swrite(0, 1);
  __syncthreads();
  if (nkb > 1) {
    gload(1, 0);
    gload(1, 1);
  }
  int kb = 0;
  if constexpr (KFULL) {
    // k a multiple of 64: no bound checks on the loads, and stages in pairs
    // so that the LDS buffer of every stage is a compile-time constant (its
    // offset rides in the instructions' immediates).  kb is even after the
    // loop and at most three stages remain.
    for (; kb + 3 < nkb; kb += 2) {
      stage(kb, B0{}, true, true);
      stage(kb + 1, B1{}, true, true);
    }
    if (kb < nkb) stage(kb, B0{}, kb + 1 < nkb, kb + 2 < nkb);
    if (kb + 1 < nkb) stage(kb + 1, B1{}, kb + 2 < nkb, kb + 3 < nkb);
    if (kb + 2 < nkb) stage(kb + 2, B0{}, false, false);
  } else {
    for (; kb + 2 < nkb; ++kb) stage(kb, BR{}, true, true);
    if (kb + 1 < nkb) stage(kb++, BR{}, true, false);
    stage(kb, BR{}, false, false);
  }

  }
  // The epilogue's lane-derived values are recomputed from the lane index
  // rather than kept live across the k loop (which runs at the register limit).
  const int lane_e = lane_fresh();
  {
  const int lane = lane_e, tid = wave * 64 + lane_e;
  const int g = lane >> 5, c32 = lane & 31;
  const int g16 = lane >> 4, c16 = lane & 15;
  int urow16[GPW];
#pragma unroll
  for (int gg = 0; gg < GPW; ++gg) urow16[gg] = wm * WTI + 16 * (wn * GPW + gg) + c16;
  // ---- epilogue (LDS is free after the loop's last barrier).  Regions:
  // [0, XCH) the exchange of the k-half partial sums, later the per-wave
  // staging of the bf16 output block; then Us [2][BM][RP] fp32 (the two
  // k-half partials of U, summed in fixed order) and Bs [BN][RP] bf16 (B rows
  // of the tile, zero beyond r and n, staged in the prologue).  Two
  // barriers in all.
  float* Us = reinterpret_cast<float*>(smem + XCH);
  // Exchange region of (pair, destination half h): the partner's fragments
  // [fjl][fi][q4] as float4 x 64 lanes; wave wk keeps feature fragments
  // 2 wk, 2 wk + 1 and sends the other two.
  float4* xb = reinterpret_cast<float4*>(smem);
  const int pair = wm * 2 + wn;
  auto region = [&](int h) LORA_INLINE { return xb + (size_t)((pair * 2 + h) * 16) * 64; };
  {
    float4* dst = region(1 - wk);
#pragma unroll
    for (int fjl = 0; fjl < 2; ++fjl)
#pragma unroll
      for (int fi = 0; fi < FI; ++fi) {
        const floatx16 v = wk == 0 ? acc[2 + fjl][fi] : acc[fjl][fi];
#pragma unroll
        for (int q4 = 0; q4 < 4; ++q4)
          dst[((fjl * FI + fi) * 4 + q4) * 64 + lane] = float4{v[4 * q4], v[4 * q4 + 1], v[4 * q4 + 2], v[4 * q4 + 3]};
      }
  }
  if (!UPRE) {
#pragma unroll
    for (int gg = 0; gg < GPW; ++gg)
#pragma unroll
      for (int q = 0; q < 4; ++q) Us[(wk * BM + urow16[gg]) * RP + 4 * g16 + q] = uacc16[gg][q];
  }
  __syncthreads();
  {
    const float4* src = region(wk);
#pragma unroll
    for (int fjl = 0; fjl < 2; ++fjl)
#pragma unroll
      for (int fi = 0; fi < FI; ++fi)
#pragma unroll
        for (int q4 = 0; q4 < 4; ++q4) {
          const float4 o = src[((fjl * FI + fi) * 4 + q4) * 64 + lane];
          if (wk == 0) {
            acc[fjl][fi][4 * q4] += o.x; acc[fjl][fi][4 * q4 + 1] += o.y;
            acc[fjl][fi][4 * q4 + 2] += o.z; acc[fjl][fi][4 * q4 + 3] += o.w;
          } else {
            acc[2 + fjl][fi][4 * q4] += o.x; acc[2 + fjl][fi][4 * q4 + 1] += o.y;
            acc[2 + fjl][fi][4 * q4 + 2] += o.z; acc[2 + fjl][fi][4 * q4 + 3] += o.w;
          }
        }
  }
  if (UPRE) {   // U of the tile's tokens from the U pass (zero beyond r and m), all loads issued before the first use
    constexpr int UPT = BM * RP / NT;
    static_assert(BM * RP % NT == 0, "U values per thread");
    const __amdgpu_buffer_rsrc_t rsU = make_rsrc(U + (size_t)m0 * r, (uint64_t)min(BM, m - m0) * r * 4);
    float uv[UPT];
#pragma unroll
    for (int i = 0; i < UPT; ++i) {
      const int e = tid + i * NT, il = e / RP, t = e - il * RP;
      uv[i] = buf_load4f(rsU, t < r ? (uint32_t)(il * r + t) * 4 : kOOB);
    }
#pragma unroll
    for (int i = 0; i < UPT; ++i) Us[tid + i * NT] = uv[i];
  } else {
    // (the partial of half 1 is read here and written before the barrier above)
    for (int e = tid; e < BM * RP; e += NT) Us[e] = Us[e] + Us[BM * RP + e];
  }
  __syncthreads();
  if (n0 == 0 && !UPRE) {
    for (int e = tid; e < BM * RP; e += NT) {
      const int il = e / RP, t = e - il * RP;
      if (m0 + il < m && t < r) U[(size_t)(m0 + il) * r + t] = Us[e];
    }
  }
  // acc += s U B^T (high and low bf16 parts of s U), then Y rounded to bf16
  // on the wave's 64 x 64 block: features wn WTJ + 64 wk + 32 fjl, tokens
  // wm WTI + 32 fi, stored through a wave-private LDS region (the exchange
  // region is free after the barrier above).
  auto finish = [&](floatx16 (&a2)[FI], floatx16 (&b2)[FI]) {
    floatx16* own[2] = {a2, b2};
    const int t0 = 8 * g;
    short8 bfr[2];
#pragma unroll
    for (int fjl = 0; fjl < 2; ++fjl) {
      const int jl = wn * WTJ + 64 * wk + 32 * fjl + c32;
      bfr[fjl] = *reinterpret_cast<const short8*>(Bs + jl * RP + t0);
    }
#pragma unroll
    for (int fi = 0; fi < FI; ++fi) {
      const int il = wm * WTI + 32 * fi + c32;
      const float* up = Us + il * RP + t0;
      short8 uh, ul;
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const float v = s * up[e];
        const u16 hi = f32_to_bf16(v);
        uh[e] = (short)hi;
        ul[e] = (short)f32_to_bf16(v - bf16_to_f32(hi));
      }
#pragma unroll
      for (int fjl = 0; fjl < 2; ++fjl) {
        own[fjl][fi] = mfma32x32x16(bfr[fjl], uh, own[fjl][fi]);
        own[fjl][fi] = mfma32x32x16(bfr[fjl], ul, own[fjl][fi]);
      }
    }
    const int j0 = n0 + wn * WTJ + 64 * wk;
#pragma unroll
    for (int fi = 0; fi < FI; ++fi) {
      const int i0 = m0 + wm * WTI + 32 * fi;
      store_block_32x64(a2[fi], b2[fi], smem + wave * kYsBytes, Y + (size_t)i0 * n + j0, (size_t)n, m - i0, n - j0,
                        lane);
    }
  };
  static_assert(8 * kYsBytes <= XCH, "output staging fits the exchange region");
  if (wk == 0) finish(acc[0], acc[1]);
  else finish(acc[2], acc[3]);
  }
}

// ---------------------------------------------------------------------------
// Launchers: execute the plans of lora_plan.hpp.

// Instantiations a plan can name (any other combination is refused): U from
// the U pass for single projections of rank above 16, on the 256 x 256 tile
// and under dropout (where the pass applies the keep mask), in the tile for
// groups and rank 16 otherwise; the 128 x 256 tile at rank 16 is the k-split
// kernel's.
template <int BM, int BN, int RP, bool GRP, bool UPRE, bool KFULL, bool DMA>
constexpr bool fwd_instantiated() {
  return !(BM == 128 && BN == 256 && RP == 16) && (UPRE ? !GRP : (RP == 16 || GRP)) &&
         DMA == (KFULL && BM == 256 && BN == 256);
}

static hipError_t run_fwd_launch(const Launch& L, const FwdArgs& a, const FwdGroup& grp, hipStream_t st) {
  const dim3 grid((unsigned)L.grid), block((unsigned)L.block);
  if (L.id == K_UPASS) {
    return with_int<16, 32, 64>(L.rp, [&](auto rc) {
      return with_int<8, 16, 32>(L.tpw, [&](auto tc) {
        return with_bool(L.drop, [&](auto kc) {
          hipLaunchKernelGGL((lora_u_kernel<decltype(rc)::value, decltype(tc)::value, decltype(kc)::value>), grid,
                             block, 0, st, a.X, a.A, a.keep, a.U, (int)a.m, (int)a.k, (int)a.r, a.inv_keep);
          return hipGetLastError();
        });
      });
    });
  }
  if (L.id == K_FWD_KS) {
    return with_bool(L.grp, [&](auto gc) {
      return with_bool(L.full, [&](auto fc) {
        return with_bool(L.dma, [&](auto dc) {
          return with_bool(L.upre, [&](auto uc) {
            constexpr bool G = decltype(gc)::value, F = decltype(fc)::value, D = decltype(dc)::value,
                           UP = decltype(uc)::value;
            if constexpr ((D && (G || !F)) || (UP && (G || !F))) {   // (dropout: k a multiple of 64)
              return hipErrorInvalidValue;
            } else {
              hipLaunchKernelGGL((lora_fwd_ks_kernel<G, F, D, UP>), grid, block, 0, st, a.X, a.W, a.A, a.B, a.Y,
                                 a.U, (int)a.m, (int)a.n, (int)a.k, (int)a.r, a.s, L.tiles_m, L.tiles_n,
                                 (int)L.col_begin, grp);
              return hipGetLastError();
            }
          });
        });
      });
    });
  }
  if (L.id != K_FWD) return hipErrorInvalidValue;
  return with_int<0, 1, 2>(tile_code(L), [&](auto tc) {
    constexpr int T = decltype(tc)::value;
    constexpr int BM = T == 0 ? 256 : 128, BN = T == 2 ? 128 : 256, WN = T == 2 ? 2 : 4;
    return with_int<16, 32, 64>(L.rp, [&](auto rc) {
      return with_bool(L.grp, [&](auto gr) {
        return with_bool(L.upre, [&](auto up) {
          return with_bool(L.full, [&](auto kf) {
            return with_bool(L.dma, [&](auto dm) {
              constexpr int RP = decltype(rc)::value;
              constexpr bool GRP = decltype(gr)::value, UPRE = decltype(up)::value, KF = decltype(kf)::value,
                             DMA = decltype(dm)::value;
              if constexpr (!fwd_instantiated<BM, BN, RP, GRP, UPRE, KF, DMA>()) {
                return hipErrorInvalidValue;
              } else {
                hipLaunchKernelGGL((lora_fwd_kernel<BM, BN, 2, WN, RP, GRP, UPRE, KF, DMA>), grid, block, 0, st,
                                   a.X, a.W, a.A, a.B, a.Y, a.U, (int)a.m, (int)a.n, (int)a.k, (int)a.r, a.s,
                                   L.tiles_m, L.tiles_n, (int)L.col_begin, grp);
                return hipGetLastError();
              }
            });
          });
        });
      });
    });
  });
}

hipError_t launch_fwd(const FwdArgs& a, hipStream_t st) {
  const Plan p = plan_fwd(a.m, a.n, a.k, a.r, a.keep != nullptr);
  const FwdGroup none{};
  for (int i = 0; i < p.count; ++i) {
    const hipError_t e = run_fwd_launch(p.l[i], a, none, st);
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

// One launch for the whole group: each projection owns a run of column tiles
// (tile0 filled here for the plan's tile width).
hipError_t launch_fwd_group(const GroupFwdArgs& a, hipStream_t st) {
  const Plan p = plan_group_fwd(a.count, a.n, a.m, a.k, a.r);
  if (a.count == 1) {   // a group of one is the single projection
    FwdArgs f{};
    f.X = a.X; f.W = a.W[0]; f.A = a.A[0]; f.B = a.B[0]; f.Y = a.Y[0]; f.U = a.U[0];
    f.m = a.m; f.n = a.n[0]; f.k = a.k; f.r = a.r; f.s = a.s;
    return launch_fwd(f, st);
  }
  FwdGroup grp{};
  for (int g = 0; g < a.count; ++g) {
    grp.W[g] = a.W[g]; grp.A[g] = a.A[g]; grp.B[g] = a.B[g]; grp.Y[g] = a.Y[g]; grp.U[g] = a.U[g];
    grp.n[g] = (int)a.n[g];
  }
  grp.count = a.count;
  FwdArgs f{};
  f.X = a.X;
  f.m = a.m; f.n = 0; f.k = a.k; f.r = a.r; f.s = a.s;
  for (int i = 0; i < p.count; ++i) {
    const Launch& L = p.l[i];
    int t0 = 0;
    for (int g = 0; g < a.count; ++g) {
      grp.tile0[g] = t0;
      t0 += (grp.n[g] + L.bn - 1) / L.bn;
    }
    const hipError_t e = run_fwd_launch(L, f, grp, st);
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

}  // namespace lora
