// Forward of the LoRA-adapted linear layer (Eq. 1 of JORA, Section 3):
//   U = X A^T,   Y = X W^T + s U B^T,   s = alpha / r.
//
// One kernel.  Each workgroup owns a BM x BN tile of Y (BM tokens x BN output
// features) and walks k in steps of 64.  Per step it stages three
// k-contiguous tiles in LDS -- X[BM rows], W[BN rows] and the padded LoRA
// down-projection A[RP rows] -- so each X tile is read from memory once and
// feeds both the W columns and the r extra "U columns".  Matrix-core products
// are formed transposed (W and A as the A operand, X as the B operand), so a
// lane's accumulator holds 4 consecutive output features of one token.
//
// U work is split over the waves that share a token range.  After the k loop
// the epilogue parks U in LDS, writes it out (tile column 0 only), and adds
// s U B^T to the accumulators with one more matrix-core pass in which s U
// enters as a bf16 high part and a bf16 low part (K = 2 x 16 per pass), then
// rounds Y to bf16.
#include "lora_device.hpp"
#include "lora_launch.hpp"

namespace lora {

template <int BM, int BN, int WM, int WN, int RP>
__global__ __launch_bounds__(64 * WM * WN) void lora_fwd_kernel(
    const u16* __restrict__ X, const u16* __restrict__ W, const u16* __restrict__ A,
    const u16* __restrict__ B, u16* __restrict__ Y, float* __restrict__ U,
    int m, int n, int k, int r, float s, int tiles_m, int tiles_n) {
  constexpr int NT = 64 * WM * WN;
  constexpr int WTM = BM / WM, WTN = BN / WN;
  constexpr int FI = WTM / 16;   // token fragments per wave (B operand)
  constexpr int FJ = WTN / 16;   // feature fragments per wave (A operand)
  constexpr int FT = RP / 16;    // U row fragments
  constexpr int FU = FI / WN;    // token fragments of U per wave
  constexpr int ROWS = BM + BN + RP;
  constexpr int STAGE = ROWS * 128;
  constexpr int CHUNKS = ROWS * 8;
  constexpr int LOADS = (CHUNKS + NT - 1) / NT;
  static_assert(BM % (16 * WM) == 0 && BN % (16 * WN) == 0, "tile/wave split");
  static_assert(FI % WN == 0 && FU >= 1, "U fragments must split evenly over waves");
  static_assert(CHUNKS % 64 == 0, "a wave's 64 chunks are 8 whole rows");
  static_assert(BM % 8 == 0 && BN % 8 == 0 && RP % 16 == 0, "row groups of 8 stay in one matrix");
  static_assert(2 * STAGE <= 160 * 1024, "LDS budget");
  static_assert(BM * RP * 4 + BN * RP * 2 <= 2 * STAGE, "epilogue LDS reuse");

  __shared__ __attribute__((aligned(16))) char smem[2 * STAGE];

  int tm, tn;
  tile_coords(tiles_m, tiles_n, 8, tm, tn);
  const int m0 = tm * BM, n0 = tn * BN;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave / WN, wn = wave % WN;
  const int g = lane >> 4, c16 = lane & 15;

  const uint32_t rowbytes = (uint32_t)k * 2;
  const __amdgpu_buffer_rsrc_t rsX = make_rsrc(X + (size_t)m0 * k, (uint64_t)min(BM, m - m0) * rowbytes);
  const __amdgpu_buffer_rsrc_t rsW = make_rsrc(W + (size_t)n0 * k, (uint64_t)min(BN, n - n0) * rowbytes);
  const __amdgpu_buffer_rsrc_t rsA = make_rsrc(A, (uint64_t)r * rowbytes);

  // Per-thread staging: chunk id q = tid + i*NT -> row q/8, k-chunk q%8.
  int4v stage_regs[LOADS];
  auto gload = [&](int kb) {
    const int k0 = kb * 64;
#pragma unroll
    for (int i = 0; i < LOADS; ++i) {
      const int q = tid + i * NT;
      if (CHUNKS % NT != 0 && q >= CHUNKS) break;  // wave-uniform
      const int row = q >> 3, ch = q & 7;
      const int kk = k0 + ch * 8;
      // rows in groups of 8 never straddle X/W/A, so the choice below is wave-uniform
      if (row < BM) {
        uint32_t off = (kk < k) ? (uint32_t)row * rowbytes + (uint32_t)kk * 2 : kOOB;
        stage_regs[i] = buf_load16(rsX, off);
      } else if (row < BM + BN) {
        uint32_t off = (kk < k) ? (uint32_t)(row - BM) * rowbytes + (uint32_t)kk * 2 : kOOB;
        stage_regs[i] = buf_load16(rsW, off);
      } else {
        uint32_t off = (kk < k) ? (uint32_t)(row - BM - BN) * rowbytes + (uint32_t)kk * 2 : kOOB;
        stage_regs[i] = buf_load16(rsA, off);
      }
    }
  };
  auto swrite = [&](int buf) {
    char* sb = smem + buf * STAGE;
#pragma unroll
    for (int i = 0; i < LOADS; ++i) {
      const int q = tid + i * NT;
      if (CHUNKS % NT != 0 && q >= CHUNKS) break;
      *reinterpret_cast<int4v*>(sb + kc_offset(q >> 3, q & 7)) = stage_regs[i];
    }
  };

  floatx4 acc[FJ][FI];
  floatx4 uacc[FT][FU];
#pragma unroll
  for (int a = 0; a < FJ; ++a)
#pragma unroll
    for (int b = 0; b < FI; ++b) acc[a][b] = floatx4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int a = 0; a < FT; ++a)
#pragma unroll
    for (int b = 0; b < FU; ++b) uacc[a][b] = floatx4{0.f, 0.f, 0.f, 0.f};

  const int nkb = (k + 63) / 64;
  gload(0);
  swrite(0);
  __syncthreads();

  for (int kb = 0; kb < nkb; ++kb) {
    const bool more = kb + 1 < nkb;
    if (more) gload(kb + 1);
    const char* sb = smem + (kb & 1) * STAGE;
    const char* Xs = sb;
    const char* Ws = sb + BM * 128;
    const char* As = sb + (BM + BN) * 128;
#pragma unroll
    for (int ks = 0; ks < 2; ++ks) {
      const int ch = 4 * ks + g;
      short8 wf[FJ];
#pragma unroll
      for (int fj = 0; fj < FJ; ++fj) wf[fj] = kc_read(Ws, wn * WTN + 16 * fj + c16, ch);
#pragma unroll
      for (int fi = 0; fi < FI; ++fi) {
        const short8 xf = kc_read(Xs, wm * WTM + 16 * fi + c16, ch);
#pragma unroll
        for (int fj = 0; fj < FJ; ++fj) acc[fj][fi] = mfma16x16x32(wf[fj], xf, acc[fj][fi]);
      }
      short8 af[FT];
#pragma unroll
      for (int ft = 0; ft < FT; ++ft) af[ft] = kc_read(As, 16 * ft + c16, ch);
#pragma unroll
      for (int fu = 0; fu < FU; ++fu) {
        const short8 xf = kc_read(Xs, wm * WTM + 16 * (wn * FU + fu) + c16, ch);
#pragma unroll
        for (int ft = 0; ft < FT; ++ft) uacc[ft][fu] = mfma16x16x32(af[ft], xf, uacc[ft][fu]);
      }
    }
    if (more) swrite((kb + 1) & 1);
    __syncthreads();
  }

  // ---- epilogue ------------------------------------------------------------
  // LDS reuse: Us [BM][RP] fp32, then Bs [BN][RP] bf16 (B rows of this tile,
  // zero beyond r and n).
  float* Us = reinterpret_cast<float*>(smem);
  u16* Bs = reinterpret_cast<u16*>(smem + BM * RP * 4);
  const bool write_u = (tn == 0);
#pragma unroll
  for (int ft = 0; ft < FT; ++ft)
#pragma unroll
    for (int fu = 0; fu < FU; ++fu) {
      const int il = wm * WTM + 16 * (wn * FU + fu) + c16;
      const int i = m0 + il;
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const int t = 16 * ft + 4 * g + q;
        Us[il * RP + t] = uacc[ft][fu][q];
        if (write_u && i < m && t < r) U[(size_t)i * r + t] = uacc[ft][fu][q];
      }
    }
  for (int e = tid; e < BN * RP; e += NT) {
    const int j = e / RP, t = e - j * RP;
    Bs[e] = (n0 + j < n && t < r) ? B[(size_t)(n0 + j) * r + t] : (u16)0;
  }
  __syncthreads();

  // acc += s U B^T as Y^T += B (sU)^T, K = [t block of 16: hi | lo]
#pragma unroll
  for (int tb = 0; tb < FT; ++tb) {
    const int t0 = 16 * tb + 8 * (g & 1);
    short8 bfr[FJ];
#pragma unroll
    for (int fj = 0; fj < FJ; ++fj) {
      const int jl = wn * WTN + 16 * fj + c16;
      bfr[fj] = *reinterpret_cast<const short8*>(Bs + jl * RP + t0);
    }
#pragma unroll
    for (int fi = 0; fi < FI; ++fi) {
      const int il = wm * WTM + 16 * fi + c16;
      const float* up = Us + il * RP + t0;
      short8 uf;
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const float v = s * up[e];
        const u16 hi = f32_to_bf16(v);
        const u16 lo = f32_to_bf16(v - bf16_to_f32(hi));
        uf[e] = (short)(g < 2 ? hi : lo);
      }
#pragma unroll
      for (int fj = 0; fj < FJ; ++fj) acc[fj][fi] = mfma16x16x32(bfr[fj], uf, acc[fj][fi]);
    }
  }

  // store Y: lane holds token (column c16) and 4 consecutive features (rows 4g..4g+3)
#pragma unroll
  for (int fi = 0; fi < FI; ++fi) {
    const int i = m0 + wm * WTM + 16 * fi + c16;
    if (i >= m) continue;
#pragma unroll
    for (int fj = 0; fj < FJ; ++fj) {
      const int j = n0 + wn * WTN + 16 * fj + 4 * g;
      if (j >= n) continue;
      const uint32_t lo = (uint32_t)f32_to_bf16(acc[fj][fi][0]) | ((uint32_t)f32_to_bf16(acc[fj][fi][1]) << 16);
      const uint32_t hi = (uint32_t)f32_to_bf16(acc[fj][fi][2]) | ((uint32_t)f32_to_bf16(acc[fj][fi][3]) << 16);
      *reinterpret_cast<uint2*>(Y + (size_t)i * n + j) = uint2{lo, hi};
    }
  }
}

template <int BM, int BN, int WM, int WN, int RP>
static hipError_t launch_fwd_cfg(const FwdArgs& a, hipStream_t st) {
  const int tiles_m = (int)((a.m + BM - 1) / BM), tiles_n = (int)((a.n + BN - 1) / BN);
  const int blocks = tiles_m * tiles_n;
  hipLaunchKernelGGL((lora_fwd_kernel<BM, BN, WM, WN, RP>), dim3(blocks), dim3(64 * WM * WN), 0, st,
                     a.X, a.W, a.A, a.B, a.Y, a.U, (int)a.m, (int)a.n, (int)a.k, (int)a.r, a.s,
                     tiles_m, tiles_n);
  return hipGetLastError();
}

template <int BM, int BN, int WM, int WN>
static hipError_t launch_fwd_rp(const FwdArgs& a, hipStream_t st) {
  switch (pad_rank(a.r)) {
    case 16: return launch_fwd_cfg<BM, BN, WM, WN, 16>(a, st);
    case 32: return launch_fwd_cfg<BM, BN, WM, WN, 32>(a, st);
    case 48: return launch_fwd_cfg<BM, BN, WM, WN, 48>(a, st);
    default: return launch_fwd_cfg<BM, BN, WM, WN, 64>(a, st);
  }
}

hipError_t launch_fwd(const FwdArgs& a, hipStream_t st) {
  switch (choose_gemm_tile(a.m, a.n)) {
    case TILE_256x256: return launch_fwd_rp<256, 256, 2, 4>(a, st);
    case TILE_256x128: return launch_fwd_rp<256, 128, 4, 2>(a, st);
    default: return launch_fwd_rp<128, 128, 2, 2>(a, st);
  }
}

}  // namespace lora
