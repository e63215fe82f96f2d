// Backward of the LoRA-adapted linear layer (chain rule through Eq. 1 of JORA,
// Section 3, for the trainable A and B; W0 is frozen so no dW is formed):
//   dU = s dY B,   dX = dY W + dU A,   dB = s dY^T U,   dA = dU^T X.
//
// Kernels, in stream order:
//   prep      Bt = B^T (rank padded to RP with zeros); Ut2 = U^T split into a
//             bf16 high part and a bf16 low part (tokens padded to mp).
//   du        dU = s dY B, reducing over n.  Writes dU2 (token-major, high |
//             low) for the dX GEMM and dUt2 (its transpose) for dA.
//   tokred    dB^T partials = Ut2 . dY over token ranges (split-K over m).
//   dx        dX = [dY | dU2] . [W ; A ; A]: one GEMM whose k loop runs over
//             n and then over the 2 RP wide slab (high and low part of dU
//             against the same A rows).  W is read through LDS with the
//             transposing ds_read_b64_tr_b16, since the product contracts
//             W over its rows.
//   tokred    dA partials = dUt2 . X over token ranges.
//   finalize  sums the partials of dB and dA in a fixed order (no atomics, so
//             results are bit-identical from run to run) and applies s to dB.
#include "lora_device.hpp"
#include "lora_launch.hpp"

namespace lora {

// ---------------------------------------------------------------------------
__global__ __launch_bounds__(256) void lora_bwd_prep_kernel(
    const u16* __restrict__ B, const float* __restrict__ U, u16* __restrict__ Bt,
    u16* __restrict__ Ut2, int m, int n, int r, int rp, int mp) {
  const int64_t nbt = (int64_t)rp * n;
  const int64_t nut = (int64_t)2 * rp * mp;
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; e < nbt + nut; e += stride) {
    if (e < nbt) {
      const int t = (int)(e / n);
      const int j = (int)(e - (int64_t)t * n);
      Bt[e] = (t < r) ? B[(int64_t)j * r + t] : (u16)0;
    } else {
      const int64_t f = e - nbt;
      const int tt = (int)(f / mp);
      const int i = (int)(f - (int64_t)tt * mp);
      const int t = tt % rp;
      const float v = (i < m && t < r) ? U[(int64_t)i * r + t] : 0.f;
      const u16 h = f32_to_bf16(v);
      Ut2[f] = (tt >= rp) ? f32_to_bf16(v - bf16_to_f32(h)) : h;
    }
  }
}

// ---------------------------------------------------------------------------
// dU for 16 tokens per workgroup; the 4 waves take interleaved 32-wide chunks
// of n and their partial sums are added in wave order through LDS.
template <int RP>
__global__ __launch_bounds__(256) void lora_bwd_du_kernel(
    const u16* __restrict__ dY, const u16* __restrict__ Bt, u16* __restrict__ dU2,
    u16* __restrict__ dUt2, int m, int n, int mp, float s) {
  constexpr int FT = RP / 16;
  __shared__ floatx4 red[4][FT][64];
  const int i0 = blockIdx.x * 16;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int g = lane >> 4, c16 = lane & 15;
  const uint32_t rowbytes = (uint32_t)n * 2;
  const int rows = max(0, min(16, m - i0));
  const __amdgpu_buffer_rsrc_t rsY = make_rsrc(dY + (size_t)i0 * n, (uint64_t)rows * rowbytes);
  const __amdgpu_buffer_rsrc_t rsB = make_rsrc(Bt, (uint64_t)RP * rowbytes);

  floatx4 acc[FT];
#pragma unroll
  for (int ft = 0; ft < FT; ++ft) acc[ft] = floatx4{0.f, 0.f, 0.f, 0.f};

  const int nch = (n + 31) / 32;
#pragma unroll 4
  for (int c = wave; c < nch; c += 4) {
    const int j = c * 32 + 8 * g;
    const bool ok = j < n;
    const short8 yf = __builtin_bit_cast(short8, buf_load16(rsY, ok ? (uint32_t)c16 * rowbytes + (uint32_t)j * 2 : kOOB));
#pragma unroll
    for (int ft = 0; ft < FT; ++ft) {
      const short8 bf = __builtin_bit_cast(
          short8, buf_load16(rsB, ok ? (uint32_t)(16 * ft + c16) * rowbytes + (uint32_t)j * 2 : kOOB));
      acc[ft] = mfma16x16x32(bf, yf, acc[ft]);
    }
  }
#pragma unroll
  for (int ft = 0; ft < FT; ++ft) red[wave][ft][lane] = acc[ft];
  __syncthreads();
  if (wave != 0) return;
  const int i = i0 + c16;  // < mp: the grid covers exactly mp tokens
#pragma unroll
  for (int ft = 0; ft < FT; ++ft) {
    const floatx4 v = ((red[0][ft][lane] + red[1][ft][lane]) + red[2][ft][lane]) + red[3][ft][lane];
    u16 hi[4], lo[4];
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const float d = s * v[q];
      hi[q] = f32_to_bf16(d);
      lo[q] = f32_to_bf16(d - bf16_to_f32(hi[q]));
    }
    const int t = 16 * ft + 4 * g;
    u16* row = dU2 + (size_t)i * (2 * RP);
    *reinterpret_cast<uint2*>(row + t) =
        uint2{(uint32_t)hi[0] | ((uint32_t)hi[1] << 16), (uint32_t)hi[2] | ((uint32_t)hi[3] << 16)};
    *reinterpret_cast<uint2*>(row + RP + t) =
        uint2{(uint32_t)lo[0] | ((uint32_t)lo[1] << 16), (uint32_t)lo[2] | ((uint32_t)lo[3] << 16)};
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      dUt2[(size_t)(t + q) * mp + i] = hi[q];
      dUt2[(size_t)(RP + t + q) * mp + i] = lo[q];
    }
  }
}

// ---------------------------------------------------------------------------
// Token reduction part[sp][t][c] = sum over tokens i of split sp of
// P[t][i] * Q[i][c], t < RP (the high and low rows of P are summed), for a
// tile of kRedCols columns.  P ([2RP][mp], token-contiguous) is read straight
// into matrix-core A operands; Q ([m][cols]) is staged in LDS 64 tokens at a
// time and read transposed.
template <int NW, int RP>
__global__ __launch_bounds__(64 * NW) void lora_tokred_kernel(
    const u16* __restrict__ P, const u16* __restrict__ Q, float* __restrict__ part,
    int m, int mp, int ncols, int span) {
  constexpr int BNC = kRedCols;
  constexpr int NT = 64 * NW;
  constexpr int WC = BNC / NW;
  constexpr int FC = WC / 16;
  constexpr int FH = RP / 16;     // high-part row fragments; low part follows
  constexpr int FP = 2 * FH;
  constexpr int CPR = BNC / 8;    // 16-byte chunks per Q row
  constexpr int STAGE = 64 * BNC * 2;
  constexpr int CH = 64 * CPR;
  constexpr int LOADS = CH / NT;
  static_assert(CH % NT == 0 && WC % 16 == 0, "shape split");
  __shared__ __attribute__((aligned(16))) char smem[2 * STAGE];

  const int c0 = blockIdx.x * BNC;
  const int sp = blockIdx.y;
  const int tb = sp * span;
  const int te = min(mp, tb + span);
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int g = lane >> 4, c16 = lane & 15;
  const uint32_t qrow = (uint32_t)ncols * 2;
  const __amdgpu_buffer_rsrc_t rsP = make_rsrc(P, (uint64_t)2 * RP * mp * 2);

  int4v qregs[LOADS];
  short8 pcur[2][FP], pnext[2][FP];
  auto gload = [&](int tc, short8 (&pf)[2][FP]) {
    const int rows = max(0, min(64, m - tc));
    const __amdgpu_buffer_rsrc_t rsQ = make_rsrc(Q + (size_t)tc * ncols, (uint64_t)rows * qrow);
#pragma unroll
    for (int i = 0; i < LOADS; ++i) {
      const int q = tid + i * NT;
      const int rho = q / CPR, c = q % CPR;
      const int cc = c0 + 8 * c;
      qregs[i] = buf_load16(rsQ, cc < ncols ? (uint32_t)rho * qrow + (uint32_t)cc * 2 : kOOB);
    }
#pragma unroll
    for (int ks = 0; ks < 2; ++ks)
#pragma unroll
      for (int f = 0; f < FP; ++f)
        pf[ks][f] = __builtin_bit_cast(
            short8, buf_load16(rsP, ((uint32_t)(16 * f + c16) * (uint32_t)mp + (uint32_t)(tc + 32 * ks + 8 * g)) * 2));
  };
  auto swrite = [&](int buf) {
    char* sb = smem + buf * STAGE;
#pragma unroll
    for (int i = 0; i < LOADS; ++i) {
      const int q = tid + i * NT;
      *reinterpret_cast<int4v*>(sb + mc_offset<BNC>(q / CPR, q % CPR)) = qregs[i];
    }
  };

  floatx4 acc[FP][FC];
#pragma unroll
  for (int f = 0; f < FP; ++f)
#pragma unroll
    for (int fc = 0; fc < FC; ++fc) acc[f][fc] = floatx4{0.f, 0.f, 0.f, 0.f};

  if (tb < te) {
    gload(tb, pcur);
    swrite(0);
    __syncthreads();
    int buf = 0;
    for (int tc = tb; tc < te; tc += 64) {
      const bool more = tc + 64 < te;
      if (more) gload(tc + 64, pnext);
      const char* Qs = smem + buf * STAGE;
#pragma unroll
      for (int ks = 0; ks < 2; ++ks) {
#pragma unroll
        for (int fc = 0; fc < FC; ++fc) {
          const short8 qf = mc_read_tr<BNC>(Qs, 32 * ks, wave * WC + 16 * fc, lane);
#pragma unroll
          for (int f = 0; f < FP; ++f) acc[f][fc] = mfma16x16x32(pcur[ks][f], qf, acc[f][fc]);
        }
      }
      if (more) {
        swrite(buf ^ 1);
#pragma unroll
        for (int ks = 0; ks < 2; ++ks)
#pragma unroll
          for (int f = 0; f < FP; ++f) pcur[ks][f] = pnext[ks][f];
      }
      __syncthreads();
      buf ^= 1;
    }
  }

  // lane holds column c16 of fragment fc, rows 4g..4g+3 of fragment f
#pragma unroll
  for (int fc = 0; fc < FC; ++fc) {
    const int col = c0 + wave * WC + 16 * fc + c16;
    if (col >= ncols) continue;
#pragma unroll
    for (int f = 0; f < FH; ++f)
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const int t = 16 * f + 4 * g + q;
        part[((size_t)sp * RP + t) * ncols + col] = acc[f][fc][q] + acc[f + FH][fc][q];
      }
  }
}

// ---------------------------------------------------------------------------
__global__ __launch_bounds__(256) void lora_bwd_finalize_kernel(
    const float* __restrict__ pb, const float* __restrict__ pa, float* __restrict__ dB,
    float* __restrict__ dA, int n, int k, int r, int rp, int sb, int sa, float s) {
  const int64_t nb = (int64_t)n * r, na = (int64_t)r * k;
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; e < nb + na; e += stride) {
    if (e < nb) {  // e = t * n + j: partial reads along j are contiguous
      const int t = (int)(e / n), j = (int)(e - (int64_t)t * n);
      float v = 0.f;
      for (int p = 0; p < sb; ++p) v += pb[((size_t)p * rp + t) * n + j];
      dB[(size_t)j * r + t] = s * v;
    } else {
      const int64_t f = e - nb;
      const int t = (int)(f / k), l = (int)(f - (int64_t)t * k);
      float v = 0.f;
      for (int p = 0; p < sa; ++p) v += pa[((size_t)p * rp + t) * k + l];
      dA[f] = v;
    }
  }
}

// ---------------------------------------------------------------------------
// dX tile of BM tokens x BN input features.  Stages: dY [BM][64] (k = n
// contiguous) and W [64 rows of n][BN] (mn-contiguous, read transposed); after
// the n loop, NSLAB stages of the 2RP slab: dU2 [BM][2RP] and A rows repeated
// for the high and low parts.
template <int BM, int BN, int WM, int WN, int RP>
__global__ __launch_bounds__(64 * WM * WN) void lora_bwd_dx_kernel(
    const u16* __restrict__ dY, const u16* __restrict__ W, const u16* __restrict__ dU2,
    const u16* __restrict__ A, u16* __restrict__ dX, int m, int n, int k, int r, int mp,
    int tiles_m, int tiles_n) {
  constexpr int NT = 64 * WM * WN;
  constexpr int WTM = BM / WM, WTN = BN / WN;
  constexpr int FI = WTM / 16, FJ = WTN / 16;
  constexpr int STAGE = (BM + BN) * 128;
  constexpr int CH_Y = BM * 8;
  constexpr int CPR = BN / 8;
  constexpr int CH = CH_Y + 64 * CPR;
  constexpr int LOADS = (CH + NT - 1) / NT;
  constexpr int KS2 = 2 * RP;
  constexpr int NSLAB = (KS2 + 63) / 64;
  static_assert(BM % (16 * WM) == 0 && BN % (16 * WN) == 0, "tile/wave split");
  static_assert(CH_Y % 64 == 0 && CH % 64 == 0 && BN >= 128, "wave-uniform staging");
  static_assert(2 * STAGE <= 160 * 1024, "LDS budget");
  __shared__ __attribute__((aligned(16))) char smem[2 * STAGE];

  int tm, tn;
  tile_coords(tiles_m, tiles_n, 8, tm, tn);
  const int m0 = tm * BM, l0 = tn * BN;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave / WN, wn = wave % WN;
  const int g = lane >> 4, c16 = lane & 15;
  const uint32_t yrow = (uint32_t)n * 2, wrow = (uint32_t)k * 2, urow = (uint32_t)KS2 * 2;
  const __amdgpu_buffer_rsrc_t rsY = make_rsrc(dY + (size_t)m0 * n, (uint64_t)min(BM, m - m0) * yrow);
  const __amdgpu_buffer_rsrc_t rsU = make_rsrc(dU2 + (size_t)m0 * KS2, (uint64_t)min(BM, mp - m0) * urow);
  const __amdgpu_buffer_rsrc_t rsA = make_rsrc(A, (uint64_t)r * wrow);
  const int nkb = (n + 63) / 64;
  const int nst = nkb + NSLAB;

  int4v regs[LOADS];
  auto gload = [&](int st) {
    if (st < nkb) {
      const int n0 = st * 64;
      const __amdgpu_buffer_rsrc_t rsW = make_rsrc(W + (size_t)n0 * k, (uint64_t)min(64, n - n0) * wrow);
#pragma unroll
      for (int i = 0; i < LOADS; ++i) {
        const int q = tid + i * NT;
        if (CH % NT != 0 && q >= CH) break;  // wave-uniform
        if (q < CH_Y) {
          const int row = q >> 3, nn = n0 + 8 * (q & 7);
          regs[i] = buf_load16(rsY, nn < n ? (uint32_t)row * yrow + (uint32_t)nn * 2 : kOOB);
        } else {
          const int q2 = q - CH_Y, rho = q2 / CPR, ll = l0 + 8 * (q2 % CPR);
          regs[i] = buf_load16(rsW, ll < k ? (uint32_t)rho * wrow + (uint32_t)ll * 2 : kOOB);
        }
      }
    } else {
      const int kk0 = (st - nkb) * 64;
#pragma unroll
      for (int i = 0; i < LOADS; ++i) {
        const int q = tid + i * NT;
        if (CH % NT != 0 && q >= CH) break;
        if (q < CH_Y) {
          const int row = q >> 3, kk = kk0 + 8 * (q & 7);
          regs[i] = buf_load16(rsU, kk < KS2 ? (uint32_t)row * urow + (uint32_t)kk * 2 : kOOB);
        } else {
          const int q2 = q - CH_Y, kk = kk0 + q2 / CPR, ll = l0 + 8 * (q2 % CPR);
          const int t = kk % RP;
          const bool ok = kk < KS2 && t < r && ll < k;
          regs[i] = buf_load16(rsA, ok ? (uint32_t)t * wrow + (uint32_t)ll * 2 : kOOB);
        }
      }
    }
  };
  auto swrite = [&](int buf) {
    char* sb = smem + buf * STAGE;
#pragma unroll
    for (int i = 0; i < LOADS; ++i) {
      const int q = tid + i * NT;
      if (CH % NT != 0 && q >= CH) break;
      if (q < CH_Y) {
        *reinterpret_cast<int4v*>(sb + kc_offset(q >> 3, q & 7)) = regs[i];
      } else {
        const int q2 = q - CH_Y;
        *reinterpret_cast<int4v*>(sb + BM * 128 + mc_offset<BN>(q2 / CPR, q2 % CPR)) = regs[i];
      }
    }
  };

  floatx4 acc[FJ][FI];
#pragma unroll
  for (int a = 0; a < FJ; ++a)
#pragma unroll
    for (int b = 0; b < FI; ++b) acc[a][b] = floatx4{0.f, 0.f, 0.f, 0.f};

  gload(0);
  swrite(0);
  __syncthreads();
  for (int st = 0; st < nst; ++st) {
    const bool more = st + 1 < nst;
    if (more) gload(st + 1);
    const char* sb = smem + (st & 1) * STAGE;
    const char* Ys = sb;
    const char* Ws = sb + BM * 128;
#pragma unroll
    for (int ks = 0; ks < 2; ++ks) {
      short8 wf[FJ];
#pragma unroll
      for (int fj = 0; fj < FJ; ++fj) wf[fj] = mc_read_tr<BN>(Ws, 32 * ks, wn * WTN + 16 * fj, lane);
#pragma unroll
      for (int fi = 0; fi < FI; ++fi) {
        const short8 yf = kc_read(Ys, wm * WTM + 16 * fi + c16, 4 * ks + g);
#pragma unroll
        for (int fj = 0; fj < FJ; ++fj) acc[fj][fi] = mfma16x16x32(wf[fj], yf, acc[fj][fi]);
      }
    }
    if (more) swrite((st + 1) & 1);
    __syncthreads();
  }

#pragma unroll
  for (int fi = 0; fi < FI; ++fi) {
    const int i = m0 + wm * WTM + 16 * fi + c16;
    if (i >= m) continue;
#pragma unroll
    for (int fj = 0; fj < FJ; ++fj) {
      const int l = l0 + wn * WTN + 16 * fj + 4 * g;
      if (l >= k) continue;
      const uint32_t lo = (uint32_t)f32_to_bf16(acc[fj][fi][0]) | ((uint32_t)f32_to_bf16(acc[fj][fi][1]) << 16);
      const uint32_t hi = (uint32_t)f32_to_bf16(acc[fj][fi][2]) | ((uint32_t)f32_to_bf16(acc[fj][fi][3]) << 16);
      *reinterpret_cast<uint2*>(dX + (size_t)i * k + l) = uint2{lo, hi};
    }
  }
}

// ---------------------------------------------------------------------------
template <int BM, int BN, int WM, int WN, int RP>
static hipError_t launch_dx_cfg(const BwdArgs& a, const BwdLayout& L, hipStream_t st) {
  const int tiles_m = (int)((a.m + BM - 1) / BM), tiles_n = (int)((a.k + BN - 1) / BN);
  hipLaunchKernelGGL((lora_bwd_dx_kernel<BM, BN, WM, WN, RP>), dim3(tiles_m * tiles_n), dim3(64 * WM * WN), 0, st,
                     a.dY, a.W, reinterpret_cast<const u16*>(a.ws + L.du2), a.A, a.dX, (int)a.m, (int)a.n,
                     (int)a.k, (int)a.r, (int)L.mp, tiles_m, tiles_n);
  return hipGetLastError();
}

template <int RP>
static hipError_t launch_bwd_rp(const BwdArgs& a, const BwdLayout& L, hipStream_t st) {
  const int m = (int)a.m, n = (int)a.n, k = (int)a.k, r = (int)a.r, mp = (int)L.mp;
  u16* Bt = reinterpret_cast<u16*>(a.ws + L.bt);
  u16* Ut2 = reinterpret_cast<u16*>(a.ws + L.ut2);
  u16* dU2 = reinterpret_cast<u16*>(a.ws + L.du2);
  u16* dUt2 = reinterpret_cast<u16*>(a.ws + L.dut2);
  float* pb = reinterpret_cast<float*>(a.ws + L.pb);
  float* pa = reinterpret_cast<float*>(a.ws + L.pa);
  hipError_t e;

  {
    const int64_t total = (int64_t)RP * n + (int64_t)2 * RP * mp;
    const int blocks = (int)std::min<int64_t>((total + 255) / 256, 4096);
    hipLaunchKernelGGL(lora_bwd_prep_kernel, dim3(blocks), dim3(256), 0, st, a.B, a.U, Bt, Ut2, m, n, r, RP, mp);
    if ((e = hipGetLastError()) != hipSuccess) return e;
  }
  hipLaunchKernelGGL((lora_bwd_du_kernel<RP>), dim3(mp / 16), dim3(256), 0, st, a.dY, Bt, dU2, dUt2, m, n, mp, a.s);
  if ((e = hipGetLastError()) != hipSuccess) return e;

  hipLaunchKernelGGL((lora_tokred_kernel<4, RP>), dim3(L.plan_b.col_tiles, L.plan_b.splits), dim3(256), 0, st,
                     Ut2, a.dY, pb, m, mp, n, (int)L.plan_b.span);
  if ((e = hipGetLastError()) != hipSuccess) return e;

  switch (choose_gemm_tile(a.m, a.k)) {
    case TILE_256x256: e = launch_dx_cfg<256, 256, 2, 4, RP>(a, L, st); break;
    case TILE_256x128: e = launch_dx_cfg<256, 128, 4, 2, RP>(a, L, st); break;
    default: e = launch_dx_cfg<128, 128, 2, 2, RP>(a, L, st); break;
  }
  if (e != hipSuccess) return e;

  hipLaunchKernelGGL((lora_tokred_kernel<4, RP>), dim3(L.plan_a.col_tiles, L.plan_a.splits), dim3(256), 0, st,
                     dUt2, a.X, pa, m, mp, k, (int)L.plan_a.span);
  if ((e = hipGetLastError()) != hipSuccess) return e;

  {
    const int64_t total = (int64_t)n * r + (int64_t)r * k;
    const int blocks = (int)std::min<int64_t>((total + 255) / 256, 4096);
    hipLaunchKernelGGL(lora_bwd_finalize_kernel, dim3(blocks), dim3(256), 0, st, pb, pa, a.dB, a.dA, n, k, r, RP,
                       L.plan_b.splits, L.plan_a.splits, a.s);
    if ((e = hipGetLastError()) != hipSuccess) return e;
  }
  return hipSuccess;
}

hipError_t launch_bwd(const BwdArgs& a, hipStream_t st) {
  const BwdLayout L = bwd_layout(a.m, a.n, a.k, a.r);
  switch (L.rp) {
    case 16: return launch_bwd_rp<16>(a, L, st);
    case 32: return launch_bwd_rp<32>(a, L, st);
    case 48: return launch_bwd_rp<48>(a, L, st);
    default: return launch_bwd_rp<64>(a, L, st);
  }
}

}  // namespace lora
