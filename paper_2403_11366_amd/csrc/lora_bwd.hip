// Backward of the LoRA-adapted linear layer (chain rule through Eq. 1 of JORA,
// Section 3, for the trainable A and B; W0 is frozen so no dW is formed):
//   dU = s dY B,   dX = dY W + dU A,   dB = s dY^T U,   dA = dU^T X.
//
// Kernels, in stream order (three launches, four when the dX columns are
// split between two tiles; each launch costs a few microseconds on its own,
// so small steps share launches):
//   du        dU = s dY B, reducing over n.  Writes dU2 (token-major, high |
//             low) for the dX GEMM, dUt2 (dU^T rounded to bf16) for dA and
//             Ut2 (U^T rounded to bf16, tokens padded to mp) for dB.
//   tokred    one launch, two token reductions split over token ranges:
//             dB^T partials = Ut2 . dY and dA partials = dUt2 . X; the
//             waves of a workgroup split its tokens.
//   dx        dX = [dY | dU2] . [W ; A ; A]: one GEMM whose k loop runs over
//             n and then over the 2 RP wide slab (high and low part of dU
//             against the same A rows).  W is read through LDS with the
//             transposing ds_read_b64_tr_b16, since the product contracts
//             W over its rows.  The 128 x 256 and 256 x 256 tiles with whole
//             stages copy them straight into LDS and issue their fragment
//             reads as inline assembly with explicit waits.  After its tile, each workgroup of this launch
//             (the first one of a split) sums a slice of the dB and dA
//             partials in a fixed order (no atomics, so results are
//             bit-identical from run to run) and applies s to dB.
#include <mutex>
#include <type_traits>

#include "lora_device.hpp"
#include "lora_launch.hpp"
#include "lora_plan.hpp"

namespace lora {

// ---------------------------------------------------------------------------
// 16x16x32 A operand (16 columns x 32 k) from a small row-major LDS tile
// whose rows are k (no swizzle, `pitch` bytes per row): lane (g = l/16,
// c = l%16) receives column col0 + c, k rows 8g .. 8g+7.
__device__ __forceinline__ short8 tr16_read(const char* tile, int pitch, int col0, int lane) {
  const int g = lane >> 4, j = lane & 15;
  const int e = j >> 2, q = j & 3;
  const char* p0 = tile + (8 * g + e) * pitch + (col0 + 4 * q) * 2;
  return join4(__builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_short4v*)p0),
               __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_short4v*)(p0 + 4 * pitch)));
}

// U^T of the tokens i0 .. i0+TPW-1 rounded to bf16 into Ut2 [RP][mp] (tokens
// at or past m and ranks at or past r zero), by NTH threads; each thread
// issues all of its loads before its first store.
template <int RP, int TPW, int NTH>
__device__ __forceinline__ void store_ut2(const float* __restrict__ U, u16* __restrict__ Ut2, int i0, int m, int r,
                                          int mp, int tid) {
  constexpr int UPT = (RP * TPW + NTH - 1) / NTH;
  const __amdgpu_buffer_rsrc_t rsU = make_rsrc(U + (size_t)i0 * r, (uint64_t)max(0, min(TPW, m - i0)) * r * 4);
  float uv[UPT];
#pragma unroll
  for (int q = 0; q < UPT; ++q) {
    const int e = tid + q * NTH, t = e / TPW, il = e % TPW;
    uv[q] = buf_load4f(rsU, (e < RP * TPW && t < r) ? (uint32_t)(il * r + t) * 4 : kOOB);
  }
#pragma unroll
  for (int q = 0; q < UPT; ++q) {
    const int e = tid + q * NTH, t = e / TPW;
    if (e < RP * TPW) Ut2[(size_t)t * mp + i0 + e % TPW] = f32_to_bf16(uv[q]);
  }
}

// ---------------------------------------------------------------------------
// dU = s dY B for TPW (8, 16 or 32) tokens per workgroup, reducing over all
// of n, plus the U^T high/low split of the same tokens.  The launch takes the
// largest TPW that still gives every compute unit a workgroup: each
// workgroup reads all of B (n x r), so more tokens per workgroup means less B
// traffic per token (at rank 64 B is 4 times the dY bytes of 16 tokens).
// TPW = 8 carries 8 zero token columns in the matrix-core B operand.  The 8
// waves take interleaved 32-wide chunks of n, UNR chunks per batch with all
// of a batch's loads issued together.  A chunk's B rows (32 x r, contiguous
// in B) are staged in a wave-private LDS slot as [32][RP] (columns t >= r
// stay zero) and read back transposed into matrix-core A operands, each used
// for the TG = TPW / 16 groups of 16 tokens; dY rows go straight into B
// operands.  The waves' sums are added in wave order through LDS, so the
// result is bit-identical from run to run.  (A split of n over workgroups
// would need a cross-workgroup reduction, whose device-scope fences write
// back the per-XCD L2s -- far dearer than the work.)  Writes dU2 (token-major,
// high | low parts), dUt2 (dU^T rounded to bf16, rows of mp tokens; for a
// group whose members share one dA reduction, the member's rows of the
// stacked dU^T) and Ut2 (U^T rounded to bf16).  Index math is 32-bit:
// validation bounds every index below 2^30.
template <int RP, int TPW>
__global__ __launch_bounds__(512) void lora_bwd_du_kernel(
    const u16* __restrict__ dY, const u16* __restrict__ B, const float* __restrict__ U,
    u16* __restrict__ dU2, u16* __restrict__ dUt2, u16* __restrict__ Ut2,
    int m, int n, int r, int mp, float s) {
  constexpr int FT = RP / 16;
  constexpr int TG = TPW >= 16 ? TPW / 16 : 1;      // 16-token groups
  constexpr int NWV = 8;
  // Chunks per batch: deep batches pay off only for the short n runs of the
  // 8-token workgroups; with 16 or more tokens, batches of one or two chunks
  // keep more of them in flight across the loop (7B up_proj dU 29.8 -> 24.0 us).
  constexpr int UNR = TPW == 8 ? (RP <= 16 ? 8 : (RP <= 32 ? 4 : 2)) : (RP <= 32 && TG == 1 ? 2 : 1);
  constexpr int SLOT = 32 * RP * 2;                 // bytes of one staged chunk of B
  constexpr int BL = RP / 16;                       // 16-byte B loads per lane per chunk (4r <= 4 RP)
  constexpr int STAGE_BYTES = NWV * UNR * SLOT, RED_BYTES = NWV * TG * FT * 64 * 16;
  __shared__ __attribute__((aligned(1024))) char sm[STAGE_BYTES > RED_BYTES ? STAGE_BYTES : RED_BYTES];
  static_assert(TPW == 32 || TPW == 16 || TPW == 8, "tokens per workgroup");
  static_assert(TG * FT <= NWV, "one wave per output fragment in the epilogue");
  const int i0 = blockIdx.x * TPW;
  const int tid = threadIdx.x, lane = tid & 63, wave = uniform(tid >> 6);
  const int g = lane >> 4, c16 = lane & 15;
  const uint32_t rowbytes = (uint32_t)n * 2;
  const int rows = uniform(max(0, min(TPW, m - i0)));
  const __amdgpu_buffer_rsrc_t rsY = make_rsrc(dY + (size_t)i0 * n, (uint64_t)rows * rowbytes);
  const __amdgpu_buffer_rsrc_t rsB = make_rsrc(B, (uint64_t)n * r * 2);
  char* slots = sm + wave * UNR * SLOT;

  for (int e = lane; e < UNR * SLOT / 16; e += 64) reinterpret_cast<int4v*>(slots)[e] = int4v{0, 0, 0, 0};

  floatx4 acc[TG][FT];
#pragma unroll
  for (int tg = 0; tg < TG; ++tg)
#pragma unroll
    for (int ft = 0; ft < FT; ++ft) acc[tg][ft] = floatx4{0.f, 0.f, 0.f, 0.f};

  const int nbch = 4 * r;                           // 16-byte chunks in 32 rows of B
  const bool fast = (r & 7) == 0;                   // a chunk then lies inside one row of B
  const float rinv = 1.0f / (float)r;
  // Batch b of this wave covers chunks j = 32 wave + 32 NWV (UNR b + u); the
  // loads of batch b+1 are in flight while batch b multiplies.
  short8 yf[2][UNR][TG];
  int4v bq[2][UNR][BL];
  auto load = [&](int bt, int p) LORA_INLINE {
#pragma unroll
    for (int u = 0; u < UNR; ++u) {
      const int j = 32 * wave + 32 * NWV * (UNR * bt + u);
      const int jy = j + 8 * g;
#pragma unroll
      for (int tg = 0; tg < TG; ++tg)
        yf[p][u][tg] = __builtin_bit_cast(
            short8, buf_load16(rsY, jy < n ? (uint32_t)(16 * tg + c16) * rowbytes + (uint32_t)jy * 2 : kOOB));
#pragma unroll
      for (int v = 0; v < BL; ++v) {
        const int c = lane + 64 * v;
        bq[p][u][v] = buf_load16(rsB, (j < n && c < nbch) ? (uint32_t)j * r * 2 + (uint32_t)c * 16 : kOOB);
      }
    }
  };
  auto process = [&](int p) LORA_INLINE {
#pragma unroll
    for (int u = 0; u < UNR; ++u) {
      char* slot = slots + u * SLOT;
#pragma unroll
      for (int v = 0; v < BL; ++v) {
        const int c = lane + 64 * v;
        if (c < nbch) {
          if (fast) {
            const int e0 = 8 * c, jj = e0 / r;
            *reinterpret_cast<int4v*>(slot + (jj * RP + e0 - jj * r) * 2) = bq[p][u][v];
          } else {
#pragma unroll
            for (int x = 0; x < 8; ++x) {   // quotient from a float product at least 0.5/r from an integer
              const int e = 8 * c + x;
              const int jj = (int)(((float)e + 0.5f) * rinv);
              *reinterpret_cast<u16*>(slot + (jj * RP + e - jj * r) * 2) =
                  (u16)((uint32_t)bq[p][u][v][x >> 1] >> (16 * (x & 1)));
            }
          }
        }
      }
#pragma unroll
      for (int ft = 0; ft < FT; ++ft) {
        const short8 bt = tr16_read(slot, RP * 2, 16 * ft, lane);
#pragma unroll
        for (int tg = 0; tg < TG; ++tg) acc[tg][ft] = mfma16x16x32(bt, yf[p][u][tg], acc[tg][ft]);
      }
    }
  };
  const int nbt = uniform(32 * wave < n ? (n - 32 * wave + 32 * NWV * UNR - 1) / (32 * NWV * UNR) : 0);
  if (nbt > 0) load(0, 0);
  for (int bt = 0; bt < nbt; bt += 2) {
    if (bt + 1 < nbt) load(bt + 1, 1);
    process(0);
    if (bt + 1 >= nbt) break;
    if (bt + 2 < nbt) load(bt + 2, 0);
    process(1);
  }

  store_ut2<RP, TPW, 64 * NWV>(U, Ut2, i0, m, r, mp, tid);   // U^T of this workgroup's tokens in bf16

  __syncthreads();
  floatx4* red = reinterpret_cast<floatx4*>(sm);   // [NWV][TG][FT][64]
#pragma unroll
  for (int tg = 0; tg < TG; ++tg)
#pragma unroll
    for (int ft = 0; ft < FT; ++ft) red[((wave * TG + tg) * FT + ft) * 64 + lane] = acc[tg][ft];
  __syncthreads();
  if (wave >= TG * FT) return;
  const int tg = wave / FT, ft = wave - tg * FT;   // one wave per 16 x 16 fragment of dU^T
  floatx4 v = red[(tg * FT + ft) * 64 + lane];
#pragma unroll
  for (int w = 1; w < NWV; ++w) v += red[((w * TG + tg) * FT + ft) * 64 + lane];
  if (16 * tg + c16 >= TPW) return;   // the zero token columns of TPW = 8
  const int i = i0 + 16 * tg + c16;   // < mp: the grid covers exactly mp tokens
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
  for (int q = 0; q < 4; ++q) dUt2[(size_t)(t + q) * mp + i] = hi[q];
}

// ---------------------------------------------------------------------------
// Wait until at most N LDS operations of this wave are outstanding, in an asm
// statement that takes a substep's fragment registers as operands (so no use
// of them can move above it): TG dY fragments, FT pairs of B^T halves.
template <int N, int FT, int TG>
__device__ __forceinline__ void du_frag_wait(short8 (&y)[TG], short4v (&bl)[FT], short4v (&bh)[FT]) {
  static_assert(N >= 0 && N <= 15, "lgkmcnt range");
#define LORA_DU_WAIT(...) asm volatile("s_waitcnt lgkmcnt(%[cnt])" : __VA_ARGS__ : [cnt] "i"(N))
  if constexpr (FT == 1 && TG == 1) LORA_DU_WAIT("+v"(y[0]), "+v"(bl[0]), "+v"(bh[0]));
  else if constexpr (FT == 1 && TG == 2) LORA_DU_WAIT("+v"(y[0]), "+v"(y[1]), "+v"(bl[0]), "+v"(bh[0]));
  else if constexpr (FT == 2 && TG == 1) LORA_DU_WAIT("+v"(y[0]), "+v"(bl[0]), "+v"(bh[0]), "+v"(bl[1]), "+v"(bh[1]));
  else if constexpr (FT == 2 && TG == 2)
    LORA_DU_WAIT("+v"(y[0]), "+v"(y[1]), "+v"(bl[0]), "+v"(bh[0]), "+v"(bl[1]), "+v"(bh[1]));
  else if constexpr (FT == 3 && TG == 1)
    LORA_DU_WAIT("+v"(y[0]), "+v"(bl[0]), "+v"(bh[0]), "+v"(bl[1]), "+v"(bh[1]), "+v"(bl[2]), "+v"(bh[2]));
  else if constexpr (FT == 3 && TG == 2)
    LORA_DU_WAIT("+v"(y[0]), "+v"(y[1]), "+v"(bl[0]), "+v"(bh[0]), "+v"(bl[1]), "+v"(bh[1]), "+v"(bl[2]),
                 "+v"(bh[2]));
  else if constexpr (FT == 4 && TG == 1)
    LORA_DU_WAIT("+v"(y[0]), "+v"(bl[0]), "+v"(bh[0]), "+v"(bl[1]), "+v"(bh[1]), "+v"(bl[2]), "+v"(bh[2]),
                 "+v"(bl[3]), "+v"(bh[3]));
  else {
    static_assert(FT == 4 && TG == 2, "fragment shapes");
    LORA_DU_WAIT("+v"(y[0]), "+v"(y[1]), "+v"(bl[0]), "+v"(bh[0]), "+v"(bl[1]), "+v"(bh[1]), "+v"(bl[2]),
                 "+v"(bh[2]), "+v"(bl[3]), "+v"(bh[3]));
  }
#undef LORA_DU_WAIT
}

// ---------------------------------------------------------------------------
// dU = s dY B for ranks that are multiples of 8 (each 16-byte piece of B then
// lies inside one row), fed by copies straight into LDS.  TPW (8, 16 or 32)
// tokens per workgroup, four waves; the n loop runs in stages of 64: wave w
// takes stages w, w + 4, ... and copies each of them (its TPW dY rows, 8 rows
// of 128 bytes per copy instruction with the swizzle of kc_offset applied to
// the global addresses, and the stage's 64 rows of B as a [64][RP] block,
// zero past r) straight into a private ring of NSW LDS stages, NSW - 1
// stages ahead, waiting only for its own copies (no barrier in the loop).
// (The register-loading kernel above reads 16 rows x 64 bytes of dY per
// instruction, which keeps the L1 busy translating addresses.)  Each wave
// accumulates all of dU^T for its stages on 16x16x32 products: B^T fragments
// by transposing reads of the B block, dY fragments as the second operand
// (TPW = 8 leaves token columns 8..15 zero); the fragment reads are issued as
// inline assembly with counted waits, since the compiler would otherwise wait
// for every copy in flight before each transposing read.  The four partial
// sums are added in wave order through LDS, then written as the register
// kernel does (dU2, dUt2, Ut2).
template <int RP, int TPW>
__global__ __launch_bounds__(256) void lora_bwd_du_dma_kernel(
    const u16* __restrict__ dY, const u16* __restrict__ B, const float* __restrict__ U,
    u16* __restrict__ dU2, u16* __restrict__ dUt2, u16* __restrict__ Ut2,
    int m, int n, int r, int mp, float s) {
  constexpr int NWV = 4;
  constexpr int FT = RP / 16;
  constexpr int TG = TPW >= 16 ? TPW / 16 : 1;
  constexpr int YR = TG * 16;                    // dY rows per stage in LDS (TPW = 8: rows 8..15 stay zero)
  constexpr int BOFF = YR * 128;                 // the B block [64][RP] after the dY rows
  constexpr int STAGE = BOFF + 64 * RP * 2;
  constexpr int CY = TPW / 8, CB = RP / 8;       // 1 KB copies per stage: dY rows, B block
  constexpr int CPW = CY + CB;
  constexpr int NSW = (156 * 1024) / (NWV * STAGE) < 6 ? (156 * 1024) / (NWV * STAGE) : 6;
  constexpr int RED = NWV * TG * FT * 64 * 16;   // cross-wave sum [NWV][TG][FT][64] float4
  constexpr int SMEM = NWV * NSW * STAGE > RED ? NWV * NSW * STAGE : RED;
  constexpr int NRD = TG + 2 * FT;               // LDS reads per wave and 32-wide substep
  static_assert(TPW == 8 || TPW == 16 || TPW == 32, "tokens per workgroup");
  static_assert(NSW >= 3 && CPW * (NSW - 2) < 64, "copies in flight fit the wait counter");
  static_assert(NRD <= 15, "reads of one substep fit the LDS wait counter");
  __shared__ __attribute__((aligned(1024))) char sm[SMEM];
  const int i0 = blockIdx.x * TPW;
  const int tid = threadIdx.x, lane = tid & 63, wave = uniform(tid >> 6);
  const int g = lane >> 4, c16 = lane & 15;
  const uint32_t rowbytes = (uint32_t)n * 2;
  const int rows = uniform(max(0, min(TPW, m - i0)));
  const __amdgpu_buffer_rsrc_t rsY = make_rsrc(dY + (size_t)i0 * n, (uint64_t)rows * rowbytes);
  const __amdgpu_buffer_rsrc_t rsB = make_rsrc(B, (uint64_t)n * r * 2);
  char* ring = sm + wave * NSW * STAGE;
  if (YR > TPW) {   // the zero token rows of TPW = 8, in every stage of the ring
    for (int e = lane; e < NSW * (YR - TPW) * 8; e += 64) {
      const int st = e / ((YR - TPW) * 8), q = e % ((YR - TPW) * 8);
      reinterpret_cast<int4v*>(ring + st * STAGE + TPW * 128)[q] = int4v{0, 0, 0, 0};
    }
  }

  // Copy c of the dY rows: rows 8c + lane/8 at physical chunk lane%8, which
  // holds logical chunk (lane%8) ^ kc_swz(row).  Copy c of the B block: its
  // bytes 1024c + 16 lane, i.e. row (1024c + 16 lane) / (2 RP) of the stage
  // and 8-element chunk ((1024c + 16 lane) % (2 RP)) / 16.
  const int nst = (n + 63) / 64;
  auto issue = [&](int j, int buf) LORA_INLINE {
    const int st = wave + NWV * j;
    const int j0 = st * 64;
    const bool live = st < nst;
    char* sb = ring + buf * STAGE;
#pragma unroll
    for (int c = 0; c < CY; ++c) {
      const int row = 8 * c + (lane >> 3);
      const int jj = j0 + 8 * ((lane & 7) ^ kc_swz(row));
      dma16(rsY, live && jj < n ? (uint32_t)row * rowbytes + (uint32_t)jj * 2 : kOOB, 0, sb + c * 1024);
    }
#pragma unroll
    for (int c = 0; c < CB; ++c) {
      const int byte = 1024 * c + 16 * lane;
      const int row = byte / (2 * RP), t0 = (byte % (2 * RP)) / 2;
      const int jb = j0 + row;
      dma16(rsB, live && jb < n && t0 < r ? ((uint32_t)jb * (uint32_t)r + (uint32_t)t0) * 2 : kOOB, 0,
            sb + BOFF + c * 1024);
    }
  };

  // Lane addresses in stage 0 of the wave's ring.  dY fragment (second
  // operand, 32 n x 16 tokens) of substep kk: row c16 (+ 2048 bytes per token
  // group), chunk 4 kk + g.  B^T fragment (first operand, 16 t x 32 n) as in
  // tr16_read: rows 8 g + e (+ 4 rows for the second read, + 32 rows for kk),
  // columns 16 ft + 4 q.
  uint32_t ya[2], ba;
#pragma unroll
  for (int kk = 0; kk < 2; ++kk) ya[kk] = lds_addr(ring + kc_offset(c16, 4 * kk + g));
  {
    const int j = lane & 15, e = j >> 2, q = j & 3;
    ba = lds_addr(ring + BOFF + (8 * g + e) * (2 * RP) + 4 * q * 2);
  }
  floatx4 acc[TG][FT];
#pragma unroll
  for (int tg = 0; tg < TG; ++tg)
#pragma unroll
    for (int ft = 0; ft < FT; ++ft) acc[tg][ft] = floatx4{0.f, 0.f, 0.f, 0.f};
  short8 fy[2][TG];
  short4v fbl[2][FT], fbh[2][FT];
  auto reads = [&](uint32_t boff, auto kkc) LORA_INLINE {
    constexpr int kk = decltype(kkc)::value;
    ds_read_b128_asm<0>(fy[kk][0], ya[kk] + boff);
    if constexpr (TG > 1) ds_read_b128_asm<2048>(fy[kk][1], ya[kk] + boff);
#pragma unroll
    for (int ft = 0; ft < FT; ++ft) {
      // (ft, kk) immediates: 32 ft bytes of columns, 32 rows of 2 RP bytes per kk
      const uint32_t a = ba + boff + (uint32_t)(32 * ft);
      ds_read_tr_b64_asm<kk * 32 * 2 * RP>(fbl[kk][ft], a);
      ds_read_tr_b64_asm<kk * 32 * 2 * RP + 4 * 2 * RP>(fbh[kk][ft], a);
    }
  };
  auto mult = [&](int kk) LORA_INLINE {
#pragma unroll
    for (int ft = 0; ft < FT; ++ft) {
      const short8 bt = join4(fbl[kk][ft], fbh[kk][ft]);
#pragma unroll
      for (int tg = 0; tg < TG; ++tg) acc[tg][ft] = mfma16x16x32(bt, fy[kk][tg], acc[tg][ft]);
    }
  };
  using K0 = std::integral_constant<int, 0>;
  using K1 = std::integral_constant<int, 1>;
  auto compute = [&](int buf) LORA_INLINE {
    const uint32_t boff = (uint32_t)buf * STAGE;
    if constexpr (2 * NRD <= 15) {   // both substeps' reads in flight, then the products
      reads(boff, K0{});
      reads(boff, K1{});
      du_frag_wait<NRD, FT, TG>(fy[0], fbl[0], fbh[0]);   // only substep 1's reads outstanding
      mult(0);
      du_frag_wait<0, FT, TG>(fy[1], fbl[1], fbh[1]);
      mult(1);
    } else {
      reads(boff, K0{});
      du_frag_wait<0, FT, TG>(fy[0], fbl[0], fbh[0]);
      mult(0);
      reads(boff, K1{});
      du_frag_wait<0, FT, TG>(fy[1], fbl[1], fbh[1]);
      mult(1);
    }
  };

  const int nsw = wave < nst ? (nst - wave + NWV - 1) / NWV : 0;   // this wave's stages
#pragma unroll
  for (int j = 0; j < NSW - 1; ++j) issue(j, j);
  for (int j = 0; j < nsw; ++j) {
    wait_vmcnt<CPW * (NSW - 2)>();   // the wave's stage j has landed
    issue(j + NSW - 1, (j + NSW - 1) % NSW);   // into the buffer of stage j - 1, read already
    compute(j % NSW);
  }
  wait_vmcnt<0>();   // the trailing copies (zeros) land before the LDS is reused

  store_ut2<RP, TPW, 64 * NWV>(U, Ut2, i0, m, r, mp, tid);   // U^T of this workgroup's tokens in bf16

  __syncthreads();
  floatx4* red = reinterpret_cast<floatx4*>(sm);   // [NWV][TG][FT][64]
#pragma unroll
  for (int tg = 0; tg < TG; ++tg)
#pragma unroll
    for (int ft = 0; ft < FT; ++ft) red[((wave * TG + tg) * FT + ft) * 64 + lane] = acc[tg][ft];
  __syncthreads();
  for (int e = wave; e < TG * FT; e += NWV) {   // fragment e of dU^T, summed in wave order
    const int tg = e / FT, ft = e - tg * FT;
    floatx4 v = red[(tg * FT + ft) * 64 + lane];
#pragma unroll
    for (int w = 1; w < NWV; ++w) v += red[((w * TG + tg) * FT + ft) * 64 + lane];
    if (16 * tg + c16 >= TPW) continue;   // the zero token columns of TPW = 8
    const int i = i0 + 16 * tg + c16;     // < mp: the grid covers exactly mp tokens
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
    for (int q = 0; q < 4; ++q) dUt2[(size_t)(t + q) * mp + i] = hi[q];
  }
}

// ---------------------------------------------------------------------------
// Token reduction part[sp][t][c] = sum over the tokens i of split sp of
// P[t][i] * Q[i][c], t < RP, for a tile of kRedCols = 128 columns.  P is the
// rank-r operand rounded to bf16 (U^T or s dU^T, [RP][mp]); its rounding
// error (relative 2^-9 per element) averages out in the sums to about 1e-3 of
// dA and dB.  One launch serves two such problems (dB^T from Ut2 and dY, dA
// from dUt2 and X): workgroups [0, nb0) take the first.
//
// The four waves of a workgroup take interleaved 32-token slices of the
// split.  Each reads its P fragments straight from the token-contiguous P
// into matrix-core A operands and stages its 32 x 128 slice of Q
// ([m][cols]) in a private LDS region that it reads back transposed, so the
// token loop has no barriers; the next slice is loaded while the current one
// multiplies.  At the end the four waves' sums are added in wave order
// through LDS (bit-identical from run to run).
struct RedProblem {
  const u16* P;
  const u16* Q;
  float* part;
  int ncols, span, col_tiles;
  const uint8_t* keep;   // dropout keep bits of Q ([m][ncols/8]) or null: masked Q elements count as 0
};

// Launched with KEEP, for the masked-Q path of LoRA dropout: the mask is
// applied to the Q chunks in registers before they are staged.  Without a
// mask the launch takes lora_tokred_dma_kernel below.
template <int RP, bool KEEP>
__global__ __launch_bounds__(256) void lora_tokred_kernel(RedProblem p0, RedProblem p1, int nb0, int m, int mp) {
  constexpr int CB = kRedCols;                // columns per workgroup
  constexpr int FC = CB / 16;                 // column fragments
  constexpr int FP = RP / 16;                 // row fragments
  constexpr int CPR = CB / 8;                 // 16-byte chunks per Q row
  constexpr int QL = 32 * CPR / 64;           // Q loads per lane per slice
  constexpr int REG = 32 * CB * 2;            // bytes of one staged Q slice
  // column fragments per reduction pass: the largest power of two dividing FC
  // whose partial sums (4 waves x FP x FCP fragments) fit the staging LDS
  constexpr int FCP = 16 / FP >= 8 ? 8 : (16 / FP >= 4 ? 4 : (16 / FP >= 2 ? 2 : 1));
  static_assert(FC % FCP == 0, "reduction passes cover the column fragments");
  static_assert(CB == 128 && QL * 64 == 32 * CPR, "slice shape");
  static_assert(4 * FP * FCP * 64 * 16 <= 4 * 2 * REG, "reduction fits the staging LDS");
  __shared__ __attribute__((aligned(1024))) char smem[4 * 2 * REG];

  const bool first = (int)blockIdx.x < nb0;
  const RedProblem& pr = first ? p0 : p1;
  const int bid = first ? (int)blockIdx.x : (int)blockIdx.x - nb0;
  const u16* __restrict__ P = pr.P;
  const u16* __restrict__ Q = pr.Q;
  const int ncols = pr.ncols;
  const int c0 = (bid % pr.col_tiles) * CB;
  const int sp = bid / pr.col_tiles;
  const int tb = sp * pr.span;
  const int te = min(mp, tb + pr.span);
  const int tid = threadIdx.x, lane = tid & 63, wave = uniform(tid >> 6);
  const int g = lane >> 4, c16 = lane & 15;
  const uint32_t qrow = (uint32_t)ncols * 2;
  const __amdgpu_buffer_rsrc_t rsP = make_rsrc(P, (uint64_t)RP * mp * 2);
  char* wreg = smem + wave * 2 * REG;

  floatx4 acc[FP][FC];
#pragma unroll
  for (int f = 0; f < FP; ++f)
#pragma unroll
    for (int fc = 0; fc < FC; ++fc) acc[f][fc] = floatx4{0.f, 0.f, 0.f, 0.f};

  // Slice loads: Q chunk u of this lane is row (lane + 64u) / CPR, chunk
  // (lane + 64u) % CPR; P fragment f is row 16f + c16, tokens ts + 8g .. +7.
  int4v qv[2][QL];
  uint32_t kq[KEEP ? 2 : 1][KEEP ? QL : 1];   // keep byte of each Q chunk (dropout)
  short8 pv[2][FP];
  const uint8_t* keep = KEEP ? pr.keep : nullptr;
  const uint32_t kb8 = (uint32_t)ncols / 8;
  auto load = [&](int ts, int b) LORA_INLINE {
    const int rows = uniform(max(0, min(32, m - ts)));   // keeps the resource in scalar registers
    const __amdgpu_buffer_rsrc_t rsQ = make_rsrc(Q + (size_t)ts * ncols, (uint64_t)rows * qrow);
#pragma unroll
    for (int u = 0; u < QL; ++u) {
      const int q = lane + 64 * u;
      const int cc = c0 + 8 * (q % CPR);
      qv[b][u] = buf_load16(rsQ, cc < ncols ? (uint32_t)(q / CPR) * qrow + (uint32_t)cc * 2 : kOOB);
    }
    if (KEEP && keep) {   // workgroup-uniform
      const __amdgpu_buffer_rsrc_t rsK = make_rsrc(keep + (size_t)ts * kb8, (uint64_t)rows * kb8);
#pragma unroll
      for (int u = 0; u < QL; ++u) {
        const int q = lane + 64 * u;
        const int cc = c0 + 8 * (q % CPR);
        kq[KEEP ? b : 0][KEEP ? u : 0] = buf_load_u8(rsK, cc < ncols ? (uint32_t)(q / CPR) * kb8 + (uint32_t)cc / 8 : kOOB);
      }
    }
#pragma unroll
    for (int f = 0; f < FP; ++f)
      pv[b][f] = __builtin_bit_cast(
          short8, buf_load16(rsP, ((uint32_t)(16 * f + c16) * (uint32_t)mp + (uint32_t)(ts + 8 * g)) * 2));
  };
  auto step = [&](int b) LORA_INLINE {
    char* qs = wreg + b * REG;
#pragma unroll
    for (int u = 0; u < QL; ++u) {
      const int q = lane + 64 * u;
      int4v v = qv[b][u];
      if (KEEP && keep)
        v = __builtin_bit_cast(int4v, keep_mask8(__builtin_bit_cast(short8, v), kq[KEEP ? b : 0][KEEP ? u : 0]));
      *reinterpret_cast<int4v*>(qs + mc16_offset<CB>(q / CPR, q % CPR)) = v;
    }
#pragma unroll
    for (int fc = 0; fc < FC; ++fc) {
      const short8 qf = mc16_read_tr<CB>(qs, 0, 16 * fc, lane);
#pragma unroll
      for (int f = 0; f < FP; ++f) acc[f][fc] = mfma16x16x32(pv[b][f], qf, acc[f][fc]);
    }
  };

  // Slices of this wave: ts0 + 128 j < te, ts0 = tb + 32 wave (te - tb is a
  // multiple of 64, so slices never straddle te).
  const int ts0 = tb + 32 * wave;
  const int ns = ts0 < te ? (te - ts0 + 127) / 128 : 0;
  if (ns > 0) load(ts0, 0);
  int j = 0;
  for (; j + 2 <= ns; j += 2) {
    load(ts0 + 128 * (j + 1), 1);
    step(0);
    if (j + 2 < ns) load(ts0 + 128 * (j + 2), 0);
    step(1);
  }
  if (j < ns) step(0);

  // Cross-wave sum in wave order, FCP column fragments per pass; lane holds
  // column c16 of fragment fc, rows 4g .. 4g+3 of fragment f.
  floatx4* red = reinterpret_cast<floatx4*>(smem);   // [4 waves][FP][FCP][64]
  float* part = pr.part;
#pragma unroll
  for (int f0 = 0; f0 < FC; f0 += FCP) {
    __syncthreads();
#pragma unroll
    for (int f = 0; f < FP; ++f)
#pragma unroll
      for (int q = 0; q < FCP; ++q) red[((wave * FP + f) * FCP + q) * 64 + lane] = acc[f][f0 + q];
    __syncthreads();
    for (int e = wave; e < FP * FCP; e += 4) {
      const int f = e / FCP, q = e - f * FCP;
      floatx4 v = red[((0 * FP + f) * FCP + q) * 64 + lane];
#pragma unroll
      for (int w = 1; w < 4; ++w) v += red[((w * FP + f) * FCP + q) * 64 + lane];
      const int col = c0 + 16 * (f0 + q) + c16;
      if (col < ncols) {
#pragma unroll
        for (int qq = 0; qq < 4; ++qq) part[((size_t)sp * RP + 16 * f + 4 * g + qq) * ncols + col] = v[qq];
      }
    }
  }
}

// ---------------------------------------------------------------------------
// The same token reduction without a keep mask, fed by copies straight into
// LDS.  Stages of 64 tokens: the stage's P block (RP rows x 64 tokens, 128
// bytes a row, kc_offset swizzle) and Q block (64 tokens x 128 columns, 256
// bytes a row, mc16_offset swizzle) are copied from global memory into a ring
// of NS LDS stages, NS - 1 stages ahead, in whole row pieces (8 rows of P or 4
// rows of Q per copy instruction; the swizzles applied to the global
// addresses), one barrier per stage.  (Register loads of 16 rows x 64 bytes
// per instruction kept the L1 busy translating addresses.)  The four waves
// split the columns, two 16-column fragments each, over all tokens of the
// split, so no cross-wave sum is needed.  The fragment reads are issued as
// inline assembly with explicit lgkmcnt waits: the compiler would otherwise
// wait for every copy still in flight before each transposing read of Q.
// At most 80 KB of LDS, so two workgroups share a compute unit.
template <int RP>
__global__ __launch_bounds__(256) void lora_tokred_dma_kernel(RedProblem p0, RedProblem p1, int nb0, int m,
                                                              int mp) {
  constexpr int CB = kRedCols, NWV = 4, TS = 64;
  constexpr int FP = RP / 16;
  constexpr int PB = RP * 128;                // P block bytes
  constexpr int QB = TS * CB * 2;             // Q block bytes
  constexpr int STAGE = PB + QB;
  constexpr int NS = (80 * 1024) / STAGE;     // ring stages
  constexpr int NP = RP / 8, NQ = TS / 4;     // 1 KB copies per stage: P rows / 8, Q rows / 4
  constexpr int QPW = NQ / NWV;               // Q copies per wave
  constexpr int NRD = FP + 4;                 // LDS reads per wave and substep
  static_assert(CB == 128 && NQ % NWV == 0 && NS >= 3, "stage shape");
  static_assert((NS - 2) * (NP / NWV + 1 + QPW) < 64, "copies in flight fit the wait counter");
  __shared__ __attribute__((aligned(1024))) char smem[NS * STAGE];

  const bool first = (int)blockIdx.x < nb0;
  const RedProblem& pr = first ? p0 : p1;
  const int bid = first ? (int)blockIdx.x : (int)blockIdx.x - nb0;
  const u16* __restrict__ P = pr.P;
  const u16* __restrict__ Q = pr.Q;
  const int ncols = pr.ncols;
  const int c0 = (bid % pr.col_tiles) * CB;
  const int sp = bid / pr.col_tiles;
  const int tb = sp * pr.span;
  const int te = min(mp, tb + pr.span);       // te - tb is a multiple of 64
  const int nst = (te - tb) / TS;
  const int tid = threadIdx.x, lane = tid & 63, wave = uniform(tid >> 6);
  const int g = lane >> 4, c16 = lane & 15;
  const uint32_t qrow = (uint32_t)ncols * 2;
  const __amdgpu_buffer_rsrc_t rsP = make_rsrc(P, (uint64_t)RP * mp * 2);

  // Copies of stage st into buffer buf.  P copy j (j = wave mod 4): rows
  // 8j + lane/8 at physical chunk lane%8; Q copy j = wave + 4i: rows
  // 4j + lane/16 at physical chunk lane%16.  Each position holds the logical
  // chunk given by the swizzle.  Tokens at or past m, columns past ncols and
  // stages past the split read zero.
  int pcol[NP / NWV + 1];
  uint32_t qoff[QPW];
  int qcol[QPW];
#pragma unroll
  for (int i = 0; i * NWV < NP; ++i) {
    const int row = 8 * (wave + NWV * i) + (lane >> 3);
    pcol[i] = 8 * ((lane & 7) ^ kc_swz(row));
  }
#pragma unroll
  for (int i = 0; i < QPW; ++i) {
    const int row = 4 * (wave + NWV * i) + (lane >> 4);
    const int c = (lane & 15) ^ mc16_swz(row);
    qcol[i] = c0 + 8 * c;
    qoff[i] = (uint32_t)row * qrow + (uint32_t)qcol[i] * 2;
  }
  auto issue = [&](int st, int buf) LORA_INLINE {
    const int ts = tb + TS * st;
    const bool live = st < nst;
    char* sb = smem + buf * STAGE;
#pragma unroll
    for (int i = 0; i * NWV < NP; ++i) {
      const int j = wave + NWV * i;
      if (j < NP) {   // wave-uniform
        const int row = 8 * j + (lane >> 3);
        dma16(rsP, live ? ((uint32_t)row * (uint32_t)mp + (uint32_t)(ts + pcol[i])) * 2 : kOOB, 0, sb + j * 1024);
      }
    }
    const int rows = uniform(live ? max(0, min(TS, m - ts)) : 0);
    const __amdgpu_buffer_rsrc_t rsQ = make_rsrc(Q + (size_t)ts * ncols, (uint64_t)rows * qrow);
#pragma unroll
    for (int i = 0; i < QPW; ++i)
      dma16(rsQ, qcol[i] < ncols ? qoff[i] : kOOB, 0, sb + PB + (wave + NWV * i) * 1024);
  };
  auto stage_barrier = [&]() LORA_INLINE {   // this wave's copies of the stage waited for: NS - 2 stages stay in flight
    if (wave < NP % NWV) copy_barrier<(NS - 2) * (NP / NWV + 1 + QPW)>();
    else copy_barrier<(NS - 2) * (NP / NWV + QPW)>();
  };

  // Lane addresses in buffer 0.  P fragment f (A operand, 16 rank rows x 32
  // tokens) of substep kk: row 16 f + c16, chunk 4 kk + g (f adds 2048 bytes;
  // the swizzle of kk depends on the lane).  Q fragment j of this wave
  // (column tile 2 wave + j; B operand, 32 tokens x 16 columns) as in
  // mc16_read_tr: two transposing reads 4 rows apart (+1024 bytes), substep kk
  // 32 rows further (+8192 bytes).
  uint32_t pa[2], qa[2];
#pragma unroll
  for (int kk = 0; kk < 2; ++kk) pa[kk] = lds_addr(smem + kc_offset(c16, 4 * kk + g));
  {
    const int j = lane & 15, e = j >> 2, q = j & 3;
#pragma unroll
    for (int jf = 0; jf < 2; ++jf) {
      const int col = 16 * (2 * wave + jf) + 4 * q;
      qa[jf] = lds_addr(smem + PB + mc16_offset<CB>(8 * g + e, col >> 3) + (col & 7) * 2);
    }
  }
  floatx4 acc[FP][2];
#pragma unroll
  for (int f = 0; f < FP; ++f) acc[f][0] = acc[f][1] = floatx4{0.f, 0.f, 0.f, 0.f};
  short8 fp[2][FP];
  short4v fql[2][2], fqh[2][2];
  auto reads = [&](uint32_t boff, int kk) LORA_INLINE {
    const uint32_t a = pa[kk] + boff;
    ds_read_b128_asm<0>(fp[kk][0], a);
    if constexpr (FP > 1) ds_read_b128_asm<2048>(fp[kk][1], a);
    if constexpr (FP > 2) ds_read_b128_asm<4096>(fp[kk][2], a);
    if constexpr (FP > 3) ds_read_b128_asm<6144>(fp[kk][3], a);
#pragma unroll
    for (int jf = 0; jf < 2; ++jf) {
      const uint32_t b = qa[jf] + boff;
      if (kk == 0) {
        ds_read_tr_b64_asm<0>(fql[kk][jf], b);
        ds_read_tr_b64_asm<1024>(fqh[kk][jf], b);
      } else {
        ds_read_tr_b64_asm<8192>(fql[kk][jf], b);
        ds_read_tr_b64_asm<9216>(fqh[kk][jf], b);
      }
    }
  };
  static_assert(FP <= 4, "rank rows per stage");
  auto mult = [&](int kk) LORA_INLINE {
#pragma unroll
    for (int jf = 0; jf < 2; ++jf) {
      const short8 qf = join4(fql[kk][jf], fqh[kk][jf]);
#pragma unroll
      for (int f = 0; f < FP; ++f) acc[f][jf] = mfma16x16x32(fp[kk][f], qf, acc[f][jf]);
    }
  };
  auto compute = [&](int buf) LORA_INLINE {
    const uint32_t boff = (uint32_t)buf * STAGE;
    reads(boff, 0);
    reads(boff, 1);
    // substep 0 once only the NRD reads of substep 1 are outstanding
    if constexpr (FP == 1)
      asm volatile("s_waitcnt lgkmcnt(5)" : "+v"(fp[0][0]), "+v"(fql[0][0]), "+v"(fqh[0][0]), "+v"(fql[0][1]),
                   "+v"(fqh[0][1]));
    else if constexpr (FP == 2)
      asm volatile("s_waitcnt lgkmcnt(6)" : "+v"(fp[0][0]), "+v"(fp[0][1]), "+v"(fql[0][0]), "+v"(fqh[0][0]),
                   "+v"(fql[0][1]), "+v"(fqh[0][1]));
    else if constexpr (FP == 3)
      asm volatile("s_waitcnt lgkmcnt(7)" : "+v"(fp[0][0]), "+v"(fp[0][1]), "+v"(fp[0][2]), "+v"(fql[0][0]),
                   "+v"(fqh[0][0]), "+v"(fql[0][1]), "+v"(fqh[0][1]));
    else
      asm volatile("s_waitcnt lgkmcnt(8)" : "+v"(fp[0][0]), "+v"(fp[0][1]), "+v"(fp[0][2]), "+v"(fp[0][3]),
                   "+v"(fql[0][0]), "+v"(fqh[0][0]), "+v"(fql[0][1]), "+v"(fqh[0][1]));
    static_assert(NRD == FP + 4, "wait counts above");
    mult(0);
    if constexpr (FP == 1)
      asm volatile("s_waitcnt lgkmcnt(0)" : "+v"(fp[1][0]), "+v"(fql[1][0]), "+v"(fqh[1][0]), "+v"(fql[1][1]),
                   "+v"(fqh[1][1]));
    else if constexpr (FP == 2)
      asm volatile("s_waitcnt lgkmcnt(0)" : "+v"(fp[1][0]), "+v"(fp[1][1]), "+v"(fql[1][0]), "+v"(fqh[1][0]),
                   "+v"(fql[1][1]), "+v"(fqh[1][1]));
    else if constexpr (FP == 3)
      asm volatile("s_waitcnt lgkmcnt(0)" : "+v"(fp[1][0]), "+v"(fp[1][1]), "+v"(fp[1][2]), "+v"(fql[1][0]),
                   "+v"(fqh[1][0]), "+v"(fql[1][1]), "+v"(fqh[1][1]));
    else
      asm volatile("s_waitcnt lgkmcnt(0)" : "+v"(fp[1][0]), "+v"(fp[1][1]), "+v"(fp[1][2]), "+v"(fp[1][3]),
                   "+v"(fql[1][0]), "+v"(fqh[1][0]), "+v"(fql[1][1]), "+v"(fqh[1][1]));
    mult(1);
  };

#pragma unroll
  for (int st = 0; st < NS - 1; ++st) issue(st, st);
  for (int st = 0; st < nst; ++st) {
    stage_barrier();   // stage st has landed; every wave is done with stage st - 1
    issue(st + NS - 1, (st + NS - 1) % NS);
    compute(st % NS);
  }
  copy_barrier<0>();   // the trailing copies land before the workgroup ends

  // lane of (f, jf): rank rows 16 f + 4 g .. +3 of column c0 + 16 (2 wave + jf) + c16
  float* part = pr.part;
#pragma unroll
  for (int jf = 0; jf < 2; ++jf) {
    const int col = c0 + 16 * (2 * wave + jf) + c16;
    if (col < ncols) {
#pragma unroll
      for (int f = 0; f < FP; ++f)
#pragma unroll
        for (int qq = 0; qq < 4; ++qq) part[((size_t)sp * RP + 16 * f + 4 * g + qq) * ncols + col] = acc[f][jf][qq];
    }
  }
}

// ---------------------------------------------------------------------------
// Fixed-order sum of the split partials of dB and dA (s applied to dB), no
// atomics.  Runs at the end of the dX workgroups, after the token reductions
// have completed in stream order.
struct FinalizeArgs {
  const float* pb;
  const float* pa;
  float* dB;
  float* dA;
  int n, k, r, rp, sb, sa;
  float s;
  float sa_scale;   // 1, or 1 / (1 - p) with dropout (dA = dU^T keep X / (1 - p))
  int rpa;          // rows of one split's dA partial block (rp, or a group's stacked rank)
};

// Sum of `count` partials spaced `step` floats apart, in index order; the
// loads of each group of eight are all issued before the first add.
__device__ __forceinline__ float sum_partials(const float* p, size_t step, int count) {
  float v = 0.f;
  for (int p0 = 0; p0 < count; p0 += 8) {
    float x[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) x[u] = p0 + u < count ? p[(size_t)(p0 + u) * step] : 0.f;
#pragma unroll
    for (int u = 0; u < 8; ++u)
      if (p0 + u < count) v += x[u];
  }
  return v;
}

__device__ __forceinline__ void finalize_partials(const FinalizeArgs& f, int first, int stride) {
  const int nb = f.n * f.r, na = f.r * f.k;
  for (int e = first; e < nb + na; e += stride) {
    if (e < nb) {  // e = t * n + j: partial reads along j are contiguous
      const int t = e / f.n, j = e - t * f.n;
      const float v = sum_partials(f.pb + (size_t)t * f.n + j, (size_t)f.rp * f.n, f.sb);
      f.dB[(size_t)j * f.r + t] = f.s * v;
    } else {
      const int g = e - nb;
      const int t = g / f.k, l = g - t * f.k;
      f.dA[g] = f.sa_scale * sum_partials(f.pa + (size_t)t * f.k + l, (size_t)f.rpa * f.k, f.sa);
    }
  }
}

// Element q of a per-projection argument array (q uniform); compile-time
// indices only, so the kernel argument is never indexed dynamically.
template <typename T>
__device__ __forceinline__ T pick(const T (&v)[kMaxGroup], int q) {
  T x = v[0];
#pragma unroll
  for (int i = 1; i < kMaxGroup; ++i)
    if (q == i) x = v[i];
  return x;
}

// Kernel argument (by value) of the grouped dX GEMM of projections that read
// one X: dX = sum_g (dY_g W_g + dU_g A_g).  The n stages of every projection
// run back to back in one k loop (ceil(n_g / 64) stages each, nkb in all);
// the rank-r terms dU_g A_g are added after the loop,
// and the workgroup tails finalize every projection's dA_g and dB_g.
struct DxGroup {
  const u16* dY[kMaxGroup];
  const u16* W[kMaxGroup];
  const u16* dU2[kMaxGroup];
  const u16* A[kMaxGroup];
  int n[kMaxGroup];
  int count, nkb;
  FinalizeArgs fin[kMaxGroup];
};

// ---------------------------------------------------------------------------
// dX tile of BM tokens x BN input features, formed as dX^T = W^T dY^T with
// v_mfma_f32_32x32x16_bf16 (W as the A operand, dY as the B operand).  Stages
// of 64 along n: dY [BM rows][64] (k-contiguous) and W [64 rows of n][BN]
// (mn-contiguous, read with the transposing LDS read).  After the n stages,
// NSLAB stages cover the 2 RP wide slab: dU2 [BM][2RP] against A's rows, once
// for the high and once for the low part.  Global loads run two stages ahead
// in registers and are stored to the free LDS buffer piece by piece during
// the stage before their use (one barrier per stage).
//
// With dropout (DROP) the LoRA term is keep * (dU A) / (1 - p): the mask acts
// after the rank-r product, so it cannot ride in the k loop.  The slab stages
// are skipped; after the n stages the tile's dU2 rows, A columns and keep bits
// are staged in LDS, dU A is formed per fragment into a temporary
// accumulator, and added under the mask with the 1 / (1 - p) scale.
//
// With GRP (DxGroup) the n stages of all projections of a group form the k
// loop, each stage loading from its own projection's dY_g and W_g; the slab
// stages are skipped and each dU_g A_g is added after the loop from LDS.
//
// FULL (every n a multiple of 64 and the launch's columns a multiple of BN):
// the n-stage loads carry no bound checks.  With BN = 256 the stages are then
// copied straight into LDS (DMA below); on the 128 x 128 tile they keep the
// register staging and run in pairs with compile-time LDS buffers.
template <int BM, int BN, int WM, int WN, int RP, bool DROP, bool GRP, bool FULL>
__global__ __launch_bounds__(64 * WM * WN) void lora_bwd_dx_kernel(
    const u16* __restrict__ dY, const u16* __restrict__ W, const u16* __restrict__ dU2,
    const u16* __restrict__ A, const uint8_t* __restrict__ keep, u16* __restrict__ dX, int m, int n, int k,
    int r, int mp, float inv_keep, int tiles_m, int tiles_n, int l_begin, FinalizeArgs fin, DxGroup grp) {
  constexpr int NW = WM * WN;
  constexpr int NT = 64 * NW;
  constexpr int WTI = BM / WM, WTJ = BN / WN;

  constexpr int FI = WTI / 32, FJ = WTJ / 32;
  constexpr int STAGE = BM * 128 + 64 * BN * 2;
  constexpr int KS2 = 2 * RP;
  constexpr int NSLAB = (KS2 + 63) / 64;
  constexpr int CPR = BN / 8;                       // 16-byte chunks per W tile row
  constexpr int CY = BM * 8, CW = 64 * CPR;          // chunks per stage
  constexpr int LY = (CY + NT - 1) / NT, LW = (CW + NT - 1) / NT;
  static_assert(WTI % 32 == 0 && WTJ % 32 == 0, "32x32 fragments");
  static_assert(BN == 128 || BN == 256, "W tile rows of 256 or 512 bytes");
  static_assert(NSLAB == 1 || NSLAB == 2, "slab stages of the unrolled tail");
  // DMA: the 256-wide tiles with FULL copy their stages straight into
  // LDS (128 x 256: three buffers, two stages ahead; 256 x 256: two buffers,
  // one stage ahead), see the k loop below.  (The 128 x 128 tile with two
  // buffers measured slower than with register staging: 13B q_proj step
  // 462 -> 467 us.)
  constexpr bool DMA = FULL && BN == 256;
  constexpr int NBUF = DMA && BM == 128 ? 3 : 2;
  static_assert(NBUF * STAGE <= 160 * 1024, "LDS budget");
  __shared__ __attribute__((aligned(1024))) char smem[NBUF * STAGE];

  int tm, tn;
  tile_coords(tiles_m, tiles_n, 8, (int)blockIdx.x, tm, tn);
  const int m0 = tm * BM, l0 = l_begin + tn * BN;
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = uniform(tid >> 6);
  const int wm = wave / WN, wn = wave % WN;
  const int g = lane >> 5, c32 = lane & 31;
  const uint32_t yrow = (uint32_t)n * 2, wrow = (uint32_t)k * 2, urow = (uint32_t)KS2 * 2;
  const __amdgpu_buffer_rsrc_t rsY = make_rsrc(dY + (size_t)m0 * n, (uint64_t)min(BM, m - m0) * yrow);
  const __amdgpu_buffer_rsrc_t rsU = make_rsrc(dU2 + (size_t)m0 * KS2, (uint64_t)min(BM, mp - m0) * urow);
  const __amdgpu_buffer_rsrc_t rsA = make_rsrc(A, (uint64_t)r * wrow);
  const int nkb = GRP ? grp.nkb : (n + 63) / 64;

  // Staging registers move in pieces, one per 16-wide substep of the stage
  // that stores them: 0 = the dY (or dU2) rows, 1 and 2 = the two halves of
  // the W (or A) rows.
  constexpr int LW1 = (LW + 1) / 2;
  int4v gy[LY], gw[LW];
  // Loads of W stage st (dY columns and W rows st*64 ..) and of slab stage sl
  // (dU2 columns and the matching A rows, high part then low part).
  // With GRP the stages are loaded in order (piece 0 of a stage first), so a
  // load cursor -- projection, its stage, its dY rows -- advances by one stage
  // at each piece 0 and switches projection only at a boundary.
  int cur_g = 0, cur_sl = -1, cur_n = GRP ? grp.n[0] : n;
  const u16* cur_W = GRP ? grp.W[0] : W;
  uint32_t cur_yr = GRP ? (uint32_t)grp.n[0] * 2 : yrow;
  __amdgpu_buffer_rsrc_t cur_rsY =
      GRP ? make_rsrc(grp.dY[0] + (size_t)m0 * grp.n[0], (uint64_t)min(BM, m - m0) * cur_yr) : rsY;
  auto gload_w = [&](int st, int piece) LORA_INLINE {
    const u16* Wp = W;
    int ns = n, sl = st;
    if (GRP) {
      if (piece == 0) {
        ++cur_sl;
        if (cur_sl * 64 >= cur_n) {   // next projection (uniform, taken count - 1 times)
          ++cur_g;
          cur_sl = 0;
          cur_n = pick(grp.n, cur_g);
          cur_W = pick(grp.W, cur_g);
          cur_yr = (uint32_t)cur_n * 2;
          cur_rsY = make_rsrc(pick(grp.dY, cur_g) + (size_t)m0 * cur_n, (uint64_t)min(BM, m - m0) * cur_yr);
        }
      }
      Wp = cur_W;
      ns = cur_n;
      sl = cur_sl;
    }
    const int n0 = sl * 64;
    if (piece == 0) {
      const uint32_t yr = GRP ? cur_yr : yrow;
      const __amdgpu_buffer_rsrc_t rsYs = GRP ? cur_rsY : rsY;
#pragma unroll
      for (int i = 0; i < LY; ++i) {
        const int q = tid + i * NT;
        if (CY % NT != 0 && wave * 64 + i * NT >= CY) break;   // wave-uniform
        const int nn = n0 + 8 * (q & 7);
        gy[i] = buf_load16(rsYs, (FULL || nn < ns) ? (uint32_t)(q >> 3) * yr + (uint32_t)nn * 2 : kOOB);
      }
    } else if (piece <= 2) {
      const __amdgpu_buffer_rsrc_t rsW = make_rsrc(Wp + (size_t)n0 * k, (uint64_t)min(64, ns - n0) * wrow);
#pragma unroll
      for (int i = piece == 1 ? 0 : LW1; i < (piece == 1 ? LW1 : LW); ++i) {
        const int q = tid + i * NT;
        if (CW % NT != 0 && wave * 64 + i * NT >= CW) break;   // wave-uniform
        const int ll = l0 + 8 * (q % CPR);
        gw[i] = buf_load16(rsW, (FULL || ll < k) ? (uint32_t)(q / CPR) * wrow + (uint32_t)ll * 2 : kOOB);
      }
    }
  };
  auto gload_s = [&](int sl, int piece) LORA_INLINE {
    const int kk0 = sl * 64;
    if (piece == 0) {
#pragma unroll
      for (int i = 0; i < LY; ++i) {
        const int q = tid + i * NT;
        if (CY % NT != 0 && wave * 64 + i * NT >= CY) break;   // wave-uniform
        const int kk = kk0 + 8 * (q & 7);
        gy[i] = buf_load16(rsU, kk < KS2 ? (uint32_t)(q >> 3) * urow + (uint32_t)kk * 2 : kOOB);
      }
    } else if (piece <= 2) {
#pragma unroll
      for (int i = piece == 1 ? 0 : LW1; i < (piece == 1 ? LW1 : LW); ++i) {
        const int q = tid + i * NT;
        if (CW % NT != 0 && wave * 64 + i * NT >= CW) break;   // wave-uniform
        const int kk = kk0 + q / CPR;
        const int t = kk % RP;
        const int ll = l0 + 8 * (q % CPR);
        const bool ok = kk < KS2 && t < r && ll < k;
        gw[i] = buf_load16(rsA, ok ? (uint32_t)t * wrow + (uint32_t)ll * 2 : kOOB);
      }
    }
  };
  auto swrite = [&](int buf, int piece) LORA_INLINE {
    char* sb = smem + buf * STAGE;
    if (piece == 0) {
#pragma unroll
      for (int i = 0; i < LY; ++i) {
        const int q = tid + i * NT;
        if (CY % NT != 0 && wave * 64 + i * NT >= CY) break;
        *reinterpret_cast<int4v*>(sb + kc_offset(q >> 3, q & 7)) = gy[i];
      }
    } else if (piece <= 2) {
#pragma unroll
      for (int i = piece == 1 ? 0 : LW1; i < (piece == 1 ? LW1 : LW); ++i) {
        const int q = tid + i * NT;
        if (CW % NT != 0 && wave * 64 + i * NT >= CW) break;
        *reinterpret_cast<int4v*>(sb + BM * 128 + mc32_offset<BN>(q / CPR, q % CPR)) = gw[i];
      }
    }
  };

  floatx16 acc[FJ][FI];
#pragma unroll
  for (int a = 0; a < FJ; ++a)
#pragma unroll
    for (int b = 0; b < FI; ++b) acc[a][b] = floatx16{};

  // Fragments of the next 16-wide substep are read while the current one
  // multiplies (two register sets, p = substep parity).
  short8 fw[2][FJ], fy[2][FI];
  auto read_frags = [&](const char* sb, int ks, int p) LORA_INLINE {
    const char* Ys = sb;
    const char* Ws = sb + BM * 128;
#pragma unroll
    for (int fj = 0; fj < FJ; ++fj) fw[p][fj] = mc32_read_tr<BN>(Ws, 16 * ks, wn * WTJ + 32 * fj, lane);
#pragma unroll
    for (int fi = 0; fi < FI; ++fi) fy[p][fi] = kc_read(Ys, wm * WTI + 32 * fi + c32, 2 * ks + g);
  };
  auto multiply = [&](int p) LORA_INLINE {
#pragma unroll
    for (int fi = 0; fi < FI; ++fi)
#pragma unroll
      for (int fj = 0; fj < FJ; ++fj) acc[fj][fi] = mfma32x32x16(fw[p][fj], fy[p][fi], acc[fj][fi]);
  };

  if constexpr (DMA) {
    // Stages 0 .. nkb-1 over n, then the NSLAB slab stages; each stage is
    // copied from global memory straight into an LDS buffer without staging
    // registers (three or two buffers, two stages or one ahead): copy
    // instruction j of a wave fills 1 KB of the
    // buffer (dY region: rows 8j .. 8j+7; W region: rows WRK j ..), lane l its
    // 16-byte position l, which holds the logical chunk given by the tile's
    // swizzle (applied to the global address).  The fragment reads are issued
    // as inline assembly with explicit lgkmcnt waits: the compiler would
    // otherwise wait for every copy still in flight (s_waitcnt vmcnt(0))
    // before each transposing read, which undoes the prefetch.  Per substep a
    // wave issues NRD LDS reads (2 FJ transposing reads of W, FI of dY); the
    // products of substep ks wait until only the reads of substep ks+1 are
    // outstanding.  Each stage ends with a barrier that waits only for this
    // wave's copies of the next stage (copy_barrier).
    constexpr int NRD = 2 * FJ + FI;
    constexpr int CYW = BM / 8 / NW;        // dY-region copies per wave and stage
    constexpr int CWW = BN / 8 / NW;        // W-region copies per wave and stage
    constexpr int WRK = 512 / BN;           // W rows per 1 KB copy
    constexpr int WRB = BN * 2;             // bytes of a W tile row
    static_assert(CYW * NW * 8 == BM && CWW * NW * 8 == BN, "copies per stage");
    const int T = nkb + ((GRP || DROP) ? 0 : NSLAB);   // (group and dropout epilogues add dU A)
    // With GRP the copies walk the projections' stages in order (dload is
    // called once per stage, in stage order): cursor = projection, its stage,
    // its dY rows.
    int dc_g = 0, dc_sl = -1, dc_n = GRP ? grp.n[0] : n;
    const u16* dc_W = GRP ? grp.W[0] : W;
    uint32_t dc_yr = GRP ? (uint32_t)grp.n[0] * 2 : yrow;
    __amdgpu_buffer_rsrc_t dc_rsY =
        GRP ? make_rsrc(grp.dY[0] + (size_t)m0 * grp.n[0], (uint64_t)min(BM, m - m0) * dc_yr) : rsY;
    const int dl_r8 = lane >> 3, dl_c8 = lane & 7, dl_rw = lane / (BN / 8), dl_cw = lane % (BN / 8);
    auto dload = [&](int kb, int buf) LORA_INLINE {
      char* sb = smem + buf * STAGE;
      if (kb < nkb) {
        const u16* Wp = W;
        uint32_t yr = yrow;
        __amdgpu_buffer_rsrc_t rsYs = rsY;
        int sl = kb;
        if (GRP) {
          ++dc_sl;
          if (dc_sl * 64 >= dc_n) {   // next projection (uniform)
            ++dc_g;
            dc_sl = 0;
            dc_n = pick(grp.n, dc_g);
            dc_W = pick(grp.W, dc_g);
            dc_yr = (uint32_t)dc_n * 2;
            dc_rsY = make_rsrc(pick(grp.dY, dc_g) + (size_t)m0 * dc_n, (uint64_t)min(BM, m - m0) * dc_yr);
          }
          Wp = dc_W;
          yr = dc_yr;
          rsYs = dc_rsY;
          sl = dc_sl;
        }
        const __amdgpu_buffer_rsrc_t rsW = make_rsrc(Wp + (size_t)sl * 64 * k, (uint64_t)64 * wrow);
#pragma unroll
        for (int i = 0; i < CYW; ++i) {
          const int j = wave + NW * i, row = 8 * j + dl_r8;
          dma16(rsYs, (uint32_t)row * yr + (uint32_t)((dl_c8 ^ kc_swz(row)) << 4), (uint32_t)sl * 128,
                sb + j * 1024);
        }
#pragma unroll
        for (int i = 0; i < CWW; ++i) {
          const int j = wave + NW * i, row = WRK * j + dl_rw;
          const int c = dl_cw ^ mc32_swz(row);
          dma16(rsW, (uint32_t)row * wrow + (uint32_t)(l0 + 8 * c) * 2, 0, sb + BM * 128 + j * 1024);
        }
      } else {
        const int kk0 = (kb - nkb) * 64;
#pragma unroll
        for (int i = 0; i < CYW; ++i) {
          const int j = wave + NW * i, row = 8 * j + dl_r8;
          const int kk = kk0 + 8 * (dl_c8 ^ kc_swz(row));
          dma16(rsU, kk < KS2 ? (uint32_t)row * urow + (uint32_t)kk * 2 : kOOB, 0, sb + j * 1024);
        }
#pragma unroll
        for (int i = 0; i < CWW; ++i) {
          const int j = wave + NW * i, row = WRK * j + dl_rw;
          const int c = dl_cw ^ mc32_swz(row);
          const int kk = kk0 + row, t = kk % RP;
          dma16(rsA, (kk < KS2 && t < r) ? (uint32_t)t * wrow + (uint32_t)(l0 + 8 * c) * 2 : kOOB, 0,
                sb + BM * 128 + j * 1024);
        }
      }
    };
    constexpr int NCOPY = CYW + CWW;   // copies per wave and stage
    // Lane addresses of the fragment reads in buffer 0, substep 0: W fragment
    // fj (the second read of a pair is 4 rows further; substep ks adds 16
    // rows, the swizzle depending only on row % 4), dY fragment fi at substep
    // ks (fi adds 32 rows = 4096 bytes).
    uint32_t wa[FJ], ya[4];
    {
      const int h = (lane >> 4) & 1, j = lane & 15, e = j >> 2, q = j & 3;
#pragma unroll
      for (int fj = 0; fj < FJ; ++fj) {
        const int col = wn * WTJ + 32 * fj + 16 * h + 4 * q;
        wa[fj] = lds_addr(smem + BM * 128 + mc32_offset<BN>(8 * g + e, col >> 3) + (col & 7) * 2);
      }
#pragma unroll
      for (int ks = 0; ks < 4; ++ks) ya[ks] = lds_addr(smem + kc_offset(wm * WTI + c32, 2 * ks + g));
    }
    short4v fwl[2][FJ], fwh[2][FJ];
    auto reads = [&](uint32_t boff, int ks, int p) LORA_INLINE {
#pragma unroll
      for (int fj = 0; fj < FJ; ++fj) {
        const uint32_t a0 = wa[fj] + boff + (uint32_t)(16 * WRB) * ks;
        ds_read_tr_b64_asm<0>(fwl[p][fj], a0);
        ds_read_tr_b64_asm<4 * WRB>(fwh[p][fj], a0);
      }
      const uint32_t y0 = ya[ks] + boff;
      ds_read_b128_asm<0>(fy[p][0], y0);
      ds_read_b128_asm<4096>(fy[p][1], y0);
      if constexpr (FI == 4) {
        ds_read_b128_asm<8192>(fy[p][2], y0);
        ds_read_b128_asm<12288>(fy[p][3], y0);
      }
    };
    static_assert(FJ == 2 && (FI == 2 || FI == 4), "reads per substep");
    auto mult = [&](int p, bool last) LORA_INLINE {
      if constexpr (FI == 2) {
        if (last)
          asm volatile("s_waitcnt lgkmcnt(0)"
                       : "+v"(fwl[p][0]), "+v"(fwh[p][0]), "+v"(fwl[p][1]), "+v"(fwh[p][1]), "+v"(fy[p][0]),
                         "+v"(fy[p][1]));
        else
          asm volatile("s_waitcnt lgkmcnt(6)"
                       : "+v"(fwl[p][0]), "+v"(fwh[p][0]), "+v"(fwl[p][1]), "+v"(fwh[p][1]), "+v"(fy[p][0]),
                         "+v"(fy[p][1]));
      } else {
        if (last)
          asm volatile("s_waitcnt lgkmcnt(0)"
                       : "+v"(fwl[p][0]), "+v"(fwh[p][0]), "+v"(fwl[p][1]), "+v"(fwh[p][1]), "+v"(fy[p][0]),
                         "+v"(fy[p][1]), "+v"(fy[p][2]), "+v"(fy[p][3]));
        else
          asm volatile("s_waitcnt lgkmcnt(8)"
                       : "+v"(fwl[p][0]), "+v"(fwh[p][0]), "+v"(fwl[p][1]), "+v"(fwh[p][1]), "+v"(fy[p][0]),
                         "+v"(fy[p][1]), "+v"(fy[p][2]), "+v"(fy[p][3]));
      }
      static_assert(NRD == (FI == 2 ? 6 : 8), "wait counts above");
#pragma unroll
      for (int fj = 0; fj < FJ; ++fj) {
        const short8 w8 = join4(fwl[p][fj], fwh[p][fj]);
#pragma unroll
        for (int fi = 0; fi < FI; ++fi) acc[fj][fi] = mfma32x32x16(w8, fy[p][fi], acc[fj][fi]);
      }
    };
    auto compute = [&](uint32_t boff) LORA_INLINE {
      reads(boff, 0, 0);
#pragma unroll
      for (int ks = 0; ks < 4; ++ks) {
        if (ks < 3) reads(boff, ks + 1, (ks + 1) & 1);
        mult(ks & 1, ks == 3);
      }
    };
    using D0 = std::integral_constant<int, 0>;
    using D1 = std::integral_constant<int, 1>;
    using D2 = std::integral_constant<int, 2>;
    if constexpr (NBUF == 3) {
      auto dstage = [&](int kb, auto bufc, bool load_next) LORA_INLINE {
        constexpr int BUF = decltype(bufc)::value;
        if (load_next) dload(kb + 2, (BUF + 2) % 3);
        compute((uint32_t)BUF * STAGE);
        if (load_next) copy_barrier<NCOPY>();
        else copy_barrier<0>();
      };
      dload(0, 0);
      if (T > 1) dload(1, 1);
      copy_barrier<0>();
      int kb = 0;
      for (; kb + 5 < T; kb += 3) {
        dstage(kb, D0{}, true);
        dstage(kb + 1, D1{}, true);
        dstage(kb + 2, D2{}, true);
      }
      if (kb < T) dstage(kb, D0{}, kb + 2 < T);
      if (kb + 1 < T) dstage(kb + 1, D1{}, kb + 3 < T);
      if (kb + 2 < T) dstage(kb + 2, D2{}, kb + 4 < T);
      if (kb + 3 < T) dstage(kb + 3, D0{}, false);
      if (kb + 4 < T) dstage(kb + 4, D1{}, false);
    } else {
      // two buffers: stage kb+1 is copied into the other buffer (read in
      // stage kb-1, before the last barrier) while stage kb multiplies
      auto dstage = [&](int kb, auto bufc, bool load_next) LORA_INLINE {
        constexpr int BUF = decltype(bufc)::value;
        if (load_next) dload(kb + 1, BUF ^ 1);
        compute((uint32_t)BUF * STAGE);
        copy_barrier<0>();
      };
      dload(0, 0);
      copy_barrier<0>();
      int kb = 0;
      for (; kb + 1 < T; kb += 2) {
        dstage(kb, D0{}, true);
        dstage(kb + 1, D1{}, kb + 2 < T);
      }
      if (kb < T) dstage(kb, D0{}, false);
    }
  } else {
  // Same pipeline as the forward GEMM: at the top of stage st the registers
  // hold stage st+1; piece ks goes to the free LDS buffer at substep ks and
  // its registers then receive the loads of stage st+2.  With ROT the
  // products of substep 3 run after the barrier (zero operands before stage
  // 0).  Stages 0 .. nkb-1 run over n, the NSLAB (1 or 2) slab stages follow;
  // the tail is unrolled so every load is of a known kind.
  constexpr bool ROT = BM * BN < 256 * 256;
  if (ROT) {
#pragma unroll
    for (int j = 0; j < FJ; ++j) fw[1][j] = short8{};
#pragma unroll
    for (int j = 0; j < FI; ++j) fy[1][j] = short8{};
  }
  enum { LD_NONE, LD_W, LD_S0, LD_S1 };
  // bufc: the stage's LDS buffer as a compile-time constant, or -1 for the
  // parity of st at run time
  auto stage = [&](int st, auto bufc, bool write_next, int load) LORA_INLINE {
    constexpr int BUF = decltype(bufc)::value;
    const int cur = BUF >= 0 ? BUF : (st & 1);
    const char* sb = smem + cur * STAGE;
    read_frags(sb, 0, 0);
    if (ROT) multiply(1);
#pragma unroll
    for (int ks = 0; ks < 4; ++ks) {
      if (write_next) swrite(cur ^ 1, ks);
      if (load == LD_W) gload_w(st + 2, ks);
      if (load == LD_S0) gload_s(0, ks);
      if (load == LD_S1) gload_s(1, ks);
      if (ks < 3) read_frags(sb, ks + 1, (ks + 1) & 1);
      if (ks < 3 || !ROT) multiply(ks & 1);
    }
    __syncthreads();
  };
#pragma unroll
  for (int pc = 0; pc < 3; ++pc) gload_w(0, pc);
#pragma unroll
  for (int pc = 0; pc < 3; ++pc) swrite(0, pc);
  __syncthreads();
  constexpr int NSL = (DROP || GRP) ? 0 : NSLAB;   // slab stages in the k loop
  using B0 = std::integral_constant<int, 0>;
  using B1 = std::integral_constant<int, 1>;
  using BR = std::integral_constant<int, -1>;
  int st = 0;
  if (nkb >= 2) {
#pragma unroll
    for (int pc = 0; pc < 3; ++pc) gload_w(1, pc);
    if constexpr (FULL) {
      for (; st + 3 < nkb; st += 2) {
        stage(st, B0{}, true, LD_W);
        stage(st + 1, B1{}, true, LD_W);
      }
    }
    for (; st + 2 < nkb; ++st) stage(st, BR{}, true, LD_W);
    stage(st, BR{}, true, NSL > 0 ? LD_S0 : LD_NONE);   // st = nkb - 2
    ++st;
  } else if (NSL > 0) {
#pragma unroll
    for (int pc = 0; pc < 3; ++pc) gload_s(0, pc);
  }
  if (NSL > 0) stage(st++, BR{}, true, NSL > 1 ? LD_S1 : LD_NONE);   // writes slab 0
  if (NSL > 1) stage(st++, BR{}, true, LD_NONE);                     // writes slab 1
  stage(st, BR{}, false, LD_NONE);
  if (ROT) multiply(1);
  }

  if (GRP) {
    // LDS after the k loop, per projection: Us2 [BM][UP] bf16 (dU_g high |
    // low of the tile's tokens), As2 [RP][BN] bf16 mn-contiguous (A_g rows,
    // zero beyond r and k).  acc += [dU_hi | dU_lo] [A_g; A_g].
    constexpr int UP = 2 * RP + 8;
    constexpr int US_BYTES = BM * UP * 2, AS_BYTES = RP * BN * 2;
    static_assert(US_BYTES + AS_BYTES <= 2 * STAGE, "group epilogue fits the stage LDS");
    u16* Us2 = reinterpret_cast<u16*>(smem);
    char* As2 = smem + US_BYTES;
    for (int pq = 0; pq < grp.count; ++pq) {
      if (pq > 0) __syncthreads();                  // the previous projection's reads are done
      const __amdgpu_buffer_rsrc_t rsU2 =
          make_rsrc(pick(grp.dU2, pq) + (size_t)m0 * KS2, (uint64_t)min(BM, mp - m0) * urow);
      const __amdgpu_buffer_rsrc_t rsAq = make_rsrc(pick(grp.A, pq), (uint64_t)r * wrow);
      constexpr int UCH = BM * (RP / 4);            // 16-byte chunks of the dU2 rows
      for (int q = tid; q < UCH; q += NT) {
        const int i = q / (RP / 4), c = q % (RP / 4);
        *reinterpret_cast<int4v*>(Us2 + i * UP + 8 * c) = buf_load16(rsU2, (uint32_t)i * urow + (uint32_t)c * 16);
      }
      constexpr int ACH = RP * (BN / 8);
      for (int q = tid; q < ACH; q += NT) {
        const int t = q / (BN / 8), c = q % (BN / 8);
        const int ll = l0 + 8 * c;
        *reinterpret_cast<int4v*>(As2 + mc32_offset<BN>(t, c)) =
            buf_load16(rsAq, (t < r && ll < k) ? (uint32_t)t * wrow + (uint32_t)ll * 2 : kOOB);
      }
      __syncthreads();
      // (kk unrolled by two only: fully unrolled, the fragment reads of all
      // 2 RP / 16 steps are issued ahead and spill beside the accumulators)
#pragma unroll
      for (int fj = 0; fj < FJ; ++fj)
#pragma unroll 2
        for (int kk = 0; kk < KS2 / 16; ++kk) {
          const short8 af = mc32_read_tr<BN>(As2, (16 * kk) % RP, wn * WTJ + 32 * fj, lane);
#pragma unroll
          for (int fi = 0; fi < FI; ++fi) {
            const short8 bf =
                *reinterpret_cast<const short8*>(Us2 + (wm * WTI + 32 * fi + c32) * UP + 16 * kk + 8 * g);
            acc[fj][fi] = mfma32x32x16(af, bf, acc[fj][fi]);
          }
        }
    }
  }

  if (DROP) {
    // LDS after the k loop: Us2 [BM][UP] bf16 (dU high | low of the tile's
    // tokens), As2 [RP][BN] bf16 mn-contiguous (A rows, zero beyond r and k),
    // Kb [BM][BN/8] keep bytes of the tile.
    constexpr int UP = 2 * RP + 8;                  // Us2 row pitch in elements (16-byte multiple)
    constexpr int US_BYTES = BM * UP * 2, AS_BYTES = RP * BN * 2;
    static_assert(US_BYTES + AS_BYTES + BM * BN / 8 <= 2 * STAGE, "dropout epilogue fits the stage LDS");
    u16* Us2 = reinterpret_cast<u16*>(smem);
    char* As2 = smem + US_BYTES;
    uint8_t* Kb = reinterpret_cast<uint8_t*>(smem + US_BYTES + AS_BYTES);
    const uint32_t kb8 = (uint32_t)k / 8;
    {
      constexpr int UCH = BM * (RP / 4);            // 16-byte chunks of the dU2 rows
      const __amdgpu_buffer_rsrc_t rsU2 = make_rsrc(dU2 + (size_t)m0 * KS2, (uint64_t)min(BM, mp - m0) * urow);
      for (int q = tid; q < UCH; q += NT) {
        const int i = q / (RP / 4), c = q % (RP / 4);
        *reinterpret_cast<int4v*>(Us2 + i * UP + 8 * c) = buf_load16(rsU2, (uint32_t)i * urow + (uint32_t)c * 16);
      }
      constexpr int ACH = RP * (BN / 8);
      for (int q = tid; q < ACH; q += NT) {
        const int t = q / (BN / 8), c = q % (BN / 8);
        const int ll = l0 + 8 * c;
        *reinterpret_cast<int4v*>(As2 + mc32_offset<BN>(t, c)) =
            buf_load16(rsA, (t < r && ll < k) ? (uint32_t)t * wrow + (uint32_t)ll * 2 : kOOB);
      }
      constexpr int KCH = BM * (BN / 64);           // 8-byte chunks of keep bits
      const __amdgpu_buffer_rsrc_t rsK = make_rsrc(keep + (size_t)m0 * kb8, (uint64_t)min(BM, m - m0) * kb8);
      for (int q = tid; q < KCH; q += NT) {
        const int i = q / (BN / 64), c = q % (BN / 64);
        *reinterpret_cast<uint2*>(Kb + i * (BN / 8) + 8 * c) =
            buf_load8(rsK, (uint32_t)i * kb8 + (uint32_t)l0 / 8 + 8 * c);
      }
    }
    __syncthreads();
#pragma unroll
    for (int fj = 0; fj < FJ; ++fj) {
      floatx16 tmp[FI];
#pragma unroll
      for (int fi = 0; fi < FI; ++fi) tmp[fi] = floatx16{};
#pragma unroll
      for (int kk = 0; kk < KS2 / 16; ++kk) {        // k = t of [dU_hi | dU_lo] against [A; A]
        const short8 af = mc32_read_tr<BN>(As2, (16 * kk) % RP, wn * WTJ + 32 * fj, lane);
#pragma unroll
        for (int fi = 0; fi < FI; ++fi) {
          const short8 bf = *reinterpret_cast<const short8*>(Us2 + (wm * WTI + 32 * fi + c32) * UP + 16 * kk + 8 * g);
          tmp[fi] = mfma32x32x16(af, bf, tmp[fi]);
        }
      }
      // lane: token column c32 of fragment fi, features 8 qq + 4 g + q4 of
      // fragment fj -> keep byte (wn WTJ + 32 fj) / 8 + qq, bit 4 g + q4
#pragma unroll
      for (int fi = 0; fi < FI; ++fi) {
        const uint8_t* kr = Kb + (wm * WTI + 32 * fi + c32) * (BN / 8) + (wn * WTJ + 32 * fj) / 8;
#pragma unroll
        for (int qq = 0; qq < 4; ++qq) {
          const uint32_t byte = kr[qq];
#pragma unroll
          for (int q4 = 0; q4 < 4; ++q4)
            if ((byte >> (4 * g + q4)) & 1u) acc[fj][fi][4 * qq + q4] += inv_keep * tmp[fi][4 * qq + q4];
        }
      }
    }
  }

  // store dX: each wave's 32-token blocks of its 64 features through a
  // wave-private LDS region (the k loop ended with a barrier; the group and
  // dropout epilogues read LDS until here)
  static_assert(FJ == 2 && NW * kYsBytes <= 2 * STAGE, "output staging");
  if (GRP || DROP) __syncthreads();
  {
    const int j0 = l0 + wn * WTJ;
#pragma unroll
    for (int fi = 0; fi < FI; ++fi) {
      const int i0 = m0 + wm * WTI + 32 * fi;
      store_block_32x64(acc[0][fi], acc[1][fi], smem + wave * kYsBytes, dX + (size_t)i0 * k + j0, (size_t)k,
                        m - i0, k - j0, lane);
    }
  }
  // After its tile, every workgroup sums a slice of the dA, dB partials
  // (complete: the token reductions ran before this launch in stream order).
  const int first = (int)blockIdx.x * NT + (int)threadIdx.x, stride = (int)gridDim.x * NT;
  if (GRP) {
    for (int pq = 0; pq < grp.count; ++pq) finalize_partials(pick(grp.fin, pq), first, stride);
  } else {
    finalize_partials(fin, first, stride);
  }
}

// ---------------------------------------------------------------------------
// Fused backward for ranks up to 16 (no dropout): the dX GEMM also forms dU
// and the dB partials from the dY tiles it stages, so no other launch reads
// dY.  Tile of 128 tokens x 256 input features, waves and k loop as in
// lora_bwd_dx_kernel (stages of 64 along n, loads two stages ahead in
// registers, the products of the last substep after the barrier).
//   dU^T = B^T dY^T: each stage also stages its 64 B rows ([64][16] bf16,
//     zero beyond r and n); at substep wn of every stage, wave (wm, wn)
//     multiplies the transposed B rows (rows t >= 16 of the operand zero)
//     with its own dY fragments.  After the loop the four partial sums of each
//     token are added in wn order, s dU is split into bf16 high and low parts
//     in LDS, and the rank-r term [dU_hi | dU_lo] [A; A] is added to the dX
//     tile.  The workgroups of column tile 0 also store the parts transposed
//     (dUt2 [16][mp], the bf16 high part) for the dA reduction.
//   dB^T partials: at the stages st with st % tiles_n == tn, four waves (the
//     lower or upper four, alternately) each form U^T dY for 16 of the stage's
//     64 n over the tile's 128 tokens, with U^T as high and low bf16 parts
//     (staged in LDS in the prologue), and store the tile row's partial
//     pbt [tm][16][n] (s is applied by the finalize).
// FULL: n a multiple of 64 and k of 256 (no bound checks on the loads).
// FASTB: r a multiple of 8 (B rows staged with 16-byte loads).
template <bool FULL, bool FASTB>
__global__ __launch_bounds__(512) void lora_bwd_dxf_kernel(
    const u16* __restrict__ dY, const u16* __restrict__ W, const u16* __restrict__ A, const u16* __restrict__ B,
    const float* __restrict__ U, u16* __restrict__ dX, u16* __restrict__ dUt2, float* __restrict__ pbt, int m, int n,
    int k, int r, int mp, float s, int tiles_m, int tiles_n) {
  constexpr int BM = 128, BN = 256, WM = 2, WN = 4, RP = 16;
  constexpr int NW = WM * WN, NT = 64 * NW;
  constexpr int WTI = BM / WM, WTJ = BN / WN;
  constexpr int FI = WTI / 32, FJ = WTJ / 32;
  constexpr int YB = BM * 128, WB = 64 * BN * 2, BB = 64 * RP * 2;
  constexpr int STAGE = YB + WB + BB;
  constexpr int CPR = BN / 8;                       // 16-byte chunks per W tile row
  constexpr int CY = BM * 8, CW = 64 * CPR;
  constexpr int LY = CY / NT, LW = CW / NT, LW1 = LW / 2;
  constexpr int UTP = BM * 2 + 16;                  // U^T row pitch in bytes
  constexpr int UT_OFF = 2 * STAGE;
  static_assert(CY % NT == 0 && CW % NT == 0 && UT_OFF + 2 * RP * UTP <= 160 * 1024, "tile shape and LDS budget");
  __shared__ __attribute__((aligned(1024))) char smem[UT_OFF + 2 * RP * UTP];

  int tm, tn;
  tile_coords(tiles_m, tiles_n, 8, (int)blockIdx.x, tm, tn);
  const int m0 = tm * BM, l0 = tn * BN;
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = uniform(tid >> 6);
  const int wm = wave / WN, wn = wave % WN;
  const int g = lane >> 5, c32 = lane & 31;
  const int g16 = lane >> 4, c16 = lane & 15;
  const uint32_t yrow = (uint32_t)n * 2, wrow = (uint32_t)k * 2;
  const __amdgpu_buffer_rsrc_t rsY = make_rsrc(dY + (size_t)m0 * n, (uint64_t)min(BM, m - m0) * yrow);
  const __amdgpu_buffer_rsrc_t rsA = make_rsrc(A, (uint64_t)r * wrow);
  const __amdgpu_buffer_rsrc_t rsB = make_rsrc(B, (uint64_t)n * r * 2);
  const int nkb = (n + 63) / 64;

  // U^T of the tile's tokens: high parts in rows 0..15, low parts in rows
  // 16..31 (zero beyond r and m), for the dB products.
  char* Uts = smem + UT_OFF;
  {
    constexpr int UPT = BM * RP / NT;   // all loads issued before the first store
    static_assert(BM * RP % NT == 0, "U values per thread");
    const __amdgpu_buffer_rsrc_t rsU = make_rsrc(U + (size_t)m0 * r, (uint64_t)min(BM, m - m0) * r * 4);
    float uv[UPT];
#pragma unroll
    for (int q = 0; q < UPT; ++q) {
      const int e = tid + q * NT, i = e / RP, t = e - i * RP;
      uv[q] = buf_load4f(rsU, t < r ? (uint32_t)(i * r + t) * 4 : kOOB);
    }
#pragma unroll
    for (int q = 0; q < UPT; ++q) {
      const int e = tid + q * NT, i = e / RP, t = e - i * RP;
      const u16 h = f32_to_bf16(uv[q]);
      *reinterpret_cast<u16*>(Uts + t * UTP + i * 2) = h;
      *reinterpret_cast<u16*>(Uts + (RP + t) * UTP + i * 2) = f32_to_bf16(uv[q] - bf16_to_f32(h));
    }
  }

  // Staging registers, stored in pieces: 0 = the dY rows and (threads below
  // 128) one 16-byte half of a B row, 1 and 2 = the two halves of the W rows.
  int4v gy[LY], gw[LW], gb = int4v{0, 0, 0, 0};
  auto gload = [&](int st, int piece) LORA_INLINE {
    const int n0 = st * 64;
    if (piece == 0) {
#pragma unroll
      for (int i = 0; i < LY; ++i) {
        const int q = tid + i * NT;
        const int nn = n0 + 8 * (q & 7);
        gy[i] = buf_load16(rsY, (FULL || nn < n) ? (uint32_t)(q >> 3) * yrow + (uint32_t)nn * 2 : kOOB);
      }
      if (tid < 128) {   // waves 0 and 1: row n0 + tid / 2, ranks 8 (tid % 2) .. +7
        const int row = n0 + (tid >> 1), t0 = 8 * (tid & 1);
        if constexpr (FASTB) {
          gb = buf_load16(rsB, (row < n && t0 < r) ? ((uint32_t)row * r + t0) * 2 : kOOB);
        } else {
          uint32_t w[4];
#pragma unroll
          for (int x = 0; x < 4; ++x) {
            const int t = t0 + 2 * x;
            const uint32_t lo = (row < n && t < r) ? B[(size_t)row * r + t] : 0u;
            const uint32_t hi = (row < n && t + 1 < r) ? B[(size_t)row * r + t + 1] : 0u;
            w[x] = lo | (hi << 16);
          }
          gb = int4v{(int)w[0], (int)w[1], (int)w[2], (int)w[3]};
        }
      }
    } else if (piece <= 2) {
      const __amdgpu_buffer_rsrc_t rsW = make_rsrc(W + (size_t)n0 * k, (uint64_t)min(64, n - n0) * wrow);
#pragma unroll
      for (int i = piece == 1 ? 0 : LW1; i < (piece == 1 ? LW1 : LW); ++i) {
        const int q = tid + i * NT;
        const int ll = l0 + 8 * (q % CPR);
        gw[i] = buf_load16(rsW, (FULL || ll < k) ? (uint32_t)(q / CPR) * wrow + (uint32_t)ll * 2 : kOOB);
      }
    }
  };
  auto swrite = [&](int buf, int piece) LORA_INLINE {
    char* sb = smem + buf * STAGE;
    if (piece == 0) {
#pragma unroll
      for (int i = 0; i < LY; ++i) {
        const int q = tid + i * NT;
        *reinterpret_cast<int4v*>(sb + kc_offset(q >> 3, q & 7)) = gy[i];
      }
      if (tid < 128) *reinterpret_cast<int4v*>(sb + YB + WB + tid * 16) = gb;   // Bs [64][16]
    } else if (piece <= 2) {
#pragma unroll
      for (int i = piece == 1 ? 0 : LW1; i < (piece == 1 ? LW1 : LW); ++i) {
        const int q = tid + i * NT;
        *reinterpret_cast<int4v*>(sb + YB + mc32_offset<BN>(q / CPR, q % CPR)) = gw[i];
      }
    }
  };

  floatx16 acc[FJ][FI], dacc[FI];
#pragma unroll
  for (int a = 0; a < FJ; ++a)
#pragma unroll
    for (int b = 0; b < FI; ++b) acc[a][b] = floatx16{};
#pragma unroll
  for (int b = 0; b < FI; ++b) dacc[b] = floatx16{};

  // Fragments of substep ks (16 n): W and dY as in lora_bwd_dx_kernel, and at
  // this wave's substep (ks == wn) the B^T operand: lane (g, c32) row t = c32
  // (zero for c32 >= 16), k = n 16 ks + 8g .. +7, read transposed from Bs
  // (rows of 32 bytes, no swizzle: a 16-lane read covers 128 contiguous bytes).
  short8 fw[2][FJ], fy[2][FI], fb = short8{};
  auto read_frags = [&](const char* sb, int ks, int p) LORA_INLINE {
    const char* Ys = sb;
    const char* Ws = sb + YB;
#pragma unroll
    for (int fj = 0; fj < FJ; ++fj) fw[p][fj] = mc32_read_tr<BN>(Ws, 16 * ks, wn * WTJ + 32 * fj, lane);
#pragma unroll
    for (int fi = 0; fi < FI; ++fi) fy[p][fi] = kc_read(Ys, wm * WTI + 32 * fi + c32, 2 * ks + g);
    if (ks == wn) {
      const int j = lane & 15;
      const char* p0 = sb + YB + WB + (16 * ks + 8 * g + (j >> 2)) * (RP * 2) + (j & 3) * 8;
      const short8 v = join4(__builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_short4v*)p0),
                             __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_short4v*)(p0 + 4 * RP * 2)));
      fb = ((lane >> 4) & 1) ? short8{} : v;
    }
  };
  auto multiply = [&](int p, int ks) LORA_INLINE {
#pragma unroll
    for (int fi = 0; fi < FI; ++fi)
#pragma unroll
      for (int fj = 0; fj < FJ; ++fj) acc[fj][fi] = mfma32x32x16(fw[p][fj], fy[p][fi], acc[fj][fi]);
    if (ks == wn) {
#pragma unroll
      for (int fi = 0; fi < FI; ++fi) dacc[fi] = mfma32x32x16(fb, fy[p][fi], dacc[fi]);
    }
  };
  // dB^T partial of stage st (its buffer sb): wave set (st / tiles_n) % 2,
  // wave f of the set takes n columns 16 f .. 16 f + 15 of the stage.
  auto dB_part = [&](const char* sb, int st) LORA_INLINE {
    const int f = wave - 4 * ((st / tiles_n) & 1);
    if (f < 0 || f >= 4) return;
    floatx4 d = floatx4{0.f, 0.f, 0.f, 0.f};
    const int j = lane & 15, col = 16 * f + 4 * (j & 3);
#pragma unroll
    for (int kt = 0; kt < BM / 32; ++kt) {
      // B operand: lane (g16, c16) column n 16 f + c16, k = tokens 32 kt + 8 g16 .. +7
      const int r0 = 32 * kt + 8 * g16 + (j >> 2);
      const char* p0 = sb + kc_offset(r0, col >> 3) + (col & 7) * 2;
      const char* p1 = sb + kc_offset(r0 + 4, col >> 3) + (col & 7) * 2;
      const short8 yb = join4(__builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_short4v*)p0),
                              __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_short4v*)p1));
      const short8 uh = *reinterpret_cast<const short8*>(Uts + c16 * UTP + (32 * kt + 8 * g16) * 2);
      const short8 ul = *reinterpret_cast<const short8*>(Uts + (RP + c16) * UTP + (32 * kt + 8 * g16) * 2);
      d = mfma16x16x32(uh, yb, d);
      d = mfma16x16x32(ul, yb, d);
    }
    const int cn = st * 64 + 16 * f + c16;   // lane: column cn, ranks 4 g16 .. +3
    if (FULL || cn < n) {
#pragma unroll
      for (int q = 0; q < 4; ++q) pbt[((size_t)tm * RP + 4 * g16 + q) * n + cn] = d[q];
    }
  };

#pragma unroll
  for (int j = 0; j < FJ; ++j) fw[1][j] = short8{};
#pragma unroll
  for (int j = 0; j < FI; ++j) fy[1][j] = short8{};
  auto stage = [&](int st, auto bufc, bool write_next, bool load_next) LORA_INLINE {
    constexpr int BUF = decltype(bufc)::value;
    const int cur = BUF >= 0 ? BUF : (st & 1);
    const char* sb = smem + cur * STAGE;
    read_frags(sb, 0, 0);
    multiply(1, 3);   // substep 3 of the previous stage (zero operands before stage 0)
#pragma unroll
    for (int ks = 0; ks < 4; ++ks) {
      if (write_next) swrite(cur ^ 1, ks);
      if (load_next) gload(st + 2, ks);
      if (ks < 3) {
        read_frags(sb, ks + 1, (ks + 1) & 1);
        multiply(ks & 1, ks);
      }
    }
    if (st % tiles_n == tn) dB_part(sb, st);
    __syncthreads();
  };
#pragma unroll
  for (int pc = 0; pc < 3; ++pc) gload(0, pc);
#pragma unroll
  for (int pc = 0; pc < 3; ++pc) swrite(0, pc);
  __syncthreads();
  // (stages with run-time buffer parity: the paired loop of lora_bwd_dx_kernel
  // spills here)
  using BR = std::integral_constant<int, -1>;
  int st = 0;
  if (nkb >= 2) {
#pragma unroll
    for (int pc = 0; pc < 3; ++pc) gload(1, pc);
    for (; st + 2 < nkb; ++st) stage(st, BR{}, true, true);
    stage(st++, BR{}, true, false);   // st = nkb - 2: stores the last stage
  }
  stage(st, BR{}, false, false);
  multiply(1, 3);

  // ---- epilogue (LDS stage buffers free after the loop's last barrier):
  // red [NW][FI][8][64] fp32 (rows t < 16 of each wave's dU^T partials), Us2
  // [BM][UP] bf16 (s dU high | low), As2 [RP][BN] bf16 mn-contiguous (A rows
  // of the tile, zero beyond r and k).
  constexpr int RED = NW * FI * 8 * 64 * 4;
  constexpr int UP = 2 * RP + 8;
  static_assert(RED + BM * UP * 2 + RP * BN * 2 <= UT_OFF && NW * kYsBytes <= UT_OFF, "epilogue fits the stage LDS");
  float* red = reinterpret_cast<float*>(smem);
  u16* Us2 = reinterpret_cast<u16*>(smem + RED);
  char* As2 = smem + RED + BM * UP * 2;
#pragma unroll
  for (int fi = 0; fi < FI; ++fi)
#pragma unroll
    for (int q = 0; q < 8; ++q) red[((wave * FI + fi) * 8 + q) * 64 + lane] = dacc[fi][q];
  for (int q = tid; q < RP * (BN / 8); q += NT) {
    const int t = q / (BN / 8), c = q % (BN / 8);
    const int ll = l0 + 8 * c;
    *reinterpret_cast<int4v*>(As2 + mc32_offset<BN>(t, c)) =
        buf_load16(rsA, (t < r && ll < k) ? (uint32_t)t * wrow + (uint32_t)ll * 2 : kOOB);
  }
  __syncthreads();
  // entry e: lane ln of (token half wh, fragment fi), result row q: token
  // wh 64 + 32 fi + ln % 32, rank 8 (q / 4) + 4 (ln / 32) + q % 4
  for (int e = tid; e < WM * FI * 8 * 64; e += NT) {
    const int ln = e & 63, q = (e >> 6) & 7, fi = (e >> 9) & 1, wh = e >> 10;
    float v = 0.f;
#pragma unroll
    for (int w4 = 0; w4 < WN; ++w4) v += red[(((wh * WN + w4) * FI + fi) * 8 + q) * 64 + ln];
    const int i = wh * WTI + 32 * fi + (ln & 31);
    const int t = 8 * (q >> 2) + 4 * (ln >> 5) + (q & 3);
    const float d = s * v;
    const u16 hi = f32_to_bf16(d), lo = f32_to_bf16(d - bf16_to_f32(hi));
    Us2[i * UP + t] = hi;
    Us2[i * UP + RP + t] = lo;
    if (tn == 0 && m0 + i < mp) dUt2[(size_t)t * mp + m0 + i] = hi;
  }
  __syncthreads();
#pragma unroll
  for (int fj = 0; fj < FJ; ++fj) {
    const short8 af = mc32_read_tr<BN>(As2, 0, wn * WTJ + 32 * fj, lane);
#pragma unroll
    for (int kk = 0; kk < 2; ++kk)   // k = t of [dU_hi | dU_lo] against [A; A]
#pragma unroll
      for (int fi = 0; fi < FI; ++fi) {
        const short8 bf = *reinterpret_cast<const short8*>(Us2 + (wm * WTI + 32 * fi + c32) * UP + 16 * kk + 8 * g);
        acc[fj][fi] = mfma32x32x16(af, bf, acc[fj][fi]);
      }
  }
  __syncthreads();
  {
    const int j0 = l0 + wn * WTJ;
#pragma unroll
    for (int fi = 0; fi < FI; ++fi) {
      const int i0 = m0 + wm * WTI + 32 * fi;
      store_block_32x64(acc[0][fi], acc[1][fi], smem + wave * kYsBytes, dX + (size_t)i0 * k + j0, (size_t)k,
                        m - i0, k - j0, lane);
    }
  }
}

// Fixed-order sum of the dA and dB partials as a launch of its own (the fused
// backward's token reduction runs after its dX launch).
__global__ __launch_bounds__(256) void lora_finalize_kernel(FinalizeArgs f) {
  finalize_partials(f, (int)(blockIdx.x * 256 + threadIdx.x), (int)(gridDim.x * 256));
}

// ---------------------------------------------------------------------------
// Launchers: execute the plans of lora_plan.hpp.

// dX instantiations a plan can name: no dropout in groups or on the 256 x 256
// tile, and the 256 x 256 tile only with whole stages (FULL).
template <int BM, int BN, int RP, bool DROP, bool GRP, bool FULL>
constexpr bool dx_instantiated() {
  return !(DROP && GRP) && !(DROP && BM == 256) && !(BM == 256 && !FULL);
}

static hipError_t run_dx(const Launch& L, const BwdArgs& a, const u16* dU2, int mp, const FinalizeArgs& fin,
                         const DxGroup& grp, hipStream_t st) {
  const dim3 grid((unsigned)L.grid), block((unsigned)L.block);
  return with_int<0, 1, 2>(tile_code(L), [&](auto tc) {
    constexpr int T = decltype(tc)::value;
    constexpr int BM = T == 0 ? 256 : 128, BN = T == 2 ? 128 : 256, WN = T == 2 ? 2 : 4;
    return with_int<16, 32, 48, 64>(L.rp, [&](auto rc) {
      return with_bool(L.drop, [&](auto dr) {
        return with_bool(L.grp, [&](auto gr) {
          return with_bool(L.full, [&](auto fu) {
            constexpr int RP = decltype(rc)::value;
            constexpr bool DROP = decltype(dr)::value, GRP = decltype(gr)::value, FULL = decltype(fu)::value;
            if constexpr (!dx_instantiated<BM, BN, RP, DROP, GRP, FULL>()) {
              return hipErrorInvalidValue;
            } else {
              hipLaunchKernelGGL((lora_bwd_dx_kernel<BM, BN, 2, WN, RP, DROP, GRP, FULL>), grid, block, 0, st, a.dY,
                                 a.W, dU2, a.A, a.keep, a.dX, (int)a.m, (int)a.n, (int)a.k, (int)a.r, mp, a.inv_keep,
                                 L.tiles_m, L.tiles_n, (int)L.col_begin, L.finalize ? fin : FinalizeArgs{}, grp);
              return hipGetLastError();
            }
          });
        });
      });
    });
  });
}

// dUt2: where dU^T goes (the projection's own region, or its rows of a
// group's stacked region).
static hipError_t run_du(const Launch& L, const BwdArgs& a, const BwdLayout& BL, hipStream_t st,
                         u16* dUt2 = nullptr) {
  u16* Ut2 = reinterpret_cast<u16*>(a.ws + BL.ut2);
  u16* dU2 = reinterpret_cast<u16*>(a.ws + BL.du2);
  if (!dUt2) dUt2 = reinterpret_cast<u16*>(a.ws + BL.dut2);
  return with_int<16, 32, 48, 64>(L.rp, [&](auto rc) {
    return with_int<8, 16, 32>(L.tpw, [&](auto tc) {
      constexpr int RP = decltype(rc)::value, TPW = decltype(tc)::value;
      if (L.fastb)
        hipLaunchKernelGGL((lora_bwd_du_dma_kernel<RP, TPW>), dim3((unsigned)L.grid), dim3((unsigned)L.block), 0, st,
                           a.dY, a.B, a.U, dU2, dUt2, Ut2, (int)a.m, (int)a.n, (int)a.r, (int)BL.mp, a.s);
      else
        hipLaunchKernelGGL((lora_bwd_du_kernel<RP, TPW>), dim3((unsigned)L.grid), dim3((unsigned)L.block), 0, st,
                           a.dY, a.B, a.U, dU2, dUt2, Ut2, (int)a.m, (int)a.n, (int)a.r, (int)BL.mp, a.s);
      return hipGetLastError();
    });
  });
}

// The two token reductions of one projection in one launch: dB^T partials =
// Ut2 . dY, then dA partials = dUt2 . X (masked X under dropout).
// L.part: 0 both reductions, 1 dB only (a group member whose dA is reduced
// with the group's), 2 the group's stacked dA (pap given by the caller).
static hipError_t run_tokred(const Launch& L, const BwdArgs& a, const BwdLayout& BL, hipStream_t st,
                             const RedProblem* stacked = nullptr) {
  const u16* Ut2 = reinterpret_cast<const u16*>(a.ws + BL.ut2);
  const u16* dUt2 = reinterpret_cast<const u16*>(a.ws + BL.dut2);
  float* pb = reinterpret_cast<float*>(a.ws + BL.pb);
  float* pa = reinterpret_cast<float*>(a.ws + BL.pa);
  const RedProblem pbp0{Ut2, a.dY, pb, (int)a.n, (int)BL.plan_b.span, BL.plan_b.col_tiles, nullptr};
  const RedProblem pap0{dUt2, a.X, pa, (int)a.k, (int)BL.plan_a.span, BL.plan_a.col_tiles, a.keep};
  const RedProblem pbp = L.part == 2 ? *stacked : pbp0;
  const RedProblem pap = L.part == 0 ? pap0 : pbp;
  const int nb0 = L.part == 0 ? BL.plan_b.col_tiles * BL.plan_b.splits : (int)L.grid;
  return with_int<16, 32, 48, 64>(L.rp, [&](auto rc) {
    constexpr int RP = decltype(rc)::value;
    if (L.drop)
      hipLaunchKernelGGL((lora_tokred_kernel<RP, true>), dim3((unsigned)L.grid), dim3((unsigned)L.block), 0, st, pbp,
                         pap, nb0, (int)a.m, (int)BL.mp);
    else
      hipLaunchKernelGGL((lora_tokred_dma_kernel<RP>), dim3((unsigned)L.grid), dim3((unsigned)L.block), 0, st, pbp,
                         pap, nb0, (int)a.m, (int)BL.mp);
    return hipGetLastError();
  });
}

static FinalizeArgs finalize_args(const BwdArgs& a, const BwdLayout& L) {
  return FinalizeArgs{reinterpret_cast<const float*>(a.ws + L.pb), reinterpret_cast<const float*>(a.ws + L.pa),
                      a.dB, a.dA, (int)a.n, (int)a.k, (int)a.r, L.rp, L.plan_b.splits, L.plan_a.splits, a.s,
                      a.keep ? a.inv_keep : 1.0f, L.rp};
}

hipError_t launch_bwd(const BwdArgs& a, hipStream_t st) {
  const BwdLayout BL = bwd_layout(a.m, a.n, a.k, a.r);
  const Plan p = plan_bwd(a.m, a.n, a.k, a.r, a.keep != nullptr);
  const FinalizeArgs fin = finalize_args(a, BL);
  const DxGroup none{};
  const u16* dU2 = reinterpret_cast<const u16*>(a.ws + BL.du2);
  for (int i = 0; i < p.count; ++i) {
    const Launch& L = p.l[i];
    hipError_t e = hipErrorInvalidValue;
    switch (L.id) {
      case K_DU: e = run_du(L, a, BL, st); break;
      case K_TOKRED: e = run_tokred(L, a, BL, st); break;
      case K_DX: e = run_dx(L, a, dU2, (int)BL.mp, fin, none, st); break;
      default: break;
    }
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

// Fused backward: the dX launch (dU, the dB partials, dX), the dA token
// reduction, then the finalize of dA and dB.
hipError_t launch_bwd_fused(const BwdArgs& a, hipStream_t st) {
  const BwdFusedLayout BL = bwd_fused_layout(a.m, a.n, a.k, a.r);
  const Plan p = plan_bwd_fused(a.m, a.n, a.k, a.r);
  u16* dUt2 = reinterpret_cast<u16*>(a.ws + BL.dut2);
  float* pb = reinterpret_cast<float*>(a.ws + BL.pb);
  float* pa = reinterpret_cast<float*>(a.ws + BL.pa);
  const int m = (int)a.m, n = (int)a.n, k = (int)a.k, r = (int)a.r, mp = (int)BL.mp;
  for (int i = 0; i < p.count; ++i) {
    const Launch& L = p.l[i];
    const dim3 grid((unsigned)L.grid), block((unsigned)L.block);
    if (L.id == K_DXF) {
      const hipError_t e = with_bool(L.full, [&](auto fc) {
        return with_bool(L.fastb, [&](auto bc) {
          constexpr bool F = decltype(fc)::value, FB = decltype(bc)::value;
          if constexpr (F && !FB) {
            return hipErrorInvalidValue;
          } else {
            hipLaunchKernelGGL((lora_bwd_dxf_kernel<F, FB>), grid, block, 0, st, a.dY, a.W, a.A, a.B, a.U, a.dX, dUt2,
                               pb, m, n, k, r, mp, a.s, L.tiles_m, L.tiles_n);
            return hipGetLastError();
          }
        });
      });
      if (e != hipSuccess) return e;
    } else if (L.id == K_TOKRED) {
      const RedProblem pap{dUt2, a.X, pa, k, (int)BL.plan_a.span, BL.plan_a.col_tiles, nullptr};
      hipLaunchKernelGGL((lora_tokred_dma_kernel<16>), grid, block, 0, st, pap, pap, (int)L.grid, m, mp);
      const hipError_t e = hipGetLastError();
      if (e != hipSuccess) return e;
    } else if (L.id == K_FINALIZE) {
      const FinalizeArgs fin{pb, pa, a.dB, a.dA, n, k, r, 16, BL.tiles_m, BL.plan_a.splits, a.s, 1.0f, 16};
      hipLaunchKernelGGL(lora_finalize_kernel, grid, block, 0, st, fin);
      const hipError_t e = hipGetLastError();
      if (e != hipSuccess) return e;
    } else {
      return hipErrorInvalidValue;
    }
  }
  return hipSuccess;
}

// ---------------------------------------------------------------------------
// Backward without a caller-provided workspace: the workspace regions live in
// a fixed device array of this library, one per GPU, whose address is looked
// up once per device (with that device current) on the first call there.
// Host code never passes the array's name itself to a kernel or a copy: in
// host code it stands for a host-side shadow, not the device address.
static __device__ __align__(256) char scratch[kNoAllocScratchBytes];

namespace {
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};
}  // namespace

hipError_t noalloc_scratch(void** out) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    if (!p) return hipErrorInvalidSymbol;
    g_scratch_ptr[dev] = p;
  }
  *out = g_scratch_ptr[dev];
  return hipSuccess;
}

hipError_t launch_bwd_noalloc(const BwdArgs& a, hipStream_t st) {
  if (bwd_layout(a.m, a.n, a.k, a.r).total > kNoAllocScratchBytes) return hipErrorInvalidValue;
  void* ws = nullptr;
  const hipError_t e = noalloc_scratch(&ws);
  if (e != hipSuccess) return e;
  BwdArgs b = a;
  b.ws = static_cast<char*>(ws);
  return launch_bwd(b, st);
}

// Grouped backward: per projection the dU and token-reduction launches (each
// in its own workspace region), then one dX launch over the whole group whose
// tails (of the first column range) finalize every projection's dA and dB.
hipError_t launch_bwd_group(const GroupBwdArgs& a, hipStream_t st) {
  auto member_args = [&](int g, const GroupBwdLayout& GL) {
    BwdArgs b{};
    b.dY = a.dY[g]; b.X = a.X; b.W = a.W[g]; b.A = a.A[g]; b.B = a.B[g]; b.U = a.U[g];
    b.dX = a.dX; b.dA = a.dA[g]; b.dB = a.dB[g]; b.ws = a.ws + GL.off[g];
    b.m = a.m; b.n = a.n[g]; b.k = a.k; b.r = a.r; b.s = a.s;
    return b;
  };
  if (a.count == 1) {   // a group of one is the single projection (workspace sizes agree)
    BwdArgs b{};
    b.dY = a.dY[0]; b.X = a.X; b.W = a.W[0]; b.A = a.A[0]; b.B = a.B[0]; b.U = a.U[0];
    b.dX = a.dX; b.dA = a.dA[0]; b.dB = a.dB[0]; b.ws = a.ws;
    b.m = a.m; b.n = a.n[0]; b.k = a.k; b.r = a.r; b.s = a.s;
    return launch_bwd(b, st);
  }
  const GroupBwdLayout GL = group_bwd_layout(a.count, a.n, a.m, a.k, a.r);
  const Plan p = plan_group_bwd(a.count, a.n, a.m, a.k, a.r);
  const int rp = GL.L[0].rp;
  u16* dut_stack = GL.stacked ? reinterpret_cast<u16*>(a.ws + GL.dut_stack) : nullptr;
  float* pa_stack = GL.stacked ? reinterpret_cast<float*>(a.ws + GL.pa_stack) : nullptr;
  DxGroup grp{};
  int nkb = 0;
  for (int g = 0; g < a.count; ++g) {
    const BwdArgs b = member_args(g, GL);
    grp.dY[g] = a.dY[g];
    grp.W[g] = a.W[g];
    grp.dU2[g] = reinterpret_cast<const u16*>(b.ws + GL.L[g].du2);
    grp.A[g] = a.A[g];
    grp.n[g] = (int)a.n[g];
    nkb += (int)((a.n[g] + 63) / 64);
    grp.fin[g] = finalize_args(b, GL.L[g]);
    if (GL.stacked) {   // member g's dA rows of the stacked reduction
      grp.fin[g].pa = pa_stack + (size_t)g * rp * a.k;
      grp.fin[g].rpa = GL.rpt;
      grp.fin[g].sa = GL.plan_a.splits;
    }
  }
  grp.count = a.count;
  grp.nkb = nkb;
  DxGroup rest = grp;   // later column ranges finalize nothing
  for (int g = 0; g < kMaxGroup; ++g) rest.fin[g] = FinalizeArgs{};
  BwdArgs d{};
  d.X = a.X; d.dX = a.dX; d.ws = a.ws;
  d.m = a.m; d.n = 0; d.k = a.k; d.r = a.r; d.s = a.s;
  for (int i = 0; i < p.count; ++i) {
    const Launch& L = p.l[i];
    hipError_t e = hipErrorInvalidValue;
    if (L.id == K_TOKRED && L.part == 2) {   // the stacked dA reduction over X
      const RedProblem pap{dut_stack, a.X, pa_stack, (int)a.k, (int)GL.plan_a.span, GL.plan_a.col_tiles, nullptr};
      const BwdArgs b = member_args(0, GL);
      e = with_int<32, 48, 64>(L.rp, [&](auto rc) {
        hipLaunchKernelGGL((lora_tokred_dma_kernel<decltype(rc)::value>), dim3((unsigned)L.grid),
                           dim3((unsigned)L.block), 0, st, pap, pap, (int)L.grid, (int)b.m, (int)GL.L[0].mp);
        return hipGetLastError();
      });
    } else if (L.id == K_DU) {
      const BwdArgs b = member_args(L.member, GL);
      e = GL.stacked ? run_du(L, b, GL.L[L.member], st, dut_stack + (size_t)L.member * rp * GL.L[0].mp)
                     : run_du(L, b, GL.L[L.member], st);
    } else if (L.id == K_TOKRED) {
      const BwdArgs b = member_args(L.member, GL);
      e = run_tokred(L, b, GL.L[L.member], st);
    } else if (L.id == K_DX) {
      e = run_dx(L, d, nullptr, (int)GL.L[0].mp, FinalizeArgs{}, L.finalize ? grp : rest, st);
    }
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

}  // namespace lora
