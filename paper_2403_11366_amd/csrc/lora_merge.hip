// Merge and unmerge of the LoRA adapter into the frozen weight.  Eq. 1 of
// JORA (Section 3) writes the adapted layer both as W0 x + B A x and as
// (W0 + B A) x; with the LoRA scale s = alpha / r the merged weight is
//   W_out = W + sign * s * B A        (sign = +1 merges, -1 unmerges),
// rounded once to bf16 (nearest-even) after fp32 accumulation.
//
// One kernel.  Each workgroup owns a 128 x 128 tile of W (rows j = output
// features, columns l = input features).  It stages the tile's A columns
// ([RP][128], mn-contiguous, read back transposed) and B rows ([128][RP],
// rank padded with zeros) in LDS, forms D^T = A^T B^T for the tile on the
// matrix cores (v_mfma_f32_32x32x16_bf16, K = RP), parks D in LDS, and then
// adds sign * s * D to W (loaded in coalesced 16-byte chunks at the start, so
// the load latency overlaps the product) and writes W_out in the same chunks.
// W_out may be W itself: every element is read and written by one thread, all
// of a thread's reads come before its writes, and W carries no no-alias
// qualifier.
// HBM traffic is one read and one write of W, so the kernel is HBM-bound.
#include "lora_device.hpp"
#include "lora_launch.hpp"
#include "lora_plan.hpp"

namespace lora {

template <int RP, int BJ>
__global__ __launch_bounds__(256) void lora_merge_kernel(const u16* W, const u16* __restrict__ A,
                                                         const u16* __restrict__ B, u16* Wout, int n, int k,
                                                         int r, float ss, int tiles_j, int tiles_l) {
  constexpr int BL = 128, NT = 256;
  constexpr int FJN = BJ / 32;                 // 32-row blocks of j per wave
  constexpr int BP = RP + 8;                   // Bs row pitch in elements (16-byte multiple)
  constexpr int DP = BL + 4;                   // Ds row pitch in floats
  constexpr int AS_BYTES = RP * BL * 2;
  constexpr int BS_BYTES = BJ * BP * 2;
  static_assert(AS_BYTES + BS_BYTES <= BJ * DP * 4, "Ds reuses the staging LDS");
  __shared__ __attribute__((aligned(1024))) char smem[BJ * DP * 4];
  char* As = smem;
  u16* Bs = reinterpret_cast<u16*>(smem + AS_BYTES);
  float* Ds = reinterpret_cast<float*>(smem);   // [BJ][DP]: D of the tile, after the products

  int tj, tl;
  tile_coords(tiles_j, tiles_l, 8, (int)blockIdx.x, tj, tl);
  const int j0 = tj * BJ, l0 = tl * BL;
  const int tid = threadIdx.x, lane = tid & 63, wave = uniform(tid >> 6);
  const int g = lane >> 5, c32 = lane & 31;
  const uint32_t wrow = (uint32_t)k * 2;

  // This thread's 16-byte chunks of the W tile (chunk q is row q / 16, columns
  // 8 (q % 16) ..), loaded first so their latency overlaps the product.
  constexpr int WCH = BJ * (BL / 8) / NT;     // BJ / 16 chunks per thread
  int4v wv[WCH];
#pragma unroll
  for (int i = 0; i < WCH; ++i) {
    const int q = tid + i * NT;
    const int jj = q >> 4, c = q & 15;
    const int j = j0 + jj, l = l0 + 8 * c;
    wv[i] = (j < n && l < k) ? *reinterpret_cast<const int4v*>(W + (size_t)j * k + l) : int4v{0, 0, 0, 0};
  }

  // A tile: rows t < r, columns l0 .. l0+127 (zero beyond r and k).
  constexpr int ACH = RP * (BL / 8);
  const __amdgpu_buffer_rsrc_t rsA = make_rsrc(A, (uint64_t)r * wrow);
#pragma unroll
  for (int i = 0; i < (ACH + NT - 1) / NT; ++i) {
    const int q = tid + i * NT;
    if (ACH % NT != 0 && q >= ACH) break;
    const int t = q / (BL / 8), c = q % (BL / 8);
    const int l = l0 + 8 * c;
    const int4v v = buf_load16(rsA, (t < r && l < k) ? (uint32_t)t * wrow + (uint32_t)l * 2 : kOOB);
    *reinterpret_cast<int4v*>(As + mc32_offset<BL>(t, c)) = v;
  }
  // B rows j0 .. j0+jn-1 are contiguous in B: fetch them as 16-byte chunks of
  // 8 elements and scatter into Bs[j][t] (columns t >= r stay zero).
  const int jn = min(BJ, n - j0);
  const int nch = jn * r / 8;                          // exact: n and j0 are multiples of 8
  constexpr int BCH = (BJ * RP / 8 + NT - 1) / NT;
  const __amdgpu_buffer_rsrc_t rsB = make_rsrc(B + (size_t)j0 * r, (uint64_t)nch * 16);
  int4v bv[BCH];
#pragma unroll
  for (int i = 0; i < BCH; ++i) {
    const int q = tid + i * NT;
    bv[i] = buf_load16(rsB, q < nch ? (uint32_t)q * 16 : kOOB);
  }
  for (int e = tid; e < BS_BYTES / 16; e += NT) reinterpret_cast<int4v*>(Bs)[e] = int4v{0, 0, 0, 0};
  __syncthreads();
  {
    const float rinv = 1.0f / (float)r;
#pragma unroll
    for (int i = 0; i < BCH; ++i) {
      const int q = tid + i * NT;
      if (q < nch) {
#pragma unroll
        for (int e = 0; e < 8; ++e) {   // quotient from a float product at least 0.5/r from an integer
          const int idx = 8 * q + e;
          const int jj = (int)(((float)idx + 0.5f) * rinv);
          Bs[jj * BP + idx - jj * r] = (u16)((uint32_t)bv[i][e >> 1] >> (16 * (e & 1)));
        }
      }
    }
  }
  __syncthreads();

  // D^T[l][j] = sum_t A[t][l] B[j][t]: wave w takes the 32 columns
  // l0 + 32w .. and all BJ / 32 row blocks of j.
  floatx16 acc[FJN];
#pragma unroll
  for (int fj = 0; fj < FJN; ++fj) acc[fj] = floatx16{};
#pragma unroll
  for (int kk = 0; kk < RP / 16; ++kk) {
    const short8 af = mc32_read_tr<BL>(As, 16 * kk, 32 * wave, lane);
#pragma unroll
    for (int fj = 0; fj < FJN; ++fj) {
      const short8 bf = *reinterpret_cast<const short8*>(Bs + (32 * fj + c32) * BP + 16 * kk + 8 * g);
      acc[fj] = mfma32x32x16(af, bf, acc[fj]);
    }
  }
  __syncthreads();   // staging LDS is reused for Ds
  // lane holds column j = 32 fj + c32, rows l = 32 w + 8(q/4) + 4g + q%4
#pragma unroll
  for (int fj = 0; fj < FJN; ++fj)
#pragma unroll
    for (int q = 0; q < 16; ++q) {
      const int l = 32 * wave + 8 * (q >> 2) + 4 * g + (q & 3);
      Ds[(32 * fj + c32) * DP + l] = acc[fj][q];
    }
  __syncthreads();

  // W_out = W + ss * D in 16-byte chunks: chunk q is row q / 16, columns 8 (q % 16) ..
#pragma unroll
  for (int i = 0; i < WCH; ++i) {
    const int q = tid + i * NT;
    const int jj = q >> 4, c = q & 15;
    const int j = j0 + jj, l = l0 + 8 * c;
    if (j < n && l < k) {
      const floatx4 da = *reinterpret_cast<const floatx4*>(Ds + jj * DP + 8 * c);
      const floatx4 db = *reinterpret_cast<const floatx4*>(Ds + jj * DP + 8 * c + 4);
      const float d[8] = {da[0], da[1], da[2], da[3], db[0], db[1], db[2], db[3]};
      int4v o;
#pragma unroll
      for (int h = 0; h < 4; ++h) {
        const uint32_t w2 = (uint32_t)wv[i][h];
        const float d0 = d[2 * h], d1 = d[2 * h + 1];
        const u16 o0 = f32_to_bf16(fmaf(ss, d0, bf16_to_f32((u16)(w2 & 0xFFFF))));
        const u16 o1 = f32_to_bf16(fmaf(ss, d1, bf16_to_f32((u16)(w2 >> 16))));
        o[h] = (int)((uint32_t)o0 | ((uint32_t)o1 << 16));
      }
      *reinterpret_cast<int4v*>(Wout + (size_t)j * k + l) = o;
    }
  }
}

hipError_t launch_merge(const MergeArgs& a, hipStream_t st) {
  const Plan p = plan_merge(a.n, a.k, a.r);
  const Launch& L = p.l[0];
  return with_int<16, 32, 48, 64>(L.rp, [&](auto rc) {
    hipLaunchKernelGGL((lora_merge_kernel<decltype(rc)::value, kMergeRows>), dim3((unsigned)L.grid),
                       dim3((unsigned)L.block), 0, st, a.W, a.A, a.B, a.Wout, (int)a.n, (int)a.k, (int)a.r, a.ss,
                       L.tiles_m, L.tiles_n);
    return hipGetLastError();
  });
}

}  // namespace lora
