// Keep mask of LoRA dropout (the configuration of Listing 3 carries
// LORA_DROPOUT) drawn on the device from a counter-based generator, in the
// packed layout the *_dropout entry points read: byte (i, q) of keep [m][k/8]
// holds the keep bits of elements 8q .. 8q + 7 of row i of X.
//
// Generator: Philox4x64-10 (Salmon, Moraes, Dror and Shaw, "Parallel random
// numbers: as easy as 1, 2, 3", SC 2011).  A 256-bit counter (c0, c1, c2, c3)
// and a 128-bit key (k0, k1) go through ten rounds; each round multiplies c0
// and c2 by the two round constants into 128-bit products (hi, lo) and forms
//   (c0, c1, c2, c3) <- (hi(M1 c2) ^ c1 ^ k0, lo(M1 c2), hi(M0 c0) ^ c3 ^ k1, lo(M0 c0)),
// and between rounds the key is advanced by the two Weyl constants.
//
// Bytes 2t and 2t + 1 of the call's mask (byte b = i (k/8) + q holds the
// bits of elements 8q .. 8q + 7 of row i) come from one block: counter =
// offset + t as a 128-bit integer in (c0, c1), c2 = c3 = 0; key = (seed, 0).
// Its four output words split into sixteen 16-bit values u_e (u_{4h+j} = bits
// 16j .. 16j + 15 of word h); bit e of the byte pair (byte 2t: e = 0..7, byte
// 2t + 1: e = 8..15) is set, i.e. the element kept, iff u_e < T with
// T = floor((1 - p) 2^16 + 1/2), so an element is kept with probability
// T / 2^16 (exactly 1 for p = 0).  A call uses the counters offset ..
// offset + ceil(m k / 16) - 1; successive masks of one seed take disjoint
// ranges.
//
// One thread makes 4 bytes (2 blocks, one 4-byte store), so that enough
// waves run to hide the latency of the multiply chains.  The kernel only
// writes m k / 8 bytes; its cost is the generator arithmetic (64-bit
// multiplies, each from four 32 x 32 products), half of it saved by drawing
// 16 bits per element.
#include "lora_device.hpp"
#include "lora_launch.hpp"
#include "lora_plan.hpp"

namespace lora {

// The 128-bit product of two 64-bit words from four 32 x 32 -> 64 products,
// each with a 32-bit addend (v_mad_u64_u32), none of which can overflow:
// the low word is lo32(a_l b_l) + 2^32 lo32(v), the high word
// a_h b_h + hi32(u) + hi32(v), with u = a_l b_h + hi32(a_l b_l) and
// v = a_h b_l + lo32(u).
__device__ __forceinline__ void mulhilo64(uint64_t a, uint64_t b, uint64_t& hi, uint64_t& lo) {
  const uint32_t al = (uint32_t)a, ah = (uint32_t)(a >> 32), bl = (uint32_t)b, bh = (uint32_t)(b >> 32);
  const uint64_t t = (uint64_t)al * bl;
  const uint64_t u = (uint64_t)al * bh + (t >> 32);
  const uint64_t v = (uint64_t)ah * bl + (uint32_t)u;
  lo = (uint32_t)t | (v << 32);
  hi = (uint64_t)ah * bh + (u >> 32) + (v >> 32);
}

__device__ __forceinline__ void philox4x64_10(uint64_t (&c)[4], uint64_t k0, uint64_t k1) {
  constexpr uint64_t M0 = 0xD2E7470EE14C6C93ull, M1 = 0xCA5A826395121157ull;   // round multipliers
  constexpr uint64_t W0 = 0x9E3779B97F4A7C15ull, W1 = 0xBB67AE8584CAA73Bull;   // key increments
#pragma unroll
  for (int rnd = 0; rnd < 10; ++rnd) {
    uint64_t hi0, lo0, hi1, lo1;
    mulhilo64(M0, c[0], hi0, lo0);
    mulhilo64(M1, c[2], hi1, lo1);
    const uint64_t n0 = hi1 ^ c[1] ^ k0, n2 = hi0 ^ c[3] ^ k1;
    c[0] = n0;
    c[1] = lo1;
    c[2] = n2;
    c[3] = lo0;
    k0 += W0;
    k1 += W1;
  }
}

__global__ __launch_bounds__(256) void lora_keep_mask_kernel(uint64_t seed, uint64_t offset, uint32_t thr,
                                                             uint8_t* __restrict__ keep, int64_t nbytes) {
  const int64_t b0 = ((int64_t)blockIdx.x * 256 + threadIdx.x) * kMaskBytesPerThread;   // even
  if (b0 >= nbytes) return;
  const int nb = (int)min((int64_t)kMaskBytesPerThread, nbytes - b0);
  uint32_t w = 0u;
#pragma unroll
  for (int q = 0; q < kMaskBytesPerThread / 2; ++q) {   // block t = b0 / 2 + q: bytes b0 + 2q, b0 + 2q + 1
    if (2 * q < nb) {
      const uint64_t ctr = offset + (uint64_t)(b0 / 2 + q);
      uint64_t c[4] = {ctr, ctr < offset ? 1ull : 0ull, 0ull, 0ull};   // offset + t as a 128-bit counter
      philox4x64_10(c, seed, 0ull);
      uint32_t pair = 0;
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        const uint32_t u = (uint32_t)(c[e >> 2] >> (16 * (e & 3))) & 0xFFFFu;
        pair |= (u < thr ? 1u : 0u) << e;
      }
      w |= pair << (16 * q);
    }
  }
  static_assert(kMaskBytesPerThread == 2 || kMaskBytesPerThread == 4, "one 2- or 4-byte store");
  if (nb == kMaskBytesPerThread) {
    if constexpr (kMaskBytesPerThread == 4) *reinterpret_cast<uint32_t*>(keep + b0) = w;
    else *reinterpret_cast<uint16_t*>(keep + b0) = (uint16_t)w;
  } else {
    for (int q = 0; q < nb; ++q) keep[b0 + q] = (uint8_t)(w >> (8 * q));
  }
}

hipError_t launch_keep_mask(const MaskArgs& a, hipStream_t st) {
  const Plan p = plan_keep_mask(a.m, a.k);
  const Launch& L = p.l[0];
  hipLaunchKernelGGL(lora_keep_mask_kernel, dim3((unsigned)L.grid), dim3((unsigned)L.block), 0, st, a.seed,
                     a.offset, a.thr, a.keep, a.m * (a.k / 8));
  return hipGetLastError();
}

}  // namespace lora
