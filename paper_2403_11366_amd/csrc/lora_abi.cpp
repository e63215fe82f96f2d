// C ABI of the LoRA-linear library: argument validation, workspace sizing and
// dispatch to the kernel launchers.  Every check runs before the first HIP
// call, so an invalid call launches nothing and leaves its outputs untouched.
#include <stdint.h>

#include <new>

#include "lora_linear.h"
#include "lora_launch.hpp"

namespace {

constexpr int64_t kMaxDim = int64_t(1) << 22;       // m, n, k each at most 4M
constexpr int64_t kMaxElems = int64_t(1) << 30;     // any one bf16 matrix at most 2 GiB

struct Range {
  uintptr_t lo, hi;  // [lo, hi)
};

inline Range span(const void* p, int64_t rows, int64_t cols, int64_t elem) {
  const uintptr_t a = reinterpret_cast<uintptr_t>(p);
  return Range{a, a + (uintptr_t)(rows * cols * elem)};
}

inline bool overlap(const Range& x, const Range& y) { return x.lo < y.hi && y.lo < x.hi; }

inline bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

lora_status check_shape(int64_t m, int64_t n, int64_t k, int64_t r) {
  if (m < 1 || n < 8 || k < 8 || r < 1) return LORA_ERR_SHAPE;
  if (n % 8 != 0 || k % 8 != 0) return LORA_ERR_SHAPE;
  if (r > 64) return LORA_ERR_UNSUPPORTED;
  if (m > kMaxDim || n > kMaxDim || k > kMaxDim) return LORA_ERR_UNSUPPORTED;
  if (m * k > kMaxElems || n * k > kMaxElems || m * n > kMaxElems) return LORA_ERR_UNSUPPORTED;
  return LORA_OK;
}

}  // namespace

extern "C" {

const char* lora_status_string(lora_status s) {
  switch (s) {
    case LORA_OK: return "ok";
    case LORA_ERR_NULL: return "null pointer argument";
    case LORA_ERR_SHAPE: return "invalid shape (need m >= 1, n and k >= 8 and multiples of 8, r >= 1; merge sign +1 or -1)";
    case LORA_ERR_ALIGN: return "matrix pointer not 16-byte aligned";
    case LORA_ERR_UNSUPPORTED: return "unsupported size (r > 64, a dimension > 2^22, or a matrix > 2^30 elements)";
    case LORA_ERR_WORKSPACE: return "workspace missing or too small";
    case LORA_ERR_ALIAS: return "an output overlaps an input or another output";
    case LORA_ERR_HIP: return "HIP runtime error at launch";
  }
  return "unknown status";
}

lora_status lora_linear_fwd(const lora_bf16* X, const lora_bf16* W, const lora_bf16* A,
                            const lora_bf16* B, lora_bf16* Y, float* U,
                            int64_t m, int64_t n, int64_t k, int64_t r, float alpha,
                            void* stream) {
  if (!X || !W || !A || !B || !Y || !U) return LORA_ERR_NULL;
  lora_status st = check_shape(m, n, k, r);
  if (st != LORA_OK) return st;
  if (!aligned16(X) || !aligned16(W) || !aligned16(A) || !aligned16(B) || !aligned16(Y) || !aligned16(U))
    return LORA_ERR_ALIGN;
  const Range in[4] = {span(X, m, k, 2), span(W, n, k, 2), span(A, r, k, 2), span(B, n, r, 2)};
  const Range ry = span(Y, m, n, 2), ru = span(U, m, r, 4);
  for (const Range& x : in)
    if (overlap(ry, x) || overlap(ru, x)) return LORA_ERR_ALIAS;
  if (overlap(ry, ru)) return LORA_ERR_ALIAS;

  lora::FwdArgs a{X, W, A, B, Y, U, m, n, k, r, (float)alpha / (float)r};
  hipError_t e = lora::launch_fwd(a, reinterpret_cast<hipStream_t>(stream));
  return e == hipSuccess ? LORA_OK : LORA_ERR_HIP;
}

lora_status lora_linear_fwd_dropout(const lora_bf16* X, const lora_bf16* W, const lora_bf16* A,
                                    const lora_bf16* B, const uint8_t* keep, float p, lora_bf16* Y, float* U,
                                    int64_t m, int64_t n, int64_t k, int64_t r, float alpha, void* stream) {
  if (!X || !W || !A || !B || !keep || !Y || !U) return LORA_ERR_NULL;
  lora_status st = check_shape(m, n, k, r);
  if (st != LORA_OK) return st;
  if (k % 64 != 0 || !(p >= 0.0f && p < 1.0f)) return LORA_ERR_SHAPE;
  if (!aligned16(X) || !aligned16(W) || !aligned16(A) || !aligned16(B) || !aligned16(keep) || !aligned16(Y) ||
      !aligned16(U))
    return LORA_ERR_ALIGN;
  const Range in[5] = {span(X, m, k, 2), span(W, n, k, 2), span(A, r, k, 2), span(B, n, r, 2),
                       span(keep, m, k / 8, 1)};
  const Range ry = span(Y, m, n, 2), ru = span(U, m, r, 4);
  for (const Range& x : in)
    if (overlap(ry, x) || overlap(ru, x)) return LORA_ERR_ALIAS;
  if (overlap(ry, ru)) return LORA_ERR_ALIAS;

  lora::FwdArgs a{X, W, A, B, Y, U, m, n, k, r, (float)alpha / (float)r, keep, 1.0f / (1.0f - p)};
  hipError_t e = lora::launch_fwd(a, reinterpret_cast<hipStream_t>(stream));
  return e == hipSuccess ? LORA_OK : LORA_ERR_HIP;
}

size_t lora_linear_bwd_workspace_size(int64_t m, int64_t n, int64_t k, int64_t r) {
  if (check_shape(m, n, k, r) != LORA_OK) return 0;
  return lora::bwd_layout(m, n, k, r).total;
}

lora_status lora_linear_bwd(const lora_bf16* dY, const lora_bf16* X, const lora_bf16* W,
                            const lora_bf16* A, const lora_bf16* B, const float* U,
                            lora_bf16* dX, float* dA, float* dB,
                            void* workspace, size_t workspace_bytes,
                            int64_t m, int64_t n, int64_t k, int64_t r, float alpha,
                            void* stream) {
  if (!dY || !X || !W || !A || !B || !U || !dX || !dA || !dB) return LORA_ERR_NULL;
  lora_status st = check_shape(m, n, k, r);
  if (st != LORA_OK) return st;
  if (!aligned16(dY) || !aligned16(X) || !aligned16(W) || !aligned16(A) || !aligned16(B) ||
      !aligned16(U) || !aligned16(dX) || !aligned16(dA) || !aligned16(dB))
    return LORA_ERR_ALIGN;
  const size_t need = lora::bwd_layout(m, n, k, r).total;
  if (!workspace || workspace_bytes < need) return LORA_ERR_WORKSPACE;
  if (!aligned16(workspace)) return LORA_ERR_ALIGN;

  const Range in[6] = {span(dY, m, n, 2), span(X, m, k, 2), span(W, n, k, 2),
                       span(A, r, k, 2),  span(B, n, r, 2), span(U, m, r, 4)};
  const Range out[4] = {span(dX, m, k, 2), span(dA, r, k, 4), span(dB, n, r, 4),
                        Range{reinterpret_cast<uintptr_t>(workspace),
                              reinterpret_cast<uintptr_t>(workspace) + need}};
  for (int i = 0; i < 4; ++i) {
    for (const Range& x : in)
      if (overlap(out[i], x)) return LORA_ERR_ALIAS;
    for (int j = i + 1; j < 4; ++j)
      if (overlap(out[i], out[j])) return LORA_ERR_ALIAS;
  }

  lora::BwdArgs a{dY, X, W, A, B, U, dX, dA, dB, static_cast<char*>(workspace),
                  m, n, k, r, (float)alpha / (float)r};
  hipError_t e = lora::launch_bwd(a, reinterpret_cast<hipStream_t>(stream));
  return e == hipSuccess ? LORA_OK : LORA_ERR_HIP;
}

lora_status lora_linear_bwd_dropout(const lora_bf16* dY, const lora_bf16* X, const lora_bf16* W,
                                    const lora_bf16* A, const lora_bf16* B, const float* U, const uint8_t* keep,
                                    float p, lora_bf16* dX, float* dA, float* dB, void* workspace,
                                    size_t workspace_bytes, int64_t m, int64_t n, int64_t k, int64_t r, float alpha,
                                    void* stream) {
  if (!dY || !X || !W || !A || !B || !U || !keep || !dX || !dA || !dB) return LORA_ERR_NULL;
  lora_status st = check_shape(m, n, k, r);
  if (st != LORA_OK) return st;
  if (k % 64 != 0 || !(p >= 0.0f && p < 1.0f)) return LORA_ERR_SHAPE;
  if (!aligned16(dY) || !aligned16(X) || !aligned16(W) || !aligned16(A) || !aligned16(B) ||
      !aligned16(U) || !aligned16(keep) || !aligned16(dX) || !aligned16(dA) || !aligned16(dB))
    return LORA_ERR_ALIGN;
  const size_t need = lora::bwd_layout(m, n, k, r).total;
  if (!workspace || workspace_bytes < need) return LORA_ERR_WORKSPACE;
  if (!aligned16(workspace)) return LORA_ERR_ALIGN;

  const Range in[7] = {span(dY, m, n, 2), span(X, m, k, 2), span(W, n, k, 2), span(A, r, k, 2),
                       span(B, n, r, 2),  span(U, m, r, 4), span(keep, m, k / 8, 1)};
  const Range out[4] = {span(dX, m, k, 2), span(dA, r, k, 4), span(dB, n, r, 4),
                        Range{reinterpret_cast<uintptr_t>(workspace),
                              reinterpret_cast<uintptr_t>(workspace) + need}};
  for (int i = 0; i < 4; ++i) {
    for (const Range& x : in)
      if (overlap(out[i], x)) return LORA_ERR_ALIAS;
    for (int j = i + 1; j < 4; ++j)
      if (overlap(out[i], out[j])) return LORA_ERR_ALIAS;
  }

  lora::BwdArgs a{dY, X, W, A, B, U, dX, dA, dB, static_cast<char*>(workspace),
                  m, n, k, r, (float)alpha / (float)r, keep, 1.0f / (1.0f - p)};
  hipError_t e = lora::launch_bwd(a, reinterpret_cast<hipStream_t>(stream));
  return e == hipSuccess ? LORA_OK : LORA_ERR_HIP;
}

lora_status lora_linear_merge(const lora_bf16* W, const lora_bf16* A, const lora_bf16* B, lora_bf16* W_out,
                              int64_t n, int64_t k, int64_t r, float alpha, int sign, void* stream) {
  if (!W || !A || !B || !W_out) return LORA_ERR_NULL;
  lora_status st = check_shape(1, n, k, r);
  if (st != LORA_OK) return st;
  if (sign != 1 && sign != -1) return LORA_ERR_SHAPE;
  if (!aligned16(W) || !aligned16(A) || !aligned16(B) || !aligned16(W_out)) return LORA_ERR_ALIGN;
  const Range rw = span(W, n, k, 2), ro = span(W_out, n, k, 2);
  if (overlap(ro, span(A, r, k, 2)) || overlap(ro, span(B, n, r, 2))) return LORA_ERR_ALIAS;
  if (overlap(ro, rw) && W_out != W) return LORA_ERR_ALIAS;   // in place is allowed, a shifted overlap is not

  lora::MergeArgs a{W, A, B, W_out, n, k, r, (float)sign * ((float)alpha / (float)r)};
  hipError_t e = lora::launch_merge(a, reinterpret_cast<hipStream_t>(stream));
  return e == hipSuccess ? LORA_OK : LORA_ERR_HIP;
}

}  // extern "C"
