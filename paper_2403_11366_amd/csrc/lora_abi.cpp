// C ABI of the LoRA-linear library: argument validation, workspace sizing and
// dispatch to the kernel launchers.  Every check runs before the first HIP
// call, so an invalid call launches nothing and leaves its outputs untouched.
#include <cmath>
#include <stdint.h>
#include <string.h>

#include <new>

#include "lora_linear.h"
#include "lora_launch.hpp"
#include "lora_plan.hpp"

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

// True if any output range overlaps an input range or another output range.
bool any_alias(const Range* out, int n_out, const Range* in, int n_in) {
  for (int i = 0; i < n_out; ++i) {
    for (int j = 0; j < n_in; ++j)
      if (overlap(out[i], in[j])) return true;
    for (int j = i + 1; j < n_out; ++j)
      if (overlap(out[i], out[j])) return true;
  }
  return false;
}

// Shape checks of a group of projections sharing X: the count, the host
// array of output widths and each projection's shape.
lora_status check_group(int64_t group, const int64_t* n, int64_t m, int64_t k, int64_t r) {
  if (!n) return LORA_ERR_NULL;
  if (group < 1) return LORA_ERR_SHAPE;
  if (group > lora::kMaxGroup) return LORA_ERR_UNSUPPORTED;
  int64_t total = 0;
  for (int64_t g = 0; g < group; ++g) {
    const lora_status st = check_shape(m, n[g], k, r);
    if (st != LORA_OK) return st;
    total += n[g];
  }
  if (total > kMaxDim) return LORA_ERR_UNSUPPORTED;
  return LORA_OK;
}

template <typename T>
bool all_set(const T* const* p, int64_t group) {
  if (!p) return false;
  for (int64_t g = 0; g < group; ++g)
    if (!p[g]) return false;
  return true;
}

template <typename T>
bool all_aligned(const T* const* p, int64_t group) {
  for (int64_t g = 0; g < group; ++g)
    if (!aligned16(p[g])) return false;
  return true;
}

}  // namespace

extern "C" {

const char* lora_status_string(lora_status s) {
  // A C caller may pass any int.  Its bits are read as an int: in C++, loading
  // a lora_status object that holds a value past the enumerators is undefined.
  static_assert(sizeof(lora_status) == sizeof(int), "lora_status is int-sized");
  int code;
  memcpy(&code, &s, sizeof code);
  switch (code) {
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

// HIP keeps the last runtime error of the calling thread until it is read,
// and the launchers read it after each launch.  An error left pending by an
// earlier call would be reported by a call's first launch after that kernel
// was enqueued, so it is reported before anything is enqueued instead (and
// left pending for the caller to read).
static bool hip_error_pending() { return hipPeekAtLastError() != hipSuccess; }

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
  if (hip_error_pending()) return LORA_ERR_HIP;
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
  if (hip_error_pending()) return LORA_ERR_HIP;
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
  if (hip_error_pending()) return LORA_ERR_HIP;
  hipError_t e = lora::launch_bwd(a, reinterpret_cast<hipStream_t>(stream));
  return e == hipSuccess ? LORA_OK : LORA_ERR_HIP;
}

lora_status lora_linear_bwd_noalloc(const lora_bf16* dY, const lora_bf16* X, const lora_bf16* W,
                                    const lora_bf16* A, const lora_bf16* B, const float* U,
                                    lora_bf16* dX, float* dA, float* dB,
                                    int64_t m, int64_t n, int64_t k, int64_t r, float alpha, void* stream) {
  if (!dY || !X || !W || !A || !B || !U || !dX || !dA || !dB) return LORA_ERR_NULL;
  lora_status st = check_shape(m, n, k, r);
  if (st != LORA_OK) return st;
  if (!aligned16(dY) || !aligned16(X) || !aligned16(W) || !aligned16(A) || !aligned16(B) ||
      !aligned16(U) || !aligned16(dX) || !aligned16(dA) || !aligned16(dB))
    return LORA_ERR_ALIGN;
  if (lora::bwd_layout(m, n, k, r).total > lora::kNoAllocScratchBytes) return LORA_ERR_WORKSPACE;
  const Range in[6] = {span(dY, m, n, 2), span(X, m, k, 2), span(W, n, k, 2),
                       span(A, r, k, 2),  span(B, n, r, 2), span(U, m, r, 4)};
  const Range out[3] = {span(dX, m, k, 2), span(dA, r, k, 4), span(dB, n, r, 4)};
  if (any_alias(out, 3, in, 6)) return LORA_ERR_ALIAS;

  lora::BwdArgs a{dY, X, W, A, B, U, dX, dA, dB, nullptr, m, n, k, r, (float)alpha / (float)r};
  if (hip_error_pending()) return LORA_ERR_HIP;
  hipError_t e = lora::launch_bwd_noalloc(a, reinterpret_cast<hipStream_t>(stream));
  return e == hipSuccess ? LORA_OK : LORA_ERR_HIP;
}

size_t lora_linear_bwd_fused_workspace_size(int64_t m, int64_t n, int64_t k, int64_t r) {
  if (check_shape(m, n, k, r) != LORA_OK || r > 16) return 0;
  return lora::bwd_fused_layout(m, n, k, r).total;
}

lora_status lora_linear_bwd_fused(const lora_bf16* dY, const lora_bf16* X, const lora_bf16* W,
                                  const lora_bf16* A, const lora_bf16* B, const float* U,
                                  lora_bf16* dX, float* dA, float* dB,
                                  void* workspace, size_t workspace_bytes,
                                  int64_t m, int64_t n, int64_t k, int64_t r, float alpha,
                                  void* stream) {
  if (!dY || !X || !W || !A || !B || !U || !dX || !dA || !dB) return LORA_ERR_NULL;
  lora_status st = check_shape(m, n, k, r);
  if (st != LORA_OK) return st;
  if (r > 16) return LORA_ERR_UNSUPPORTED;
  if (!aligned16(dY) || !aligned16(X) || !aligned16(W) || !aligned16(A) || !aligned16(B) ||
      !aligned16(U) || !aligned16(dX) || !aligned16(dA) || !aligned16(dB))
    return LORA_ERR_ALIGN;
  const size_t need = lora::bwd_fused_layout(m, n, k, r).total;
  if (!workspace || workspace_bytes < need) return LORA_ERR_WORKSPACE;
  if (!aligned16(workspace)) return LORA_ERR_ALIGN;

  const Range in[6] = {span(dY, m, n, 2), span(X, m, k, 2), span(W, n, k, 2),
                       span(A, r, k, 2),  span(B, n, r, 2), span(U, m, r, 4)};
  const Range out[4] = {span(dX, m, k, 2), span(dA, r, k, 4), span(dB, n, r, 4),
                        Range{reinterpret_cast<uintptr_t>(workspace),
                              reinterpret_cast<uintptr_t>(workspace) + need}};
  if (any_alias(out, 4, in, 6)) return LORA_ERR_ALIAS;

  lora::BwdArgs a{dY, X, W, A, B, U, dX, dA, dB, static_cast<char*>(workspace),
                  m, n, k, r, (float)alpha / (float)r};
  if (hip_error_pending()) return LORA_ERR_HIP;
  hipError_t e = lora::launch_bwd_fused(a, reinterpret_cast<hipStream_t>(stream));
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
  if (hip_error_pending()) return LORA_ERR_HIP;
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
  if (hip_error_pending()) return LORA_ERR_HIP;
  hipError_t e = lora::launch_merge(a, reinterpret_cast<hipStream_t>(stream));
  return e == hipSuccess ? LORA_OK : LORA_ERR_HIP;
}

lora_status lora_linear_group_fwd(const lora_bf16* X, int64_t group, const int64_t* n,
                                  const lora_bf16* const* W, const lora_bf16* const* A,
                                  const lora_bf16* const* B, lora_bf16* const* Y, float* const* U,
                                  int64_t m, int64_t k, int64_t r, float alpha, void* stream) {
  if (!X || !n) return LORA_ERR_NULL;
  lora_status st = check_group(group, n, m, k, r);
  if (st != LORA_OK) return st;
  if (!all_set(W, group) || !all_set(A, group) || !all_set(B, group) || !all_set(Y, group) || !all_set(U, group))
    return LORA_ERR_NULL;
  if (!aligned16(X) || !all_aligned(W, group) || !all_aligned(A, group) || !all_aligned(B, group) ||
      !all_aligned(Y, group) || !all_aligned(U, group))
    return LORA_ERR_ALIGN;
  Range in[1 + 3 * lora::kMaxGroup], out[2 * lora::kMaxGroup];
  int ni = 0, no = 0;
  in[ni++] = span(X, m, k, 2);
  for (int64_t g = 0; g < group; ++g) {
    in[ni++] = span(W[g], n[g], k, 2);
    in[ni++] = span(A[g], r, k, 2);
    in[ni++] = span(B[g], n[g], r, 2);
    out[no++] = span(Y[g], m, n[g], 2);
    out[no++] = span(U[g], m, r, 4);
  }
  if (any_alias(out, no, in, ni)) return LORA_ERR_ALIAS;

  lora::GroupFwdArgs a{};
  a.X = X;
  a.count = (int)group;
  for (int64_t g = 0; g < group; ++g) {
    a.n[g] = n[g]; a.W[g] = W[g]; a.A[g] = A[g]; a.B[g] = B[g]; a.Y[g] = Y[g]; a.U[g] = U[g];
  }
  a.m = m; a.k = k; a.r = r; a.s = (float)alpha / (float)r;
  if (hip_error_pending()) return LORA_ERR_HIP;
  hipError_t e = lora::launch_fwd_group(a, reinterpret_cast<hipStream_t>(stream));
  return e == hipSuccess ? LORA_OK : LORA_ERR_HIP;
}

size_t lora_linear_group_bwd_workspace_size(int64_t group, const int64_t* n, int64_t m, int64_t k, int64_t r) {
  if (check_group(group, n, m, k, r) != LORA_OK) return 0;
  return lora::group_bwd_layout((int)group, n, m, k, r).total;
}

lora_status lora_linear_group_bwd(const lora_bf16* const* dY, const lora_bf16* X, int64_t group, const int64_t* n,
                                  const lora_bf16* const* W, const lora_bf16* const* A,
                                  const lora_bf16* const* B, const float* const* U, lora_bf16* dX,
                                  float* const* dA, float* const* dB, void* workspace, size_t workspace_bytes,
                                  int64_t m, int64_t k, int64_t r, float alpha, void* stream) {
  if (!X || !n || !dX) return LORA_ERR_NULL;
  lora_status st = check_group(group, n, m, k, r);
  if (st != LORA_OK) return st;
  if (!all_set(dY, group) || !all_set(W, group) || !all_set(A, group) || !all_set(B, group) ||
      !all_set(U, group) || !all_set(dA, group) || !all_set(dB, group))
    return LORA_ERR_NULL;
  if (!aligned16(X) || !aligned16(dX) || !all_aligned(dY, group) || !all_aligned(W, group) ||
      !all_aligned(A, group) || !all_aligned(B, group) || !all_aligned(U, group) || !all_aligned(dA, group) ||
      !all_aligned(dB, group))
    return LORA_ERR_ALIGN;
  const size_t need = lora::group_bwd_layout((int)group, n, m, k, r).total;
  if (!workspace || workspace_bytes < need) return LORA_ERR_WORKSPACE;
  if (!aligned16(workspace)) return LORA_ERR_ALIGN;

  Range in[1 + 5 * lora::kMaxGroup], out[2 + 2 * lora::kMaxGroup];
  int ni = 0, no = 0;
  in[ni++] = span(X, m, k, 2);
  out[no++] = span(dX, m, k, 2);
  out[no++] = Range{reinterpret_cast<uintptr_t>(workspace), reinterpret_cast<uintptr_t>(workspace) + need};
  for (int64_t g = 0; g < group; ++g) {
    in[ni++] = span(dY[g], m, n[g], 2);
    in[ni++] = span(W[g], n[g], k, 2);
    in[ni++] = span(A[g], r, k, 2);
    in[ni++] = span(B[g], n[g], r, 2);
    in[ni++] = span(U[g], m, r, 4);
    out[no++] = span(dA[g], r, k, 4);
    out[no++] = span(dB[g], n[g], r, 4);
  }
  if (any_alias(out, no, in, ni)) return LORA_ERR_ALIAS;

  lora::GroupBwdArgs a{};
  a.X = X;
  a.count = (int)group;
  for (int64_t g = 0; g < group; ++g) {
    a.n[g] = n[g]; a.dY[g] = dY[g]; a.W[g] = W[g]; a.A[g] = A[g]; a.B[g] = B[g]; a.U[g] = U[g];
    a.dA[g] = dA[g]; a.dB[g] = dB[g];
  }
  a.dX = dX;
  a.ws = static_cast<char*>(workspace);
  a.m = m; a.k = k; a.r = r; a.s = (float)alpha / (float)r;
  if (hip_error_pending()) return LORA_ERR_HIP;
  hipError_t e = lora::launch_bwd_group(a, reinterpret_cast<hipStream_t>(stream));
  return e == hipSuccess ? LORA_OK : LORA_ERR_HIP;
}

lora_status lora_dropout_keep_mask(uint64_t seed, uint64_t offset, float p, uint8_t* keep, int64_t m, int64_t k,
                                   void* stream) {
  if (!keep) return LORA_ERR_NULL;
  lora_status st = check_shape(m, 8, k, 1);
  if (st != LORA_OK) return st;
  if (!(p >= 0.0f && p < 1.0f)) return LORA_ERR_SHAPE;
  if (!aligned16(keep)) return LORA_ERR_ALIGN;
  lora::MaskArgs a{seed, offset, (uint32_t)std::floor((1.0 - (double)p) * 65536.0 + 0.5), keep, m, k};
  if (hip_error_pending()) return LORA_ERR_HIP;
  hipError_t e = lora::launch_keep_mask(a, reinterpret_cast<hipStream_t>(stream));
  return e == hipSuccess ? LORA_OK : LORA_ERR_HIP;
}

int64_t lora_linear_plan(lora_op op, int64_t group, const int64_t* n, int64_t m, int64_t k, int64_t r,
                         lora_launch_info* out, int64_t capacity) {
  if (!n || (capacity > 0 && !out)) return -(int64_t)LORA_ERR_NULL;
  lora_status st = LORA_OK;
  lora::Plan p;
  switch (op) {
    case LORA_OP_FWD:
    case LORA_OP_FWD_DROPOUT:
    case LORA_OP_BWD:
    case LORA_OP_BWD_DROPOUT:
    case LORA_OP_BWD_FUSED: {
      if (group != 1) return -(int64_t)LORA_ERR_SHAPE;
      st = check_shape(m, n[0], k, r);
      const bool drop = op == LORA_OP_FWD_DROPOUT || op == LORA_OP_BWD_DROPOUT;
      if (st == LORA_OK && drop && k % 64 != 0) st = LORA_ERR_SHAPE;
      if (st == LORA_OK && op == LORA_OP_BWD_FUSED && r > 16) st = LORA_ERR_UNSUPPORTED;
      if (st != LORA_OK) break;
      if (op == LORA_OP_FWD || op == LORA_OP_FWD_DROPOUT) p = lora::plan_fwd(m, n[0], k, r, drop);
      else if (op == LORA_OP_BWD_FUSED) p = lora::plan_bwd_fused(m, n[0], k, r);
      else p = lora::plan_bwd(m, n[0], k, r, drop);
      break;
    }
    case LORA_OP_MERGE:
      if (group != 1) return -(int64_t)LORA_ERR_SHAPE;
      st = check_shape(1, n[0], k, r);
      if (st == LORA_OK) p = lora::plan_merge(n[0], k, r);
      break;
    case LORA_OP_KEEP_MASK:
      st = check_shape(m, 8, k, 1);
      if (st == LORA_OK) p = lora::plan_keep_mask(m, k);
      break;
    case LORA_OP_GROUP_FWD:
    case LORA_OP_GROUP_BWD:
      st = check_group(group, n, m, k, r);
      if (st != LORA_OK) break;
      p = op == LORA_OP_GROUP_FWD ? lora::plan_group_fwd((int)group, n, m, k, r)
                                  : lora::plan_group_bwd((int)group, n, m, k, r);
      break;
    default: return -(int64_t)LORA_ERR_SHAPE;
  }
  if (st != LORA_OK) return -(int64_t)st;
  for (int i = 0; i < p.count && i < capacity; ++i) {
    const lora::Launch& L = p.l[i];
    lora_launch_info& o = out[i];
    lora::launch_name(L, o.kernel, sizeof(o.kernel));
    o.grid = L.grid;
    o.block = L.block;
    o.tile_m = L.bm;
    o.tile_n = L.bn;
    o.member = L.member;
    o.col_begin = L.col_begin;
    o.col_end = L.col_end;
  }
  return p.count;
}

}  // extern "C"
