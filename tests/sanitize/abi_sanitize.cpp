// Memory- and UB-checking driver for the C-ABI layer (argument validation,
// workspace sizing and launch planning), built with
// -fsanitize=address,undefined on the host by tests/test_sanitizers.py.  It
// runs without a GPU: every entry-point call below is invalid and must be
// rejected, with the expected status, before any HIP call; the plan query and
// the workspace sizes are host-only and are swept over many shapes.  Device
// pointers are fake, 16-byte aligned addresses that validation never reads;
// host arrays (the group's widths and pointer tables) are real.
#include <stdint.h>
#include <stdio.h>
#include <string.h>

#include <vector>

#include "lora_linear.h"

extern "C" const char* status_text(int code);   // status_codes.c: the call made from C

static int failures = 0;

#define EXPECT(call, want)                                                                      \
  do {                                                                                          \
    const long got_ = (long)(call);                                                             \
    if (got_ != (long)(want)) {                                                                 \
      fprintf(stderr, "line %d: %s returned %ld, expected %ld\n", __LINE__, #call, got_, (long)(want)); \
      ++failures;                                                                               \
    }                                                                                           \
  } while (0)

template <typename T = lora_bf16>
static T* dev(int i, uintptr_t off = 0) {   // fake device address i (4 GiB apart)
  return reinterpret_cast<T*>((uintptr_t(1) << 40) + uintptr_t(i) * (uintptr_t(1) << 32) + off);
}

static void single_projection() {
  const int64_t m = 64, n = 64, k = 64, r = 8;
  const size_t ws = lora_linear_bwd_workspace_size(m, n, k, r);
  if (ws == 0) { fprintf(stderr, "zero workspace size\n"); ++failures; }
  // forward: each pointer missing, bad shapes, misaligned, aliasing
  EXPECT(lora_linear_fwd(nullptr, dev(1), dev(2), dev(3), dev(4), dev<float>(5), m, n, k, r, 16.f, nullptr), LORA_ERR_NULL);
  EXPECT(lora_linear_fwd(dev(0), dev(1), dev(2), dev(3), dev(4), nullptr, m, n, k, r, 16.f, nullptr), LORA_ERR_NULL);
  EXPECT(lora_linear_fwd(dev(0), dev(1), dev(2), dev(3), dev(4), dev<float>(5), 0, n, k, r, 16.f, nullptr), LORA_ERR_SHAPE);
  EXPECT(lora_linear_fwd(dev(0), dev(1), dev(2), dev(3), dev(4), dev<float>(5), m, 60, k, r, 16.f, nullptr), LORA_ERR_SHAPE);
  EXPECT(lora_linear_fwd(dev(0), dev(1), dev(2), dev(3), dev(4), dev<float>(5), m, n, 12, r, 16.f, nullptr), LORA_ERR_SHAPE);
  EXPECT(lora_linear_fwd(dev(0), dev(1), dev(2), dev(3), dev(4), dev<float>(5), m, n, k, 65, 16.f, nullptr), LORA_ERR_UNSUPPORTED);
  EXPECT(lora_linear_fwd(dev(0), dev(1), dev(2), dev(3), dev(4), dev<float>(5), int64_t(1) << 23, n, k, r, 16.f, nullptr), LORA_ERR_UNSUPPORTED);
  EXPECT(lora_linear_fwd(dev(0, 2), dev(1), dev(2), dev(3), dev(4), dev<float>(5), m, n, k, r, 16.f, nullptr), LORA_ERR_ALIGN);
  EXPECT(lora_linear_fwd(dev(0), dev(1), dev(2), dev(3), dev(0, 64), dev<float>(5), m, n, k, r, 16.f, nullptr), LORA_ERR_ALIAS);
  // forward with dropout: rate and k rules, missing mask
  EXPECT(lora_linear_fwd_dropout(dev(0), dev(1), dev(2), dev(3), dev<uint8_t>(6), -0.1f, dev(4), dev<float>(5), m, n, k, r, 16.f, nullptr), LORA_ERR_SHAPE);
  EXPECT(lora_linear_fwd_dropout(dev(0), dev(1), dev(2), dev(3), dev<uint8_t>(6), 1.0f, dev(4), dev<float>(5), m, n, k, r, 16.f, nullptr), LORA_ERR_SHAPE);
  EXPECT(lora_linear_fwd_dropout(dev(0), dev(1), dev(2), dev(3), dev<uint8_t>(6), 0.05f, dev(4), dev<float>(5), m, n, 72, r, 16.f, nullptr), LORA_ERR_SHAPE);
  EXPECT(lora_linear_fwd_dropout(dev(0), dev(1), dev(2), dev(3), nullptr, 0.05f, dev(4), dev<float>(5), m, n, k, r, 16.f, nullptr), LORA_ERR_NULL);
  EXPECT(lora_dropout_keep_mask(1, 0, 0.05f, nullptr, m, k, nullptr), LORA_ERR_NULL);
  EXPECT(lora_dropout_keep_mask(1, 0, 1.5f, dev<uint8_t>(6), m, k, nullptr), LORA_ERR_SHAPE);
  // backward: missing pointer, workspace, aliasing, the fused and dropout variants, the fixed workspace
  EXPECT(lora_linear_bwd(nullptr, dev(1), dev(2), dev(3), dev(4), dev<float>(5), dev(6), dev<float>(7), dev<float>(8), dev<void>(9), ws, m, n, k, r, 16.f, nullptr), LORA_ERR_NULL);
  EXPECT(lora_linear_bwd(dev(0), dev(1), dev(2), dev(3), dev(4), dev<float>(5), dev(6), dev<float>(7), dev<float>(8), dev<void>(9), ws - 16, m, n, k, r, 16.f, nullptr), LORA_ERR_WORKSPACE);
  EXPECT(lora_linear_bwd(dev(0), dev(1), dev(2), dev(3), dev(4), dev<float>(5), dev(6), dev<float>(7), dev<float>(8), dev<void>(9), ws, m, 7, k, r, 16.f, nullptr), LORA_ERR_SHAPE);
  EXPECT(lora_linear_bwd(dev(0), dev(1), dev(2), dev(3), dev(4), dev<float>(5), dev(0, 32), dev<float>(7), dev<float>(8), dev<void>(9), ws, m, n, k, r, 16.f, nullptr), LORA_ERR_ALIAS);
  EXPECT(lora_linear_bwd(dev(0), dev(1), dev(2), dev(3), dev(4), dev<float>(5), dev(6), dev<float>(7), dev<float>(7, 16), dev<void>(9), ws, m, n, k, r, 16.f, nullptr), LORA_ERR_ALIAS);
  EXPECT(lora_linear_bwd_noalloc(dev(0), dev(1), dev(2), nullptr, dev(4), dev<float>(5), dev(6), dev<float>(7), dev<float>(8), m, n, k, r, 16.f, nullptr), LORA_ERR_NULL);
  {
    const int64_t bm = 65536, bn = 4096, bk = 4096, br = 64;   // needs more than the fixed workspace
    EXPECT(lora_linear_bwd_workspace_size(bm, bn, bk, br) > (size_t(32) << 20), 1);
    EXPECT(lora_linear_bwd_noalloc(dev(0), dev(1), dev(2), dev(3), dev(4), dev<float>(5), dev(6), dev<float>(7), dev<float>(8), bm, bn, bk, br, 16.f, nullptr), LORA_ERR_WORKSPACE);
  }
  const size_t wsf = lora_linear_bwd_fused_workspace_size(m, n, k, r);
  EXPECT(lora_linear_bwd_fused(dev(0), dev(1), dev(2), dev(3), dev(4), dev<float>(5), dev(6), dev<float>(7), dev<float>(8), dev<void>(9), wsf - 16, m, n, k, r, 16.f, nullptr), LORA_ERR_WORKSPACE);
  EXPECT(lora_linear_bwd_fused(dev(0), dev(1), dev(2), dev(3), dev(4), dev<float>(5), dev(6), dev<float>(7), dev<float>(8), dev<void>(9), wsf, m, n, k, 32, 16.f, nullptr), LORA_ERR_UNSUPPORTED);
  EXPECT(lora_linear_bwd_dropout(dev(0), dev(1), dev(2), dev(3), dev(4), dev<float>(5), dev<uint8_t>(10), 1.0f, dev(6), dev<float>(7), dev<float>(8), dev<void>(9), ws, m, n, k, r, 16.f, nullptr), LORA_ERR_SHAPE);
  // merge: sign, pointers, partial overlap of the output with A
  EXPECT(lora_linear_merge(dev(0), dev(1), dev(2), dev(3), n, k, r, 16.f, 0, nullptr), LORA_ERR_SHAPE);
  EXPECT(lora_linear_merge(dev(0), nullptr, dev(2), dev(3), n, k, r, 16.f, 1, nullptr), LORA_ERR_NULL);
  EXPECT(lora_linear_merge(dev(0), dev(1), dev(2), dev(1, 128), n, k, r, 16.f, 1, nullptr), LORA_ERR_ALIAS);
}

static void groups() {
  const int64_t m = 64, k = 64, r = 8;
  int64_t n3[3] = {64, 128, 64};
  const lora_bf16* W[3] = {dev(1), dev(2), dev(3)};
  const lora_bf16* A[3] = {dev(4), dev(5), dev(6)};
  const lora_bf16* B[3] = {dev(7), dev(8), dev(9)};
  lora_bf16* Y[3] = {dev(10), dev(11), dev(12)};
  float* U[3] = {dev<float>(13), dev<float>(14), dev<float>(15)};
  EXPECT(lora_linear_group_fwd(dev(0), 0, n3, W, A, B, Y, U, m, k, r, 16.f, nullptr), LORA_ERR_SHAPE);
  EXPECT(lora_linear_group_fwd(dev(0), 9, n3, W, A, B, Y, U, m, k, r, 16.f, nullptr), LORA_ERR_UNSUPPORTED);
  EXPECT(lora_linear_group_fwd(dev(0), 3, nullptr, W, A, B, Y, U, m, k, r, 16.f, nullptr), LORA_ERR_NULL);
  EXPECT(lora_linear_group_fwd(dev(0), 3, n3, nullptr, A, B, Y, U, m, k, r, 16.f, nullptr), LORA_ERR_NULL);
  const lora_bf16* Wgap[3] = {dev(1), nullptr, dev(3)};
  EXPECT(lora_linear_group_fwd(dev(0), 3, n3, Wgap, A, B, Y, U, m, k, r, 16.f, nullptr), LORA_ERR_NULL);
  lora_bf16* Ymis[3] = {dev(10), dev(11, 8), dev(12)};
  EXPECT(lora_linear_group_fwd(dev(0), 3, n3, W, A, B, Ymis, U, m, k, r, 16.f, nullptr), LORA_ERR_ALIGN);
  int64_t nbad[3] = {64, 60, 64};
  EXPECT(lora_linear_group_fwd(dev(0), 3, nbad, W, A, B, Y, U, m, k, r, 16.f, nullptr), LORA_ERR_SHAPE);
  const size_t ws = lora_linear_group_bwd_workspace_size(3, n3, m, k, r);
  const lora_bf16* dY[3] = {dev(16), dev(17), dev(18)};
  const float* Uc[3] = {dev<float>(13), dev<float>(14), dev<float>(15)};
  float* dA[3] = {dev<float>(19), dev<float>(20), dev<float>(21)};
  float* dB[3] = {dev<float>(22), dev<float>(23), dev<float>(24)};
  EXPECT(lora_linear_group_bwd(dY, dev(0), 3, n3, W, A, B, Uc, dev(25), dA, dB, dev<void>(26), ws - 16, m, k, r, 16.f, nullptr), LORA_ERR_WORKSPACE);
  float* dAal[3] = {dev<float>(19), dev<float>(19, 64), dev<float>(21)};
  EXPECT(lora_linear_group_bwd(dY, dev(0), 3, n3, W, A, B, Uc, dev(25), dAal, dB, dev<void>(26), ws, m, k, r, 16.f, nullptr), LORA_ERR_ALIAS);
}

static void plans() {
  const int64_t ms[] = {1, 7, 64, 100, 2000, 2048, 4096, 8192};
  const int64_t ns[] = {8, 64, 200, 4000, 4096, 5120, 11008, 13824};
  const int64_t rs[] = {1, 8, 16, 17, 33, 48, 64, 65};
  std::vector<lora_launch_info> buf;
  long checked = 0;
  for (int op = LORA_OP_FWD; op <= LORA_OP_KEEP_MASK; ++op) {
    const bool grouped = op == LORA_OP_GROUP_FWD || op == LORA_OP_GROUP_BWD;
    for (int64_t m : ms)
      for (int64_t n : ns)
        for (int64_t k : ns)
          for (int64_t r : rs) {
            int64_t nn[3] = {n, n, n / 2 / 8 * 8 + 8};
            const int64_t group = grouped ? 3 : 1;
            const int64_t count = lora_linear_plan((lora_op)op, group, nn, m, k, r, nullptr, 0);
            if (count <= 0) continue;   // minus the status the entry point would return
            buf.assign((size_t)count + 1, lora_launch_info{});
            memset(buf.data(), 0xA5, sizeof(lora_launch_info) * buf.size());
            const int64_t again = lora_linear_plan((lora_op)op, group, nn, m, k, r, buf.data(), count);
            if (again != count) { fprintf(stderr, "plan count changed (op %d)\n", op); ++failures; continue; }
            for (int64_t i = 0; i < count; ++i) {
              const lora_launch_info& L = buf[(size_t)i];
              if (strnlen(L.kernel, sizeof(L.kernel)) == 0 || strnlen(L.kernel, sizeof(L.kernel)) == sizeof(L.kernel) ||
                  L.grid < 1 || L.block < 64 || L.col_begin < 0 || L.col_end < L.col_begin) {
                fprintf(stderr, "bad launch entry: op %d m %lld n %lld k %lld r %lld entry %lld\n", op, (long long)m,
                        (long long)n, (long long)k, (long long)r, (long long)i);
                ++failures;
              }
            }
            // the entry past the capacity stays untouched
            const unsigned char* tail = reinterpret_cast<const unsigned char*>(&buf[(size_t)count]);
            for (size_t b = 0; b < sizeof(lora_launch_info); ++b)
              if (tail[b] != 0xA5) { fprintf(stderr, "plan wrote past its capacity (op %d)\n", op); ++failures; break; }
            // a capacity of one writes one entry
            lora_launch_info one;
            if (lora_linear_plan((lora_op)op, group, nn, m, k, r, &one, 1) != count) ++failures;
            ++checked;
          }
  }
  printf("plans checked: %ld\n", checked);
  for (int64_t m : ms)
    for (int64_t n : ns)
      for (int64_t r : rs) {
        (void)lora_linear_bwd_workspace_size(m, n, 4096, r);
        (void)lora_linear_bwd_fused_workspace_size(m, n, 4096, r);
        int64_t nn[2] = {n, n};
        (void)lora_linear_group_bwd_workspace_size(2, nn, m, 4096, r);
      }
}

int main() {
  for (int s = 0; s <= 7; ++s)
    if (strcmp(status_text(s), "unknown status") == 0) ++failures;
  if (strcmp(status_text(8), "unknown status") != 0 || strcmp(status_text(99), "unknown status") != 0 ||
      strcmp(status_text(-1), "unknown status") != 0)
    ++failures;
  single_projection();
  groups();
  plans();
  printf(failures ? "abi sanitizer driver: %d FAILED\n" : "abi sanitizer driver: ok\n", failures);
  return failures ? 1 : 0;
}
