// A caller of the C ABI with no Python and no PyTorch: device memory from the
// HIP runtime, lora_linear_fwd then lora_linear_bwd on the default stream,
// results copied back to the host.  Test infrastructure (the GPU test
// tests/test_gpu_c_caller.py runs it and checks its outputs against the
// oracle).
//
// Usage: lora_caller DIR m n k r alpha
//   reads  DIR/X.bin [m,k], W.bin [n,k], A.bin [r,k], B.bin [n,r], dY.bin [m,n]
//          (bf16 bit patterns, uint16, row-major)
//   writes DIR/Y.bin [m,n], dX.bin [m,k] (bf16 bit patterns) and
//          DIR/U.bin [m,r], dA.bin [r,k], dB.bin [n,r] (float32)
// Exit status: 0 on success, 1 on bad arguments or files, 2 on a library
// status other than LORA_OK (printed), 3 on a HIP runtime error.
#include <hip/hip_runtime.h>

#include <cstdint>
#include <cstdio>
#include <cstdlib>
#include <string>
#include <vector>

#include "lora_linear.h"

namespace {

bool read_file(const std::string& path, void* dst, size_t bytes) {
  FILE* f = std::fopen(path.c_str(), "rb");
  if (!f) return false;
  const size_t got = std::fread(dst, 1, bytes, f);
  std::fclose(f);
  return got == bytes;
}

bool write_file(const std::string& path, const void* src, size_t bytes) {
  FILE* f = std::fopen(path.c_str(), "wb");
  if (!f) return false;
  const size_t put = std::fwrite(src, 1, bytes, f);
  std::fclose(f);
  return put == bytes;
}

#define HIP_OK(call)                                                               \
  do {                                                                             \
    const hipError_t e_ = (call);                                                  \
    if (e_ != hipSuccess) {                                                        \
      std::fprintf(stderr, "%s: %s\n", #call, hipGetErrorString(e_));              \
      std::exit(3);                                                                \
    }                                                                              \
  } while (0)

}  // namespace

int main(int argc, char** argv) {
  if (argc != 7) {
    std::fprintf(stderr, "usage: %s DIR m n k r alpha\n", argv[0]);
    return 1;
  }
  const std::string dir = argv[1];
  const int64_t m = std::atoll(argv[2]), n = std::atoll(argv[3]), k = std::atoll(argv[4]), r = std::atoll(argv[5]);
  const float alpha = (float)std::atof(argv[6]);
  if (m < 1 || n < 1 || k < 1 || r < 1) return 1;

  std::vector<uint16_t> X(m * k), W(n * k), A(r * k), B(n * r), dY(m * n);
  if (!read_file(dir + "/X.bin", X.data(), X.size() * 2) || !read_file(dir + "/W.bin", W.data(), W.size() * 2) ||
      !read_file(dir + "/A.bin", A.data(), A.size() * 2) || !read_file(dir + "/B.bin", B.data(), B.size() * 2) ||
      !read_file(dir + "/dY.bin", dY.data(), dY.size() * 2)) {
    std::fprintf(stderr, "cannot read the inputs in %s\n", dir.c_str());
    return 1;
  }

  auto upload = [](const std::vector<uint16_t>& h) {
    void* d = nullptr;
    HIP_OK(hipMalloc(&d, h.size() * 2));
    HIP_OK(hipMemcpy(d, h.data(), h.size() * 2, hipMemcpyHostToDevice));
    return static_cast<lora_bf16*>(d);
  };
  lora_bf16 *dXin = upload(X), *dW = upload(W), *dA_ = upload(A), *dB_ = upload(B), *ddY = upload(dY);
  lora_bf16 *dYout = nullptr, *ddX = nullptr;
  float *dU = nullptr, *ddA = nullptr, *ddB = nullptr;
  HIP_OK(hipMalloc((void**)&dYout, m * n * 2));
  HIP_OK(hipMalloc((void**)&ddX, m * k * 2));
  HIP_OK(hipMalloc((void**)&dU, m * r * 4));
  HIP_OK(hipMalloc((void**)&ddA, r * k * 4));
  HIP_OK(hipMalloc((void**)&ddB, n * r * 4));
  const size_t ws_bytes = lora_linear_bwd_workspace_size(m, n, k, r);
  void* ws = nullptr;
  HIP_OK(hipMalloc(&ws, ws_bytes > 0 ? ws_bytes : 16));

  lora_status st = lora_linear_fwd(dXin, dW, dA_, dB_, dYout, dU, m, n, k, r, alpha, nullptr);
  if (st == LORA_OK)
    st = lora_linear_bwd(ddY, dXin, dW, dA_, dB_, dU, ddX, ddA, ddB, ws, ws_bytes, m, n, k, r, alpha, nullptr);
  if (st != LORA_OK) {
    std::fprintf(stderr, "library status %d: %s\n", (int)st, lora_status_string(st));
    return 2;
  }
  HIP_OK(hipDeviceSynchronize());

  std::vector<uint16_t> Y(m * n), dX(m * k);
  std::vector<float> U(m * r), dA(r * k), dB(n * r);
  HIP_OK(hipMemcpy(Y.data(), dYout, Y.size() * 2, hipMemcpyDeviceToHost));
  HIP_OK(hipMemcpy(dX.data(), ddX, dX.size() * 2, hipMemcpyDeviceToHost));
  HIP_OK(hipMemcpy(U.data(), dU, U.size() * 4, hipMemcpyDeviceToHost));
  HIP_OK(hipMemcpy(dA.data(), ddA, dA.size() * 4, hipMemcpyDeviceToHost));
  HIP_OK(hipMemcpy(dB.data(), ddB, dB.size() * 4, hipMemcpyDeviceToHost));
  for (void* p : {(void*)dXin, (void*)dW, (void*)dA_, (void*)dB_, (void*)ddY, (void*)dYout, (void*)ddX, (void*)dU,
                  (void*)ddA, (void*)ddB, ws})
    HIP_OK(hipFree(p));
  if (!write_file(dir + "/Y.bin", Y.data(), Y.size() * 2) || !write_file(dir + "/dX.bin", dX.data(), dX.size() * 2) ||
      !write_file(dir + "/U.bin", U.data(), U.size() * 4) || !write_file(dir + "/dA.bin", dA.data(), dA.size() * 4) ||
      !write_file(dir + "/dB.bin", dB.data(), dB.size() * 4)) {
    std::fprintf(stderr, "cannot write the outputs in %s\n", dir.c_str());
    return 1;
  }
  std::printf("lora_caller: m=%lld n=%lld k=%lld r=%lld done\n", (long long)m, (long long)n, (long long)k,
              (long long)r);
  return 0;
}
