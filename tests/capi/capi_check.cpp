// Drives the flashdiff C ABI from C++ alone (no Python, no torch) on one GPU:
// the normalisation passes, a normalised fused product and a block Lanczos
// solve, plus one rejected call.  Test infrastructure: tests/test_gpu_capi.py
// writes the inputs, runs this program and checks what it writes against
// the oracle.
//
//   capi_check N D b k beta alpha in.bin out.bin
//
// in.bin : float32 X (N x D, row-major) then float32 V (N x b).
// out.bin: float32 q, d, s (N each); float64 s_off; float32 Y (N x b);
//          float64 evals (k); float64 residuals (k); float32 evecs (N x k);
//          int32 restarts, block_matvecs, nconv, status of the solve;
//          int32 status of a call with b = 0, int32 length of its message.
#include <hip/hip_runtime.h>

#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <vector>

#include "flashdiff.h"

#define HIP_OK(call)                                                         \
  do {                                                                       \
    hipError_t e_ = (call);                                                  \
    if (e_ != hipSuccess) {                                                  \
      std::fprintf(stderr, "%s failed: %s\n", #call, hipGetErrorString(e_)); \
      std::exit(2);                                                          \
    }                                                                        \
  } while (0)

static void fd_ok(fd_status st, const char* what) {
  if (st != FD_OK) {
    std::fprintf(stderr, "%s: %s (%s)\n", what, fd_status_string(st), fd_last_error());
    std::exit(3);
  }
}

template <typename T>
static T* dev_alloc(size_t n) {
  void* p = nullptr;
  HIP_OK(hipMalloc(&p, n * sizeof(T) + 1));
  return static_cast<T*>(p);
}

int main(int argc, char** argv) {
  if (argc != 9) {
    std::fprintf(stderr, "usage: %s N D b k beta alpha in.bin out.bin\n", argv[0]);
    return 1;
  }
  const int64_t N = std::atoll(argv[1]), D = std::atoll(argv[2]), b = std::atoll(argv[3]),
                k = std::atoll(argv[4]);
  const float beta = float(std::atof(argv[5])), alpha = float(std::atof(argv[6]));
  if (N < 2 || D < 1 || b < 1 || b > 64 || k < 1 || k > N) return 1;

  std::vector<float> X(static_cast<size_t>(N * D)), V(static_cast<size_t>(N * b));
  FILE* f = std::fopen(argv[7], "rb");
  if (f == nullptr || std::fread(X.data(), sizeof(float), X.size(), f) != X.size() ||
      std::fread(V.data(), sizeof(float), V.size(), f) != V.size())
    return 4;
  std::fclose(f);

  hipStream_t stream;
  HIP_OK(hipStreamCreate(&stream));
  float* dX = dev_alloc<float>(X.size());
  float* dV = dev_alloc<float>(V.size());
  float *dq = dev_alloc<float>(N), *dd = dev_alloc<float>(N), *ds = dev_alloc<float>(N);
  double* dsoff = dev_alloc<double>(1);
  float* dY = dev_alloc<float>(size_t(N * b));
  float* dE = dev_alloc<float>(size_t(N * k));
  HIP_OK(hipMemcpy(dX, X.data(), X.size() * sizeof(float), hipMemcpyHostToDevice));
  HIP_OK(hipMemcpy(dV, V.data(), V.size() * sizeof(float), hipMemcpyHostToDevice));

  fd_lanczos_opts opts;
  fd_lanczos_default_opts(&opts);
  const size_t ws_deg = fd_workspace_size(FD_OP_DEGREE, N, N, D, 0, 0, nullptr);
  const size_t ws_mm = fd_workspace_size(FD_OP_KERNEL_MATMUL, N, N, D, b, 0, nullptr);
  const size_t ws_lz = fd_workspace_size(FD_OP_BLOCK_LANCZOS, N, N, D, b, k, &opts);
  if (ws_deg == 0 || ws_mm == 0 || ws_lz == 0) return 5;
  size_t ws_bytes = ws_deg;
  if (ws_mm > ws_bytes) ws_bytes = ws_mm;
  if (ws_lz > ws_bytes) ws_bytes = ws_lz;
  void* ws = nullptr;
  HIP_OK(hipMalloc(&ws, ws_bytes));  // hipMalloc memory is 256-byte aligned

  fd_ok(fd_degree(dX, FD_F32, N, D, D, beta, alpha, dq, dd, ds, dsoff, ws, ws_bytes, stream),
        "fd_degree");
  fd_ok(fd_kernel_matmul(dX, N, dX, N, D, D, FD_F32, beta, ds, ds, dV, b, b, dY, b, ws, ws_bytes,
                         stream),
        "fd_kernel_matmul");
  std::vector<double> evals(static_cast<size_t>(k)), res(static_cast<size_t>(k));
  fd_lanczos_info info;
  std::memset(&info, 0, sizeof(info));
  const fd_status lst =
      fd_block_lanczos(dX, FD_F32, N, D, D, beta, alpha, b, k, nullptr, 0, 0, 1, &opts,
                       evals.data(), dE, nullptr, res.data(), &info, ws, ws_bytes, stream);
  if (lst != FD_OK && lst != FD_ERR_NOT_CONVERGED) fd_ok(lst, "fd_block_lanczos");
  // a rejected call: block width 0
  const fd_status bad = fd_kernel_matmul(dX, N, dX, N, D, D, FD_F32, beta, nullptr, nullptr, dV,
                                         0, b, dY, b, ws, ws_bytes, stream);
  const int32_t msg_len = int32_t(std::strlen(fd_last_error()));
  HIP_OK(hipStreamSynchronize(stream));

  const size_t n = static_cast<size_t>(N);
  std::vector<float> q(n), d(n), s(n), Y(n * size_t(b)), E(n * size_t(k));
  double soff = 0.0;
  HIP_OK(hipMemcpy(q.data(), dq, q.size() * sizeof(float), hipMemcpyDeviceToHost));
  HIP_OK(hipMemcpy(d.data(), dd, d.size() * sizeof(float), hipMemcpyDeviceToHost));
  HIP_OK(hipMemcpy(s.data(), ds, s.size() * sizeof(float), hipMemcpyDeviceToHost));
  HIP_OK(hipMemcpy(&soff, dsoff, sizeof(double), hipMemcpyDeviceToHost));
  HIP_OK(hipMemcpy(Y.data(), dY, Y.size() * sizeof(float), hipMemcpyDeviceToHost));
  HIP_OK(hipMemcpy(E.data(), dE, E.size() * sizeof(float), hipMemcpyDeviceToHost));

  FILE* o = std::fopen(argv[8], "wb");
  if (o == nullptr) return 6;
  std::fwrite(q.data(), sizeof(float), q.size(), o);
  std::fwrite(d.data(), sizeof(float), d.size(), o);
  std::fwrite(s.data(), sizeof(float), s.size(), o);
  std::fwrite(&soff, sizeof(double), 1, o);
  std::fwrite(Y.data(), sizeof(float), Y.size(), o);
  std::fwrite(evals.data(), sizeof(double), evals.size(), o);
  std::fwrite(res.data(), sizeof(double), res.size(), o);
  std::fwrite(E.data(), sizeof(float), E.size(), o);
  const int32_t tail[6] = {info.restarts, info.block_matvecs, info.nconv, int32_t(lst),
                           int32_t(bad), msg_len};
  std::fwrite(tail, sizeof(int32_t), 6, o);
  std::fclose(o);

  HIP_OK(hipFree(ws));
  HIP_OK(hipFree(dX));
  HIP_OK(hipFree(dV));
  HIP_OK(hipFree(dq));
  HIP_OK(hipFree(dd));
  HIP_OK(hipFree(ds));
  HIP_OK(hipFree(dsoff));
  HIP_OK(hipFree(dY));
  HIP_OK(hipFree(dE));
  HIP_OK(hipStreamDestroy(stream));
  std::printf("capi_check: ok\n");
  return 0;
}
