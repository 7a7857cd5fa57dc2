// lssvm-predict: label the points of a LIBSVM-format file with a model written
// by lssvm-train (or a binary LIBSVM model with labels 1 and -1), on one GPU.
//
//   lssvm-predict [options] test_file model_file output_file
//
// Writes one predicted label per line and reports the accuracy against the
// labels of the test file.
#include "lssvm.h"
#include "lssvm_io.h"

#include <hip/hip_runtime_api.h>

#include <algorithm>
#include <chrono>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <string>
#include <vector>

namespace {

using Clock = std::chrono::steady_clock;
double ms(Clock::time_point a, Clock::time_point b) {
  return std::chrono::duration<double, std::milli>(b - a).count();
}

void usage() {
  std::fprintf(stderr,
               "Usage: lssvm-predict [options] test_file model_file output_file\n"
               "options:\n"
               "  -p 64|32   : floating-point precision (default 64)\n"
               "  -T threads : host threads for file IO (default: all available)\n"
               "  -q         : quiet (no accuracy or times)\n");
}

int lib_error(const char* what) {
  std::fprintf(stderr, "lssvm-predict: %s: %s\n", what, lssvm_last_error());
  return 1;
}

int hip_error(const char* what, hipError_t e) {
  std::fprintf(stderr, "lssvm-predict: %s: %s\n", what, hipGetErrorString(e));
  return 1;
}

template <class T>
int run(const std::string& test, const std::string& model, const std::string& out, int32_t dtype,
        int threads, bool quiet) {
  const auto t0 = Clock::now();
  int32_t kernel = 0;
  lssvm_params kp{};
  double b = 0.0;
  int64_t n = 0, dm = 0, nt = 0, dt = 0;
  if (lssvm_model_scan(model.c_str(), &kernel, &kp, &b, &n, &dm) != LSSVM_OK)
    return lib_error("model");
  if (n < 1) {
    std::fprintf(stderr, "lssvm-predict: %s has no support vectors\n", model.c_str());
    return 1;
  }
  if (lssvm_libsvm_scan(test.c_str(), &nt, &dt, threads) != LSSVM_OK) return lib_error("test data");
  const int64_t d = std::max<int64_t>({dm, dt, 1});
  std::vector<T> Xm((size_t)n * d), alpha(n), ym(n), Xt((size_t)std::max<int64_t>(nt, 1) * d),
      yt(std::max<int64_t>(nt, 1));
  if (lssvm_model_read(model.c_str(), dtype, Xm.data(), alpha.data(), ym.data(), n, d, threads) !=
      LSSVM_OK)
    return lib_error("model");
  if (nt > 0 && lssvm_libsvm_read(test.c_str(), dtype, Xt.data(), yt.data(), nt, d, threads) !=
                    LSSVM_OK)
    return lib_error("test data");
  const auto t_read = Clock::now();

  std::vector<int32_t> labels(std::max<int64_t>(nt, 1));
  if (nt > 0) {
    const size_t ws_bytes = lssvm_predict_workspace_bytes(n, nt, d, dtype);
    void *dXm, *dalpha, *dXt, *dscores, *dlabels, *ws;
    hipError_t e;
    if ((e = hipMalloc(&dXm, Xm.size() * sizeof(T))) != hipSuccess ||
        (e = hipMalloc(&dalpha, alpha.size() * sizeof(T))) != hipSuccess ||
        (e = hipMalloc(&dXt, Xt.size() * sizeof(T))) != hipSuccess ||
        (e = hipMalloc(&dscores, (size_t)nt * sizeof(T))) != hipSuccess ||
        (e = hipMalloc(&dlabels, (size_t)nt * sizeof(int32_t))) != hipSuccess ||
        (e = hipMalloc(&ws, ws_bytes)) != hipSuccess)
      return hip_error("device allocation", e);
    if ((e = hipMemcpy(dXm, Xm.data(), Xm.size() * sizeof(T), hipMemcpyHostToDevice)) !=
            hipSuccess ||
        (e = hipMemcpy(dalpha, alpha.data(), alpha.size() * sizeof(T), hipMemcpyHostToDevice)) !=
            hipSuccess ||
        (e = hipMemcpy(dXt, Xt.data(), Xt.size() * sizeof(T), hipMemcpyHostToDevice)) !=
            hipSuccess)
      return hip_error("upload", e);
    if (lssvm_predict(dXm, dalpha, b, n, d, dtype, kernel, &kp, dXt, nt, ws, ws_bytes, dscores,
                      static_cast<int32_t*>(dlabels), nullptr) != LSSVM_OK)
      return lib_error("predict");
    if ((e = hipMemcpy(labels.data(), dlabels, (size_t)nt * sizeof(int32_t),
                       hipMemcpyDeviceToHost)) != hipSuccess)
      return hip_error("download", e);
    (void)hipFree(ws);
    (void)hipFree(dlabels);
    (void)hipFree(dscores);
    (void)hipFree(dXt);
    (void)hipFree(dalpha);
    (void)hipFree(dXm);
  }
  const auto t_pred = Clock::now();

  FILE* f = std::fopen(out.c_str(), "w");
  if (!f) {
    std::fprintf(stderr, "lssvm-predict: cannot create %s\n", out.c_str());
    return 1;
  }
  int64_t correct = 0;
  for (int64_t i = 0; i < nt; ++i) {
    std::fprintf(f, "%d\n", labels[i]);
    correct += (double)labels[i] == (double)yt[i];
  }
  if (std::fclose(f) != 0) {
    std::fprintf(stderr, "lssvm-predict: cannot write %s\n", out.c_str());
    return 1;
  }
  if (!quiet) {
    if (nt > 0)
      std::printf("Accuracy = %.4f%% (%lld/%lld)\n", 100.0 * (double)correct / (double)nt,
                  (long long)correct, (long long)nt);
    std::printf("read %.3f ms | predict %.3f ms | total %.3f ms\n", ms(t0, t_read),
                ms(t_read, t_pred), ms(t0, Clock::now()));
  }
  return 0;
}

}  // namespace

int main(int argc, char** argv) {
  int precision = 64, threads = 0;
  bool quiet = false;
  int i = 1;
  for (; i < argc && argv[i][0] == '-' && argv[i][1] != '\0'; ++i) {
    const char opt = argv[i][1];
    if (argv[i][2] != '\0') {
      usage();
      return 2;
    }
    if (opt == 'q') {
      quiet = true;
      continue;
    }
    if (i + 1 >= argc || (opt != 'p' && opt != 'T')) {
      usage();
      return 2;
    }
    char* end = nullptr;
    const long v = std::strtol(argv[++i], &end, 10);
    if (!end || *end != '\0' || (opt == 'p' && v != 32 && v != 64) ||
        (opt == 'T' && (v < 0 || v > 1024))) {
      usage();
      return 2;
    }
    (opt == 'p' ? precision : threads) = (int)v;
  }
  if (argc - i != 3) {
    usage();
    return 2;
  }
  return precision == 64 ? run<double>(argv[i], argv[i + 1], argv[i + 2], LSSVM_F64, threads, quiet)
                         : run<float>(argv[i], argv[i + 1], argv[i + 2], LSSVM_F32, threads, quiet);
}
