// lssvm-train: train an LS-SVM on a LIBSVM-format file and write the model,
// with the options of LIBSVM's svm-train that apply to it, on one GPU.
//
//   lssvm-train [options] training_file [model_file]
//
// Prints the time of each training component (Sec. IV-E: read, transfer to
// the device, the training call's setup and CG, write, total).
#include "lssvm.h"
#include "lssvm_io.h"

#include <hip/hip_runtime_api.h>

#include <chrono>
#include <cmath>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <string>

namespace {

using Clock = std::chrono::steady_clock;
double ms(Clock::time_point a, Clock::time_point b) {
  return std::chrono::duration<double, std::milli>(b - a).count();
}

void usage() {
  std::fprintf(stderr,
               "Usage: lssvm-train [options] training_file [model_file]\n"
               "options:\n"
               "  -t kernel_type : 0 linear (default), 1 polynomial (gamma*u'*v + coef0)^degree,\n"
               "                   2 radial basis exp(-gamma*|u-v|^2)\n"
               "  -d degree      : polynomial degree (default 3)\n"
               "  -g gamma       : kernel gamma (default 1/num_features)\n"
               "  -r coef0       : polynomial coef0 (default 0)\n"
               "  -c cost        : the parameter C (default 1)\n"
               "  -e epsilon     : CG stops at relative residual epsilon (default 0.001)\n"
               "  -i max_iter    : CG iteration limit (default: number of points - 1)\n"
               "  -p 64|32       : floating-point precision (default 64)\n"
               "  -T threads     : host threads for file IO (default: all available)\n"
               "  -q             : quiet (no component times)\n");
}

struct Args {
  int kernel = LSSVM_LINEAR;
  int degree = 3;
  double gamma = -1.0, coef0 = 0.0, C = 1.0, eps = 1e-3;
  long long max_iter = 0;
  int precision = 64, threads = 0;
  bool quiet = false;
  std::string train, model;
};

bool parse_double(const char* s, double* out) {
  char* end = nullptr;
  *out = std::strtod(s, &end);
  return end && *end == '\0' && end != s;
}

bool parse_long(const char* s, long long* out) {
  char* end = nullptr;
  *out = std::strtoll(s, &end, 10);
  return end && *end == '\0' && end != s;
}

bool parse(int argc, char** argv, Args* a) {
  int i = 1;
  for (; i < argc && argv[i][0] == '-' && argv[i][1] != '\0'; ++i) {
    const char opt = argv[i][1];
    if (argv[i][2] != '\0') return false;
    if (opt == 'q') {
      a->quiet = true;
      continue;
    }
    if (i + 1 >= argc) return false;
    const char* v = argv[++i];
    long long l = 0;
    switch (opt) {
      case 't':
        if (!parse_long(v, &l) || l < 0 || l > 2) return false;
        a->kernel = (int)l;
        break;
      case 'd':
        if (!parse_long(v, &l) || l < 1 || l > 1000) return false;
        a->degree = (int)l;
        break;
      case 'g':
        if (!parse_double(v, &a->gamma)) return false;
        break;
      case 'r':
        if (!parse_double(v, &a->coef0)) return false;
        break;
      case 'c':
        if (!parse_double(v, &a->C)) return false;
        break;
      case 'e':
        if (!parse_double(v, &a->eps)) return false;
        break;
      case 'i':
        if (!parse_long(v, &a->max_iter)) return false;
        break;
      case 'p':
        if (!parse_long(v, &l) || (l != 32 && l != 64)) return false;
        a->precision = (int)l;
        break;
      case 'T':
        if (!parse_long(v, &l) || l < 0 || l > 1024) return false;
        a->threads = (int)l;
        break;
      default:
        return false;
    }
  }
  if (i >= argc || argc - i > 2) return false;
  // the library checks these too; checking here reports them before any GPU work
  if (!(a->C > 0.0) || !std::isfinite(a->C)) return false;
  if (!(a->eps > 0.0 && a->eps < 1.0)) return false;
  if (a->max_iter < 0) return false;
  if (a->gamma != -1.0 && !(a->gamma > 0.0 && std::isfinite(a->gamma))) return false;
  if (!std::isfinite(a->coef0)) return false;
  a->train = argv[i];
  if (i + 1 < argc) {
    a->model = argv[i + 1];
  } else {
    const std::string& t = a->train;
    const size_t slash = t.find_last_of('/');
    a->model = (slash == std::string::npos ? t : t.substr(slash + 1)) + ".model";
  }
  return true;
}

int lib_error(const char* what) {
  std::fprintf(stderr, "lssvm-train: %s: %s\n", what, lssvm_last_error());
  return 1;
}

int hip_error(const char* what, hipError_t e) {
  std::fprintf(stderr, "lssvm-train: %s: %s\n", what, hipGetErrorString(e));
  return 1;
}

}  // namespace

int main(int argc, char** argv) {
  Args a;
  if (!parse(argc, argv, &a)) {
    usage();
    return 2;
  }
  const auto t0 = Clock::now();
  int64_t n = 0, d = 0;
  if (lssvm_libsvm_scan(a.train.c_str(), &n, &d, a.threads) != LSSVM_OK) return lib_error("read");
  if (n < 1) {
    std::fprintf(stderr, "lssvm-train: %s holds no data points\n", a.train.c_str());
    return 1;
  }
  if (d < 1) d = 1;
  if (a.gamma < 0.0) a.gamma = 1.0 / (double)d;
  const int32_t dtype = a.precision == 64 ? LSSVM_F64 : LSSVM_F32;
  const size_t es = a.precision == 64 ? sizeof(double) : sizeof(float);
  lssvm_params kp{a.gamma, a.coef0, a.degree};

  // host buffers in pinned memory: the upload then runs at full PCIe speed
  void *hX = nullptr, *hy = nullptr, *halpha = nullptr;
  hipError_t e;
  if ((e = hipHostMalloc(&hX, (size_t)n * d * es, hipHostMallocDefault)) != hipSuccess ||
      (e = hipHostMalloc(&hy, (size_t)n * es, hipHostMallocDefault)) != hipSuccess ||
      (e = hipHostMalloc(&halpha, (size_t)n * es, hipHostMallocDefault)) != hipSuccess)
    return hip_error("host allocation", e);
  if (lssvm_libsvm_read(a.train.c_str(), dtype, hX, hy, n, d, a.threads) != LSSVM_OK)
    return lib_error("read");
  const auto t_read = Clock::now();

  const size_t ws_bytes = lssvm_workspace_bytes(n, d, dtype);
  void *dX = nullptr, *dy = nullptr, *dalpha = nullptr, *ws = nullptr;
  if ((e = hipMalloc(&dX, (size_t)n * d * es)) != hipSuccess ||
      (e = hipMalloc(&dy, (size_t)n * es)) != hipSuccess ||
      (e = hipMalloc(&dalpha, (size_t)n * es)) != hipSuccess ||
      (e = hipMalloc(&ws, ws_bytes)) != hipSuccess)
    return hip_error("device allocation", e);
  if ((e = hipMemcpy(dX, hX, (size_t)n * d * es, hipMemcpyHostToDevice)) != hipSuccess ||
      (e = hipMemcpy(dy, hy, (size_t)n * es, hipMemcpyHostToDevice)) != hipSuccess)
    return hip_error("upload", e);
  const auto t_up = Clock::now();

  lssvm_info info;
  std::memset(&info, 0, sizeof info);
  double b = 0.0;
  const int rc = lssvm_train(dX, dy, n, d, dtype, a.kernel, &kp, a.C, a.eps, a.max_iter, ws,
                             ws_bytes, dalpha, &b, &info, nullptr);
  if (rc < 0) return lib_error("train");
  if (rc == LSSVM_NOT_CONVERGED)
    std::fprintf(stderr, "lssvm-train: warning: %s\n", lssvm_last_error());
  const auto t_train = Clock::now();

  if ((e = hipMemcpy(halpha, dalpha, (size_t)n * es, hipMemcpyDeviceToHost)) != hipSuccess)
    return hip_error("download", e);
  if (lssvm_model_write(a.model.c_str(), dtype, a.kernel, &kp, b, halpha, hX, hy, n, d,
                        a.threads) != LSSVM_OK)
    return lib_error("write");
  const auto t_write = Clock::now();

  if (!a.quiet) {
    std::printf("points %lld, features %lld, fp%d, %lld CG iterations, relative residual %.3g%s\n",
                (long long)n, (long long)d, a.precision, (long long)info.iterations,
                info.rel_residual, rc == LSSVM_NOT_CONVERGED ? " (not converged)" : "");
    std::printf("read %.3f ms | transfer %.3f ms | setup %.3f ms | cg %.3f ms | "
                "train call %.3f ms | write %.3f ms | total %.3f ms\n",
                ms(t0, t_read), ms(t_read, t_up), info.t_setup_ms, info.t_cg_ms,
                ms(t_up, t_train), ms(t_train, t_write), ms(t0, t_write));
    std::printf("b = %.17g, model written to %s\n", b, a.model.c_str());
  }
  (void)hipFree(ws);
  (void)hipFree(dalpha);
  (void)hipFree(dy);
  (void)hipFree(dX);
  (void)hipHostFree(halpha);
  (void)hipHostFree(hy);
  (void)hipHostFree(hX);
  return 0;
}
