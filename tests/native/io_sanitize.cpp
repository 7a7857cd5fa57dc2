// Host-only driver for the LIBSVM-format IO of include/lssvm_io.h, built by
// tests/test_io_sanitizers.py with AddressSanitizer + UndefinedBehaviorSanitizer
// and, separately, ThreadSanitizer (the reader and writers are multi-threaded).
//
// It links io.cpp alone, so it supplies the two error helpers that the
// training runtime normally provides. Exit status 0 means every check passed
// and the sanitizers reported nothing (they abort on the first finding).
#include "lssvm.h"
#include "lssvm_error.h"
#include "lssvm_io.h"

#include <cmath>
#include <cstdarg>
#include <cstdint>
#include <cstdio>
#include <cstring>
#include <random>
#include <string>
#include <vector>

namespace lssvm {
thread_local std::string g_err;
int fail(int code, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  std::vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_err = buf;
  return code;
}
void clear_error() { g_err.clear(); }
}  // namespace lssvm

static int g_failures = 0;
static int g_read_ok = 0, g_read_bad = 0, g_scan_bad = 0, g_model_ok = 0;
#define CHECK(cond)                                                              \
  do {                                                                           \
    if (!(cond)) {                                                               \
      std::fprintf(stderr, "CHECK failed at line %d: %s (%s)\n", __LINE__, #cond, \
                   lssvm::g_err.c_str());                                        \
      ++g_failures;                                                              \
    }                                                                            \
  } while (0)

static std::string g_dir;

static std::string path(const char* name) { return g_dir + "/" + name; }

static void put_file(const std::string& p, const std::string& text) {
  FILE* f = std::fopen(p.c_str(), "wb");
  std::fwrite(text.data(), 1, text.size(), f);
  std::fclose(f);
}

template <class T>
static bool same_bits(const std::vector<T>& a, const std::vector<T>& b) {
  return a.size() == b.size() && std::memcmp(a.data(), b.data(), a.size() * sizeof(T)) == 0;
}

template <class T>
static void round_trip(int32_t dtype, int64_t n, int64_t d, double density, uint64_t seed) {
  std::mt19937_64 rng(seed);
  std::normal_distribution<double> nd(0.0, 1.0);
  std::uniform_real_distribution<double> u(0.0, 1.0);
  std::vector<T> X(n * d, T(0)), y(n);
  for (int64_t i = 0; i < n; ++i) {
    y[i] = u(rng) < 0.5 ? T(1) : T(-1);
    for (int64_t j = 0; j < d; ++j)
      if (u(rng) < density) {
        T v = T(nd(rng) * std::pow(10.0, (int)(u(rng) * 12) - 6));
        X[i * d + j] = v == T(0) ? T(1) : v;
      }
  }
  for (int threads : {1, 3, 8, 64}) {
    const std::string p = path("rt.libsvm");
    CHECK(lssvm_libsvm_write(p.c_str(), dtype, X.data(), y.data(), n, d, threads) == LSSVM_OK);
    int64_t nn = -1, dd = -1;
    CHECK(lssvm_libsvm_scan(p.c_str(), &nn, &dd, threads) == LSSVM_OK);
    CHECK(nn == n && dd <= d);
    std::vector<T> X2(n * d, T(7)), y2(n, T(7));
    CHECK(lssvm_libsvm_read(p.c_str(), dtype, X2.data(), y2.data(), n, d, threads) == LSSVM_OK);
    CHECK(same_bits(X, X2) && same_bits(y, y2));
    // model file: every point a support vector, +1 first
    std::vector<T> alpha(n);
    for (int64_t i = 0; i < n; ++i) alpha[i] = T(nd(rng));
    lssvm_params kp{0.25, 1.0, 3};
    const std::string m = path("rt.model");
    CHECK(lssvm_model_write(m.c_str(), dtype, LSSVM_POLY, &kp, -0.5, alpha.data(), X.data(),
                            y.data(), n, d, threads) == LSSVM_OK);
    int32_t kernel = -1;
    lssvm_params kp2{};
    double b = 0;
    CHECK(lssvm_model_scan(m.c_str(), &kernel, &kp2, &b, &nn, &dd) == LSSVM_OK);
    CHECK(kernel == LSSVM_POLY && kp2.gamma == 0.25 && kp2.coef0 == 1.0 && kp2.degree == 3);
    CHECK(b == -0.5 && nn == n);
    std::vector<T> Xm(n * d), am(n), ym(n);
    CHECK(lssvm_model_read(m.c_str(), dtype, Xm.data(), am.data(), ym.data(), n, d, threads) ==
          LSSVM_OK);
    int64_t k = 0;
    for (int pass = 0; pass < 2; ++pass)
      for (int64_t i = 0; i < n; ++i)
        if ((y[i] == T(1)) == (pass == 0)) {
          CHECK(std::memcmp(&Xm[k * d], &X[i * d], d * sizeof(T)) == 0);
          CHECK(std::memcmp(&am[k], &alpha[i], sizeof(T)) == 0);
          CHECK(ym[k] == y[i]);
          ++k;
        }
  }
}

static void edge_files() {
  const std::string p = path("edge.libsvm");
  int64_t n = -1, d = -1;
  put_file(p, "");
  CHECK(lssvm_libsvm_scan(p.c_str(), &n, &d, 4) == LSSVM_OK && n == 0 && d == 0);
  put_file(p, "\n \t\r\n\n");
  CHECK(lssvm_libsvm_scan(p.c_str(), &n, &d, 4) == LSSVM_OK && n == 0);
  put_file(p, "+1 1:0.5 3:-2.5e-1\r\n\n-1\t2:1E2  4:007\n1");   // no final newline
  CHECK(lssvm_libsvm_scan(p.c_str(), &n, &d, 16) == LSSVM_OK && n == 3 && d == 4);
  std::vector<double> X(3 * 4), y(3);
  CHECK(lssvm_libsvm_read(p.c_str(), LSSVM_F64, X.data(), y.data(), 3, 4, 16) == LSSVM_OK);
  CHECK(X[0] == 0.5 && X[2] == -0.25 && X[5] == 100.0 && X[7] == 7.0 && y[2] == 1.0);
  const char* bad[] = {"1 1:1 1:2\n", "1 2:1 1:1\n", "1 0:1\n", "1 1:\n", "1 1:x\n", "x\n",
                       "1 1 :2\n", "1 1:2:3\n", "1 :2\n", "1 99999999999999999999:1\n",
                       "1 1:1e\n", "1 1:++2\n", "1 -1:2\n", "1 5:1\n"};
  for (const char* t : bad) {
    put_file(p, std::string("1 1:1\n") + t);
    std::vector<double> Xb(2 * 4), yb(2);
    CHECK(lssvm_libsvm_read(p.c_str(), LSSVM_F64, Xb.data(), yb.data(), 2, 4, 2) ==
          LSSVM_EINVAL);
  }
  CHECK(lssvm_libsvm_scan((g_dir + "/missing").c_str(), &n, &d, 1) == LSSVM_EINVAL);
  CHECK(lssvm_libsvm_scan(g_dir.c_str(), &n, &d, 1) == LSSVM_EINVAL);
}

// Random bytes and mutated valid files: every call must return OK or EINVAL,
// and the sanitizers must stay quiet.
static void fuzz(uint64_t seed, int rounds) {
  std::mt19937_64 rng(seed);
  const std::string alphabet = "0123456789+-.:eE \t\r\nnaifINFAX";
  const std::string p = path("fuzz.libsvm");
  for (int r = 0; r < rounds; ++r) {
    std::string text;
    if (r % 2 == 0) {
      const int len = (int)(rng() % 400);
      for (int i = 0; i < len; ++i) text += alphabet[rng() % alphabet.size()];
    } else {
      text = "1 1:0.5 2:-1 7:3e2\n-1 3:1\n+1 2:.25 4:7\n\n-1\n";
      const int edits = 1 + (int)(rng() % 6);
      for (int e = 0; e < edits; ++e) {
        const size_t at = rng() % (text.size() + 1);
        const int kind = (int)(rng() % 3);
        if (kind == 0 && at < text.size()) text.erase(at, 1);
        else if (kind == 1) text.insert(at, 1, alphabet[rng() % alphabet.size()]);
        else if (at < text.size()) text[at] = alphabet[rng() % alphabet.size()];
      }
    }
    put_file(p, text);
    for (int threads : {1, 5}) {
      int64_t n = -1, d = -1;
      const int rc = lssvm_libsvm_scan(p.c_str(), &n, &d, threads);
      CHECK(rc == LSSVM_OK || rc == LSSVM_EINVAL);
      if (rc != LSSVM_OK) ++g_scan_bad;
      if (rc != LSSVM_OK || n > 100000 || d > 4096) continue;
      const int64_t dd = d + 1;
      std::vector<double> X(std::max<int64_t>(1, n * dd)), y(std::max<int64_t>(1, n));
      const int rr = lssvm_libsvm_read(p.c_str(), LSSVM_F64, X.data(), y.data(), n, dd, threads);
      CHECK(rr == LSSVM_OK || rr == LSSVM_EINVAL);
      ++(rr == LSSVM_OK ? g_read_ok : g_read_bad);
      std::vector<float> Xf(X.size()), yf(y.size());
      const int rf = lssvm_libsvm_read(p.c_str(), LSSVM_F32, Xf.data(), yf.data(), n, dd, threads);
      CHECK(rf == rr);
    }
    // the same text as the SV section of a model whose header counts its lines
    int64_t nsv = -1, dsv = -1;
    if (lssvm_libsvm_scan(p.c_str(), &nsv, &dsv, 1) != LSSVM_OK) nsv = (int64_t)(rng() % 4);
    const int64_t npos = nsv > 0 ? (int64_t)(rng() % (nsv + 1)) : 0;
    put_file(p, "svm_type c_svc\nkernel_type rbf\ngamma 0.5\nnr_class 2\ntotal_sv " +
                    std::to_string(nsv) + "\nrho 0\nlabel " + (rng() % 2 ? "1 -1" : "-1 1") +
                    "\nnr_sv " + std::to_string(npos) + " " + std::to_string(nsv - npos) +
                    "\nSV\n" + text);
    int32_t kernel;
    lssvm_params kp;
    double b;
    int64_t n = -1, d = -1;
    const int rc = lssvm_model_scan(p.c_str(), &kernel, &kp, &b, &n, &d);
    CHECK(rc == LSSVM_OK || rc == LSSVM_EINVAL);
    if (rc == LSSVM_OK && n <= 100000 && d < 4096) {
      std::vector<double> X(std::max<int64_t>(1, n * (d + 1))), a(std::max<int64_t>(1, n)),
          y(std::max<int64_t>(1, n));
      const int rm = lssvm_model_read(p.c_str(), LSSVM_F64, X.data(), a.data(), y.data(), n,
                                      d + 1, 3);
      CHECK(rm == LSSVM_OK || rm == LSSVM_EINVAL);
      if (rm == LSSVM_OK) ++g_model_ok;
    }
  }
}

int main(int argc, char** argv) {
  if (argc < 2) {
    std::fprintf(stderr, "usage: %s <scratch dir> [fuzz rounds]\n", argv[0]);
    return 2;
  }
  g_dir = argv[1];
  const int rounds = argc > 2 ? std::atoi(argv[2]) : 400;
  round_trip<double>(LSSVM_F64, 257, 19, 0.7, 1);
  round_trip<float>(LSSVM_F32, 131, 33, 0.5, 2);
  round_trip<double>(LSSVM_F64, 3, 1, 1.0, 3);
  edge_files();
  fuzz(7, rounds);
  std::printf("io_sanitize: %d failures; fuzz: %d scans rejected, %d reads ok, %d reads "
              "rejected, %d models read\n", g_failures, g_scan_bad, g_read_ok, g_read_bad,
              g_model_ok);
  return g_failures == 0 ? 0 : 1;
}
