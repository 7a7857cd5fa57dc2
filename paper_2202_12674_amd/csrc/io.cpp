// Host IO of include/lssvm_io.h: LIBSVM-format data files and model files
// around the training path (Sec. III, steps (1) and (4) of training; timed as
// "read" and "write" in Sec. IV-E).
//
// The paper's reader builds an irregular 2D structure and a later step
// transforms it into one contiguous vector. Here the reader parses straight
// into the caller's dense row-major buffer (zero-filled where a feature is
// absent), so the only layout change left is the on-device panel layout of
// the training call. Files are memory-mapped and split at line boundaries into
// one byte range per thread; a counting pass gives each range its first row,
// then every range is parsed in parallel. Writers format disjoint row ranges
// in parallel and place them with positioned writes.
//
// Numbers are converted with std::from_chars / std::to_chars: parsing rounds
// the decimal text once, correctly, to the requested type, and writing emits
// the shortest text that reads back to the same value.
#include "lssvm.h"
#include "lssvm_error.h"
#include "lssvm_io.h"

#include <errno.h>
#include <fcntl.h>
#include <locale.h>
#include <sched.h>
#include <stdlib.h>
#include <sys/mman.h>
#include <sys/stat.h>
#include <unistd.h>

#include <algorithm>
#include <charconv>
#include <cmath>
#include <cstdint>
#include <cstring>
#include <exception>
#include <limits>
#include <string>
#include <thread>
#include <vector>

namespace lssvm {
namespace {

constexpr int64_t kMaxDim = int64_t(1) << 31;     // largest feature index accepted

// ------------------------------------------------------------------ threads --

int resolve_threads(int32_t requested) {
  if (requested > 0) return std::min<int32_t>(requested, 1024);
  cpu_set_t set;
  if (sched_getaffinity(0, sizeof set, &set) == 0) {
    int c = CPU_COUNT(&set);
    if (c > 0) return c;
  }
  unsigned h = std::thread::hardware_concurrency();
  return h ? int(h) : 1;
}

// Run f(0..nt-1), f(0) on the calling thread.
template <class F>
void parallel_for(int nt, F&& f) {
  if (nt <= 1) {
    f(0);
    return;
  }
  std::vector<std::thread> pool;
  pool.reserve(nt - 1);
  for (int t = 1; t < nt; ++t) pool.emplace_back([&f, t] { f(t); });
  f(0);
  for (auto& th : pool) th.join();
}

// ------------------------------------------------------------- text helpers --

inline bool is_blank(char c) { return c == ' ' || c == '\t' || c == '\r'; }

locale_t c_locale() {
  static locale_t loc = newlocale(LC_ALL_MASK, "C", locale_t(0));
  return loc;
}

inline void strto_c(const char* s, double& v) { v = strtod_l(s, nullptr, c_locale()); }
inline void strto_c(const char* s, float& v) { v = strtof_l(s, nullptr, c_locale()); }

// Parse one real number at [s, e): an optional '+' or '-', then a decimal
// number with optional fraction and exponent, or inf / infinity / nan. The
// value is the decimal rounded once to T (overflow gives +-inf, underflow a
// subnormal or zero). Returns the end of the number or nullptr.
template <class T>
const char* parse_real(const char* s, const char* e, T& out) {
  if (s < e && *s == '+') {
    ++s;
    if (s < e && (*s == '+' || *s == '-')) return nullptr;
  }
  auto r = std::from_chars(s, e, out, std::chars_format::general);
  if (r.ec == std::errc()) return r.ptr;
  if (r.ec == std::errc::result_out_of_range) {
    std::string tok(s, r.ptr);
    strto_c(tok.c_str(), out);
    return r.ptr;
  }
  return nullptr;
}

// Parse a decimal integer token that must end at a blank, the line end or `stop`.
const char* parse_int(const char* s, const char* e, int64_t& out) {
  auto r = std::from_chars(s, e, out, 10);
  if (r.ec != std::errc()) return nullptr;
  return r.ptr;
}

inline const char* skip_blank(const char* s, const char* e) {
  while (s < e && is_blank(*s)) ++s;
  return s;
}

inline bool token_ends(const char* s, const char* e) { return s == e || is_blank(*s); }

// ---------------------------------------------------------------- mmap file --

struct MappedFile {
  int fd = -1;
  const char* p = nullptr;
  size_t size = 0;
  ~MappedFile() {
    if (p) munmap(const_cast<char*>(p), size);
    if (fd >= 0) close(fd);
  }
};

int map_file(const char* path, MappedFile& m) {
  if (!path) return fail(LSSVM_EINVAL, "path is NULL");
  m.fd = open(path, O_RDONLY | O_CLOEXEC);
  if (m.fd < 0) return fail(LSSVM_EINVAL, "cannot open %s: %s", path, strerror(errno));
  struct stat st;
  if (fstat(m.fd, &st) != 0) return fail(LSSVM_EINVAL, "cannot stat %s: %s", path, strerror(errno));
  if (!S_ISREG(st.st_mode)) return fail(LSSVM_EINVAL, "%s is not a regular file", path);
  m.size = size_t(st.st_size);
  if (m.size == 0) return LSSVM_OK;
  void* p = mmap(nullptr, m.size, PROT_READ, MAP_PRIVATE, m.fd, 0);
  if (p == MAP_FAILED) return fail(LSSVM_EINVAL, "cannot map %s: %s", path, strerror(errno));
  madvise(p, m.size, MADV_WILLNEED);
  m.p = static_cast<const char*>(p);
  return LSSVM_OK;
}

// Split [from, size) into `parts` ranges that each start at a line start.
std::vector<size_t> split_lines(const char* p, size_t size, size_t from, int parts) {
  std::vector<size_t> b(parts + 1, size);
  b[0] = from;
  for (int c = 1; c < parts; ++c) {
    size_t s = from + (size - from) / parts * c;
    size_t cut = from;
    if (s > from) {
      const void* nl = memchr(p + s - 1, '\n', size - (s - 1));
      cut = nl ? size_t(static_cast<const char*>(nl) - p) + 1 : size;
    }
    b[c] = std::max(cut, b[c - 1]);
  }
  return b;
}

// Call f(line_begin, line_end) for every line of [b, e) (line_end excludes '\n').
template <class F>
void for_lines(const char* p, size_t b, size_t e, F&& f) {
  size_t q = b;
  while (q < e) {
    const void* nl = memchr(p + q, '\n', e - q);
    size_t le = nl ? size_t(static_cast<const char*>(nl) - p) : e;
    f(p + q, p + le);
    q = le + 1;
  }
}

int pick_parts(size_t bytes, int threads) {
  size_t by_size = bytes / (size_t(1) << 16) + 1;  // at least 64 KiB per range
  return int(std::max<size_t>(1, std::min<size_t>(size_t(threads), by_size)));
}

// Per-range result of a pass; errors carry the line number within the range.
struct RangeStats {
  int64_t lines = 0, points = 0, max_index = 0;
  int64_t err_line = -1;
  const char* err = nullptr;
};

// Report the earliest error over all ranges, numbering lines from first_line.
int first_error(const std::vector<RangeStats>& st, int64_t first_line, const char* path) {
  int64_t before = first_line;
  for (const auto& r : st) {
    if (r.err) return fail(LSSVM_EINVAL, "%s:%lld: %s", path, (long long)(before + r.err_line + 1),
                           r.err);
    before += r.lines;
  }
  return LSSVM_OK;
}

// Largest feature index of a data line (its last "<index>:"; indices increase).
int64_t last_index(const char* s, const char* e, const char** err) {
  const void* c = memrchr(s, ':', size_t(e - s));
  if (!c) return 0;
  const char* colon = static_cast<const char*>(c);
  const char* q = colon;
  while (q > s && q[-1] >= '0' && q[-1] <= '9') --q;
  int64_t v = 0;
  if (q == colon || parse_int(q, colon, v) != colon) {
    *err = "expected <index>:<value>";
    return -1;
  }
  return v;
}

// Counting pass over the data lines of [from, size).
int scan_lines(const MappedFile& m, size_t from, int threads, int64_t first_line, const char* path,
               std::vector<size_t>& bounds, std::vector<RangeStats>& st) {
  int parts = pick_parts(m.size - from, threads);
  bounds = split_lines(m.p, m.size, from, parts);
  st.assign(parts, RangeStats{});
  parallel_for(parts, [&](int c) {
    RangeStats& r = st[c];
    for_lines(m.p, bounds[c], bounds[c + 1], [&](const char* s, const char* e) {
      const char* q = skip_blank(s, e);
      if (q != e) {
        if (!r.err) {
          const char* why = nullptr;
          int64_t k = last_index(q, e, &why);
          if (why) {
            r.err = why;
            r.err_line = r.lines;
          } else {
            r.max_index = std::max(r.max_index, k);
          }
        }
        ++r.points;
      }
      ++r.lines;
    });
  });
  return first_error(st, first_line, path);
}

// Parse one non-blank data line "<head> <index>:<value> ..." into head and the
// zero-filled dense row. Returns nullptr or the reason the line is malformed.
template <class T>
const char* parse_line(const char* s, const char* e, T& head, T* row, int64_t d) {
  const char* q = parse_real(s, e, head);
  if (!q || !token_ends(q, e)) return "the first token is not a number";
  std::fill(row, row + d, T(0));
  int64_t prev = 0;
  for (;;) {
    q = skip_blank(q, e);
    if (q == e) return nullptr;
    int64_t idx = 0;
    q = parse_int(q, e, idx);
    if (!q || q == e || *q != ':') return "expected <index>:<value>";
    if (idx < 1) return "feature indices start at 1";
    if (idx <= prev) return "feature indices must increase along a line";
    if (idx > d) return "feature index exceeds d";
    T v;
    q = parse_real(q + 1, e, v);
    if (!q || !token_ends(q, e)) return "feature value is not a number";
    row[idx - 1] = v;
    prev = idx;
  }
}

// Parsing pass: rows of X and heads (labels, or model coefficients) per line.
template <class T>
int parse_lines(const MappedFile& m, const std::vector<size_t>& bounds,
                const std::vector<RangeStats>& counted, int64_t first_line, const char* path,
                T* X, T* heads, int64_t d) {
  int parts = int(counted.size());
  std::vector<int64_t> row0(parts + 1, 0);
  for (int c = 0; c < parts; ++c) row0[c + 1] = row0[c] + counted[c].points;
  std::vector<RangeStats> st(parts);
  parallel_for(parts, [&](int c) {
    RangeStats& r = st[c];
    int64_t row = row0[c];
    for_lines(m.p, bounds[c], bounds[c + 1], [&](const char* s, const char* e) {
      if (r.err) return;
      const char* q = skip_blank(s, e);
      if (q != e) {
        const char* why = parse_line(q, e, heads[row], X + row * d, d);
        if (why) {
          r.err = why;
          r.err_line = r.lines;
        }
        ++row;
      }
      ++r.lines;
    });
  });
  return first_error(st, first_line, path);
}

// ------------------------------------------------------------------ writing --

struct OutBuf {
  char* p = nullptr;
  size_t len = 0, cap = 0;
  ~OutBuf() { free(p); }
  char* reserve(size_t more) {
    if (len + more > cap) {
      size_t nc = std::max(cap * 2, len + more);
      char* np = static_cast<char*>(realloc(p, nc));
      if (!np) throw std::bad_alloc();
      p = np;
      cap = nc;
    }
    return p + len;
  }
};

constexpr size_t kNumChars = 32;  // room for any shortest double / float / int64

template <class T>
char* put_real(char* o, T v) {
  return std::to_chars(o, o + kNumChars, v).ptr;
}

// "<head> <j+1>:<x_j> ...\n" with zero features left out.
template <class T>
void format_row(OutBuf& out, T head, const T* row, int64_t d) {
  char* o = out.reserve(kNumChars + 1 + size_t(d) * (2 * kNumChars + 2));
  char* start = o;
  o = put_real(o, head);
  for (int64_t j = 0; j < d; ++j) {
    T v = row[j];
    if (v == T(0)) continue;
    *o++ = ' ';
    o = std::to_chars(o, o + kNumChars, j + 1).ptr;
    *o++ = ':';
    o = put_real(o, v);
  }
  *o++ = '\n';
  out.len += size_t(o - start);
}

bool pwrite_all(int fd, const char* p, size_t n, off_t off) {
  while (n) {
    ssize_t w = pwrite(fd, p, n, off);
    if (w < 0) {
      if (errno == EINTR) continue;
      return false;
    }
    p += w;
    n -= size_t(w);
    off += w;
  }
  return true;
}

// Write `header` then the buffers in order, the buffers concurrently.
int write_file(const char* path, const std::string& header, std::vector<OutBuf>& bufs) {
  int fd = open(path, O_WRONLY | O_CREAT | O_TRUNC | O_CLOEXEC, 0644);
  if (fd < 0) return fail(LSSVM_EINVAL, "cannot create %s: %s", path, strerror(errno));
  std::vector<off_t> off(bufs.size() + 1, off_t(header.size()));
  for (size_t i = 0; i < bufs.size(); ++i) off[i + 1] = off[i] + off_t(bufs[i].len);
  bool ok = pwrite_all(fd, header.data(), header.size(), 0);
  std::vector<int> good(bufs.size(), 1);
  parallel_for(int(bufs.size()), [&](int t) {
    good[t] = pwrite_all(fd, bufs[t].p, bufs[t].len, off[t]) ? 1 : 0;
  });
  for (int g : good) ok = ok && g;
  int err = ok ? 0 : errno;
  if (close(fd) != 0 && ok) {
    ok = false;
    err = errno;
  }
  if (!ok) return fail(LSSVM_EINVAL, "cannot write %s: %s", path, strerror(err));
  return LSSVM_OK;
}

std::string fmt_double(double v) {
  char b[kNumChars];
  return std::string(b, std::to_chars(b, b + kNumChars, v).ptr);
}

// --------------------------------------------------------------- data files --

template <class T>
int write_data(const char* path, const T* X, const T* y, int64_t n, int64_t d, int threads) {
  int parts = int(std::max<int64_t>(1, std::min<int64_t>(threads, n)));
  std::vector<OutBuf> bufs(parts);
  parallel_for(parts, [&](int t) {
    int64_t r0 = n * t / parts, r1 = n * (t + 1) / parts;
    for (int64_t i = r0; i < r1; ++i) format_row(bufs[t], y[i], X + i * d, d);
  });
  return write_file(path, std::string(), bufs);
}

template <class T>
int read_data(const char* path, T* X, T* y, int64_t n, int64_t d, int threads) {
  MappedFile m;
  int rc = map_file(path, m);
  if (rc != LSSVM_OK) return rc;
  std::vector<size_t> bounds;
  std::vector<RangeStats> st;
  if (m.size) {
    int parts = pick_parts(m.size, threads);
    bounds = split_lines(m.p, m.size, 0, parts);
    st.assign(parts, RangeStats{});
    parallel_for(parts, [&](int c) {
      RangeStats& r = st[c];
      for_lines(m.p, bounds[c], bounds[c + 1], [&](const char* s, const char* e) {
        if (skip_blank(s, e) != e) ++r.points;
        ++r.lines;
      });
    });
  }
  int64_t points = 0;
  for (const auto& r : st) points += r.points;
  if (points != n)
    return fail(LSSVM_EINVAL, "%s holds %lld points, n is %lld", path, (long long)points,
                (long long)n);
  if (n == 0) return LSSVM_OK;
  return parse_lines(m, bounds, st, 0, path, X, y, d);
}

// -------------------------------------------------------------- model files --

struct ModelHeader {
  int32_t kernel = -1;
  lssvm_params kp{1.0, 0.0, 3};
  bool have_gamma = false, have_rho = false, have_svm_type = false;
  double rho = 0.0;
  int64_t nr_class = -1, total_sv = -1, nr_sv[2] = {-1, -1};
  int64_t label[2] = {0, 0};
  bool have_label = false;
  size_t sv_offset = 0;   // byte offset of the first support-vector line
  int64_t sv_line = 0;    // number of lines before it
};

// The values after the key of a header line, as whitespace-separated tokens.
std::vector<std::string> tokens(const char* s, const char* e) {
  std::vector<std::string> out;
  while ((s = skip_blank(s, e)) < e) {
    const char* t = s;
    while (s < e && !is_blank(*s)) ++s;
    out.emplace_back(t, s);
  }
  return out;
}

bool to_double(const std::string& t, double& v) {
  const char* e = t.data() + t.size();
  return parse_real(t.data(), e, v) == e;
}

bool to_int(const std::string& t, int64_t& v) {
  const char* e = t.data() + t.size();
  return parse_int(t.data(), e, v) == e;
}

int parse_header(const MappedFile& m, const char* path, ModelHeader& h) {
  size_t q = 0;
  int64_t line = 0;
  bool saw_sv = false;
  while (q < m.size && !saw_sv) {
    const void* nl = memchr(m.p + q, '\n', m.size - q);
    size_t le = nl ? size_t(static_cast<const char*>(nl) - m.p) : m.size;
    auto tok = tokens(m.p + q, m.p + le);
    ++line;
    q = le + 1;
    if (tok.empty()) continue;
    const std::string& key = tok[0];
    size_t nv = tok.size() - 1;
    auto bad = [&](const char* what) {
      return fail(LSSVM_EINVAL, "%s:%lld: %s", path, (long long)line, what);
    };
    if (key == "SV") {
      if (nv) return bad("nothing may follow SV on its line");
      saw_sv = true;
    } else if (key == "svm_type") {
      if (nv != 1 || tok[1] != "c_svc") return bad("svm_type must be c_svc");
      h.have_svm_type = true;
    } else if (key == "kernel_type") {
      if (nv != 1) return bad("kernel_type takes one value");
      if (tok[1] == "linear") h.kernel = LSSVM_LINEAR;
      else if (tok[1] == "polynomial") h.kernel = LSSVM_POLY;
      else if (tok[1] == "rbf") h.kernel = LSSVM_RBF;
      else return bad("kernel_type must be linear, polynomial or rbf");
    } else if (key == "degree") {
      int64_t v;
      if (nv != 1 || !to_int(tok[1], v) || v < 1 || v > std::numeric_limits<int32_t>::max())
        return bad("degree must be a positive integer");
      h.kp.degree = int32_t(v);
    } else if (key == "gamma") {
      if (nv != 1 || !to_double(tok[1], h.kp.gamma)) return bad("gamma must be a number");
      h.have_gamma = true;
    } else if (key == "coef0") {
      if (nv != 1 || !to_double(tok[1], h.kp.coef0)) return bad("coef0 must be a number");
    } else if (key == "nr_class") {
      if (nv != 1 || !to_int(tok[1], h.nr_class) || h.nr_class != 2)
        return bad("nr_class must be 2 (binary classification)");
    } else if (key == "total_sv") {
      if (nv != 1 || !to_int(tok[1], h.total_sv) || h.total_sv < 0)
        return bad("total_sv must be a non-negative integer");
    } else if (key == "rho") {
      if (nv != 1 || !to_double(tok[1], h.rho) || !std::isfinite(h.rho))
        return bad("rho must be one finite number");
      h.have_rho = true;
    } else if (key == "label") {
      if (nv != 2 || !to_int(tok[1], h.label[0]) || !to_int(tok[2], h.label[1]) ||
          !((h.label[0] == 1 && h.label[1] == -1) || (h.label[0] == -1 && h.label[1] == 1)))
        return bad("label must list the classes 1 and -1");
      h.have_label = true;
    } else if (key == "nr_sv") {
      if (nv != 2 || !to_int(tok[1], h.nr_sv[0]) || !to_int(tok[2], h.nr_sv[1]) ||
          h.nr_sv[0] < 0 || h.nr_sv[1] < 0)
        return bad("nr_sv must be two non-negative integers");
    } else if (key == "probA" || key == "probB") {
      // probability estimates are not used by this library
    } else {
      return bad("unknown model header key");
    }
  }
  if (!saw_sv) return fail(LSSVM_EINVAL, "%s: no SV section", path);
  if (!h.have_svm_type || h.kernel < 0 || h.nr_class != 2 || h.total_sv < 0 || !h.have_rho ||
      !h.have_label || h.nr_sv[0] < 0)
    return fail(LSSVM_EINVAL,
                "%s: header needs svm_type, kernel_type, nr_class, total_sv, rho, label, nr_sv",
                path);
  if (h.kernel != LSSVM_LINEAR && !h.have_gamma)
    return fail(LSSVM_EINVAL, "%s: gamma missing for this kernel", path);
  if (h.nr_sv[0] + h.nr_sv[1] != h.total_sv)
    return fail(LSSVM_EINVAL, "%s: nr_sv does not add up to total_sv", path);
  h.sv_offset = std::min(q, m.size);
  h.sv_line = line;
  return LSSVM_OK;
}

// +1 when the first listed class is +1: the file's decision value
// sum coef_i k(x_i, x) - rho then is f(x) = sum alpha_i k(x_i, x) + b directly.
double orientation(const ModelHeader& h) { return h.label[0] == 1 ? 1.0 : -1.0; }

template <class T>
int write_model(const char* path, int32_t kernel, const lssvm_params& kp, double b,
                const T* alpha, const T* X, const T* y, int64_t n, int64_t d, int threads) {
  std::vector<int64_t> order;
  order.reserve(size_t(n));
  for (int64_t i = 0; i < n; ++i) {
    if (y[i] != T(1) && y[i] != T(-1)) return fail(LSSVM_EBADLABEL, "labels must be +1 or -1");
    if (y[i] == T(1)) order.push_back(i);
  }
  int64_t npos = int64_t(order.size());
  for (int64_t i = 0; i < n; ++i)
    if (y[i] == T(-1)) order.push_back(i);
  std::string hd = "svm_type c_svc\nkernel_type ";
  hd += kernel == LSSVM_LINEAR ? "linear\n" : kernel == LSSVM_POLY ? "polynomial\n" : "rbf\n";
  if (kernel == LSSVM_POLY) hd += "degree " + std::to_string(kp.degree) + "\n";
  if (kernel != LSSVM_LINEAR) hd += "gamma " + fmt_double(kp.gamma) + "\n";
  if (kernel == LSSVM_POLY) hd += "coef0 " + fmt_double(kp.coef0) + "\n";
  hd += "nr_class 2\ntotal_sv " + std::to_string(n) + "\nrho " + fmt_double(-b) +
        "\nlabel 1 -1\nnr_sv " + std::to_string(npos) + " " + std::to_string(n - npos) + "\nSV\n";
  int parts = int(std::max<int64_t>(1, std::min<int64_t>(threads, n)));
  std::vector<OutBuf> bufs(parts);
  parallel_for(parts, [&](int t) {
    int64_t r0 = n * t / parts, r1 = n * (t + 1) / parts;
    for (int64_t k = r0; k < r1; ++k) {
      int64_t i = order[size_t(k)];
      format_row(bufs[t], alpha[i], X + i * d, d);
    }
  });
  return write_file(path, hd, bufs);
}

int scan_model(const char* path, int32_t* kernel, lssvm_params* kp, double* b, int64_t* n_out,
               int64_t* d_out, int threads) {
  MappedFile m;
  int rc = map_file(path, m);
  if (rc != LSSVM_OK) return rc;
  ModelHeader h;
  if ((rc = parse_header(m, path, h)) != LSSVM_OK) return rc;
  std::vector<size_t> bounds;
  std::vector<RangeStats> st;
  if ((rc = scan_lines(m, h.sv_offset, threads, h.sv_line, path, bounds, st)) != LSSVM_OK)
    return rc;
  int64_t points = 0, dmax = 0;
  for (const auto& r : st) {
    points += r.points;
    dmax = std::max(dmax, r.max_index);
  }
  if (points != h.total_sv)
    return fail(LSSVM_EINVAL, "%s: total_sv is %lld but %lld support vectors follow", path,
                (long long)h.total_sv, (long long)points);
  *kernel = h.kernel;
  *kp = h.kp;
  *b = -orientation(h) * h.rho;
  *n_out = points;
  *d_out = dmax;
  return LSSVM_OK;
}

template <class T>
int read_model(const char* path, T* X, T* alpha, T* y, int64_t n, int64_t d, int threads) {
  MappedFile m;
  int rc = map_file(path, m);
  if (rc != LSSVM_OK) return rc;
  ModelHeader h;
  if ((rc = parse_header(m, path, h)) != LSSVM_OK) return rc;
  if (h.total_sv != n)
    return fail(LSSVM_EINVAL, "%s holds %lld support vectors, n is %lld", path,
                (long long)h.total_sv, (long long)n);
  std::vector<size_t> bounds;
  std::vector<RangeStats> st;
  if ((rc = scan_lines(m, h.sv_offset, threads, h.sv_line, path, bounds, st)) != LSSVM_OK)
    return rc;
  int64_t points = 0;
  for (const auto& r : st) points += r.points;
  if (points != n)
    return fail(LSSVM_EINVAL, "%s: total_sv is %lld but %lld support vectors follow", path,
                (long long)n, (long long)points);
  if (n == 0) return LSSVM_OK;
  if ((rc = parse_lines(m, bounds, st, h.sv_line, path, X, alpha, d)) != LSSVM_OK) return rc;
  const T s = T(orientation(h));
  const T first = T(h.label[0]), second = T(h.label[1]);
  for (int64_t i = 0; i < n; ++i) {
    alpha[i] *= s;
    y[i] = i < h.nr_sv[0] ? first : second;
  }
  return LSSVM_OK;
}

// ------------------------------------------------------------------- checks --

int check_dims(int64_t n, int64_t d, bool allow_empty) {
  if (n < (allow_empty ? 0 : 1))
    return fail(LSSVM_EINVAL, "n must be >= 1 (got %lld)", (long long)n);
  if (d < 0 || d > kMaxDim) return fail(LSSVM_EINVAL, "d out of range (got %lld)", (long long)d);
  if (n > 0 && d > 0 && n > std::numeric_limits<int64_t>::max() / d)
    return fail(LSSVM_EINVAL, "n * d overflows");
  return LSSVM_OK;
}

bool valid_dtype(int32_t t) { return t == LSSVM_F64 || t == LSSVM_F32; }

template <class F>
int guarded(F&& f) {
  clear_error();
  try {
    return f();
  } catch (const std::bad_alloc&) {
    return fail(LSSVM_EINVAL, "out of host memory");
  } catch (const std::exception& e) {
    return fail(LSSVM_EINVAL, "%s", e.what());
  }
}

}  // namespace
}  // namespace lssvm

using namespace lssvm;

extern "C" {

int lssvm_libsvm_scan(const char* path, int64_t* n_out, int64_t* d_out, int32_t num_threads) {
  return guarded([&] {
    if (!n_out || !d_out) return fail(LSSVM_EINVAL, "NULL output argument");
    MappedFile m;
    int rc = map_file(path, m);
    if (rc != LSSVM_OK) return rc;
    int64_t points = 0, dmax = 0;
    if (m.size) {
      std::vector<size_t> bounds;
      std::vector<RangeStats> st;
      rc = scan_lines(m, 0, resolve_threads(num_threads), 0, path, bounds, st);
      if (rc != LSSVM_OK) return rc;
      for (const auto& r : st) {
        points += r.points;
        dmax = std::max(dmax, r.max_index);
      }
    }
    if (dmax > kMaxDim) return fail(LSSVM_EINVAL, "%s: feature index too large", path);
    *n_out = points;
    *d_out = dmax;
    return int(LSSVM_OK);
  });
}

int lssvm_libsvm_read(const char* path, int32_t dtype, void* X, void* y, int64_t n, int64_t d,
                      int32_t num_threads) {
  return guarded([&] {
    if (!valid_dtype(dtype)) return fail(LSSVM_EINVAL, "unknown dtype %d", int(dtype));
    int rc = check_dims(n, d, true);
    if (rc != LSSVM_OK) return rc;
    if (n > 0 && (!y || (d > 0 && !X))) return fail(LSSVM_EINVAL, "NULL array argument");
    int nt = resolve_threads(num_threads);
    return dtype == LSSVM_F64
               ? read_data(path, static_cast<double*>(X), static_cast<double*>(y), n, d, nt)
               : read_data(path, static_cast<float*>(X), static_cast<float*>(y), n, d, nt);
  });
}

int lssvm_libsvm_write(const char* path, int32_t dtype, const void* X, const void* y, int64_t n,
                       int64_t d, int32_t num_threads) {
  return guarded([&] {
    if (!path) return fail(LSSVM_EINVAL, "path is NULL");
    if (!valid_dtype(dtype)) return fail(LSSVM_EINVAL, "unknown dtype %d", int(dtype));
    int rc = check_dims(n, d, true);
    if (rc != LSSVM_OK) return rc;
    if (n > 0 && (!y || (d > 0 && !X))) return fail(LSSVM_EINVAL, "NULL array argument");
    int nt = resolve_threads(num_threads);
    return dtype == LSSVM_F64 ? write_data(path, static_cast<const double*>(X),
                                           static_cast<const double*>(y), n, d, nt)
                              : write_data(path, static_cast<const float*>(X),
                                           static_cast<const float*>(y), n, d, nt);
  });
}

int lssvm_model_write(const char* path, int32_t dtype, int32_t kernel, const lssvm_params* kp,
                      double b, const void* alpha, const void* X, const void* y, int64_t n,
                      int64_t d, int32_t num_threads) {
  return guarded([&] {
    if (!path) return fail(LSSVM_EINVAL, "path is NULL");
    if (!valid_dtype(dtype)) return fail(LSSVM_EINVAL, "unknown dtype %d", int(dtype));
    if (kernel != LSSVM_LINEAR && kernel != LSSVM_POLY && kernel != LSSVM_RBF)
      return fail(LSSVM_EINVAL, "unknown kernel %d", int(kernel));
    lssvm_params p{1.0, 0.0, 1};
    if (kernel != LSSVM_LINEAR) {
      if (!kp) return fail(LSSVM_EINVAL, "kernel parameters required for kernel %d", int(kernel));
      p = *kp;
      if (!(std::isfinite(p.gamma) && p.gamma > 0))
        return fail(LSSVM_EINVAL, "gamma must be finite and > 0 (got %g)", p.gamma);
      if (kernel == LSSVM_POLY && (p.degree < 1 || !std::isfinite(p.coef0)))
        return fail(LSSVM_EINVAL, "degree must be >= 1 and coef0 finite");
    }
    if (!std::isfinite(b)) return fail(LSSVM_EINVAL, "b must be finite");
    int rc = check_dims(n, d, false);
    if (rc != LSSVM_OK) return rc;
    if (!alpha || !y || (d > 0 && !X)) return fail(LSSVM_EINVAL, "NULL array argument");
    int nt = resolve_threads(num_threads);
    return dtype == LSSVM_F64
               ? write_model(path, kernel, p, b, static_cast<const double*>(alpha),
                             static_cast<const double*>(X), static_cast<const double*>(y), n, d,
                             nt)
               : write_model(path, kernel, p, b, static_cast<const float*>(alpha),
                             static_cast<const float*>(X), static_cast<const float*>(y), n, d, nt);
  });
}

int lssvm_model_scan(const char* path, int32_t* kernel, lssvm_params* kp, double* b,
                     int64_t* n_out, int64_t* d_out) {
  return guarded([&] {
    if (!kernel || !kp || !b || !n_out || !d_out) return fail(LSSVM_EINVAL, "NULL output argument");
    return scan_model(path, kernel, kp, b, n_out, d_out, resolve_threads(0));
  });
}

int lssvm_model_read(const char* path, int32_t dtype, void* X, void* alpha, void* y, int64_t n,
                     int64_t d, int32_t num_threads) {
  return guarded([&] {
    if (!valid_dtype(dtype)) return fail(LSSVM_EINVAL, "unknown dtype %d", int(dtype));
    int rc = check_dims(n, d, true);
    if (rc != LSSVM_OK) return rc;
    if (n > 0 && (!alpha || !y || (d > 0 && !X))) return fail(LSSVM_EINVAL, "NULL array argument");
    int nt = resolve_threads(num_threads);
    return dtype == LSSVM_F64 ? read_model(path, static_cast<double*>(X),
                                           static_cast<double*>(alpha), static_cast<double*>(y),
                                           n, d, nt)
                              : read_model(path, static_cast<float*>(X),
                                           static_cast<float*>(alpha), static_cast<float*>(y), n,
                                           d, nt);
  });
}

}  // extern "C"
