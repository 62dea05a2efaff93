// Reader of sparse multi-label datasets in the text format of the Extreme
// Classification Repository, the source of the paper's datasets (Sec. 5.1,
// Table 1; they are stored in libSVM format): an optional header line
// "n_rows n_features n_labels", then one row per line,
//     l1,l2,...  f1:v1 f2:v2 ...
// (comma-separated label ids, possibly none, then feature:value pairs).  Two
// calls: asgd_libsvm_scan sizes the arrays, asgd_libsvm_read fills them; rows
// are sorted by feature id and by label id.
#include <errno.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include <algorithm>
#include <string>
#include <utility>
#include <vector>

#include "../../include/asgd.h"

namespace asgd {
asgd_status set_error(asgd_status s, const char* msg);
}

namespace {

asgd_status io_fail(asgd_status s, const std::string& msg) { return asgd::set_error(s, msg.c_str()); }

struct Parsed {
  std::vector<int32_t> labels;
  std::vector<std::pair<int32_t, float>> feats;
};

// One data line; false (with *why set) on a syntax error.
bool parse_line(const char* p, int one_based, Parsed* out, const char** why) {
  out->labels.clear();
  out->feats.clear();
  while (*p == ' ' || *p == '\t') ++p;
  // labels: a comma-separated list before the first space, unless the first
  // token is already a feature (contains ':')
  const char* tok_end = p;
  while (*tok_end && *tok_end != ' ' && *tok_end != '\t' && *tok_end != '\n' && *tok_end != '\r') ++tok_end;
  const bool first_is_feature = memchr(p, ':', (size_t)(tok_end - p)) != nullptr;
  if (!first_is_feature) {
    while (p < tok_end) {
      char* e = nullptr;
      errno = 0;
      const long v = strtol(p, &e, 10);
      if (e == p || errno || v < 0 || v > INT32_MAX) {
        *why = "bad label id";
        return false;
      }
      out->labels.push_back((int32_t)v);
      p = e;
      if (p < tok_end) {
        if (*p != ',') {
          *why = "labels must be separated by commas";
          return false;
        }
        ++p;
      }
    }
  }
  for (;;) {
    while (*p == ' ' || *p == '\t') ++p;
    if (!*p || *p == '\n' || *p == '\r' || *p == '#') break;
    char* e = nullptr;
    errno = 0;
    long f = strtol(p, &e, 10);
    if (e == p || *e != ':' || errno) {
      *why = "expected feature:value";
      return false;
    }
    f -= one_based ? 1 : 0;
    if (f < 0 || f > INT32_MAX) {
      *why = "feature id out of range";
      return false;
    }
    p = e + 1;
    errno = 0;
    const float v = strtof(p, &e);
    if (e == p || errno) {
      *why = "bad feature value";
      return false;
    }
    out->feats.emplace_back((int32_t)f, v);
    p = e;
  }
  return true;
}

// Reads the file line by line: calls on_header(n, F, L) for a header line
// and on_row(parsed) for every data row.
template <typename H, typename R>
asgd_status scan_file(const char* path, int one_based, H on_header, R on_row) {
  FILE* f = fopen(path, "rb");
  if (!f) return io_fail(ASGD_EINVAL, std::string("cannot open ") + path);
  std::string line;
  std::vector<char> buf(1 << 16);
  Parsed row;
  int64_t lineno = 0;
  bool first = true;
  asgd_status st = ASGD_OK;
  for (;;) {
    line.clear();
    bool got = false;
    while (fgets(buf.data(), (int)buf.size(), f)) {
      got = true;
      line += buf.data();
      if (!line.empty() && line.back() == '\n') break;
    }
    if (!got) break;
    ++lineno;
    const char* s = line.c_str();
    while (*s == ' ' || *s == '\t') ++s;
    if (!*s || *s == '\n' || *s == '\r' || *s == '#') continue;
    if (first) {
      first = false;
      long long a = 0, b = 0, c = 0;
      char tail = 0;
      if (sscanf(s, "%lld %lld %lld %c", &a, &b, &c, &tail) == 3 && !strchr(s, ':') && !strchr(s, ',')) {
        on_header(a, b, c);
        continue;
      }
    }
    const char* why = nullptr;
    if (!parse_line(s, one_based, &row, &why)) {
      st = io_fail(ASGD_EINVAL, std::string(path) + ":" + std::to_string(lineno) + ": " + why);
      break;
    }
    st = on_row(row, lineno);
    if (st) break;
  }
  fclose(f);
  return st;
}

}  // namespace

extern "C" {

asgd_status asgd_libsvm_scan(const char* path, int32_t one_based, asgd_libsvm_info* info) {
  if (!path || !info) return io_fail(ASGD_EINVAL, "NULL argument");
  *info = asgd_libsvm_info{};
  int64_t hdr[3] = {-1, -1, -1};
  int64_t max_f = -1, max_l = -1;
  asgd_status s = scan_file(
      path, one_based, [&](long long a, long long b, long long c) { hdr[0] = a, hdr[1] = b, hdr[2] = c; },
      [&](const Parsed& r, int64_t) {
        ++info->n_rows;
        info->nnz += (int64_t)r.feats.size();
        info->label_nnz += (int64_t)r.labels.size();
        for (const auto& fv : r.feats) max_f = std::max<int64_t>(max_f, fv.first);
        for (int32_t l : r.labels) max_l = std::max<int64_t>(max_l, l);
        return ASGD_OK;
      });
  if (s) return s;
  info->n_features = hdr[1] >= 0 ? hdr[1] : max_f + 1;
  info->n_labels = hdr[2] >= 0 ? hdr[2] : max_l + 1;
  info->header_rows = hdr[0];
  if (max_f >= info->n_features || max_l >= info->n_labels)
    return io_fail(ASGD_EINVAL, std::string(path) + ": an id exceeds the header's feature or label count");
  if (hdr[0] >= 0 && hdr[0] != info->n_rows)
    return io_fail(ASGD_EINVAL, std::string(path) + ": the header's row count does not match the rows");
  return ASGD_OK;
}

asgd_status asgd_libsvm_read(const char* path, int32_t one_based, const asgd_libsvm_info* info,
                             int64_t* indptr, int32_t* indices, float* values, int64_t* label_indptr,
                             int32_t* label_indices) {
  if (!path || !info || !indptr || !label_indptr || (info->nnz && (!indices || !values)) ||
      (info->label_nnz && !label_indices))
    return io_fail(ASGD_EINVAL, "NULL argument");
  int64_t r = 0, q = 0, ql = 0;
  indptr[0] = 0;
  label_indptr[0] = 0;
  std::vector<std::pair<int32_t, float>> fs;
  std::vector<int32_t> ls;
  asgd_status s = scan_file(
      path, one_based, [](long long, long long, long long) {},
      [&](const Parsed& p, int64_t lineno) {
        if (r >= info->n_rows || q + (int64_t)p.feats.size() > info->nnz ||
            ql + (int64_t)p.labels.size() > info->label_nnz)
          return io_fail(ASGD_ESTATE, std::string(path) + ": the file changed since it was scanned");
        fs = p.feats;
        ls = p.labels;
        std::sort(fs.begin(), fs.end(), [](const auto& a, const auto& b) { return a.first < b.first; });
        std::sort(ls.begin(), ls.end());
        for (size_t k = 1; k < fs.size(); ++k)
          if (fs[k].first == fs[k - 1].first)
            return io_fail(ASGD_EINVAL, std::string(path) + ":" + std::to_string(lineno) + ": repeated feature id");
        for (size_t k = 1; k < ls.size(); ++k)
          if (ls[k] == ls[k - 1])
            return io_fail(ASGD_EINVAL, std::string(path) + ":" + std::to_string(lineno) + ": repeated label id");
        for (const auto& fv : fs) {
          indices[q] = fv.first;
          values[q] = fv.second;
          ++q;
        }
        for (int32_t l : ls) label_indices[ql++] = l;
        ++r;
        indptr[r] = q;
        label_indptr[r] = ql;
        return ASGD_OK;
      });
  if (s) return s;
  if (r != info->n_rows || q != info->nnz || ql != info->label_nnz)
    return io_fail(ASGD_ESTATE, std::string(path) + ": the file changed since it was scanned");
  return ASGD_OK;
}

}  // extern "C"
