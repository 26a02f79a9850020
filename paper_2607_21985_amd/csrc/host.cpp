// Host side of libspdp: the Tiled-CBC encoder (Sec. 4.1), global magnitude
// pruning (Sec. 2.2), TEAL-style threshold calibration (Sec. 5.1), the
// integer threshold code the kernels compare against, and error reporting.
// Plain C++17: no HIP headers, so this file also builds with g++ alone.

#include <algorithm>
#include <atomic>
#include <cmath>
#include <cstring>
#include <new>
#include <thread>

#include "internal.h"

namespace spdp {

namespace {

thread_local std::string g_last_error;

// Runs fn(i) for i in [0, n) on up to hardware_concurrency() threads (at most
// 16), handing out indices dynamically so that uneven items balance.
template <class Fn>
void parallel_for(int64_t n, Fn fn) {
  unsigned hw = std::thread::hardware_concurrency();
  int64_t nt = std::min<int64_t>({n, (int64_t)(hw ? hw : 1), 16});
  if (nt <= 1) {
    for (int64_t i = 0; i < n; ++i) fn(i);
    return;
  }
  std::atomic<int64_t> next{0};
  auto worker = [&]() {
    for (int64_t i = next.fetch_add(1); i < n; i = next.fetch_add(1)) fn(i);
  };
  std::vector<std::thread> pool;
  pool.reserve(nt - 1);
  for (int64_t t = 1; t < nt; ++t) pool.emplace_back(worker);
  worker();
  for (auto& th : pool) th.join();
}

// Exact value of an IEEE binary16 bit pattern.
double half_value(uint16_t h) {
  const int e = (h >> 10) & 0x1F;
  const int f = h & 0x3FF;
  double v;
  if (e == 0)
    v = std::ldexp((double)f, -24);
  else if (e == 31)
    v = f ? NAN : INFINITY;
  else
    v = std::ldexp((double)(f | 0x400), e - 25);
  return (h & 0x8000) ? -v : v;
}

constexpr uint32_t kMagInf = 0x7C00;  // magnitude bits of +-inf; above: NaN

bool valid_tile(int32_t tile_m, int32_t tile_k) {
  return tile_m >= 64 && tile_m <= 256 && tile_m % 64 == 0 && tile_k >= 1 &&
         tile_k <= 256 && (tile_k & (tile_k - 1)) == 0 &&
         (int64_t)(tile_k - 1) * tile_m <= 0xFFFF;
}

}  // namespace

int fail(int status, const std::string& detail) {
  g_last_error = detail;
  return status;
}

void clear_error() { g_last_error.clear(); }

// Tiled-CBC encoder. Row stripes are independent, so each worker takes one
// stripe at a time: it transposes the stripe into a column-major buffer
// (blocked, so the row-major reads stay contiguous), then walks the GTiles of
// the stripe left to right and each GTile's columns left to right, building
// the bitmap words, ColInfo entries and the packed, 8-element-padded values.
// A serial prefix sum over GTile sizes gives TileOffset, and the per-stripe
// value runs are then copied into place in parallel.
namespace {

int check_shape(const uint16_t* W, int64_t rows, int64_t cols, int32_t tile_m, int32_t tile_k) {
  if (!W) return fail(SPDP_ERR_INVALID_ARG, "W is NULL");
  if (rows < 1 || cols < 1) return fail(SPDP_ERR_INVALID_ARG, "rows and cols must be >= 1");
  if (!valid_tile(tile_m, tile_k)) {
    if (tile_m > 256 && tile_m <= 1024 && tile_m % 64 == 0)
      return fail(SPDP_ERR_UNSUPPORTED, "tile_m above 256 is not supported by this library");
    return fail(SPDP_ERR_INVALID_ARG,
                "tile_m must be a multiple of 64 in [64, 256] and tile_k a power of two in [1, 256]");
  }
  if ((rows + tile_m - 1) / tile_m > 65535) return fail(SPDP_ERR_UNSUPPORTED, "more than 65535 row stripes");
  if ((cols + tile_k - 1) / tile_k * tile_k > (int64_t)1 << 31) return fail(SPDP_ERR_UNSUPPORTED, "too many columns");
  return SPDP_OK;
}

// The stripe walk for either value type: T = uint16_t (fp16 bits, columns
// padded to 8 elements) or int8_t (codes, padded to 16); both pads are 16
// bytes. value_of(row, h) is the element stored for the nonzero of `row`
// whose fp16 bits are h (it is also called, and its result discarded, for
// zeros and for the padding rows past the last one).
template <typename T, typename ValueOf>
int walk(const uint16_t* W, int64_t rows, int64_t cols, int32_t tile_m, int32_t tile_k, ValueOf value_of,
         spdp_matrix* m, std::vector<T>* values) {
  constexpr uint32_t kPad = 16 / sizeof(T);
  const int64_t R = (rows + tile_m - 1) / tile_m;
  const int64_t C = (cols + tile_k - 1) / tile_k;
  const int64_t NGT = R * C;
  const int wpc = tile_m / 64;
  const int64_t kpad = C * tile_k;

  try {
    m->col_info.assign((size_t)(NGT * tile_k), 0u);
    m->bitmap.assign((size_t)(NGT * tile_k * wpc), 0ull);
    m->tile_offset.assign((size_t)(NGT + 1), 0u);
  } catch (const std::bad_alloc&) {
    return fail(SPDP_ERR_OOM, "host allocation for the format arrays failed");
  }
  std::vector<std::vector<T>> stripe_vals((size_t)R);
  std::vector<uint64_t> gtile_size((size_t)NGT, 0);
  std::atomic<bool> oom{false};

  parallel_for(R, [&](int64_t r) {
    std::vector<uint16_t> colbuf;
    std::vector<T> vals;
    try {
      colbuf.assign((size_t)(kpad * tile_m), 0);
      vals.resize((size_t)(kpad * tile_m));
    } catch (const std::bad_alloc&) {
      oom = true;
      return;
    }
    const int64_t m0 = r * tile_m;
    const int64_t mrows = std::min<int64_t>(tile_m, rows - m0);
    for (int64_t kb = 0; kb < cols; kb += 64) {
      const int64_t kn = std::min<int64_t>(64, cols - kb);
      for (int64_t i = 0; i < mrows; ++i) {
        const uint16_t* src = W + (m0 + i) * cols + kb;
        uint16_t* dst = colbuf.data() + kb * tile_m + i;
        for (int64_t k = 0; k < kn; ++k) dst[k * tile_m] = src[k];
      }
    }
    size_t pos = 0;
    for (int64_t c = 0; c < C; ++c) {
      const int64_t g = r * C + c;
      uint32_t off = 0;
      for (int j = 0; j < tile_k; ++j) {
        const int64_t k = c * tile_k + j;
        const uint16_t* col = colbuf.data() + k * tile_m;
        uint32_t nnz = 0;
        for (int w = 0; w < wpc; ++w) {
          uint64_t word = 0;
          for (int i = 0; i < 64; ++i) {
            const uint16_t h = col[64 * w + i];
            const uint64_t nz = (h & 0x7FFF) != 0;
            word |= nz << i;
            vals[pos] = value_of(m0 + 64 * w + i, h);
            pos += nz;
          }
          m->bitmap[(size_t)((g * tile_k + j) * wpc + w)] = word;
          nnz += (uint32_t)__builtin_popcountll(word);
        }
        const uint32_t padded = (nnz + kPad - 1) & ~(kPad - 1);
        for (uint32_t z = nnz; z < padded; ++z) vals[pos++] = 0;
        m->col_info[(size_t)(g * tile_k + j)] = (off << 16) | nnz;
        off += padded;
      }
      gtile_size[(size_t)g] = off;
    }
    vals.resize(pos);
    vals.shrink_to_fit();
    stripe_vals[(size_t)r] = std::move(vals);
  });
  if (oom) return fail(SPDP_ERR_OOM, "host allocation during encoding failed");

  uint64_t total = 0;
  for (int64_t g = 0; g < NGT; ++g) {
    total += gtile_size[(size_t)g];
    if (total > 0xFFFFFFFFull)
      return fail(SPDP_ERR_UNSUPPORTED, "encoded matrix would hold 2^32 or more values");
    m->tile_offset[(size_t)(g + 1)] = (uint32_t)total;
  }
  try {
    values->resize((size_t)total);
  } catch (const std::bad_alloc&) {
    return fail(SPDP_ERR_OOM, "host allocation for values failed");
  }
  parallel_for(R, [&](int64_t r) {
    const auto& v = stripe_vals[(size_t)r];
    if (!v.empty())
      std::memcpy(values->data() + m->tile_offset[(size_t)(r * C)], v.data(), v.size() * sizeof(T));
  });
  m->rows = rows;
  m->cols = cols;
  m->tile_m = tile_m;
  m->tile_k = tile_k;
  m->n_stripes = R;
  m->n_colblocks = C;
  m->n_gtiles = NGT;
  return SPDP_OK;
}

}  // namespace

int encode_host_arrays(const uint16_t* W, int64_t rows, int64_t cols,
                       int32_t tile_m, int32_t tile_k, spdp_matrix* m) {
  const int st = check_shape(W, rows, cols, tile_m, tile_k);
  if (st != SPDP_OK) return st;
  m->value_bits = 16;
  return walk<uint16_t>(W, rows, cols, tile_m, tile_k, [](int64_t, uint16_t h) { return h; }, m, &m->values);
}

// Round-to-nearest quantization after pruning (Sec. 5.1 quantization setup:
// symmetric, one scale per row): s = fp32(max |w| of the row's nonzeros) /
// (2^(bits-1) - 1), code = clamp(rint(fp32(w) / s)) with fp32 division and
// ties to even; the sparsity pattern stays the pruning's (a nonzero whose
// code is 0 is still stored), and a row with no nonzero has scale 0.
int encode_host_arrays_rtn(const uint16_t* W, int64_t rows, int64_t cols,
                           int32_t tile_m, int32_t tile_k, int32_t bits, spdp_matrix* m) {
  int st = check_shape(W, rows, cols, tile_m, tile_k);
  if (st != SPDP_OK) return st;
  if (bits < 2 || bits > 8) return fail(SPDP_ERR_INVALID_ARG, "bits must be in [2, 8]");
  const float qmax = (float)((1 << (bits - 1)) - 1);
  try {
    m->scales.assign((size_t)rows, 0.0f);
  } catch (const std::bad_alloc&) {
    return fail(SPDP_ERR_OOM, "host allocation for the scales failed");
  }
  std::atomic<bool> non_finite{false};
  parallel_for(rows, [&](int64_t r) {
    float amax = 0.0f;
    for (int64_t k = 0; k < cols; ++k) {
      const uint16_t h = W[r * cols + k];
      if ((h & 0x7FFF) == 0) continue;
      if ((h & 0x7C00) == 0x7C00) {
        non_finite = true;
        return;
      }
      amax = std::max(amax, (float)std::fabs(half_value(h)));
    }
    m->scales[(size_t)r] = amax / qmax;
  });
  if (non_finite) return fail(SPDP_ERR_INVALID_ARG, "weights must be finite (inf or NaN found)");
  const float* sc = m->scales.data();
  auto code = [sc, rows, qmax](int64_t row, uint16_t h) -> int8_t {
    const float s = sc[std::min(row, rows - 1)];
    if ((h & 0x7FFF) == 0 || !(s > 0.0f)) return 0;
    const float q = std::nearbyint((float)half_value(h) / s);
    return (int8_t)std::min(std::max(q, -qmax), qmax);
  };
  m->value_bits = bits;
  return walk<int8_t>(W, rows, cols, tile_m, tile_k, code, m, &m->codes);
}

}  // namespace spdp

using spdp::fail;
using spdp::half_value;
using spdp::kMagInf;
using spdp::parallel_for;

extern "C" {

const char* spdp_strerror(int status) {
  switch (status) {
    case SPDP_OK: return "success";
    case SPDP_ERR_INVALID_ARG: return "invalid argument";
    case SPDP_ERR_UNSUPPORTED: return "unsupported";
    case SPDP_ERR_OOM: return "out of memory";
    case SPDP_ERR_HIP: return "HIP runtime error";
    default: return "unknown status";
  }
}

const char* spdp_last_error(void) { return spdp::g_last_error.c_str(); }

int spdp_encode_host(const uint16_t* W, int64_t rows, int64_t cols,
                     int32_t tile_m, int32_t tile_k, spdp_handle_t* out) {
  spdp::clear_error();
  if (!out) return fail(SPDP_ERR_INVALID_ARG, "out is NULL");
  *out = nullptr;
  spdp_matrix* m = new (std::nothrow) spdp_matrix();
  if (!m) return fail(SPDP_ERR_OOM, "host allocation failed");
  const int st = spdp::encode_host_arrays(W, rows, cols, tile_m, tile_k, m);
  if (st != SPDP_OK) {
    delete m;
    return st;
  }
  *out = m;
  return SPDP_OK;
}

int spdp_encode_rtn_host(const uint16_t* W, int64_t rows, int64_t cols, int32_t tile_m, int32_t tile_k,
                         int32_t bits, spdp_handle_t* out) {
  spdp::clear_error();
  if (!out) return fail(SPDP_ERR_INVALID_ARG, "out is NULL");
  *out = nullptr;
  spdp_matrix* m = new (std::nothrow) spdp_matrix();
  if (!m) return fail(SPDP_ERR_OOM, "host allocation failed");
  const int st = spdp::encode_host_arrays_rtn(W, rows, cols, tile_m, tile_k, bits, m);
  if (st != SPDP_OK) {
    delete m;
    return st;
  }
  *out = m;
  return SPDP_OK;
}

int spdp_format(spdp_handle_t h, spdp_format_t* out) {
  spdp::clear_error();
  if (!h || !out) return fail(SPDP_ERR_INVALID_ARG, "handle or out is NULL");
  out->rows = h->rows;
  out->cols = h->cols;
  out->tile_m = h->tile_m;
  out->tile_k = h->tile_k;
  out->n_stripes = h->n_stripes;
  out->n_colblocks = h->n_colblocks;
  out->n_gtiles = h->n_gtiles;
  const bool q = h->value_bits < 16;
  out->n_values = (int64_t)(q ? h->codes.size() : h->values.size());
  out->tile_offset = h->tile_offset.data();
  out->col_info = h->col_info.data();
  out->bitmap = h->bitmap.data();
  out->values = q ? nullptr : h->values.data();
  out->d_tile_offset = h->d_tile_offset;
  out->d_col_info = h->d_col_info;
  out->d_bitmap = h->d_bitmap;
  out->d_values = h->d_values;
  out->device = h->device;
  out->value_bits = h->value_bits;
  out->codes = q ? h->codes.data() : nullptr;
  out->scales = q ? h->scales.data() : nullptr;
  out->d_scales = h->d_scales;
  return SPDP_OK;
}

// Magnitude order of non-NaN fp16 values is the order of their magnitude bits,
// so a 31745-bin histogram of (h & 0x7FFF) locates the pruning cut exactly.
// Entries below the cut are zeroed; entries equal to the cut are zeroed in
// index order until the count is met (each worker learns how many tied entries
// precede its chunk from a prefix sum over chunks).
int spdp_prune_magnitude(const uint16_t* W, int64_t n, double sparsity, uint16_t* out) {
  spdp::clear_error();
  if (!W || !out) return fail(SPDP_ERR_INVALID_ARG, "W or out is NULL");
  if (n < 0) return fail(SPDP_ERR_INVALID_ARG, "n must be >= 0");
  if (!(sparsity >= 0.0 && sparsity <= 1.0))
    return fail(SPDP_ERR_INVALID_ARG, "sparsity must lie in [0, 1]");
  const int64_t n_prune = (int64_t)std::floor(sparsity * (double)n);
  const int64_t chunk = 1 << 22;
  const int64_t nchunks = (n + chunk - 1) / chunk;
  std::vector<std::vector<int64_t>> hist((size_t)nchunks);
  std::atomic<bool> has_nan{false};
  parallel_for(nchunks, [&](int64_t c) {
    auto& hc = hist[(size_t)c];
    hc.assign(kMagInf + 1, 0);
    const int64_t e = std::min(n, (c + 1) * chunk);
    for (int64_t i = c * chunk; i < e; ++i) {
      const uint32_t mag = W[i] & 0x7FFF;
      if (mag > kMagInf) {
        has_nan = true;
        return;
      }
      hc[mag]++;
    }
  });
  if (has_nan) return fail(SPDP_ERR_INVALID_ARG, "W contains NaN");
  if (out != W) std::memcpy(out, W, (size_t)n * sizeof(uint16_t));
  if (n_prune == 0) return SPDP_OK;
  std::vector<int64_t> total(kMagInf + 1, 0);
  for (const auto& hc : hist)
    for (uint32_t b = 0; b <= kMagInf; ++b) total[b] += hc[b];
  uint32_t cut = 0;
  int64_t below = 0;
  while (below + total[cut] < n_prune) below += total[cut++];
  const int64_t tie_quota = n_prune - below;  // tied entries to zero, lowest index first
  std::vector<int64_t> ties_before((size_t)nchunks + 1, 0);
  for (int64_t c = 0; c < nchunks; ++c) ties_before[(size_t)c + 1] = ties_before[(size_t)c] + hist[(size_t)c][cut];
  parallel_for(nchunks, [&](int64_t c) {
    int64_t tie_idx = ties_before[(size_t)c];
    const int64_t e = std::min(n, (c + 1) * chunk);
    for (int64_t i = c * chunk; i < e; ++i) {
      const uint32_t mag = W[i] & 0x7FFF;
      if (mag < cut) {
        out[i] = 0;
      } else if (mag == cut) {
        if (tie_idx < tie_quota) out[i] = 0;
        ++tie_idx;
      }
    }
  });
  return SPDP_OK;
}

int spdp_calibrate_threshold(const uint16_t* X, int64_t n, double p, float* t) {
  spdp::clear_error();
  if (!t || (!X && n > 0)) return fail(SPDP_ERR_INVALID_ARG, "X or t is NULL");
  if (n < 0) return fail(SPDP_ERR_INVALID_ARG, "n must be >= 0");
  if (!(p >= 0.0 && p <= 1.0)) return fail(SPDP_ERR_INVALID_ARG, "p must lie in [0, 1]");
  std::vector<int64_t> hist(kMagInf + 1, 0);
  for (int64_t i = 0; i < n; ++i) {
    const uint32_t mag = X[i] & 0x7FFF;
    if (mag > kMagInf) return fail(SPDP_ERR_INVALID_ARG, "X contains NaN");
    hist[mag]++;
  }
  if (p == 0.0 || n == 0) {
    *t = -1.0f;
    return SPDP_OK;
  }
  const int64_t idx = (int64_t)std::ceil(p * (double)n) - 1;  // 0-based rank in ascending |X|
  uint32_t code = 0;
  int64_t seen = 0;
  while (seen + hist[code] <= idx) seen += hist[code++];
  *t = (float)half_value((uint16_t)code);
  return SPDP_OK;
}

int spdp_threshold_code(float threshold, int32_t* code) {
  spdp::clear_error();
  if (!code) return fail(SPDP_ERR_INVALID_ARG, "code is NULL");
  if (std::isnan(threshold)) return fail(SPDP_ERR_INVALID_ARG, "threshold is NaN");
  if (threshold < 0.0f) {
    *code = -1;
    return SPDP_OK;
  }
  // largest magnitude pattern h in [0, 0x7C00] whose value is <= threshold
  const double t = threshold;
  uint32_t lo = 0, hi = kMagInf;  // invariant: value(lo) <= t
  while (lo < hi) {
    const uint32_t mid = (lo + hi + 1) / 2;
    if (half_value((uint16_t)mid) <= t)
      lo = mid;
    else
      hi = mid - 1;
  }
  *code = (int32_t)lo;
  return SPDP_OK;
}

}  // extern "C"
