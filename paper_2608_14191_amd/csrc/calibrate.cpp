// Host-side calibration of one (KV head, tensor): Algorithm 1 (calibration part),
// Sec. 5.1 (decorrelating transform, PCA form of App. D) and Sec. 5.2 (attention-aware
// reverse water-filling and per-channel scales).  Pure C++17, fp64.
#include <algorithm>
#include <cmath>
#include <cstring>
#include <numeric>
#include <queue>
#include <vector>

#include "aatc.h"
#include "params.h"

// The percentile interpolation and the scale reciprocals are defined as separate
// IEEE operations; keep the compiler from fusing them.
#pragma clang fp contract(off)

namespace aatc {

// Round a double to fp16 bits, nearest-even, saturating at +-65504.
uint16_t f64_to_f16_bits(double v) {
  uint16_t sign = std::signbit(v) ? 0x8000 : 0;
  double a = std::fabs(v);
  if (std::isnan(v)) return 0x7e00;
  if (a >= 65504.0) return sign | 0x7bff;
  if (a == 0.0) return sign;
  int e;
  double m = std::frexp(a, &e);          // a = m * 2^e, m in [0.5, 1)
  int exp16 = e - 1 + 15;                // biased exponent of a normal fp16
  double scaled;
  if (exp16 >= 1) {
    scaled = std::ldexp(m, 11);          // 11 significant bits: [1024, 2048)
  } else {
    scaled = std::ldexp(a, 24);          // subnormal: units of 2^-24
    exp16 = 0;
  }
  double fl = std::floor(scaled);
  double frac = scaled - fl;
  uint32_t q = (uint32_t)fl;
  if (frac > 0.5 || (frac == 0.5 && (q & 1u))) q += 1;
  if (exp16 == 0) {
    // subnormal (q <= 1024; q == 1024 is the smallest normal)
    return sign | (uint16_t)q;
  }
  if (q == 2048) {                       // rounding carried into the next binade
    q = 1024;
    exp16 += 1;
  }
  if (exp16 >= 31) return sign | 0x7bff;
  return sign | (uint16_t)((exp16 << 10) | (q - 1024));
}

double f16_bits_to_f64(uint16_t h) {
  int e = (h >> 10) & 0x1f;
  int m = h & 0x3ff;
  double v;
  if (e == 0) v = std::ldexp((double)m, -24);
  else if (e == 31) v = m ? NAN : INFINITY;
  else v = std::ldexp((double)(m | 0x400), e - 25);
  return (h & 0x8000) ? -v : v;
}

namespace {

// Cyclic Jacobi eigendecomposition of a symmetric n x n matrix (row-major, destroyed).
// On success: w = eigenvalues (unsorted), V columns = orthonormal eigenvectors.
bool jacobi_eigen(std::vector<double>& a, int n, std::vector<double>& v,
                  std::vector<double>& w) {
  v.assign((size_t)n * n, 0.0);
  for (int i = 0; i < n; ++i) v[(size_t)i * n + i] = 1.0;
  bool converged = false;
  for (int sweep = 0; sweep < 100; ++sweep) {
    double off = 0.0, diag = 0.0;
    for (int p = 0; p < n; ++p) {
      diag += a[(size_t)p * n + p] * a[(size_t)p * n + p];
      for (int q = p + 1; q < n; ++q) off += a[(size_t)p * n + q] * a[(size_t)p * n + q];
    }
    if (off <= 1e-32 * diag || off == 0.0) {
      converged = true;
      break;
    }
    for (int p = 0; p < n - 1; ++p) {
      for (int q = p + 1; q < n; ++q) {
        double apq = a[(size_t)p * n + q];
        if (apq == 0.0) continue;
        double app = a[(size_t)p * n + p], aqq = a[(size_t)q * n + q];
        double theta = (aqq - app) / (2.0 * apq);
        double t = (theta >= 0 ? 1.0 : -1.0) / (std::fabs(theta) + std::sqrt(theta * theta + 1.0));
        double c = 1.0 / std::sqrt(t * t + 1.0), s = t * c;
        // A <- J^T A J on the symmetric matrix: rows p and q (contiguous) for k != p, q,
        // mirrored into columns p and q; then the 2 x 2 block.
        double* ap = &a[(size_t)p * n];
        double* aq = &a[(size_t)q * n];
        for (int k = 0; k < n; ++k) {
          if (k == p || k == q) continue;
          const double apk = ap[k], aqk = aq[k];
          const double np_ = c * apk - s * aqk, nq = s * apk + c * aqk;
          ap[k] = np_;
          aq[k] = nq;
          a[(size_t)k * n + p] = np_;
          a[(size_t)k * n + q] = nq;
        }
        const double npp = c * c * app - 2.0 * s * c * apq + s * s * aqq;
        const double nqq = s * s * app + 2.0 * s * c * apq + c * c * aqq;
        ap[p] = npp;
        aq[q] = nqq;
        ap[q] = 0.0;
        aq[p] = 0.0;
        // V <- V J, with V held transposed (row i = eigenvector column i): rows p and q.
        double* vp = &v[(size_t)p * n];
        double* vq = &v[(size_t)q * n];
        for (int k = 0; k < n; ++k) {
          const double vkp = vp[k], vkq = vq[k];
          vp[k] = c * vkp - s * vkq;
          vq[k] = s * vkp + c * vkq;
        }
      }
    }
  }
  w.resize(n);
  for (int i = 0; i < n; ++i) w[i] = a[(size_t)i * n + i];
  // back to V columns = eigenvectors
  for (int i = 0; i < n; ++i)
    for (int k = i + 1; k < n; ++k) std::swap(v[(size_t)i * n + k], v[(size_t)k * n + i]);
  return converged;
}

// numpy's "linear" percentile of an ascending array: virtual index (n-1) q, then
// lerp(a, b, t) = a + (b-a) t for t < 1/2, b - (b-a)(1-t) otherwise.
double percentile_linear(const std::vector<double>& sorted, double q) {
  size_t n = sorted.size();
  double vi = (double)(n - 1) * q;
  double lo = std::floor(vi);
  size_t i = (size_t)lo;
  if (i >= n - 1) return sorted[n - 1];
  double t = vi - lo;
  double a = sorted[i], b = sorted[i + 1];
  double diff = b - a;
  if (t >= 0.5) {
    double u = diff * (1.0 - t);
    return b - u;
  }
  double u = diff * t;
  return a + u;
}

}  // namespace
}  // namespace aatc

using namespace aatc;

namespace {

// The calibration of aatc_calibrate; with `bits_given` (eigen order) the widths are taken
// as they are instead of allocated, and a nonzero `record_bytes_given` pads the records.
// With `gram` the d x d matrix whose eigenvectors form the basis is given (instead of the
// covariance of the samples) and the samples are `x64` (fp64) instead of `x_calib`.
// Out is aatc_calibration (one KV head, d = 128) or aatc_group_calibration (a head group,
// d = 128 gkv up to 512); the transform is stored densely with row stride d.
template <class Out>
aatc_status calibrate_impl(const float* x_calib, int64_t n_calib, int32_t d,
                           const float* q_calib, int64_t n_q, int32_t q_group,
                           const float* w_o, int32_t d_out, double avg_bits, int32_t b_max,
                           const uint8_t* bits_given, int32_t record_bytes_given,
                           double percentile, Out* out,
                           const double* gram = nullptr, const double* x64 = nullptr) {
  constexpr int kMaxDim = (int)(sizeof(out->bits) / sizeof(out->bits[0]));
  try {
    if ((!x_calib && !x64) || !out) return AATC_E_INVALID;
    if (kMaxDim == AATC_HEAD_DIM ? d != AATC_HEAD_DIM
                                 : (d < AATC_HEAD_DIM || d > kMaxDim || d % AATC_HEAD_DIM))
      return AATC_E_UNSUPPORTED;
    if (n_calib < 2 || b_max < 1 || b_max > AATC_MAX_BITS) return AATC_E_INVALID;
    if (!(percentile > 0.0 && percentile <= 1.0)) return AATC_E_INVALID;
    if (q_calib && w_o) return AATC_E_INVALID;
    if (q_calib && (q_group < 1 || n_q < q_group || n_q % q_group != 0)) return AATC_E_INVALID;
    if (w_o && d_out < 1) return AATC_E_INVALID;
    int64_t budget = 0;
    if (bits_given) {
      for (int c = 0; c < d; ++c) {
        if (bits_given[c] > b_max) return AATC_E_INVALID;
        budget += bits_given[c];
      }
      if (budget < 1) return AATC_E_INVALID;
    } else {
      if (!(avg_bits > 0.0) || !std::isfinite(avg_bits)) return AATC_E_INVALID;
      budget = (int64_t)std::floor(avg_bits * d + 0.5);
      if (budget < 1 || budget > (int64_t)d * b_max) return AATC_E_INVALID;
    }
    const int32_t min_rb = (int32_t)(4 * ((budget + 31) / 32));
    if (record_bytes_given != 0 &&
        (record_bytes_given < min_rb || record_bytes_given % 4 != 0 ||
         record_bytes_given > d * AATC_MAX_BITS / 8))
      return AATC_E_INVALID;

    const size_t n = (size_t)n_calib;
    auto sample = [&](size_t i, int j) -> double {
      return x64 ? x64[i * d + j] : (double)x_calib[i * d + j];
    };
    for (size_t i = 0; i < n * d; ++i)
      if (!std::isfinite(sample(i / d, (int)(i % d)))) return AATC_E_NUMERIC;

    // 1. Sigma = X^T X / n (fp64, uncentered), or the given matrix.
    std::vector<double> sigma((size_t)d * d, 0.0);
    if (gram) {
      std::copy(gram, gram + (size_t)d * d, sigma.begin());
    } else {
      std::vector<double> row(d);
      for (size_t i = 0; i < n; ++i) {
        for (int j = 0; j < d; ++j) row[j] = sample(i, j);
        for (int j = 0; j < d; ++j) {
          double xj = row[j];
          double* s = &sigma[(size_t)j * d];
          for (int k = j; k < d; ++k) s[k] += xj * row[k];
        }
      }
      for (int j = 0; j < d; ++j)
        for (int k = j; k < d; ++k) {
          double v = sigma[(size_t)j * d + k] / (double)n;
          sigma[(size_t)j * d + k] = v;
          sigma[(size_t)k * d + j] = v;
        }
    }

    // 2. Eigendecomposition, decreasing eigenvalues, canonical signs.
    std::vector<double> vec, lam_raw;
    if (!jacobi_eigen(sigma, d, vec, lam_raw)) return AATC_E_NUMERIC;
    std::vector<int> order(d);
    std::iota(order.begin(), order.end(), 0);
    std::stable_sort(order.begin(), order.end(),
                     [&](int a, int b) { return lam_raw[a] > lam_raw[b]; });
    std::vector<double> p((size_t)d * d), lam(d);   // p[j*d + c]
    for (int c = 0; c < d; ++c) {
      int src = order[c];
      lam[c] = lam_raw[src];
      int jmax = 0;
      double amax = -1.0;
      for (int j = 0; j < d; ++j) {
        double a = std::fabs(vec[(size_t)j * d + src]);
        if (a > amax) { amax = a; jmax = j; }
      }
      double sgn = vec[(size_t)jmax * d + src] < 0 ? -1.0 : 1.0;
      for (int j = 0; j < d; ++j) p[(size_t)j * d + c] = sgn * vec[(size_t)j * d + src];
    }

    // 3. Channel weights.
    std::vector<double> w(d, 1.0);
    if (q_calib) {
      for (int64_t i = 0; i < n_q * d; ++i)
        if (!std::isfinite(q_calib[i])) return AATC_E_NUMERIC;
      std::fill(w.begin(), w.end(), 0.0);
      const double t = (double)(n_q / q_group);
      for (int64_t i = 0; i < n_q; ++i) {
        const float* q = q_calib + i * d;
        for (int c = 0; c < d; ++c) {
          double acc = 0.0;
          for (int j = 0; j < d; ++j) acc += (double)q[j] * p[(size_t)j * d + c];
          w[c] += acc * acc;
        }
      }
      for (int c = 0; c < d; ++c) w[c] /= t;
    } else if (w_o) {
      for (int64_t i = 0; i < (int64_t)d * d_out; ++i)
        if (!std::isfinite(w_o[i])) return AATC_E_NUMERIC;
      for (int c = 0; c < d; ++c) {
        double acc2 = 0.0;
        for (int o = 0; o < d_out; ++o) {
          double acc = 0.0;
          for (int j = 0; j < d; ++j) acc += p[(size_t)j * d + c] * (double)w_o[(size_t)j * d_out + o];
          acc2 += acc * acc;
        }
        w[c] = acc2;
      }
    }

    // 4. Integer reverse water-filling: greedy marginal allocation (or the given widths).
    std::vector<double> wv(d);
    for (int c = 0; c < d; ++c) wv[c] = w[c] * lam[c];
    std::vector<int> b_eig(d, 0);
    if (bits_given)
      for (int c = 0; c < d; ++c) b_eig[c] = bits_given[c];
    for (int64_t step = 0; !bits_given && step < budget; ++step) {
      int best = -1;
      double gbest = 0.0;
      for (int c = 0; c < d; ++c) {
        if (b_eig[c] >= b_max) continue;
        double g = std::ldexp(wv[c], -2 * b_eig[c]);
        if (best < 0 || g > gbest) { best = c; gbest = g; }
      }
      b_eig[best] += 1;
    }

    // 5. Storage order: widest first, eigen order on ties.
    std::vector<int> perm(d);
    std::iota(perm.begin(), perm.end(), 0);
    std::stable_sort(perm.begin(), perm.end(),
                     [&](int a, int b) { return b_eig[a] > b_eig[b]; });

    std::memset(out, 0, sizeof(*out));
    out->d = d;
    out->budget_bits = (int32_t)budget;
    out->record_bytes = record_bytes_given ? record_bytes_given : min_rb;
    int d_active = 0;
    for (int c = 0; c < d; ++c) {
      int e = perm[c];
      out->perm[c] = e;
      out->bits[c] = (uint8_t)b_eig[e];
      if (b_eig[e] > 0) ++d_active;
      out->sigma2[c] = lam[c];
      out->weight[c] = w[c];
      out->bits_eig[c] = (uint8_t)b_eig[c];
      // The stored transform: each entry rounded to the nearest multiple of 2^-22 (ties
      // to even), exactly representable in fp32.
      for (int j = 0; j < d; ++j)
        out->transform[(size_t)j * d + c] =
            (float)std::ldexp(std::nearbyint(std::ldexp(p[(size_t)j * d + e], aatc::kTFrac)), -aatc::kTFrac);
    }
    out->d_active = d_active;

    // 6. Per-channel scales: percentile of |h_c| over the calibration tokens, fp16.
    std::vector<double> col(n);
    for (int c = 0; c < d; ++c) {
      if (out->bits[c] == 0) { out->scale_f16[c] = 0; continue; }
      int e = perm[c];
      for (size_t i = 0; i < n; ++i) {
        double acc = 0.0;
        for (int j = 0; j < d; ++j) acc += sample(i, j) * p[(size_t)j * d + e];
        col[i] = std::fabs(acc);
      }
      std::sort(col.begin(), col.end());
      out->scale_f16[c] = f64_to_f16_bits(percentile_linear(col, percentile));
    }
    return AATC_OK;
  } catch (...) {
    return AATC_E_INVALID;
  }
}

}  // namespace

extern "C" aatc_status aatc_calibrate_group(const float* x_calib, int64_t n_calib, int32_t d,
                                            const float* q_calib, int64_t n_q, int32_t q_group,
                                            const float* w_o, int32_t d_out, double avg_bits,
                                            int32_t b_max, double percentile,
                                            aatc_group_calibration* out) {
  return calibrate_impl(x_calib, n_calib, d, q_calib, n_q, q_group, w_o, d_out, avg_bits,
                        b_max, nullptr, 0, percentile, out);
}

extern "C" aatc_status aatc_calibrate(const float* x_calib, int64_t n_calib, int32_t d,
                                      const float* q_calib, int64_t n_q, int32_t q_group,
                                      const float* w_o, int32_t d_out, double avg_bits,
                                      int32_t b_max, double percentile,
                                      aatc_calibration* out) {
  return calibrate_impl(x_calib, n_calib, d, q_calib, n_q, q_group, w_o, d_out, avg_bits,
                        b_max, nullptr, 0, percentile, out);
}

namespace {

// Cholesky factor L (lower, row-major) of a symmetric positive definite n x n matrix;
// false if it is not numerically positive definite.
bool cholesky(const std::vector<double>& a, int n, std::vector<double>& l) {
  l.assign((size_t)n * n, 0.0);
  for (int j = 0; j < n; ++j) {
    double s = a[(size_t)j * n + j];
    for (int k = 0; k < j; ++k) s -= l[(size_t)j * n + k] * l[(size_t)j * n + k];
    if (!(s > 0.0) || !std::isfinite(s)) return false;
    const double d = std::sqrt(s);
    l[(size_t)j * n + j] = d;
    for (int i = j + 1; i < n; ++i) {
      double t = a[(size_t)i * n + j];
      for (int k = 0; k < j; ++k) t -= l[(size_t)i * n + k] * l[(size_t)j * n + k];
      l[(size_t)i * n + j] = t / d;
    }
  }
  return true;
}

}  // namespace

extern "C" aatc_status aatc_calibrate_whitened(const float* x_in, int64_t n_calib,
                                               int32_t d_model, const float* w_proj, int32_t d,
                                               const float* q_calib, int64_t n_q,
                                               int32_t q_group, const float* w_o,
                                               int32_t d_out, double avg_bits, int32_t b_max,
                                               double percentile, aatc_calibration* out) {
  try {
    if (!x_in || !w_proj || !out || d_model < 1) return AATC_E_INVALID;
    if (d != AATC_HEAD_DIM) return AATC_E_UNSUPPORTED;
    if (n_calib < 2) return AATC_E_INVALID;
    const size_t n = (size_t)n_calib, dm = (size_t)d_model;
    for (size_t i = 0; i < n * dm; ++i)
      if (!std::isfinite(x_in[i])) return AATC_E_NUMERIC;
    for (size_t i = 0; i < dm * d; ++i)
      if (!std::isfinite(w_proj[i])) return AATC_E_NUMERIC;
    // Sigma_X = X^T X / T (fp64, uncentered) and its Cholesky factor L.
    std::vector<double> sx(dm * dm, 0.0), row(dm);
    for (size_t i = 0; i < n; ++i) {
      for (size_t j = 0; j < dm; ++j) row[j] = x_in[i * dm + j];
      for (size_t j = 0; j < dm; ++j)
        for (size_t k = j; k < dm; ++k) sx[j * dm + k] += row[j] * row[k];
    }
    for (size_t j = 0; j < dm; ++j)
      for (size_t k = j; k < dm; ++k) {
        sx[j * dm + k] /= (double)n;
        sx[k * dm + j] = sx[j * dm + k];
      }
    std::vector<double> l;
    if (!cholesky(sx, d_model, l)) return AATC_E_NUMERIC;
    // The whitened weight W~ = L^T W and its Gram matrix W~^T W~: the right singular
    // vectors of W~ (the basis P) are its eigenvectors, the squared singular values its
    // eigenvalues.
    std::vector<double> wt(dm * d, 0.0);
    for (size_t j = 0; j < dm; ++j)
      for (size_t k = j; k < dm; ++k) {           // (L^T)_{jk} = L_{kj}, nonzero for k >= j
        const double lkj = l[k * dm + j];
        for (int c = 0; c < d; ++c) wt[j * d + c] += lkj * (double)w_proj[k * d + c];
      }
    std::vector<double> gram((size_t)d * d, 0.0);
    for (size_t j = 0; j < dm; ++j)
      for (int a = 0; a < d; ++a) {
        const double v = wt[j * d + a];
        for (int b = 0; b < d; ++b) gram[(size_t)a * d + b] += v * wt[j * d + b];
      }
    // The calibration samples of the cache, K = X W (fp64), for the channel scales.
    std::vector<double> k(n * d, 0.0);
    for (size_t i = 0; i < n; ++i)
      for (size_t j = 0; j < dm; ++j) {
        const double xv = x_in[i * dm + j];
        for (int c = 0; c < d; ++c) k[i * d + c] += xv * (double)w_proj[j * d + c];
      }
    return calibrate_impl(nullptr, n_calib, d, q_calib, n_q, q_group, w_o, d_out, avg_bits,
                          b_max, nullptr, 0, percentile, out, gram.data(), k.data());
  } catch (...) {
    return AATC_E_INVALID;
  }
}

extern "C" aatc_status aatc_calibrate_bits(const float* x_calib, int64_t n_calib, int32_t d,
                                           const float* q_calib, int64_t n_q, int32_t q_group,
                                           const float* w_o, int32_t d_out,
                                           const uint8_t* bits_eig, int32_t record_bytes,
                                           double percentile, aatc_calibration* out) {
  if (!bits_eig) return AATC_E_INVALID;
  return calibrate_impl(x_calib, n_calib, d, q_calib, n_q, q_group, w_o, d_out, 0.0,
                        AATC_MAX_BITS, bits_eig, record_bytes, percentile, out);
}

namespace aatc {
namespace {

// Greedy marginal allocation of `budget` bits over w_var[0..n): each bit goes to the
// channel of largest W_c 4^(-b_c) among those below b_max, the lowest index on ties.  A
// heap holds one entry per open channel with its current gain; ldexp keeps the gains
// exact, so the decisions are those of a scan for the first maximum.
void greedy_bits(const double* w_var, int64_t n, int64_t budget, int b_max, uint8_t* bits) {
  struct Entry { double gain; int64_t idx; };
  auto less = [](const Entry& a, const Entry& b) {
    return a.gain < b.gain || (a.gain == b.gain && a.idx > b.idx);
  };
  std::priority_queue<Entry, std::vector<Entry>, decltype(less)> heap(less);
  for (int64_t c = 0; c < n; ++c) {
    bits[c] = 0;
    heap.push({w_var[c], c});
  }
  for (int64_t step = 0; step < budget; ++step) {
    const Entry e = heap.top();
    heap.pop();
    const int b = ++bits[e.idx];
    if (b < b_max) heap.push({std::ldexp(w_var[e.idx], -2 * b), e.idx});
  }
}

}  // namespace
}  // namespace aatc

extern "C" aatc_status aatc_allocate_global(const double* sigma2, const double* weight,
                                            int32_t n_layers, int32_t m, double avg_bits,
                                            int32_t b_max, int32_t n_protect,
                                            int32_t protect_extra, int32_t normalize_weight,
                                            uint8_t* bits) {
  try {
    if (!sigma2 || !bits || n_layers < 1 || m < 1 || b_max < 1 || b_max > AATC_MAX_BITS ||
        n_protect < 0 || protect_extra < 0 || protect_extra > AATC_MAX_BITS ||
        !std::isfinite(avg_bits) || avg_bits < 0.0 || avg_bits > AATC_MAX_BITS)
      return AATC_E_INVALID;                       // (also keeps the budgets in int64)
    const int64_t n = (int64_t)n_layers * m;
    for (int64_t i = 0; i < n; ++i) {
      if (!(std::isfinite(sigma2[i]) && sigma2[i] >= 0.0)) return AATC_E_INVALID;
      if (weight && !(std::isfinite(weight[i]) && weight[i] >= 0.0)) return AATC_E_INVALID;
    }
    const int n_prot = std::min(n_protect, n_layers);
    const int64_t total = (int64_t)std::floor(avg_bits * m * n_layers + 0.5);
    const int64_t prot = (int64_t)std::floor((avg_bits + protect_extra) * m + 0.5);
    const int64_t rest = total - n_prot * prot;
    const int64_t cap = (int64_t)m * b_max;
    if (n_prot > 0 && prot > cap) return AATC_E_INVALID;
    if (n_layers > n_prot && (rest < 0 || rest > (n_layers - n_prot) * cap))
      return AATC_E_INVALID;
    // Per-layer scale: the layer's 95th percentile (linear interpolation), 1 if it is 0.
    auto layer_scale = [&](const double* a) {
      std::vector<double> v(a, a + m);
      std::sort(v.begin(), v.end());
      const double p = percentile_linear(v, 0.95);
      return p > 0.0 ? p : 1.0;
    };
    std::vector<double> w_var(n);
    for (int l = 0; l < n_layers; ++l) {
      const double* s2 = sigma2 + (int64_t)l * m;
      const double* w = weight ? weight + (int64_t)l * m : nullptr;
      const double ps = layer_scale(s2);
      const double pw = (w && normalize_weight) ? layer_scale(w) : 1.0;
      for (int c = 0; c < m; ++c) {
        const double wc = w ? (normalize_weight ? w[c] / pw : w[c]) : 1.0;
        w_var[(int64_t)l * m + c] = wc * (s2[c] / ps);
      }
    }
    for (int l = 0; l < n_prot; ++l)
      greedy_bits(w_var.data() + (int64_t)l * m, m, prot, b_max, bits + (int64_t)l * m);
    if (n_layers > n_prot)
      greedy_bits(w_var.data() + (int64_t)n_prot * m, n - (int64_t)n_prot * m, rest, b_max,
                  bits + (int64_t)n_prot * m);
    return AATC_OK;
  } catch (...) {
    return AATC_E_INVALID;
  }
}
