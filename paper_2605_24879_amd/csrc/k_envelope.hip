// Envelope CDF of the Hutchinson estimate (privacy analysis, proposition on the
// extremal envelope; appendix algorithms cdf-grid and binary-search-xplus).
//
// MiddleRegionCDF(x): the largest P(S <= x) over the two-level forms
//   S(i, j, lam) = lam/(ik) chi^2(ik) + (1-lam)/(jk) chi^2(jk),
//   i, j >= 1, i + j <= d, lam = l / (2 (n_lambda - 1)), l = 0 .. n_lambda - 1.
// One thread per candidate (i, j, l) and point x (fp64).  A candidate's CDF is
// the convolution integral over the first term written in s = sqrt(v) (v the
// chi^2(ik) variable), where the chi density has a bulk of constant width:
//   P(S <= x) = int 2 s f_{ik}(s^2) P_reg(jk/2, (x - a s^2)/(2b)) ds,
// a = lam/(ik), b = (1-lam)/(jk), over [max(0, sqrt(ik) - 10), min(sqrt(x/a),
// sqrt(ik) + 10)] by composite Gauss-Legendre (16 panels of 16 nodes; nodes
// and weights computed on the host).  lam = 0 reduces to one regularised
// incomplete gamma.  P_reg(a, y) is the power series for y < a + 1 and
// Lentz's evaluation of the Legendre continued fraction for the complement
// otherwise (Press et al., Numerical Recipes, incomplete gamma function).
// Workgroups reduce (value, candidate index) pairs to the largest value with
// the smallest index; a second kernel reduces the workgroup results in order.
#include <algorithm>
#include "device.hpp"
#include "kernels.hpp"

namespace dprc {

constexpr int kEnvBlock = 256;

__device__ double gamma_p(double a, double y) {
  if (y <= 0.0) return 0.0;
  const double lpre = -y + a * log(y) - lgamma(a);
  if (y < a + 1.0) {
    double ap = a, term = 1.0 / a, sum = term;
    for (int n = 0; n < 100000; ++n) {
      ap += 1.0;
      term *= y / ap;
      sum += term;
      if (fabs(term) < fabs(sum) * 1e-17) break;
    }
    return fmin(1.0, sum * exp(lpre));
  }
  const double tiny = 1e-300;
  double b = y + 1.0 - a, c = 1.0 / tiny, d = 1.0 / b, h = d;
  for (int i = 1; i < 100000; ++i) {
    const double an = -i * (i - a);
    b += 2.0;
    d = an * d + b;
    if (fabs(d) < tiny) d = tiny;
    c = b + an / c;
    if (fabs(c) < tiny) c = tiny;
    d = 1.0 / d;
    const double del = d * c;
    h *= del;
    if (fabs(del - 1.0) < 1e-16) break;
  }
  return fmax(0.0, 1.0 - exp(lpre) * h);
}

__device__ double two_level_cdf(double x, int i, int j, double lam, int k, const EnvArgs& g) {
  const int panels = g.panels;
  if (x <= 0.0) return 0.0;
  const double n1 = (double)i * k, n2 = (double)j * k;
  const double b = (1.0 - lam) / n2;
  if (lam == 0.0) return gamma_p(n2 / 2.0, x / (2.0 * b));
  const double a = lam / n1;
  const double smax = sqrt(x / a), c = sqrt(n1);
  const double lo = fmax(0.0, c - 10.0), hi = fmin(smax, c + 10.0);
  if (hi <= lo) return 0.0;
  // log of the chi density 2 s f_{n1}(s^2) = 2 s^(n1-1) e^(-s^2/2) / (2^(n1/2) Gamma(n1/2))
  const double lc = log(2.0) - (n1 / 2.0) * log(2.0) - lgamma(n1 / 2.0);
  // When the range runs to the end of the support (s = sqrt(x/a)) the second CDF
  // vanishes there like (sqrt(x/a) - s)^(n2/2); with s = sqrt(x/a) - t^2 the
  // integrand is smooth in t for every n2.
  const bool edge = hi >= smax;
  const double tlo = edge ? 0.0 : lo, thi = edge ? sqrt(smax - lo) : hi;
  const double pw = (thi - tlo) / panels;
  double sum = 0.0;
  for (int pn = 0; pn < panels; ++pn) {
    const double mid = tlo + (pn + 0.5) * pw, half = 0.5 * pw;
    double ps = 0.0;
#pragma unroll 4
    for (int q = 0; q < kEnvNodes; ++q) {
      const double t = mid + half * g.gx[q];
      const double s = edge ? smax - t * t : t;
      const double jac = edge ? 2.0 * t : 1.0;
      if (s <= 0.0) continue;
      const double dens = exp(lc + (n1 - 1.0) * log(s) - 0.5 * s * s);
      const double rest = x - a * s * s;
      if (rest <= 0.0) continue;
      ps += g.gw[q] * jac * dens * gamma_p(n2 / 2.0, rest / (2.0 * b));
    }
    sum += half * ps;
  }
  return fmin(fmax(sum, 0.0), 1.0);
}

// candidate c -> (i, j, l): pairs in (i, then j) order, lam index fastest
__device__ void candidate(int64_t c, int d, int nl, int& i, int& j, int& l) {
  l = (int)(c % nl);
  int64_t pr = c / nl;
  // row i (1-based) holds d - i pairs; offset(i) = (i-1) d - (i-1) i / 2
  int lo = 1, hi = d - 1;
  while (lo < hi) {
    const int m = (lo + hi + 1) / 2;
    const int64_t off = (int64_t)(m - 1) * d - (int64_t)(m - 1) * m / 2;
    if (off <= pr) lo = m;
    else hi = m - 1;
  }
  i = lo;
  j = 1 + (int)(pr - ((int64_t)(i - 1) * d - (int64_t)(i - 1) * i / 2));
}

__device__ __forceinline__ void better(double v, int64_t c, double& bv, int64_t& bc) {
  if (v > bv || (v == bv && c < bc)) { bv = v; bc = c; }
}

__global__ __launch_bounds__(kEnvBlock) void env_middle_kernel(EnvArgs a) {
  __shared__ double sv[kEnvBlock];
  __shared__ int64_t sc[kEnvBlock];
  const int xi = blockIdx.y;
  const double x = a.x[xi];
  double bv = -1.0;
  int64_t bc = INT64_MAX;
  for (int64_t c = (int64_t)blockIdx.x * kEnvBlock + threadIdx.x; c < a.ncand;
       c += (int64_t)gridDim.x * kEnvBlock) {
    int i, j, l;
    candidate(c, a.d, a.n_lambda, i, j, l);
    const double lam = a.n_lambda > 1 ? 0.5 * l / (a.n_lambda - 1) : 0.0;
    better(two_level_cdf(x, i, j, lam, a.k, a), c, bv, bc);
  }
  sv[threadIdx.x] = bv;
  sc[threadIdx.x] = bc;
  __syncthreads();
  for (int off = kEnvBlock / 2; off > 0; off >>= 1) {
    if (threadIdx.x < off) {
      double v = sv[threadIdx.x];
      int64_t c = sc[threadIdx.x];
      better(sv[threadIdx.x + off], sc[threadIdx.x + off], v, c);
      sv[threadIdx.x] = v;
      sc[threadIdx.x] = c;
    }
    __syncthreads();
  }
  if (threadIdx.x == 0) {
    a.part_v[(int64_t)xi * gridDim.x + blockIdx.x] = sv[0];
    a.part_c[(int64_t)xi * gridDim.x + blockIdx.x] = sc[0];
  }
}

__global__ void env_reduce_kernel(EnvArgs a, int nblk) {
  const int xi = blockIdx.x * blockDim.x + threadIdx.x;
  if (xi >= a.nx) return;
  double bv = -1.0;
  int64_t bc = INT64_MAX;
  for (int b = 0; b < nblk; ++b) better(a.part_v[(int64_t)xi * nblk + b], a.part_c[(int64_t)xi * nblk + b], bv, bc);
  a.best[xi] = bv;
  if (a.arg) {
    int i, j, l;
    candidate(bc, a.d, a.n_lambda, i, j, l);
    a.arg[3 * xi] = i;
    a.arg[3 * xi + 1] = j;
    a.arg[3 * xi + 2] = l;
  }
}

__global__ void chi2_cdf_kernel(const double* x, int64_t n, double dof, double scale, double* out) {
  for (int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; e < n; e += (int64_t)gridDim.x * blockDim.x)
    out[e] = gamma_p(dof / 2.0, x[e] * scale / 2.0);
}

hipError_t launch_chi2_cdf(const double* x, int64_t n, double dof, double scale, double* out, hipStream_t st) {
  if (n <= 0) return hipSuccess;
  const unsigned blocks = (unsigned)std::min<int64_t>(4096, ceil_div(n, 256));
  DPRC_LAUNCH(chi2_cdf_kernel, dim3(blocks), dim3(256), 0, st, x, n, dof, scale, out);
  return hipGetLastError();
}

int env_blocks(int64_t ncand) { return (int)std::min<int64_t>(2048, ceil_div(ncand, kEnvBlock)); }

hipError_t launch_env_middle(const EnvArgs& a, hipStream_t st) {
  const int nblk = env_blocks(a.ncand);
  DPRC_LAUNCH(env_middle_kernel, dim3((unsigned)nblk, (unsigned)a.nx), dim3(kEnvBlock), 0, st, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  DPRC_LAUNCH(env_reduce_kernel, dim3((unsigned)ceil_div(a.nx, 64)), dim3(64), 0, st, a, nblk);
  return hipGetLastError();
}

}  // namespace dprc
