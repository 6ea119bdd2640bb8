// Privacy accounting with an envelope CDF (appendix: Algorithm accounting and the
// binning of the envelope law that feeds it), fp64.
//
// * envelope_bins_kernel: the envelope law of Y as bins.  From F(y_0..y_M) on an
//   even grid it takes the running maximum (a CDF evaluated numerically may dip),
//   clips to [0, 1], takes the increments as bin weights, clamps them at zero,
//   normalises them to sum to one, and puts each bin's weight at its midpoint.
// * pld_survival_kernel: one subsampled step's privacy-loss survival function
//   S(t) = P(L > t) at the cut points t = (c - n + 1/2) h, c = 0 .. 2n - 1.  With
//   amplification by subsampling at rate p, S(t) = p betabar(t + s(t)) +
//   (1 - p) alpha(t + s(t)), s(t) = log(1/p - (1-p)/p e^-t), above the support
//   bound log(1 - p), and S = 1 at and below it.  alpha and betabar are the
//   Gaussian test errors at signal-to-noise mu = a / sigma averaged over the
//   envelope bins with a_i = 1 / sqrt(ybar_i) (or a = 1 without an envelope):
//   alpha(u) = sum_i w_i Phi(-u/mu_i - mu_i/2), betabar(u) = sum_i w_i Phi(-u/mu_i + mu_i/2).
//   One thread per cut point; the bins are summed in bin order.
// * pld_masses_kernel: cell masses of the grid t_j = (j - n + 1) h, j < 2n - 1,
//   as decrements of S between the cuts around each cell (clamped at zero); the
//   mass below the first cut joins the lowest cell, S at the last cut is the atom
//   at +infinity; everything is normalised to total one.
// * pld_fold_kernel: after a linear convolution of two such distributions (an FFT
//   product computed by the caller), negatives are clipped, the centred L cells
//   are kept, mass below them is folded into the lowest cell, mass above joins the
//   +infinity atom (whose mass composes as 1 - (1 - a)(1 - b)), and the finite
//   cells are rescaled so that the total stays one.
// * pld_delta_kernel: delta(eps) = sum over t_j >= eps of q_j (1 - e^(eps - t_j))
//   plus the atom, clipped to [0, 1], for a batch of eps values (one workgroup each).
//
// Every reduction runs in one workgroup in a fixed order, so results are
// deterministic.  Phi is the standard normal CDF, 0.5 erfc(-x / sqrt 2).
#include <algorithm>
#include "device.hpp"
#include "kernels.hpp"

namespace dprc {

constexpr int kPldBlock = 1024;

__device__ __forceinline__ double norm_cdf(double x) { return 0.5 * erfc(-x * 0.70710678118654752440); }

// Sum of the workgroup's `v` (fixed order: lanes within each wave, then waves in order).
__device__ double block_sum(double v, double* red) {
  v = wave_sum(v);
  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6, nw = blockDim.x >> 6;
  __syncthreads();
  if (lane == 0) red[wv] = v;
  __syncthreads();
  double s = 0.0;
  for (int q = 0; q < nw; ++q) s += red[q];
  return s;
}

__global__ __launch_bounds__(kPldBlock) void envelope_bins_kernel(const double* F, int32_t M, double y_min,
                                                                  double y_max, double* ybar, double* w) {
  __shared__ double cmax[kPldBlock];
  __shared__ double red[kPldBlock / 64];
  const int tid = threadIdx.x;
  const int64_t npts = (int64_t)M + 1;
  const int64_t chunk = (npts + kPldBlock - 1) / kPldBlock;
  const int64_t b0 = tid * chunk, b1 = min(npts, b0 + chunk);
  // running maximum: each thread's chunk maximum, then a prefix maximum over the chunks
  double m = -INFINITY;
  for (int64_t j = b0; j < b1; ++j) m = fmax(m, F[j]);
  cmax[tid] = m;
  __syncthreads();
  for (int off = 1; off < kPldBlock; off <<= 1) {   // inclusive prefix maximum (Hillis-Steele)
    const double o = tid >= off ? cmax[tid - off] : -INFINITY;
    __syncthreads();
    cmax[tid] = fmax(cmax[tid], o);
    __syncthreads();
  }
  const double before = tid > 0 ? cmax[tid - 1] : -INFINITY;
  // weights of bins j = b0 .. b1 - 1 (bin j spans points j, j + 1); a chunk's last bin
  // needs the next chunk's first point, which the running maximum through it gives
  double run = before, local = 0.0;
  for (int64_t j = b0; j < b1 && j < M; ++j) {
    run = fmax(run, F[j]);
    const double g0 = fmin(fmax(run, 0.0), 1.0);
    const double g1 = fmin(fmax(fmax(run, F[j + 1]), 0.0), 1.0);
    const double wj = fmax(g1 - g0, 0.0);
    w[j] = wj;
    local += wj;
  }
  const double tot = block_sum(local, red);
  const double step = (y_max - y_min) / (double)M;
  for (int64_t j = b0; j < b1 && j < M; ++j) {
    w[j] = w[j] / tot;
    ybar[j] = y_min + ((double)j + 0.5) * step;
  }
}

__global__ void pld_survival_kernel(PldArgs a) {
  const int64_t c = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (c >= 2 * a.n) return;
  const double t = ((double)(c - a.n) + 0.5) * a.h;
  double S = 1.0;
  if (t > a.t_min) {
    const double u = a.p < 1.0 ? t + log(1.0 / a.p - (1.0 - a.p) / a.p * exp(-t)) : t;
    double al = 0.0, beb = 0.0;
    if (a.n_bins == 0) {
      const double mu = 1.0 / a.sigma;
      al = norm_cdf(-u / mu - 0.5 * mu);
      beb = norm_cdf(-u / mu + 0.5 * mu);
    } else {
      for (int32_t i = 0; i < a.n_bins; ++i) {
        const double wi = a.w[i];
        if (wi == 0.0) continue;
        const double mu = 1.0 / (sqrt(a.ybar[i]) * a.sigma);
        al += wi * norm_cdf(-u / mu - 0.5 * mu);
        beb += wi * norm_cdf(-u / mu + 0.5 * mu);
      }
    }
    S = a.p * beb + (1.0 - a.p) * al;
  }
  a.S[c] = S;
}

__global__ __launch_bounds__(kPldBlock) void pld_masses_kernel(PldArgs a) {
  __shared__ double red[kPldBlock / 64];
  const int64_t L = 2 * a.n - 1;
  const int64_t chunk = (L + kPldBlock - 1) / kPldBlock;
  const int64_t b0 = threadIdx.x * chunk, b1 = min(L, b0 + chunk);
  double local = 0.0;
  for (int64_t j = b0; j < b1; ++j) {
    double qj = fmax(a.S[j] - a.S[j + 1], 0.0);
    if (j == 0) qj += fmax(1.0 - a.S[0], 0.0);      // below the first cut
    a.q[j] = qj;
    local += qj;
  }
  const double atom = fmax(a.S[2 * a.n - 1], 0.0);  // above the last cut
  const double tot = block_sum(local, red) + atom;
  for (int64_t j = b0; j < b1; ++j) a.q[j] /= tot;
  if (threadIdx.x == 0) a.q_inf[0] = atom / tot;
}

__global__ __launch_bounds__(kPldBlock) void pld_fold_kernel(const double* r, int64_t L, const double* ainf,
                                                             const double* binf, double* q, double* q_inf) {
  __shared__ double red[kPldBlock / 64];
  const int64_t n = 2 * L - 1, c = (L - 1) / 2;       // r[j] sits at cell j - c of the kept grid
  const int64_t chunk = (n + kPldBlock - 1) / kPldBlock;
  const int64_t b0 = threadIdx.x * chunk, b1 = min(n, b0 + chunk);
  double below = 0.0, kept = 0.0, above = 0.0;
  for (int64_t j = b0; j < b1; ++j) {
    const double v = fmax(r[j], 0.0);
    if (j < c) below += v;
    else if (j < c + L) kept += v;
    else above += v;
  }
  below = block_sum(below, red);
  kept = block_sum(kept, red);
  above = block_sum(above, red);
  const double inf0 = 1.0 - (1.0 - ainf[0]) * (1.0 - binf[0]);
  const double fin = below + kept + above;
  const double scale = fin > 0.0 ? (1.0 - inf0) / fin : 0.0;
  for (int64_t j = max(b0, c); j < min(b1, c + L); ++j) {
    double v = fmax(r[j], 0.0);
    if (j == c) v += below;
    q[j - c] = v * scale;
  }
  if (threadIdx.x == 0) q_inf[0] = fin > 0.0 ? inf0 + above * scale : inf0;
}

__global__ __launch_bounds__(256) void pld_delta_kernel(const double* q, int64_t L, double h, const double* q_inf,
                                                        const double* eps, double* delta) {
  __shared__ double red[4];
  const double e = eps[blockIdx.x];
  const int64_t c = (L - 1) / 2;
  double s = 0.0;
  for (int64_t j = threadIdx.x; j < L; j += blockDim.x) {
    const double t = (double)(j - c) * h;
    if (t >= e) s += q[j] * (1.0 - exp(e - t));
  }
  const double tot = block_sum(s, red) + q_inf[0];
  if (threadIdx.x == 0) delta[blockIdx.x] = fmin(fmax(tot, 0.0), 1.0);
}

hipError_t launch_envelope_bins(const double* F, int32_t M, double y_min, double y_max, double* ybar, double* w,
                                hipStream_t st) {
  DPRC_LAUNCH(envelope_bins_kernel, dim3(1), dim3(kPldBlock), 0, st, F, M, y_min, y_max, ybar, w);
  return hipGetLastError();
}

hipError_t launch_pld_step(const PldArgs& a, hipStream_t st) {
  DPRC_LAUNCH(pld_survival_kernel, dim3((unsigned)ceil_div(2 * a.n, 256)), dim3(256), 0, st, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  DPRC_LAUNCH(pld_masses_kernel, dim3(1), dim3(kPldBlock), 0, st, a);
  return hipGetLastError();
}

hipError_t launch_pld_fold(const double* r, int64_t L, const double* ainf, const double* binf, double* q,
                           double* q_inf, hipStream_t st) {
  DPRC_LAUNCH(pld_fold_kernel, dim3(1), dim3(kPldBlock), 0, st, r, L, ainf, binf, q, q_inf);
  return hipGetLastError();
}

hipError_t launch_pld_delta(const double* q, int64_t L, double h, const double* q_inf, const double* eps,
                            int32_t n_eps, double* delta, hipStream_t st) {
  DPRC_LAUNCH(pld_delta_kernel, dim3((unsigned)n_eps), dim3(256), 0, st, q, L, h, q_inf, eps, delta);
  return hipGetLastError();
}

}  // namespace dprc
