// Hutch++ pieces that are not token streams (Algorithm 2, Hutch++ branch):
//  * a batched Householder QR of the sketch O S (m x s per sample) giving the
//    orthonormal basis Q; Householder keeps Q orthonormal when O S is rank
//    deficient (a Gram/Cholesky QR would break down there);
//  * the finalize step V = W_P - U (Q^T P) and the estimate
//    ||U||_F^2 + ||V||_F^2 / r.
// Both are small (m * s and n * (s + r) per sample); one workgroup per sample,
// arithmetic in fp64.
#include <algorithm>
#include "device.hpp"
#include "kernels.hpp"

namespace dprc {

constexpr int kQrThreads = 256;
constexpr int kQrGroup = 16;  // columns reduced together

// Sum over the workgroup of v[0..cnt) (cnt <= kQrGroup); every thread gets the sums.
__device__ void block_sum_vec(double* v, int cnt, double* sh /*[4][kQrGroup]*/, double* out) {
  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
  for (int q = 0; q < cnt; ++q) {
    double x = wave_sum(v[q]);
    if (lane == 0) sh[wv * kQrGroup + q] = x;
  }
  __syncthreads();
  for (int q = 0; q < cnt; ++q) out[q] = (sh[q] + sh[kQrGroup + q]) + (sh[2 * kQrGroup + q] + sh[3 * kQrGroup + q]);
  __syncthreads();
}

__global__ __launch_bounds__(kQrThreads) void qr_kernel(const float* OS, int64_t os_ld, int64_t os_ss,
                                                         int32_t m, int32_t s, double* work, float* Q,
                                                         int64_t q_ld, int64_t q_ss, uint16_t* Qhi,
                                                         uint16_t* Qlo, int64_t qh_ld, int64_t qh_ss) {
  __shared__ double sh[4 * kQrGroup];
  __shared__ double tau[64];
  const int i = blockIdx.x, tid = threadIdx.x;
  double* R = work + (int64_t)i * 2 * s * m;   // [s][m]: the factorisation, then Householder vectors
  double* W = R + (int64_t)s * m;              // [s][m]: Q being formed
  const float* os = OS + (int64_t)i * os_ss;
  for (int c = 0; c < s; ++c)
    for (int j = tid; j < m; j += kQrThreads) R[(int64_t)c * m + j] = (double)os[(int64_t)c * os_ld + j];
  __syncthreads();

  double part[kQrGroup], tot[kQrGroup];
  for (int k = 0; k < s; ++k) {
    double* x = R + (int64_t)k * m;
    part[0] = 0.0;
    for (int j = k + tid; j < m; j += kQrThreads) part[0] += x[j] * x[j];
    block_sum_vec(part, 1, sh, tot);
    const double nrm2 = tot[0];
    const double x0 = x[k];
    __syncthreads();
    if (!(nrm2 > 0.0)) {  // zero column: identity reflector
      if (tid == 0) tau[k] = 0.0;
      __syncthreads();
      continue;
    }
    const double alpha = -copysign(sqrt(nrm2), x0);
    const double v0 = x0 - alpha;
    const double vn2 = nrm2 - x0 * x0 + v0 * v0;
    const double t = vn2 > 0.0 ? 2.0 / vn2 : 0.0;
    if (tid == 0) {
      tau[k] = t;
      x[k] = v0;
    }
    __syncthreads();
    for (int c0 = k + 1; c0 < s; c0 += kQrGroup) {
      const int cnt = min(kQrGroup, s - c0);
      for (int q = 0; q < cnt; ++q) part[q] = 0.0;
      for (int j = k + tid; j < m; j += kQrThreads) {
        const double vj = x[j];
        for (int q = 0; q < cnt; ++q) part[q] += vj * R[(int64_t)(c0 + q) * m + j];
      }
      block_sum_vec(part, cnt, sh, tot);
      for (int j = k + tid; j < m; j += kQrThreads) {
        const double vj = x[j];
        for (int q = 0; q < cnt; ++q) R[(int64_t)(c0 + q) * m + j] -= t * tot[q] * vj;
      }
      __syncthreads();
    }
  }
  // Q = H_0 H_1 ... H_{s-1} [I; 0]
  for (int c = 0; c < s; ++c)
    for (int j = tid; j < m; j += kQrThreads) W[(int64_t)c * m + j] = (j == c) ? 1.0 : 0.0;
  __syncthreads();
  for (int k = s - 1; k >= 0; --k) {
    const double t = tau[k];
    if (t == 0.0) continue;
    const double* v = R + (int64_t)k * m;
    for (int c0 = 0; c0 < s; c0 += kQrGroup) {
      const int cnt = min(kQrGroup, s - c0);
      for (int q = 0; q < cnt; ++q) part[q] = 0.0;
      for (int j = k + tid; j < m; j += kQrThreads) {
        const double vj = v[j];
        for (int q = 0; q < cnt; ++q) part[q] += vj * W[(int64_t)(c0 + q) * m + j];
      }
      block_sum_vec(part, cnt, sh, tot);
      for (int j = k + tid; j < m; j += kQrThreads) {
        const double vj = v[j];
        for (int q = 0; q < cnt; ++q) W[(int64_t)(c0 + q) * m + j] -= t * tot[q] * vj;
      }
      __syncthreads();
    }
  }
  for (int c = 0; c < s; ++c) {
    if (Q)
      for (int j = tid; j < m; j += kQrThreads)
        Q[(int64_t)i * q_ss + (int64_t)c * q_ld + j] = (float)W[(int64_t)c * m + j];
    if (Qhi)
      for (int j = tid; j < qh_ld; j += kQrThreads) {
        uint32_t h = 0, l = 0;
        if (j < m) split_bf16((float)W[(int64_t)c * m + j], h, l);
        Qhi[(int64_t)i * qh_ss + (int64_t)c * qh_ld + j] = (uint16_t)h;
        Qlo[(int64_t)i * qh_ss + (int64_t)c * qh_ld + j] = (uint16_t)l;
      }
  }
}

hipError_t launch_qr(const float* OS, int64_t os_ld, int64_t os_ss, int32_t B, int32_t m,
                     int32_t s, double* work, float* Q, int64_t q_ld, int64_t q_ss, uint16_t* Qhi,
                     uint16_t* Qlo, int64_t qh_ld, int64_t qh_ss, hipStream_t st) {
  hipLaunchKernelGGL(qr_kernel, dim3(B), dim3(kQrThreads), 0, st, OS, os_ld, os_ss, m, s, work, Q,
                     q_ld, q_ss, Qhi, Qlo, qh_ld, qh_ss);
  return hipGetLastError();
}

// ---- finalize ------------------------------------------------------------------------
constexpr int kFinThreads = 256;

__global__ __launch_bounds__(kFinThreads) void hutchpp_final_kernel(
    const float* UW, int64_t uw_ld, int64_t uw_ss, const float* Q, int64_t q_ld, int64_t q_ss,
    int32_t n, int32_t m, int32_t s, int32_t r, uint32_t key0, uint32_t key1, uint32_t layer,
    int32_t wpc, float* n2, float* n2_layer, int accumulate) {
  extern __shared__ __attribute__((aligned(16))) uint32_t fsm[];
  __shared__ double dred[4];
  const int i = blockIdx.x, tid = threadIdx.x;
  float* C = reinterpret_cast<float*>(fsm);           // [s][r]
  uint32_t* zw = fsm + s * r;                          // [r][wpc]
  const float* q = Q + (int64_t)i * q_ss;
  const int npair = s * r;
  // C = Q^T P: one (a, b) pair per thread per pass, fp64 sums; probe words staged per chunk
  for (int pg = 0; pg < npair; pg += kFinThreads) {
    const int pr = pg + tid;
    const bool active = pr < npair;
    const int a = active ? pr / r : 0, b = active ? pr - (pr / r) * r : 0;
    const float* qa = q + (int64_t)a * q_ld;
    double sacc = 0.0;
    for (int64_t uc = 0; uc < m; uc += 32 * (int64_t)wpc) {
      __syncthreads();
      const int nblk = wpc >> 2;
      for (int idx = tid; idx < r * nblk; idx += kFinThreads) {
        const int bb = idx / nblk, blk = idx - bb * nblk;
        const u32x4 v = rademacher_block(key0, key1, layer, kStreamProbe, (uint32_t)(uc >> 7) + blk, (uint32_t)bb);
        uint32_t* dst = zw + bb * wpc + 4 * blk;
        dst[0] = v.x; dst[1] = v.y; dst[2] = v.z; dst[3] = v.w;
      }
      __syncthreads();
      if (active) {
        const int64_t uend = min((int64_t)m, uc + 32 * (int64_t)wpc);
        const uint32_t* zb = zw + b * wpc;
        for (int64_t u = uc; u < uend; ++u) {
          const int64_t uu = u - uc;
          const uint32_t bit = (zb[uu >> 5] >> (uu & 31)) & 1u;
          const double qv = (double)qa[u];
          sacc += bit ? -qv : qv;
        }
      }
    }
    if (active) C[pr] = (float)sacc;
  }
  __syncthreads();
  // ||U||^2 + ||W_P - U C||^2 / r
  const float* uw = UW + (int64_t)i * uw_ss;
  double su = 0.0, sv = 0.0;
  for (int j = tid; j < n; j += kFinThreads) {
    float u[64];
    for (int a = 0; a < s; ++a) {
      u[a] = uw[(int64_t)a * uw_ld + j];
      su += (double)u[a] * (double)u[a];
    }
    for (int b = 0; b < r; ++b) {
      double v = (double)uw[(int64_t)(s + b) * uw_ld + j];
      for (int a = 0; a < s; ++a) v -= (double)u[a] * (double)C[a * r + b];
      sv += v * v;
    }
  }
  su = [&] {
    double x = wave_sum(su);
    __syncthreads();
    if ((tid & 63) == 0) dred[tid >> 6] = x;
    __syncthreads();
    return (dred[0] + dred[1]) + (dred[2] + dred[3]);
  }();
  sv = [&] {
    double x = wave_sum(sv);
    __syncthreads();
    if ((tid & 63) == 0) dred[tid >> 6] = x;
    __syncthreads();
    return (dred[0] + dred[1]) + (dred[2] + dred[3]);
  }();
  if (tid == 0) {
    const float est = (float)(su + sv / (double)r);
    n2[i] = (accumulate ? n2[i] : 0.f) + est;
    if (n2_layer) n2_layer[i] = est;
  }
}

hipError_t launch_hutchpp_final(const float* UW, int64_t uw_ld, int64_t uw_ss, const float* Q,
                                int64_t q_ld, int64_t q_ss, int32_t B, int32_t n, int32_t m,
                                int32_t s, int32_t r, uint32_t key0, uint32_t key1,
                                uint32_t layer, float* n2, float* n2_layer, int accumulate,
                                hipStream_t st) {
  if (s > 64 || r < 1 || s * r > 12288) return hipErrorInvalidValue;
  int wpc = (int)std::min<int64_t>(round_up(ceil_div(m, 32), 4), std::max(4, (4096 / r) & ~3));
  const size_t lds = (size_t)s * r * 4 + (size_t)r * wpc * 4;
  hipLaunchKernelGGL(hutchpp_final_kernel, dim3(B), dim3(kFinThreads), lds, st, UW, uw_ld, uw_ss, Q,
                     q_ld, q_ss, n, m, s, r, key0, key1, layer, wpc, n2, n2_layer, accumulate);
  return hipGetLastError();
}

}  // namespace dprc
