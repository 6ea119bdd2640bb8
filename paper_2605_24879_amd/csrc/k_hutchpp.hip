// Hutch++ pieces that are not token streams (Algorithm 2, Hutch++ branch):
//
//  * Q = orthonormal basis of the sketch O S (m x s per sample) by a tall-skinny
//    Householder QR (TSQR): each workgroup factors a block of rows in LDS, one
//    workgroup per sample factors the stacked s x s R factors, and each block
//    workgroup then expands its rows of Q = Q_block * Q_stack.  Householder
//    keeps Q orthonormal when O S is rank deficient (a Gram/Cholesky QR breaks
//    down there), and the blocks make the work parallel over rows.  All in fp64.
//  * While it holds its rows of Q, a block workgroup also forms its share of
//    C = Q^T P (P the residual probes, regenerated from Philox).
//  * The finalize step V = W_P - U C and the sums ||U||^2, ||V||^2 run
//    row-parallel; a last kernel adds the row chunks in a fixed order:
//    estimate = ||U||^2 + ||V||^2 / r.
#include <algorithm>
#include "device.hpp"
#include "kernels.hpp"

namespace dprc {

constexpr int kQrThreads = 256;
constexpr int kQrGroup = 16;  // columns whose dot products are reduced together

__device__ __forceinline__ double qr_block_sum(double v, double* sh) {
  const int tid = threadIdx.x;
  v = wave_sum(v);
  __syncthreads();
  if ((tid & 63) == 0) sh[tid >> 6] = v;
  __syncthreads();
  return (sh[0] + sh[1]) + (sh[2] + sh[3]);
}

// Sum over the workgroup of v[0..kQrGroup) (entries >= cnt are zero); every
// thread gets the sums.  A reduce-scatter inside the wave halves the vector at
// each of the exchanges over lane bits 5, 4, 3, 2 (8 + 4 + 2 + 1 shuffles), so
// lane l ends with column (l >> 2) & 15 summed over 16 lanes; two more
// exchanges finish the wave, and the four waves are added in a fixed order.
__device__ __forceinline__ void qr_block_sum_vec(double* v, int cnt, double* sh /*[4][kQrGroup]*/, double* out) {
  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
#pragma unroll
  for (int st = 0, o = 32, n = kQrGroup; st < 4; ++st, o >>= 1, n >>= 1) {
    const bool up = (lane & o) != 0;
    const int half = n >> 1;
#pragma unroll
    for (int j = 0; j < kQrGroup / 2; ++j) {
      if (j < half) {
        const double send = up ? v[j] : v[j + half];
        const double keep = up ? v[j + half] : v[j];
        v[j] = keep + __shfl_xor(send, o, 64);
      }
    }
  }
  double x = v[0];
  x += __shfl_xor(x, 2, 64);
  x += __shfl_xor(x, 1, 64);
  __syncthreads();
  if ((lane & 3) == 0) sh[wv * kQrGroup + ((lane >> 2) & 15)] = x;
  __syncthreads();
#pragma unroll
  for (int q = 0; q < kQrGroup; ++q)
    out[q] = q < cnt ? (sh[q] + sh[kQrGroup + q]) + (sh[2 * kQrGroup + q] + sh[3 * kQrGroup + q]) : 0.0;
}

// In-place Householder QR of A (rows x s, column-major, leading dimension ld;
// LDS or global).  Afterwards column k holds v_k in rows k..rows-1 (v_k[k] =
// x_k - alpha_k), tau[k] = 2 / |v_k|^2 (0: identity reflector for a zero
// column), alpha[k] = R_kk, and rows 0..k-1 of column k hold R.
__device__ __forceinline__ void householder_qr(double* A, int ld, int rows, int s, double* tau, double* alpha, double* sh) {
  const int tid = threadIdx.x;
  double part[kQrGroup], tot[kQrGroup];
  for (int k = 0; k < s; ++k) {
    double* x = A + (int64_t)k * ld;
    double p = 0.0;
    for (int j = k + tid; j < rows; j += kQrThreads) p += x[j] * x[j];
    const double nrm2 = qr_block_sum(p, sh);
    const double x0 = k < rows ? x[k] : 0.0;
    __syncthreads();
    if (!(nrm2 > 0.0)) {
      if (tid == 0) { tau[k] = 0.0; alpha[k] = 0.0; }
      __syncthreads();
      continue;
    }
    const double al = -copysign(sqrt(nrm2), x0);
    const double v0 = x0 - al;
    const double vn2 = nrm2 - x0 * x0 + v0 * v0;
    const double t = vn2 > 0.0 ? 2.0 / vn2 : 0.0;
    if (tid == 0) { tau[k] = t; alpha[k] = al; x[k] = v0; }
    __syncthreads();
    for (int c0 = k + 1; c0 < s; c0 += kQrGroup) {
      const int cnt = min(kQrGroup, s - c0);
      for (int q = 0; q < kQrGroup; ++q) part[q] = 0.0;
      for (int j = k + tid; j < rows; j += kQrThreads) {
        const double vj = x[j];
#pragma unroll
        for (int q = 0; q < kQrGroup; ++q)
          if (q < cnt) part[q] += vj * A[(int64_t)(c0 + q) * ld + j];
      }
      qr_block_sum_vec(part, cnt, sh, tot);
      for (int j = k + tid; j < rows; j += kQrThreads) {
        const double vj = x[j];
#pragma unroll
        for (int q = 0; q < kQrGroup; ++q)
          if (q < cnt) A[(int64_t)(c0 + q) * ld + j] -= t * tot[q] * vj;
      }
      __syncthreads();
    }
  }
}

// W <- H_0 H_1 ... H_{s-1} W for W (rows x s, column-major, ld_w), reflectors from householder_qr.
__device__ __forceinline__ void apply_reflectors(const double* V, int ldv, const double* tau, int rows, int s, double* W,
                                 int ldw, double* sh) {
  const int tid = threadIdx.x;
  double part[kQrGroup], tot[kQrGroup];
  for (int k = s - 1; k >= 0; --k) {
    const double t = tau[k];
    if (t == 0.0) continue;
    const double* v = V + (int64_t)k * ldv;
    for (int c0 = 0; c0 < s; c0 += kQrGroup) {
      const int cnt = min(kQrGroup, s - c0);
      for (int q = 0; q < kQrGroup; ++q) part[q] = 0.0;
      for (int j = k + tid; j < rows; j += kQrThreads) {
        const double vj = v[j];
#pragma unroll
        for (int q = 0; q < kQrGroup; ++q)
          if (q < cnt) part[q] += vj * W[(int64_t)(c0 + q) * ldw + j];
      }
      qr_block_sum_vec(part, cnt, sh, tot);
      for (int j = k + tid; j < rows; j += kQrThreads) {
        const double vj = v[j];
#pragma unroll
        for (int q = 0; q < kQrGroup; ++q)
          if (q < cnt) W[(int64_t)(c0 + q) * ldw + j] -= t * tot[q] * vj;
      }
      __syncthreads();
    }
  }
}

// ---- level 1: Householder QR of each block of R rows ---------------------------------------------
__global__ __launch_bounds__(kQrThreads) void qr_blocks_kernel(QrArgs a) {
  extern __shared__ __attribute__((aligned(16))) double lds[];
  __shared__ double sh[4 * kQrGroup];
  __shared__ double tau[64], alpha[64];
  const int b = blockIdx.x, i = blockIdx.y, tid = threadIdx.x;
  const int R = a.R, s = a.s;
  const int64_t row0 = (int64_t)b * R;
  const float* os = a.OS + (int64_t)i * a.os_ss;
  for (int c = 0; c < s; ++c)
    for (int j = tid; j < R; j += kQrThreads)
      lds[c * R + j] = row0 + j < a.m ? (double)os[(int64_t)c * a.os_ld + row0 + j] : 0.0;
  __syncthreads();
  householder_qr(lds, R, R, s, tau, alpha, sh);
  __syncthreads();
  double* V = a.V + ((int64_t)i * a.nblk + b) * s * R;
  for (int e = tid; e < s * R; e += kQrThreads) V[e] = lds[e];
  double* tb = a.tau + ((int64_t)i * a.nblk + b) * s;
  if (tid < s) tb[tid] = tau[tid];
  // R_b into the stacked matrix: column c, rows b*s .. b*s+s-1
  const int ldst = a.nblk * s;
  double* st = a.Rst + (int64_t)i * s * ldst;
  for (int e = tid; e < s * s; e += kQrThreads) {
    const int c = e / s, r = e - c * s;
    st[(int64_t)c * ldst + b * s + r] = r < c ? lds[c * R + r] : (r == c ? alpha[c] : 0.0);
  }
}

// ---- level 2: QR of the stacked R factors and its explicit Q (one workgroup per sample) ---------
__global__ __launch_bounds__(kQrThreads) void qr_combine_kernel(QrArgs a, int in_lds) {
  extern __shared__ __attribute__((aligned(16))) double lds[];
  __shared__ double sh[4 * kQrGroup];
  __shared__ double tau[64], alpha[64];
  const int i = blockIdx.x, tid = threadIdx.x, s = a.s;
  const int rows = a.nblk * s;
  double* stg = a.Rst + (int64_t)i * s * rows;
  double* q2g = a.Q2 + (int64_t)i * s * rows;
  double* st = in_lds ? lds : stg;                  // LDS copies when both s x rows matrices fit
  double* q2 = in_lds ? lds + s * rows : q2g;
  if (in_lds) {
    for (int e = tid; e < s * rows; e += kQrThreads) st[e] = stg[e];
    __syncthreads();
  }
  householder_qr(st, rows, rows, s, tau, alpha, sh);
  for (int c = 0; c < s; ++c)
    for (int j = tid; j < rows; j += kQrThreads) q2[(int64_t)c * rows + j] = (j == c) ? 1.0 : 0.0;
  __syncthreads();
  apply_reflectors(st, rows, tau, rows, s, q2, rows, sh);
  if (in_lds) {
    __syncthreads();
    for (int e = tid; e < s * rows; e += kQrThreads) q2g[e] = q2[e];
  }
}

// ---- level 3: rows of Q = Q_block [Q2_b; 0], and the block's share of C = Q^T P -------------------
__global__ __launch_bounds__(kQrThreads) void qr_expand_kernel(QrArgs a) {
  extern __shared__ __attribute__((aligned(16))) double lds[];
  __shared__ double sh[4 * kQrGroup];
  __shared__ double tau[64];
  const int b = blockIdx.x, i = blockIdx.y, tid = threadIdx.x;
  const int R = a.R, s = a.s, rows2 = a.nblk * s;
  double* W = lds;                                           // [s][R]
  uint32_t* zw = reinterpret_cast<uint32_t*>(W + s * R);     // [r][R/32] probe words of this block
  const double* V = a.V + ((int64_t)i * a.nblk + b) * s * R; // reflectors (read-only, global)
  if (tid < s) tau[tid] = a.tau[((int64_t)i * a.nblk + b) * s + tid];
  const double* q2 = a.Q2 + (int64_t)i * s * rows2;
  for (int e = tid; e < s * R; e += kQrThreads) {
    const int c = e / R, j = e - c * R;
    W[e] = j < s ? q2[(int64_t)c * rows2 + b * s + j] : 0.0;
  }
  // probe words for rows b*R .. b*R+R-1 (R is a multiple of 128)
  const int wpb = R / 32;
  for (int e = tid; e < a.r * (wpb / 4); e += kQrThreads) {
    const int c = e / (wpb / 4), blk = e - c * (wpb / 4);
    const u32x4 v = rademacher_block(a.key0, a.key1, a.layer, kStreamProbe, (uint32_t)(b * (R / 128) + blk),
                                     (uint32_t)c);
    uint32_t* d = zw + c * wpb + 4 * blk;
    d[0] = v.x; d[1] = v.y; d[2] = v.z; d[3] = v.w;
  }
  __syncthreads();
  apply_reflectors(V, R, tau, R, s, W, R, sh);
  __syncthreads();
  const int64_t row0 = (int64_t)b * R;
  for (int c = 0; c < s; ++c) {
    for (int j = tid; j < R; j += kQrThreads) {
      const int64_t row = row0 + j;
      const double q = row < a.m ? W[c * R + j] : 0.0;
      if (a.Q && row < a.m) a.Q[(int64_t)i * a.q_ss + (int64_t)c * a.q_ld + row] = (float)q;
      if (a.Qhi && row < a.qh_ld) {
        uint32_t h, l;
        split_bf16((float)q, h, l);
        a.Qhi[(int64_t)i * a.qh_ss + (int64_t)c * a.qh_ld + row] = (uint16_t)h;
        a.Qlo[(int64_t)i * a.qh_ss + (int64_t)c * a.qh_ld + row] = (uint16_t)l;
      }
    }
  }
  // C_b[c][c'] = sum_j Q[j][c] z(j, c') over this block's rows (rows >= m count as zero)
  double* cp = a.Cpart + ((int64_t)i * a.nblk + b) * s * a.r;
  for (int pr = tid; pr < s * a.r; pr += kQrThreads) {
    const int c = pr / a.r, cc = pr - c * a.r;
    const double* wc = W + c * R;
    const uint32_t* zb = zw + cc * wpb;
    double acc = 0.0;
    for (int j = 0; j < R; ++j) {
      const double q = (row0 + j < a.m) ? wc[j] : 0.0;
      acc += ((zb[j >> 5] >> (j & 31)) & 1u) ? -q : q;
    }
    cp[pr] = acc;
  }
}

QrPlan qr_plan(int64_t m, int s) {
  QrPlan p;
  // block rows: R x s fp64 in LDS (64 KB), R a multiple of 128 (whole probe blocks)
  p.R = (int32_t)std::min<int64_t>(512, std::max<int64_t>(128, (8192 / std::max(s, 1)) / 128 * 128));
  p.nblk = (int32_t)ceil_div(m, p.R);
  return p;
}

static size_t qr_lds_expand(const QrArgs& a) {
  return (size_t)a.s * a.R * 8 + (size_t)a.r * (a.R / 32) * 4;
}

hipError_t launch_qr_blocks(const QrArgs& a, hipStream_t st) {
  DPRC_LAUNCH(qr_blocks_kernel, dim3((unsigned)a.nblk, (unsigned)a.B), dim3(kQrThreads),
                     (size_t)a.s * a.R * 8, st, a);
  return hipGetLastError();
}

hipError_t launch_qr_combine(const QrArgs& a, hipStream_t st) {
  const size_t bytes = (size_t)2 * a.s * a.nblk * a.s * 8;
  const int in_lds = bytes <= 96 * 1024;
  DPRC_LAUNCH(qr_combine_kernel, dim3((unsigned)a.B), dim3(kQrThreads), in_lds ? bytes : 0, st, a, in_lds);
  return hipGetLastError();
}

hipError_t launch_qr_expand(const QrArgs& a, hipStream_t st) {
  DPRC_LAUNCH(qr_expand_kernel, dim3((unsigned)a.nblk, (unsigned)a.B), dim3(kQrThreads), qr_lds_expand(a),
                     st, a);
  return hipGetLastError();
}

// ---- finalize -----------------------------------------------------------------------------------------
constexpr int kFinRows = 256;

// Rows j of one chunk: ||U_j||^2 and ||W_P,j - U_j C||^2 summed over the chunk.
__global__ __launch_bounds__(kFinRows) void hpp_rows_kernel(FinalArgs a) {
  extern __shared__ __attribute__((aligned(16))) float fs[];
  __shared__ double sh[4];
  const int ch = blockIdx.x, i = blockIdx.y, tid = threadIdx.x;
  const int s = a.s, r = a.r;
  float* C = fs;                           // [s][r]
  // C = sum over blocks of the partial C_b, in block order
  const double* cp = a.Cpart + (int64_t)i * a.nblk * s * r;
  for (int e = tid; e < s * r; e += kFinRows) {
    double v = 0.0;
    for (int b = 0; b < a.nblk; ++b) v += cp[(int64_t)b * s * r + e];
    C[e] = (float)v;
  }
  __syncthreads();
  const int64_t j = (int64_t)ch * kFinRows + tid;
  double su = 0.0, sv = 0.0;
  if (j < a.n) {
    const float* uw = a.UW + (int64_t)i * a.uw_ss + j;
    for (int b2 = 0; b2 < r; ++b2) {
      double v = (double)uw[(int64_t)(s + b2) * a.uw_ld];
      for (int c = 0; c < s; ++c) v -= (double)uw[(int64_t)c * a.uw_ld] * (double)C[c * r + b2];
      sv += v * v;
    }
    for (int c = 0; c < s; ++c) {
      const double u = (double)uw[(int64_t)c * a.uw_ld];
      su += u * u;
    }
  }
  su = qr_block_sum(su, sh);
  sv = qr_block_sum(sv, sh);
  if (tid == 0) {
    a.Fpart[((int64_t)i * a.nchunk + ch) * 2] = su;
    a.Fpart[((int64_t)i * a.nchunk + ch) * 2 + 1] = sv;
  }
}

__global__ __launch_bounds__(kQrThreads) void hpp_sum_kernel(FinalArgs a) {
  __shared__ double sh[4];
  const int i = blockIdx.x;
  double su = 0.0, sv = 0.0;
  for (int c = threadIdx.x; c < a.nchunk; c += kQrThreads) {
    su += a.Fpart[((int64_t)i * a.nchunk + c) * 2];
    sv += a.Fpart[((int64_t)i * a.nchunk + c) * 2 + 1];
  }
  su = qr_block_sum(su, sh);
  sv = qr_block_sum(sv, sh);
  if (threadIdx.x == 0) {
    const float est = (float)(su + sv / (double)a.r);
    a.n2[i] = (a.accumulate ? a.n2[i] : 0.f) + est;
    if (a.n2_layer) a.n2_layer[i] = est;
  }
}

hipError_t launch_hpp_rows(const FinalArgs& a, hipStream_t st) {
  DPRC_LAUNCH(hpp_rows_kernel, dim3((unsigned)a.nchunk, (unsigned)a.B), dim3(kFinRows),
                     (size_t)a.s * a.r * 4, st, a);
  return hipGetLastError();
}

hipError_t launch_hpp_sum(const FinalArgs& a, hipStream_t st) {
  DPRC_LAUNCH(hpp_sum_kernel, dim3((unsigned)a.B), dim3(kQrThreads), 0, st, a);
  return hipGetLastError();
}

int32_t final_chunks(int64_t n) { return (int32_t)ceil_div(n, kFinRows); }

}  // namespace dprc
