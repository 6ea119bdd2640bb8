// Hutch++ pieces that are not token streams (Algorithm 2, Hutch++ branch):
//
//  * Q = orthonormal basis of the sketch O S (m x s per sample) by a tall-skinny
//    Householder QR as a tree: one wavefront factors a block of 128 rows held in
//    registers (two rows per lane, fp64), the s x s R factors of the blocks are
//    stacked and factored the same way at the next level, until one block is
//    left.  The expansion runs back down the tree: each block starts from its s
//    rows of the level above's Q (the identity at the top) and applies its own
//    reflectors.  One launch takes the same step of up to eight layers' trees
//    (each block finds its layer from its block index), so the latency-bound tree
//    costs a few launches per call rather than a few per layer.  Householder keeps Q orthonormal when O S is rank deficient (a
//    Gram/Cholesky QR breaks down there).  Dot products over a block's rows are
//    summed across the wave through LDS in a fixed order, so the result does not
//    depend on scheduling.
//  * While it holds its rows of Q, a level-1 block also forms its share of
//    C = Q^T P (P the residual probes, regenerated from Philox).
//  * The finalize step V = W_P - U C and the sums ||U||^2, ||V||^2 run
//    row-parallel; a last kernel adds the row chunks in a fixed order:
//    estimate = ||U||^2 + ||V||^2 / r.
#include <algorithm>
#include "device.hpp"
#include "kernels.hpp"

namespace dprc {

constexpr int kQrThreads = 256;   // finalize kernels
constexpr int kRedLd = 65;        // padded row of the per-column lane sums

__device__ __forceinline__ double qr_block_sum(double v, double* sh) {
  const int tid = threadIdx.x;
  v = wave_sum(v);
  __syncthreads();
  if ((tid & 63) == 0) sh[tid >> 6] = v;
  __syncthreads();
  return (sh[0] + sh[1]) + (sh[2] + sh[3]);
}

// Orders a wave's LDS accesses around a hand-off between its lanes (LDS
// operations of one wave execute in issue order; this keeps the compiler from
// moving them across).
__device__ __forceinline__ void qr_wave_fence() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

__device__ __forceinline__ double readlane_f64(double v, int l) {
  const uint64_t u = (uint64_t)__double_as_longlong(v);
  const uint32_t lo = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)u, l);
  const uint32_t hi = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)(u >> 32), l);
  return __longlong_as_double((long long)(((uint64_t)hi << 32) | lo));
}

// x[l] + x[l ^ 16] (R = 16) or x[l] + x[l ^ 32] (R = 32) with the lane swaps of
// gfx950: the swap returns the pair's two values in the same order on both lanes
// (lane with the bit clear first), so both lanes form the same sum.
template <int R>
__device__ __forceinline__ double add_across(double x) {
  const uint64_t u = (uint64_t)__double_as_longlong(x);
  const uint32_t lo = (uint32_t)u, hi = (uint32_t)(u >> 32);
  uint32_t l0, l1, h0, h1;
  if constexpr (R == 16) {
    const auto pl = __builtin_amdgcn_permlane16_swap(lo, lo, false, false);
    const auto ph = __builtin_amdgcn_permlane16_swap(hi, hi, false, false);
    l0 = pl[0]; l1 = pl[1]; h0 = ph[0]; h1 = ph[1];
  } else {
    const auto pl = __builtin_amdgcn_permlane32_swap(lo, lo, false, false);
    const auto ph = __builtin_amdgcn_permlane32_swap(hi, hi, false, false);
    l0 = pl[0]; l1 = pl[1]; h0 = ph[0]; h1 = ph[1];
  }
  return __longlong_as_double((long long)(((uint64_t)h0 << 32) | l0)) +
         __longlong_as_double((long long)(((uint64_t)h1 << 32) | l1));
}

// v[c] <- sum over the 64 lanes of v[c], for c >= c_lo (c_lo a constant after
// unrolling).  Lane sums go to LDS column by column; lane (c, g) adds the g-th
// run of SP of them, and shuffles over the run bits finish the sum.
template <int SP>
__device__ __forceinline__ void wave_vec_sum(double (&v)[SP], int c_lo, double* red, double* tot) {
  const int lane = threadIdx.x & 63;
#pragma unroll
  for (int c = 0; c < SP; ++c)
    if (c >= c_lo) red[c * kRedLd + lane] = v[c];
  qr_wave_fence();
  const int c = lane % SP, g = lane / SP;
  double x = 0.0;
  if (c >= c_lo) {
    double t[SP];                                 // all reads in flight before the adds
#pragma unroll
    for (int q = 0; q < SP; ++q) t[q] = red[c * kRedLd + g * SP + q];
#pragma unroll
    for (int w = SP / 2; w >= 1; w >>= 1)        // pairwise tree
#pragma unroll
      for (int q = 0; q < w; ++q) t[q] += t[q + w];
    x = t[0];
  }
#pragma unroll
  for (int e = 0; e < 6; ++e) {
    const int m = SP << e;
    if (m == 16) x = add_across<16>(x);
    else if (m == 32) x = add_across<32>(x);
    else if (m < 64) x += __shfl_xor(x, m, 64);
  }
  if (g == 0) tot[c] = x;
  qr_wave_fence();
#pragma unroll
  for (int q = 0; q < SP; ++q)
    if (q >= c_lo) v[q] = tot[q];
  qr_wave_fence();
}

// The job of this block (jobs start at increasing blk0) and its (block, sample).
__device__ __forceinline__ int qr_job_index(const QrBatch& bt) {
  int jb = 0;
#pragma unroll
  for (int q = 1; q < kQrMaxJobs; ++q) jb += (q < bt.njobs && (int)blockIdx.x >= bt.job[q].blk0) ? 1 : 0;
  return jb;
}

// ---- factor one 128-row block of a level ----------------------------------------------------------
// Lane l holds rows l and l + 64 of the block.  Step k works on column k, held in
// register column 0: the columns not yet factored shift down one place after each
// step, so every register index is a constant.  v_k = x_k - alpha_k e_k over rows
// >= k, tau_k = 2 / |v_k|^2 (0: identity reflector for a zero column), alpha_k =
// R_kk; the dot products v_k . A_c come from one pass with the norm: x_k . A_c -
// alpha_k A_kc.  v_k, tau_k and row k of R are written out as each step ends.
template <int SP>
__global__ __launch_bounds__(64) void qr_factor_kernel(QrBatch bt) {
  __shared__ double red[SP * kRedLd];
  __shared__ double tot[SP];
  const QrJob& a = bt.job[qr_job_index(bt)];
  const int level = a.level;
  const int rel = (int)blockIdx.x - a.blk0;
  const int b = rel % a.L.nblk, i = rel / a.L.nblk, lane = threadIdx.x;
  const int s = a.s;
  const QrLevel L = a.L;
  // all loads are issued before the first use: masked entries read a valid address
  // and are replaced by zero
  double A[2][SP];
  if (level == 0) {
    const float* os = a.OS + (int64_t)i * a.os_ss;
#pragma unroll
    for (int u = 0; u < 2; ++u) {
      const int row = b * kQrRows + lane + 64 * u;
#pragma unroll
      for (int c = 0; c < SP; ++c) {
        const bool ok = c < s && row < L.rows;
        const float x = os[ok ? (int64_t)c * a.os_ld + row : 0];
        A[u][c] = ok ? (double)x : 0.0;
      }
    }
  } else {
    const double* ms = L.M + (int64_t)i * s * L.rows;
#pragma unroll
    for (int u = 0; u < 2; ++u) {
      const int row = b * kQrRows + lane + 64 * u;
#pragma unroll
      for (int c = 0; c < SP; ++c) {
        const bool ok = c < s && row < L.rows;
        const double x = ms[ok ? (int64_t)c * L.rows + row : 0];
        A[u][c] = ok ? x : 0.0;
      }
    }
  }
  double* V = L.V + ((int64_t)i * L.nblk + b) * s * kQrRows;
  double* tb = L.tau + ((int64_t)i * L.nblk + b) * s;
  const bool has_next = level + 1 < a.nlev;
  const QrLevel N = has_next ? a.X : a.L;
  // outputs stay in registers until the loop ends (a store costs the wave tens of
  // cycles even with one lane active): v_k and tau_k enter register column SP - 1
  // and move down one place per step, so after s steps column k sits at SP - s + k;
  // lane k keeps row k of R (offset e from the diagonal in register column e)
  double Vs[2][SP], Ts[SP], Rr[SP];
#pragma unroll
  for (int e = 0; e < SP; ++e) {
    Vs[0][e] = Vs[1][e] = 0.0;
    Ts[e] = 0.0;
    Rr[e] = 0.0;
  }
  for (int k = 0; k < s; ++k) {
    double pv[SP];
#pragma unroll
    for (int c = 0; c < SP; ++c) pv[c] = 0.0;
#pragma unroll
    for (int u = 0; u < 2; ++u) {
      const double xk = lane + 64 * u >= k ? A[u][0] : 0.0;
#pragma unroll
      for (int c = 0; c < SP; ++c) pv[c] += xk * A[u][c];
    }
    wave_vec_sum<SP>(pv, 0, red, tot);
    const double nrm2 = pv[0];
    double t = 0.0, al = 0.0;
    if (nrm2 > 0.0) {                               // uniform; a zero column keeps the identity reflector
      const double x0 = readlane_f64(A[0][0], k);  // row k < 32 sits in lane k
      al = -copysign(sqrt(nrm2), x0);
      const double v0 = x0 - al;
      const double vn2 = nrm2 - x0 * x0 + v0 * v0;
      t = vn2 > 0.0 ? 2.0 / vn2 : 0.0;
      double d[SP];
#pragma unroll
      for (int c = 1; c < SP; ++c) d[c] = pv[c] - al * readlane_f64(A[0][c], k);
#pragma unroll
      for (int u = 0; u < 2; ++u) {
        const int j = lane + 64 * u;
        if (j >= k) {
          const double vj = j == k ? v0 : A[u][0];
#pragma unroll
          for (int c = 1; c < SP; ++c) A[u][c] -= t * vj * d[c];
          A[u][0] = vj;
        }
      }
    }
    // v_k (zero above the diagonal; for a zero column the column itself, which is zero),
    // tau_k, and row k of R (R_kk = alpha_k, R_k,k+e = A[0][e]) in lane k
#pragma unroll
    for (int u = 0; u < 2; ++u) {
      const int j = lane + 64 * u;
#pragma unroll
      for (int e = 0; e + 1 < SP; ++e) Vs[u][e] = Vs[u][e + 1];
      Vs[u][SP - 1] = j >= k ? A[u][0] : 0.0;
    }
#pragma unroll
    for (int e = 0; e + 1 < SP; ++e) Ts[e] = Ts[e + 1];
    Ts[SP - 1] = t;
    if (lane == k) {
      Rr[0] = al;
#pragma unroll
      for (int e = 1; e < SP; ++e) Rr[e] = A[0][e];
    }
    // the remaining columns move down one register column
#pragma unroll
    for (int u = 0; u < 2; ++u) {
#pragma unroll
      for (int c = 0; c + 1 < SP; ++c) A[u][c] = A[u][c + 1];
      A[u][SP - 1] = 0.0;
    }
  }
  // V (column k of the block at register column SP - s + k), tau, and the rows of R
  // into rows b*s + q of the next level's input (zero left of the diagonal)
#pragma unroll
  for (int e = 0; e < SP; ++e) {
    const int k = e - (SP - s);
    if (k >= 0) {
#pragma unroll
      for (int u = 0; u < 2; ++u) V[(int64_t)k * kQrRows + lane + 64 * u] = Vs[u][e];
      if (lane == 0) tb[k] = Ts[e];
    }
  }
  if (has_next && lane < s) {
    double* nm = N.M + (int64_t)i * s * N.rows + (int64_t)b * s + lane;
#pragma unroll
    for (int e = 0; e < SP; ++e) {
      if (lane + e < s) nm[(int64_t)(lane + e) * N.rows] = Rr[e];
      if (e >= 1 && e <= lane) nm[(int64_t)(lane - e) * N.rows] = 0.0;
    }
  }
}

// ---- expand one block: W = H_0 ... H_{s-1} [Q_up rows; 0]; level 0 writes Q and C_b = Q_b^T P_b ----
template <int SP>
__global__ __launch_bounds__(64) void qr_expand_kernel(QrBatch bt) {
  __shared__ double red[SP * kRedLd];
  __shared__ double tot[SP];
  __shared__ double qs[SP * (kQrRows + 1)];
  __shared__ uint32_t zw[256 * 4];
  const QrJob& a = bt.job[qr_job_index(bt)];
  const int level = a.level;
  const int rel = (int)blockIdx.x - a.blk0;
  const int b = rel % a.L.nblk, i = rel / a.L.nblk, lane = threadIdx.x;
  const int s = a.s;
  const QrLevel L = a.L;
  const bool top = level + 1 == a.nlev;
  const QrLevel U = top ? a.L : a.X;
  // all loads are issued before the first use (masked entries read a valid address)
  double W[2][SP];
  const double* uq = U.Q + (int64_t)i * s * U.rows + (int64_t)b * s;
#pragma unroll
  for (int u = 0; u < 2; ++u) {
    const int j = lane + 64 * u;
#pragma unroll
    for (int c = 0; c < SP; ++c) {
      const bool ok = c < s && j < s;
      double w = 0.0;
      if (top) w = ok && j == c ? 1.0 : 0.0;
      else {
        const double x = uq[ok ? (int64_t)c * U.rows + j : 0];
        w = ok ? x : 0.0;
      }
      W[u][c] = w;
    }
  }
  // reflectors in reverse order: register column e holds v_{s-1-e}; the columns
  // move down one place after each step, so every register index is a constant
  const double* Vb = L.V + ((int64_t)i * L.nblk + b) * s * kQrRows;
  double Vr[2][SP];
#pragma unroll
  for (int u = 0; u < 2; ++u)
#pragma unroll
    for (int e = 0; e < SP; ++e) {
      const bool ok = e < s;
      const double x = Vb[ok ? (int64_t)(s - 1 - e) * kQrRows + lane + 64 * u : 0];
      Vr[u][e] = ok ? x : 0.0;
    }
  const double* tb = L.tau + ((int64_t)i * L.nblk + b) * s;
  for (int k = s - 1; k >= 0; --k) {
    const double t = tb[k];
    const double v0 = Vr[0][0], v1 = Vr[1][0];
#pragma unroll
    for (int u = 0; u < 2; ++u) {
#pragma unroll
      for (int e = 0; e + 1 < SP; ++e) Vr[u][e] = Vr[u][e + 1];
      Vr[u][SP - 1] = 0.0;
    }
    if (t == 0.0) continue;                       // uniform
    double pv[SP];
#pragma unroll
    for (int c = 0; c < SP; ++c) pv[c] = v0 * W[0][c] + v1 * W[1][c];
    wave_vec_sum<SP>(pv, 0, red, tot);
#pragma unroll
    for (int c = 0; c < SP; ++c) {
      W[0][c] -= t * v0 * pv[c];
      W[1][c] -= t * v1 * pv[c];
    }
  }
  if (level > 0) {
#pragma unroll
    for (int u = 0; u < 2; ++u) {
      const int row = b * kQrRows + lane + 64 * u;
      if (row < L.rows) {
#pragma unroll
        for (int c = 0; c < SP; ++c)
          if (c < s) L.Q[((int64_t)i * s + c) * L.rows + row] = W[u][c];
      }
    }
    return;
  }
  // level 0: rows of Q (rows >= m are zero: their reflector entries are zero)
#pragma unroll
  for (int u = 0; u < 2; ++u) {
    const int64_t row = (int64_t)b * kQrRows + lane + 64 * u;
#pragma unroll
    for (int c = 0; c < SP; ++c) {
      if (c < s) {
        const double q = row < a.m ? W[u][c] : 0.0;
        qs[c * (kQrRows + 1) + lane + 64 * u] = q;
        if (a.Q && row < a.m) a.Q[(int64_t)i * a.q_ss + (int64_t)c * a.q_ld + row] = (float)q;
        if (a.Qhi && row < a.qh_ld) {
          uint32_t h, l;
          split_bf16((float)q, h, l);
          a.Qhi[(int64_t)i * a.qh_ss + (int64_t)c * a.qh_ld + row] = (uint16_t)h;
          a.Qlo[(int64_t)i * a.qh_ss + (int64_t)c * a.qh_ld + row] = (uint16_t)l;
        }
      }
    }
  }
  // probe words of rows b*128 .. b*128+127 (one Philox block per column)
  for (int cc = lane; cc < a.r; cc += 64) {
    const u32x4 v = rademacher_block(a.key0, a.key1, a.layer, kStreamProbe, (uint32_t)b, (uint32_t)cc);
    zw[cc * 4 + 0] = v.x; zw[cc * 4 + 1] = v.y; zw[cc * 4 + 2] = v.z; zw[cc * 4 + 3] = v.w;
  }
  qr_wave_fence();
  // C_b[c][cc] = sum_j Q[j][c] z(j, cc) over this block's rows; a lane takes
  // outputs pr = lane + 64 t, four at a time so that four sums advance together
  double* cp = a.Cpart + ((int64_t)i * L.nblk + b) * s * a.r;
  for (int p0 = lane; p0 < s * a.r; p0 += 256) {
    const double* qc[4];
    uint32_t zoff[4];
    bool on[4];
#pragma unroll
    for (int t = 0; t < 4; ++t) {
      const int pr = p0 + 64 * t;
      on[t] = pr < s * a.r;
      const int c = on[t] ? pr / a.r : 0, cc = on[t] ? pr - c * a.r : 0;
      qc[t] = qs + c * (kQrRows + 1);
      zoff[t] = (uint32_t)cc * 4;
    }
    double acc[4] = {0.0, 0.0, 0.0, 0.0};
    for (int w = 0; w < 4; ++w) {
      uint32_t bits[4];
#pragma unroll
      for (int t = 0; t < 4; ++t) bits[t] = zw[zoff[t] + w];
#pragma unroll
      for (int jj = 0; jj < 32; ++jj) {
#pragma unroll
        for (int t = 0; t < 4; ++t) {
          const double q = qc[t][32 * w + jj];
          acc[t] += ((bits[t] >> jj) & 1u) ? -q : q;
        }
      }
    }
#pragma unroll
    for (int t = 0; t < 4; ++t)
      if (on[t]) cp[p0 + 64 * t] = acc[t];
  }
}

int32_t qr_levels(int64_t m, int s, int32_t rows[kQrMaxLevels], int32_t nblk[kQrMaxLevels], int64_t* dbl) {
  int32_t n = 0;
  int64_t r = m, total = 0;
  while (n < kQrMaxLevels) {
    rows[n] = (int32_t)r;
    nblk[n] = (int32_t)ceil_div(r, kQrRows);
    total += (int64_t)nblk[n] * s * kQrRows + (int64_t)nblk[n] * s;   // V, tau
    if (n > 0) total += 2 * r * s;                                     // M, Q
    ++n;
    if (nblk[n - 1] == 1) break;
    r = (int64_t)nblk[n - 1] * s;
  }
  if (nblk[n - 1] != 1) return 0;
  if (dbl) *dbl = total;
  return n;
}

template <template <int> class K>
static hipError_t launch_qr_sp(const QrBatch& bt, hipStream_t st) {
  if (bt.s < 1 || bt.s > 32 || bt.r > 256 || bt.njobs < 1 || bt.njobs > kQrMaxJobs || bt.blocks < 1)
    return hipErrorInvalidValue;
  const dim3 grid((unsigned)bt.blocks);
  if (bt.s <= 8) DPRC_LAUNCH(K<8>::fn, grid, dim3(64), 0, st, bt);
  else if (bt.s <= 16) DPRC_LAUNCH(K<16>::fn, grid, dim3(64), 0, st, bt);
  else DPRC_LAUNCH(K<32>::fn, grid, dim3(64), 0, st, bt);
  return hipGetLastError();
}
template <int SP>
struct QrFactorK {
  static constexpr auto fn = qr_factor_kernel<SP>;
};
template <int SP>
struct QrExpandK {
  static constexpr auto fn = qr_expand_kernel<SP>;
};

hipError_t launch_qr_factor(const QrBatch& bt, hipStream_t st) { return launch_qr_sp<QrFactorK>(bt, st); }
hipError_t launch_qr_expand(const QrBatch& bt, hipStream_t st) { return launch_qr_sp<QrExpandK>(bt, st); }

// ---- finalize -----------------------------------------------------------------------------------------
// A workgroup takes 32 rows j of U | W_P; its threads are (row, column group): group
// g handles the residual columns q = g, g + 8, ..., so a wave reads whole 128-byte
// runs of a column and every row's residuals advance in parallel.
constexpr int kFinRows = 32;                 // rows per workgroup
constexpr int kFinGroups = kQrThreads / kFinRows;

// C = sum of the block partials C_b, in block order (one thread per entry).
__device__ __forceinline__ void hpp_csum_block(const FinalArgs& a, int bx, int i) {
  const int sr = a.s * a.r;
  const int e = bx * kQrThreads + threadIdx.x;
  if (e >= sr) return;
  const double* cp = a.Cpart + (int64_t)i * a.nblk * sr + e;
  double v = 0.0;
  int b = 0;
  for (; b + 8 <= a.nblk; b += 8) {              // eight loads in flight, added in block order
    double x[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) x[u] = cp[(int64_t)(b + u) * sr];
#pragma unroll
    for (int u = 0; u < 8; ++u) v += x[u];
  }
  for (; b < a.nblk; ++b) v += cp[(int64_t)b * sr];
  a.C[(int64_t)i * sr + e] = v;
}
__global__ __launch_bounds__(kQrThreads) void hpp_csum_kernel(FinalArgs a) { hpp_csum_block(a, blockIdx.x, blockIdx.y); }

// Rows of one chunk: ||U_j||^2 and ||W_P,j - U_j C||^2 summed over the chunk.
template <int SP>
__device__ __forceinline__ void hpp_rows_block(const FinalArgs& a, int ch, int i) {
  extern __shared__ __attribute__((aligned(16))) float fs[];
  __shared__ double sh[4];
  const int tid = threadIdx.x;
  const int s = a.s, r = a.r;
  float* C = fs;                           // [s][r]
  for (int e = tid; e < s * r; e += kQrThreads) C[e] = (float)a.C[(int64_t)i * s * r + e];
  __syncthreads();
  const int grp = tid / kFinRows;
  const int64_t j = (int64_t)ch * kFinRows + (tid % kFinRows);
  double su = 0.0, sv = 0.0;
  if (j < a.n) {
    const float* uw = a.UW + (int64_t)i * a.uw_ss + j;
    double u[SP];                                  // row j of U
#pragma unroll
    for (int c = 0; c < SP; ++c) {
      const float x = uw[(int64_t)(c < s ? c : 0) * a.uw_ld];
      u[c] = c < s ? (double)x : 0.0;
      if (grp == 0) su += u[c] * u[c];
    }
    // residual columns of this group, four at a time: their loads are in flight together
    for (int q0 = grp; q0 < r; q0 += 4 * kFinGroups) {
      float w[4];
#pragma unroll
      for (int t = 0; t < 4; ++t) {
        const int q = q0 + t * kFinGroups;
        w[t] = uw[(int64_t)(s + (q < r ? q : 0)) * a.uw_ld];
      }
#pragma unroll
      for (int t = 0; t < 4; ++t) {
        const int q = q0 + t * kFinGroups;
        if (q < r) {
          double v = (double)w[t];
#pragma unroll
          for (int c = 0; c < SP; ++c)
            if (c < s) v -= u[c] * (double)C[c * r + q];
          sv += v * v;
        }
      }
    }
  }
  su = qr_block_sum(su, sh);
  sv = qr_block_sum(sv, sh);
  if (tid == 0) {
    a.Fpart[((int64_t)i * a.nchunk + ch) * 2] = su;
    a.Fpart[((int64_t)i * a.nchunk + ch) * 2 + 1] = sv;
  }
}
template <int SP>
__global__ __launch_bounds__(kQrThreads) void hpp_rows_kernel(FinalArgs a) { hpp_rows_block<SP>(a, blockIdx.x, blockIdx.y); }

// The finalize of several layers in one launch per step: block (x, sample) of job j at
// blk0[j] + sample * (x blocks of the job) + x.  The per-sample sum walks the jobs in
// order, so n2 adds the layers' estimates in layer order.
__device__ __forceinline__ int fin_job_index(const FinalBatch& bt) {
  int jb = 0;
#pragma unroll
  for (int q = 1; q < kFinMaxJobs; ++q) jb += (q < bt.njobs && (int)blockIdx.x >= bt.blk0[q]) ? 1 : 0;
  return jb;
}
__global__ __launch_bounds__(kQrThreads) void hpp_csum_batch_kernel(FinalBatch bt) {
  const int jb = fin_job_index(bt);
  const FinalArgs& a = bt.job[jb];
  const int nx = (a.s * a.r + kQrThreads - 1) / kQrThreads;
  const int rel = (int)blockIdx.x - bt.blk0[jb];
  hpp_csum_block(a, rel % nx, rel / nx);
}
template <int SP>
__global__ __launch_bounds__(kQrThreads) void hpp_rows_batch_kernel(FinalBatch bt) {
  const int jb = fin_job_index(bt);
  const FinalArgs& a = bt.job[jb];
  const int rel = (int)blockIdx.x - bt.blk0[jb];
  hpp_rows_block<SP>(a, rel % a.nchunk, rel / a.nchunk);
}

__device__ __forceinline__ void hpp_sum_block(const FinalArgs& a, int i) {
  __shared__ double sh[4];
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
__global__ __launch_bounds__(kQrThreads) void hpp_sum_kernel(FinalArgs a) { hpp_sum_block(a, blockIdx.x); }
__global__ __launch_bounds__(kQrThreads) void hpp_sum_batch_kernel(FinalBatch bt) {
  for (int j = 0; j < bt.njobs; ++j) {               // layer order; each job adds to n2 after the last
    hpp_sum_block(bt.job[j], blockIdx.x);
    __syncthreads();
  }
}

hipError_t launch_hpp_rows(const FinalArgs& a, hipStream_t st) {
  const dim3 grid((unsigned)a.nchunk, (unsigned)a.B);
  const size_t lds = (size_t)a.s * a.r * 4;
  if (a.s <= 8) DPRC_LAUNCH(hpp_rows_kernel<8>, grid, dim3(kQrThreads), lds, st, a);
  else if (a.s <= 16) DPRC_LAUNCH(hpp_rows_kernel<16>, grid, dim3(kQrThreads), lds, st, a);
  else DPRC_LAUNCH(hpp_rows_kernel<32>, grid, dim3(kQrThreads), lds, st, a);
  return hipGetLastError();
}

hipError_t launch_hpp_csum(const FinalArgs& a, hipStream_t st) {
  DPRC_LAUNCH(hpp_csum_kernel, dim3((unsigned)ceil_div((int64_t)a.s * a.r, kQrThreads), (unsigned)a.B),
              dim3(kQrThreads), 0, st, a);
  return hipGetLastError();
}

hipError_t launch_hpp_sum(const FinalArgs& a, hipStream_t st) {
  DPRC_LAUNCH(hpp_sum_kernel, dim3((unsigned)a.B), dim3(kQrThreads), 0, st, a);
  return hipGetLastError();
}

hipError_t launch_hpp_csum_batch(const FinalBatch& bt, hipStream_t st) {
  if (bt.njobs < 1 || bt.njobs > kFinMaxJobs) return hipErrorInvalidValue;
  FinalBatch b = bt;
  int blocks = 0;
  for (int j = 0; j < b.njobs; ++j) {
    b.blk0[j] = blocks;
    blocks += (int)ceil_div((int64_t)b.job[j].s * b.job[j].r, kQrThreads) * b.job[j].B;
  }
  DPRC_LAUNCH(hpp_csum_batch_kernel, dim3((unsigned)blocks), dim3(kQrThreads), 0, st, b);
  return hipGetLastError();
}

hipError_t launch_hpp_rows_batch(const FinalBatch& bt, hipStream_t st) {
  if (bt.njobs < 1 || bt.njobs > kFinMaxJobs) return hipErrorInvalidValue;
  FinalBatch b = bt;
  int blocks = 0;
  for (int j = 0; j < b.njobs; ++j) {
    b.blk0[j] = blocks;
    blocks += b.job[j].nchunk * b.job[j].B;
  }
  const int s = b.job[0].s;
  const size_t lds = (size_t)s * b.job[0].r * 4;
  if (s <= 8) DPRC_LAUNCH(hpp_rows_batch_kernel<8>, dim3((unsigned)blocks), dim3(kQrThreads), lds, st, b);
  else if (s <= 16) DPRC_LAUNCH(hpp_rows_batch_kernel<16>, dim3((unsigned)blocks), dim3(kQrThreads), lds, st, b);
  else DPRC_LAUNCH(hpp_rows_batch_kernel<32>, dim3((unsigned)blocks), dim3(kQrThreads), lds, st, b);
  return hipGetLastError();
}

hipError_t launch_hpp_sum_batch(const FinalBatch& bt, hipStream_t st) {
  if (bt.njobs < 1 || bt.njobs > kFinMaxJobs) return hipErrorInvalidValue;
  DPRC_LAUNCH(hpp_sum_batch_kernel, dim3((unsigned)bt.job[0].B), dim3(kQrThreads), 0, st, bt);
  return hipGetLastError();
}

int32_t final_chunks(int64_t n) { return (int32_t)ceil_div(n, kFinRows); }

}  // namespace dprc
