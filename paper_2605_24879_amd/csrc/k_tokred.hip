// Token reduction M_i = X_i^T Y_i on bf16 matrix cores (the A_i^T Y_i step of the
// Hutchinson estimator, Algorithm 2; also the W_S, O S and [U | W_P] steps of
// Hutch++), followed by either the squared-norm estimate or a store of M_i.
//
// A workgroup owns one sample, a 128-column tile of X and a contiguous range of
// tokens.  X tiles (64 tokens x 128 columns, 256 bytes per token row) are
// loaded with coalesced 16-byte reads, double-buffered through LDS and read
// back token-contiguous with the gfx950 LDS transpose read, which is the
// operand layout of the MFMA (the contraction runs over tokens, X is stored
// token-major).  Y (bf16 hi + lo, already token-contiguous) is read directly.
// Splits over tokens are summed in a fixed order by the last workgroup to
// finish a tile, and per-tile squares by the last tile of a sample, so the
// result does not depend on scheduling.
#include <algorithm>
#include "device.hpp"
#include "kernels.hpp"

namespace dprc {

__device__ __forceinline__ float block_sum_f(float v, float* red4) {
  v = wave_sum(v);
  const int tid = threadIdx.x;
  __syncthreads();
  if ((tid & 63) == 0) red4[tid >> 6] = v;
  __syncthreads();
  return red4[0] + red4[1] + red4[2] + red4[3];
}

__device__ __forceinline__ double block_sum_d(double v, double* red4) {
  v = wave_sum(v);
  const int tid = threadIdx.x;
  __syncthreads();
  if ((tid & 63) == 0) red4[tid >> 6] = v;
  __syncthreads();
  return (red4[0] + red4[1]) + (red4[2] + red4[3]);
}

__device__ __forceinline__ void store4(const TokredArgs& a, int i, int c, int j, const float v[4]) {
  if (c >= a.ncols) return;
  if (a.M) {
    float* dst = a.M + (int64_t)i * a.m_ss + (int64_t)c * a.m_ld;
#pragma unroll
    for (int q = 0; q < 4; ++q)
      if (j + q < a.n) dst[j + q] = v[q];
  }
  if (a.Mhi) {
    uint16_t* hi = a.Mhi + (int64_t)i * a.mh_ss + (int64_t)c * a.mh_ld;
    uint16_t* lo = a.Mlo + (int64_t)i * a.mh_ss + (int64_t)c * a.mh_ld;
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      uint32_t h, l;
      split_bf16(j + q < a.n ? v[q] : 0.f, h, l);
      hi[j + q] = (uint16_t)h;
      lo[j + q] = (uint16_t)l;
    }
  }
}

template <int NB, bool FAST>
__global__ __launch_bounds__(kBlock) void tokred_kernel(TokredArgs a) {
  __shared__ __attribute__((aligned(16))) uint16_t lds[2][kStage * kLdsLd];
  __shared__ double dred[4];
  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
  const int g = lane >> 4, l16 = lane & 15, r4 = l16 >> 2, c4 = lane & 3;
  const int i = blockIdx.y;
  const int tile = blockIdx.x / a.S, s = blockIdx.x - tile * a.S;
  const int j0 = tile * kTile;
  const int64_t tb = (int64_t)s * a.stages_per_split * kStage;
  const int64_t te = min((int64_t)a.T, tb + (int64_t)a.stages_per_split * kStage);
  const int nst = te > tb ? (int)((te - tb + kStage - 1) / kStage) : 0;

  const int lr0 = tid >> 4, lc = (tid & 15) * 8;
  const int64_t jc = (int64_t)j0 + lc;
  const uint16_t* xs = a.X + (int64_t)i * a.x_ss;

  uint4 gv[4];
  auto gload = [&](int st) {
    const int64_t tok0 = tb + (int64_t)st * kStage;
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int64_t t = tok0 + lr0 + 16 * q;
      gv[q] = load_bf16x8<FAST>(xs + (t < te ? t : 0) * a.ldx, jc, a.n, t < te, xs);
    }
  };
  auto swrite = [&](int buf) {
#pragma unroll
    for (int q = 0; q < 4; ++q)
      *reinterpret_cast<uint4*>(&lds[buf][(lr0 + 16 * q) * kLdsLd + lds_swz(lr0 + 16 * q, lc)]) = gv[q];
  };

  f32x4_t acc[2][2][NB];
#pragma unroll
  for (int x = 0; x < 2; ++x)
#pragma unroll
    for (int h = 0; h < 2; ++h)
#pragma unroll
      for (int nb = 0; nb < NB; ++nb) acc[x][h][nb] = f32x4_t{0.f, 0.f, 0.f, 0.f};

  if (nst > 0) {
    gload(0);
    swrite(0);
  }
  __syncthreads();
  const uint16_t* ybase = a.Yt + (int64_t)i * a.T_pad + 8 * g;
  for (int st = 0; st < nst; ++st) {
    const int buf = st & 1;
    if (st + 1 < nst) gload(st + 1);
    const int64_t ytok = tb + (int64_t)st * kStage;
#pragma unroll
    for (int ks = 0; ks < 2; ++ks) {
      uint4 bop[2][NB];
#pragma unroll
      for (int h = 0; h < 2; ++h)
#pragma unroll
        for (int nb = 0; nb < NB; ++nb)
          bop[h][nb] = *reinterpret_cast<const uint4*>(
              ybase + ((int64_t)h * a.ncols_pad + 16 * nb + l16) * a.yt_ld + ytok + 32 * ks);
#pragma unroll
      for (int x = 0; x < 2; ++x) {
        const int mb = 2 * wv + x;
        // rows 32ks + 8g + r4 (+4) all have bit 3 equal to g & 1
        const uint16_t* p = &lds[buf][(32 * ks + 8 * g + r4) * kLdsLd + ((16 * mb + 4 * c4) ^ ((g & 1) << 6))];
        const uint4 av = make_u4(lds_read_tr16(p), lds_read_tr16(p + 4 * kLdsLd));
#pragma unroll
        for (int h = 0; h < 2; ++h)
#pragma unroll
          for (int nb = 0; nb < NB; ++nb) acc[x][h][nb] = mfma16x16x32(av, bop[h][nb], acc[x][h][nb]);
      }
    }
    if (st + 1 < nst) swrite(buf ^ 1);
    __syncthreads();
  }

  // W = hi part + lo part; lane holds rows j0 + 16*mb + 4*g + (0..3) of column 16*nb + l16
  float w[2][NB][4];
#pragma unroll
  for (int x = 0; x < 2; ++x)
#pragma unroll
    for (int nb = 0; nb < NB; ++nb)
#pragma unroll
      for (int q = 0; q < 4; ++q) w[x][nb][q] = acc[x][0][nb][q] + acc[x][1][nb][q];

  const int64_t tslot = (int64_t)i * a.ntiles + tile;
  if (a.S == 1) {
    if (a.mode == 0) {
      double sq = 0.0;
#pragma unroll
      for (int x = 0; x < 2; ++x)
#pragma unroll
        for (int nb = 0; nb < NB; ++nb)
#pragma unroll
          for (int q = 0; q < 4; ++q) sq += (double)(w[x][nb][q] * w[x][nb][q]);
      sq = block_sum_d(sq, dred);
      if (tid == 0) a.tilesq[tslot] = sq;
    } else {
#pragma unroll
      for (int x = 0; x < 2; ++x)
#pragma unroll
        for (int nb = 0; nb < NB; ++nb) store4(a, i, 16 * nb + l16, j0 + 16 * (2 * wv + x) + 4 * g, w[x][nb]);
    }
    return;
  }
  // token splits: publish the partial tile; the finish kernel sums the splits in order
  float* mypart = a.part + (tslot * a.S + s) * (int64_t)a.ncols_pad * kTile;
#pragma unroll
  for (int x = 0; x < 2; ++x)
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) {
      float* dst = mypart + (int64_t)(16 * nb + l16) * kTile + 16 * (2 * wv + x) + 4 * g;
      *reinterpret_cast<float4*>(dst) = float4{w[x][nb][0], w[x][nb][1], w[x][nb][2], w[x][nb][3]};
    }
}

// Sum of the token splits of one tile, in split order: its squared norm (mode 0)
// or the stored tile (mode 1).
__global__ __launch_bounds__(kBlock) void tokred_splits_kernel(TokredArgs a) {
  __shared__ double dred[4];
  const int tid = threadIdx.x, tile = blockIdx.x, i = blockIdx.y;
  const int64_t tslot = (int64_t)i * a.ntiles + tile;
  const float* tp = a.part + tslot * a.S * (int64_t)a.ncols_pad * kTile;
  double sq = 0.0;
  for (int gi = tid; gi < a.ncols_pad * (kTile / 4); gi += kBlock) {
    const int c = gi / (kTile / 4), j4 = (gi - c * (kTile / 4)) * 4;
    float v[4] = {0.f, 0.f, 0.f, 0.f};
    for (int s2 = 0; s2 < a.S; ++s2) {
      const float4 pv = *reinterpret_cast<const float4*>(tp + ((int64_t)s2 * a.ncols_pad + c) * kTile + j4);
      v[0] += pv.x; v[1] += pv.y; v[2] += pv.z; v[3] += pv.w;
    }
    if (a.mode == 0) {
      if (c < a.ncols)
        for (int q = 0; q < 4; ++q) sq += (double)(v[q] * v[q]);
    } else {
      store4(a, i, c, tile * kTile + j4, v);
    }
  }
  if (a.mode == 0) {
    sq = block_sum_d(sq, dred);
    if (tid == 0) a.tilesq[tslot] = sq;
  }
}

// estimate_i = scale * sum over tiles (in tile order), into n2 and the per-layer copy
__global__ __launch_bounds__(kBlock) void tokred_sample_kernel(TokredArgs a) {
  __shared__ double dred[4];
  const int i = blockIdx.x;
  double t = 0.0;
  for (int k = threadIdx.x; k < a.ntiles; k += kBlock) t += a.tilesq[(int64_t)i * a.ntiles + k];
  t = block_sum_d(t, dred);
  if (threadIdx.x == 0) {
    const float est = (float)(t * (double)a.scale);
    a.n2[i] = (a.accumulate ? a.n2[i] : 0.f) + est;
    if (a.n2_layer) a.n2_layer[i] = est;
  }
}

hipError_t launch_tokred_splits(const TokredArgs& a, hipStream_t st) {
  DPRC_LAUNCH(tokred_splits_kernel, dim3((unsigned)a.ntiles, (unsigned)a.B), dim3(kBlock), 0, st, a);
  return hipGetLastError();
}

hipError_t launch_tokred_sample(const TokredArgs& a, hipStream_t st) {
  DPRC_LAUNCH(tokred_sample_kernel, dim3((unsigned)a.B), dim3(kBlock), 0, st, a);
  return hipGetLastError();
}

hipError_t launch_tokred(const TokredArgs& a, hipStream_t st) {
  dim3 grid((unsigned)(a.ntiles * a.S), (unsigned)a.B);
  const bool fast = a.vec && a.n % 8 == 0;
#define DPRC_TOKRED_CASE(NB)                                                                   \
  case NB:                                                                                     \
    if (fast) DPRC_LAUNCH((tokred_kernel<NB, true>), grid, dim3(kBlock), 0, st, a);     \
    else DPRC_LAUNCH((tokred_kernel<NB, false>), grid, dim3(kBlock), 0, st, a);         \
    break;
  switch (a.ncols_pad / 16) {
    DPRC_TOKRED_CASE(1)
    DPRC_TOKRED_CASE(2)
    DPRC_TOKRED_CASE(3)
    DPRC_TOKRED_CASE(4)
    DPRC_TOKRED_CASE(5)
    DPRC_TOKRED_CASE(6)
    DPRC_TOKRED_CASE(8)
    DPRC_TOKRED_CASE(12)
    DPRC_TOKRED_CASE(16)
    default: return hipErrorInvalidValue;
  }
#undef DPRC_TOKRED_CASE
  return hipGetLastError();
}

// ---- fp32 inputs (SIMT) ---------------------------------------------------------------
__global__ void tokred_f32_kernel(TokredF32Args a) {
  const int64_t total = (int64_t)a.B * a.n * a.ncols;
  const int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= total) return;
  const int j = (int)(idx % a.n);
  const int64_t r = idx / a.n;
  const int c = (int)(r % a.ncols), i = (int)(r / a.ncols);
  const float* x = a.X + (int64_t)i * a.x_ss + j;
  const float* y = a.Y + (int64_t)i * a.T * a.ncols + c;
  float s = 0.f;
  for (int t = 0; t < a.T; ++t) s = fmaf(x[(int64_t)t * a.ldx], y[(int64_t)t * a.ncols], s);
  a.M[(int64_t)i * a.m_ss + (int64_t)c * a.m_ld + j] = s;
}

hipError_t launch_tokred_f32(const TokredF32Args& a, hipStream_t st) {
  const int64_t total = (int64_t)a.B * a.n * a.ncols;
  DPRC_LAUNCH(tokred_f32_kernel, dim3((unsigned)ceil_div(total, 256)), dim3(256), 0, st, a);
  return hipGetLastError();
}

__global__ __launch_bounds__(kBlock) void sample_sq_kernel(const float* M, int64_t m_ld, int64_t m_ss,
                                                         int32_t ncols, int32_t n, float scale,
                                                         float* n2, float* n2_layer, int accumulate) {
  __shared__ double dred[4];
  const int i = blockIdx.x;
  double s = 0.0;
  for (int64_t e = threadIdx.x; e < (int64_t)ncols * n; e += kBlock) {
    const int c = (int)(e / n), j = (int)(e - (int64_t)c * n);
    const double v = M[(int64_t)i * m_ss + (int64_t)c * m_ld + j];
    s += v * v;
  }
  s = block_sum_d(s, dred);
  if (threadIdx.x == 0) {
    const float est = (float)(s * (double)scale);
    n2[i] = (accumulate ? n2[i] : 0.f) + est;
    if (n2_layer) n2_layer[i] = est;
  }
}

hipError_t launch_sample_sq(const float* M, int64_t m_ld, int64_t m_ss, int32_t B, int32_t ncols,
                            int32_t n, float scale, float* n2, float* n2_layer, int accumulate,
                            hipStream_t st) {
  DPRC_LAUNCH(sample_sq_kernel, dim3(B), dim3(kBlock), 0, st, M, m_ld, m_ss, ncols, n, scale,
                     n2, n2_layer, accumulate);
  return hipGetLastError();
}

}  // namespace dprc
