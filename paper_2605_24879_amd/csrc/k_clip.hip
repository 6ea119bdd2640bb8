// Clip factors, clipped-gradient accumulation and Gaussian noise (Algorithm 1:
// scaled loss, second backward pass, noise addition).
#include <algorithm>
#include "device.hpp"
#include "kernels.hpp"

namespace dprc {

// ---- c_i = min(1, C / sqrt(n_i)) -------------------------------------------------------
__global__ void clip_scale_kernel(const float* n2, int64_t B, float C, float* c) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= B) return;
  const float v = n2[i];
  float r;
  if (!(v >= 0.f) || isinf(v)) r = 0.f;       // NaN, negative, +inf
  else if (v <= C * C) r = 1.f;
  else r = C / sqrtf(v);
  c[i] = r;
}

hipError_t launch_clip_scale(const float* n2, int64_t B, float C, float* c, hipStream_t st) {
  DPRC_LAUNCH(clip_scale_kernel, dim3((unsigned)ceil_div(B, 256)), dim3(256), 0, st, n2, B, C, c);
  return hipGetLastError();
}

// ---- grad = sum_i c_i A_i^T E_i on bf16 matrix cores ---------------------------------------
// Workgroup tile 128 (d) x 128 (p), four waves of 64 x 64; the contraction runs
// over tokens, sample by sample.  Both operands are token-major, so 64-token
// tiles of A and E are staged in LDS and read back token-contiguous with the
// LDS transpose read.  The per-sample factor is applied to the fp32
// accumulator: before the first stage of sample i the accumulator is rescaled
// by c_prev / c_i, and by the last c at the end, so the result is
// sum_i c_i (A_i^T E_i) with no bf16 rounding of c_i * E.  Samples with c_i = 0
// are skipped.  Splits over the (sample, stage) list write fp32 partials that
// a second kernel sums in a fixed order.
constexpr int kGT = 128;                   // tile edge
constexpr int kGLd = kGT + 8;              // padded LDS row

template <bool FAST>
__global__ __launch_bounds__(kBlock) void gemm_kernel(GemmArgs a) {
  __shared__ __attribute__((aligned(16))) uint16_t la[2][kStage * kGLd];
  __shared__ __attribute__((aligned(16))) uint16_t le[2][kStage * kGLd];
  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
  const int g = lane >> 4, l16 = lane & 15, r4 = l16 >> 2, c4 = lane & 3;
  const int wm = wv >> 1, wn = wv & 1;
  const int p0 = blockIdx.x * kGT, d0 = blockIdx.y * kGT, split = blockIdx.z;
  const int sps = a.stages_per_sample;
  const int gs_begin = split * a.stages_per_split;
  const int gs_end = min(a.B * sps, gs_begin + a.stages_per_split);
  const int lr0 = tid >> 4, lc = (tid & 15) * 8;
  const int64_t ja = (int64_t)d0 + lc, je = (int64_t)p0 + lc;

  auto next_valid = [&](int gs) {
    while (gs < gs_end && a.c[gs / sps] == 0.f) gs = (gs / sps + 1) * sps;
    return gs;
  };
  uint4 ga[4], ge[4];
  auto gload = [&](int gs) {
    const int i = gs / sps;
    const int64_t tok0 = (int64_t)(gs - i * sps) * kStage;
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int64_t t = tok0 + lr0 + 16 * q;
      const bool ok = t < a.T;
      const uint16_t* as = a.A + (int64_t)i * a.a_ss;
      const uint16_t* es = a.E + (int64_t)i * a.e_ss;
      ga[q] = load_bf16x8<FAST>(as + (ok ? t : 0) * a.lda, ja, a.d, ok, as);
      ge[q] = load_bf16x8<FAST>(es + (ok ? t : 0) * a.lde, je, a.p, ok, es);
    }
  };
  auto swrite = [&](int buf) {
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      *reinterpret_cast<uint4*>(&la[buf][(lr0 + 16 * q) * kGLd + lc]) = ga[q];
      *reinterpret_cast<uint4*>(&le[buf][(lr0 + 16 * q) * kGLd + lc]) = ge[q];
    }
  };

  f32x4_t acc[4][4];
#pragma unroll
  for (int x = 0; x < 4; ++x)
#pragma unroll
    for (int y = 0; y < 4; ++y) acc[x][y] = f32x4_t{0.f, 0.f, 0.f, 0.f};

  int gs = next_valid(gs_begin);
  if (gs < gs_end) {
    gload(gs);
    swrite(0);
  }
  __syncthreads();
  int buf = 0, cur_i = -1;
  float cur_c = 0.f;
  while (gs < gs_end) {
    const int gnext = next_valid(gs + 1);
    if (gnext < gs_end) gload(gnext);
    const int si = gs / sps;
    if (si != cur_i) {
      const float ci = a.c[si];
      if (cur_i >= 0) {
        const float ratio = cur_c / ci;
#pragma unroll
        for (int x = 0; x < 4; ++x)
#pragma unroll
          for (int y = 0; y < 4; ++y) acc[x][y] *= ratio;
      }
      cur_c = ci;
      cur_i = si;
    }
#pragma unroll
    for (int ks = 0; ks < 2; ++ks) {
      uint4 av[4], bv[4];
#pragma unroll
      for (int x = 0; x < 4; ++x) {
        const uint16_t* pa = &la[buf][(32 * ks + 8 * g + r4) * kGLd + 16 * (4 * wm + x) + 4 * c4];
        av[x] = make_u4(lds_read_tr16(pa), lds_read_tr16(pa + 4 * kGLd));
        const uint16_t* pe = &le[buf][(32 * ks + 8 * g + r4) * kGLd + 16 * (4 * wn + x) + 4 * c4];
        bv[x] = make_u4(lds_read_tr16(pe), lds_read_tr16(pe + 4 * kGLd));
      }
#pragma unroll
      for (int x = 0; x < 4; ++x)
#pragma unroll
        for (int y = 0; y < 4; ++y) acc[x][y] = mfma16x16x32(av[x], bv[y], acc[x][y]);
    }
    if (gnext < gs_end) swrite(buf ^ 1);
    __syncthreads();
    buf ^= 1;
    gs = gnext;
  }

  // epilogue: lane holds rows d0 + 16*(4wm+x) + 4g + q, column p0 + 16*(4wn+y) + l16
  float* dst;
  int64_t ld;
  bool direct = a.S == 1;
  if (direct) {
    dst = a.out;
    ld = a.ldo;
  } else {
    dst = a.part + (int64_t)split * a.d * a.p;
    ld = a.p;
  }
#pragma unroll
  for (int x = 0; x < 4; ++x)
#pragma unroll
    for (int y = 0; y < 4; ++y) {
      const int col = p0 + 16 * (4 * wn + y) + l16;
      if (col >= a.p) continue;
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const int row = d0 + 16 * (4 * wm + x) + 4 * g + q;
        if (row >= a.d) continue;
        const float v = acc[x][y][q] * cur_c;
        float* o = dst + (int64_t)row * ld + col;
        if (direct && a.accumulate) *o += v;
        else *o = v;
      }
    }
}

hipError_t launch_gemm(const GemmArgs& a, hipStream_t st) {
  dim3 grid((unsigned)ceil_div(a.p, kGT), (unsigned)ceil_div(a.d, kGT), (unsigned)a.S);
  if (a.vec_a && a.vec_e && a.d % 8 == 0 && a.p % 8 == 0)
    DPRC_LAUNCH(gemm_kernel<true>, grid, dim3(kBlock), 0, st, a);
  else
    DPRC_LAUNCH(gemm_kernel<false>, grid, dim3(kBlock), 0, st, a);
  return hipGetLastError();
}

__global__ void splitk_reduce_kernel(const float* part, int32_t S, int32_t d, int32_t p, float* out,
                                     int64_t ldo, int accumulate) {
  const int64_t total = (int64_t)d * p;
  for (int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; e < total;
       e += (int64_t)gridDim.x * blockDim.x) {
    float v = 0.f;
    for (int s = 0; s < S; ++s) v += part[(int64_t)s * total + e];
    const int64_t r = e / p, c = e - r * p;
    float* o = out + r * ldo + c;
    *o = accumulate ? *o + v : v;
  }
}

hipError_t launch_splitk_reduce(const float* part, int32_t S, int32_t d, int32_t p, float* out,
                                int64_t ldo, int accumulate, hipStream_t st) {
  const int64_t total = (int64_t)d * p;
  const unsigned blocks = (unsigned)std::min<int64_t>(8192, ceil_div(total, 256));
  DPRC_LAUNCH(splitk_reduce_kernel, dim3(blocks), dim3(256), 0, st, part, S, d, p, out, ldo, accumulate);
  return hipGetLastError();
}

// ---- fp32 inputs (SIMT): one thread per gradient entry --------------------------------------
__global__ void gemm_f32_kernel(const float* A, int64_t lda, int64_t a_ss, const float* E, int64_t lde,
                                int64_t e_ss, int32_t B, int32_t T, int32_t d, int32_t p,
                                const float* c, float* out, int64_t ldo, int accumulate) {
  const int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= (int64_t)d * p) return;
  const int j = (int)(idx / p), u = (int)(idx - (int64_t)j * p);
  float total = 0.f;
  for (int i = 0; i < B; ++i) {
    const float ci = c[i];
    if (ci == 0.f) continue;
    float s = 0.f;
    for (int t = 0; t < T; ++t)
      s = fmaf(A[(int64_t)i * a_ss + (int64_t)t * lda + j], E[(int64_t)i * e_ss + (int64_t)t * lde + u], s);
    total = fmaf(ci, s, total);
  }
  float* o = out + (int64_t)j * ldo + u;
  *o = accumulate ? *o + total : total;
}

hipError_t launch_gemm_f32(const float* A, int64_t lda, int64_t a_ss, const float* E, int64_t lde,
                           int64_t e_ss, int32_t B, int32_t T, int32_t d, int32_t p,
                           const float* c, float* out, int64_t ldo, int accumulate,
                           hipStream_t st) {
  const int64_t total = (int64_t)d * p;
  DPRC_LAUNCH(gemm_f32_kernel, dim3((unsigned)ceil_div(total, 256)), dim3(256), 0, st, A, lda,
                     a_ss, E, lde, e_ss, B, T, d, p, c, out, ldo, accumulate);
  return hipGetLastError();
}

// ---- Gaussian noise ----------------------------------------------------------------------------
// Element e: Philox block e/4 of stream 2 keyed by (seed, tensor); Box-Muller on
// word pairs with uniforms (floor(x / 2^9) + 1/2) * 2^-23, exact in fp32.
__device__ __forceinline__ void box_muller(uint32_t x0, uint32_t x1, float& n0, float& n1) {
  const float u1 = ((float)(x0 >> 9) + 0.5f) * 0x1p-23f;
  const float u2 = ((float)(x1 >> 9) + 0.5f) * 0x1p-23f;
  const float r = sqrtf(-2.f * logf(u1));
  float sn, cs;
  sincospif(2.f * u2, &sn, &cs);
  n0 = r * cs;
  n1 = r * sn;
}

__global__ void noise_kernel(float* g, int64_t numel, float scale, uint32_t key0, uint32_t key1,
                             uint32_t tensor_id) {
  const int64_t nq = (numel + 3) >> 2;
  const bool vec = (reinterpret_cast<uintptr_t>(g) & 15) == 0;
  for (int64_t q = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; q < nq;
       q += (int64_t)gridDim.x * blockDim.x) {
    const u32x4 x = philox4x32_10(u32x4{(uint32_t)q, (uint32_t)((uint64_t)q >> 32), tensor_id, kStreamNoise}, key0, key1);
    float n[4];
    box_muller(x.x, x.y, n[0], n[1]);
    box_muller(x.z, x.w, n[2], n[3]);
    const int64_t e0 = q << 2;
    if (vec && e0 + 4 <= numel) {
      float4 v = *reinterpret_cast<float4*>(g + e0);
      v.x = fmaf(scale, n[0], v.x);
      v.y = fmaf(scale, n[1], v.y);
      v.z = fmaf(scale, n[2], v.z);
      v.w = fmaf(scale, n[3], v.w);
      *reinterpret_cast<float4*>(g + e0) = v;
    } else {
      for (int k = 0; k < 4; ++k)
        if (e0 + k < numel) g[e0 + k] = fmaf(scale, n[k], g[e0 + k]);
    }
  }
}

hipError_t launch_noise(float* g, int64_t numel, float scale, uint32_t key0, uint32_t key1,
                        uint32_t tensor_id, hipStream_t st) {
  const int64_t nq = (numel + 3) / 4;
  const unsigned blocks = (unsigned)std::min<int64_t>(16384, ceil_div(nq, 256));
  DPRC_LAUNCH(noise_kernel, dim3(blocks), dim3(256), 0, st, g, numel, scale, key0, key1, tensor_id);
  return hipGetLastError();
}

}  // namespace dprc
