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
  c[i] = clip_factor(n2[i], C);
}

hipError_t launch_clip_scale(const float* n2, int64_t B, float C, float* c, hipStream_t st) {
  DPRC_LAUNCH(clip_scale_kernel, dim3((unsigned)ceil_div(B, 256)), dim3(256), 0, st, n2, B, C, c);
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
// Element e: Philox block e/4 of stream 2 keyed by (seed, tensor), through box_muller.
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
