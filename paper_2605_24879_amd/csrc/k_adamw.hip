// Private AdamW step: noise, batch normalisation and one AdamW update of a
// layer's fp32 master weights in one pass (Algorithm 1's last two steps).
//
// A workgroup owns a 64 x 64 tile of the [d, p] master.  Each thread takes four
// consecutive columns of four rows (16-byte loads along the rows); the bf16
// copy of the updated tile is staged in LDS and written transposed, 64 rows of
// the [p, d] weight at 128 contiguous bytes each.  Noise element e = r*p + c
// uses Philox block e/4 of stream 2, as the standalone noise kernel does.
#include <algorithm>
#include "device.hpp"
#include "kernels.hpp"

namespace dprc {

constexpr int kAT = 64;

__device__ __forceinline__ float noise_elem(uint32_t key0, uint32_t key1, uint32_t tensor, int64_t e) {
  const uint64_t q = (uint64_t)e >> 2;
  const u32x4 x = philox4x32_10(u32x4{(uint32_t)q, (uint32_t)(q >> 32), tensor, kStreamNoise}, key0, key1);
  float n0, n1;
  if ((e & 2) == 0) box_muller(x.x, x.y, n0, n1);
  else box_muller(x.z, x.w, n0, n1);
  return (e & 1) ? n1 : n0;
}

__device__ __forceinline__ void adamw1(const AdamArgs& a, float g, float& th, float& m, float& v) {
  th *= a.decay;
  m = fmaf(a.beta1, m, a.one_minus_beta1 * g);
  v = fmaf(a.beta2, v, a.one_minus_beta2 * g * g);
  const float denom = fmaf(sqrtf(v), a.inv_sqrt_bc2, a.eps);
  th = fmaf(-a.step_size, m / denom, th);
}

// VEC: p, ldt, ldg multiples of 4 and 16-byte aligned bases (float4 access,
// whole noise blocks); otherwise element access with bounds checks.
template <bool VEC>
__global__ __launch_bounds__(256) void private_adamw_kernel(AdamArgs a) {
  __shared__ __attribute__((aligned(16))) uint16_t wt[kAT][kAT + 8];          // [column][row] of the bf16 tile
  const int tid = threadIdx.x;
  const int cq = tid & 15, rg = tid >> 4;
  const int64_t c0 = (int64_t)blockIdx.x * kAT, r0 = (int64_t)blockIdx.y * kAT;
  const int64_t c = c0 + 4 * cq;
  const bool noise = a.noise_scale != 0.f;
#pragma unroll
  for (int rr = 0; rr < 4; ++rr) {
    const int lr = rg + 16 * rr;
    const int64_t r = r0 + lr;
    float th[4] = {0.f, 0.f, 0.f, 0.f};
    if (r < a.d) {
      float* tp = a.theta + r * a.ldt + c;
      float* mp = a.m + r * a.ldt + c;
      float* vp = a.v + r * a.ldt + c;
      const float* gp = a.G + r * a.ldg + c;
      float g[4], m[4], v[4], n[4] = {0.f, 0.f, 0.f, 0.f};
      if (VEC && c + 4 <= a.p) {
        const float4 g4 = *reinterpret_cast<const float4*>(gp);
        const float4 t4 = *reinterpret_cast<const float4*>(tp);
        const float4 m4 = *reinterpret_cast<const float4*>(mp);
        const float4 v4 = *reinterpret_cast<const float4*>(vp);
        g[0] = g4.x; g[1] = g4.y; g[2] = g4.z; g[3] = g4.w;
        th[0] = t4.x; th[1] = t4.y; th[2] = t4.z; th[3] = t4.w;
        m[0] = m4.x; m[1] = m4.y; m[2] = m4.z; m[3] = m4.w;
        v[0] = v4.x; v[1] = v4.y; v[2] = v4.z; v[3] = v4.w;
        if (noise) {
          const uint64_t q = (uint64_t)(r * a.p + c) >> 2;
          const u32x4 x = philox4x32_10(u32x4{(uint32_t)q, (uint32_t)(q >> 32), a.tensor, kStreamNoise}, a.key0, a.key1);
          box_muller(x.x, x.y, n[0], n[1]);
          box_muller(x.z, x.w, n[2], n[3]);
        }
#pragma unroll
        for (int j = 0; j < 4; ++j) adamw1(a, fmaf(a.noise_scale, n[j], g[j]) * a.inv_batch, th[j], m[j], v[j]);
        *reinterpret_cast<float4*>(tp) = float4{th[0], th[1], th[2], th[3]};
        *reinterpret_cast<float4*>(mp) = float4{m[0], m[1], m[2], m[3]};
        *reinterpret_cast<float4*>(vp) = float4{v[0], v[1], v[2], v[3]};
      } else {
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          if (c + j >= a.p) break;
          float gj = gp[j], tj = tp[j], mj = mp[j], vj = vp[j];
          const float nj = noise ? noise_elem(a.key0, a.key1, a.tensor, r * a.p + c + j) : 0.f;
          adamw1(a, fmaf(a.noise_scale, nj, gj) * a.inv_batch, tj, mj, vj);
          tp[j] = tj; mp[j] = mj; vp[j] = vj;
          th[j] = tj;
        }
      }
    }
    if (a.w) {
#pragma unroll
      for (int j = 0; j < 4; ++j) wt[4 * cq + j][lr] = (uint16_t)f32_to_bf16(th[j]);
    }
  }
  if (!a.w) return;
  __syncthreads();
  // transposed write: thread -> weight row c0 + tid/4, 16 of the tile's rows (r) from 16*(tid%4)
  const int lc = tid >> 2, part = tid & 3;
  const int64_t wc = c0 + lc;
  if (wc >= a.p) return;
  uint16_t* wrow = a.w + wc * a.ldw + r0 + 16 * part;
  const uint16_t* src = &wt[lc][16 * part];
  const int64_t rbase = r0 + 16 * part;
  if (a.wvec && rbase + 16 <= a.d) {
    const uint4* s4 = reinterpret_cast<const uint4*>(src);
    reinterpret_cast<uint4*>(wrow)[0] = s4[0];
    reinterpret_cast<uint4*>(wrow)[1] = s4[1];
  } else {
    for (int j = 0; j < 16; ++j)
      if (rbase + j < a.d) wrow[j] = src[j];
  }
}

hipError_t launch_private_adamw(const AdamArgs& a, hipStream_t st) {
  if (a.d == 0 || a.p == 0) return hipSuccess;
  const dim3 grid((unsigned)ceil_div(a.p, kAT), (unsigned)ceil_div(a.d, kAT));
  if (a.vec) DPRC_LAUNCH(private_adamw_kernel<true>, grid, dim3(256), 0, st, a);
  else DPRC_LAUNCH(private_adamw_kernel<false>, grid, dim3(256), 0, st, a);
  return hipGetLastError();
}

}  // namespace dprc
