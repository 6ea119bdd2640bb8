// Gaussian Hutchinson probes (Algorithm 2 with normal-law probes, Section 3).
//
// Entry (u, j) of the m x k probe matrix: Philox block (u div 4, j, layer, 3)
// keyed by the seed; its words (x0, x1) give rows 4q, 4q+1 and (x2, x3) rows
// 4q+2, 4q+3 through Box-Muller.  The columns are written once per layer and
// step, column-major with a padded leading dimension (rows m .. ld-1 are zero),
// as bf16 hi + lo pairs for the matrix-core projection and/or as fp32.
#include <algorithm>
#include "device.hpp"
#include "kernels.hpp"

namespace dprc {

// One thread per (column j, row quad q); ld is a multiple of 4 or equals m.
__global__ void gauss_probe_kernel(uint32_t key0, uint32_t key1, uint32_t layer, int64_t m, int32_t k,
                                   int64_t ld, uint16_t* hi, uint16_t* lo, float* f32) {
  const int64_t nq = (ld + 3) >> 2;
  const int64_t total = nq * k;
  for (int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; idx < total;
       idx += (int64_t)gridDim.x * blockDim.x) {
    const int j = (int)(idx / nq);
    const int64_t q = idx - (int64_t)j * nq;
    float z[4] = {0.f, 0.f, 0.f, 0.f};
    if (4 * q < m) {
      const u32x4 x = philox4x32_10(u32x4{(uint32_t)q, (uint32_t)j, layer, kStreamGaussProbe}, key0, key1);
      box_muller(x.x, x.y, z[0], z[1]);
      box_muller(x.z, x.w, z[2], z[3]);
    }
    const int64_t r0 = 4 * q;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const int64_t r = r0 + e;
      if (r >= ld) break;
      const float v = r < m ? z[e] : 0.f;
      const int64_t o = (int64_t)j * ld + r;
      if (f32) f32[o] = v;
      if (hi) {
        uint32_t h, l;
        split_bf16(v, h, l);
        hi[o] = (uint16_t)h;
        lo[o] = (uint16_t)l;
      }
    }
  }
}

hipError_t launch_gauss_probe(uint32_t key0, uint32_t key1, uint32_t layer, int64_t m, int32_t k, int64_t ld,
                              uint16_t* hi, uint16_t* lo, float* f32, hipStream_t st) {
  const int64_t total = ((ld + 3) / 4) * k;
  if (total == 0) return hipSuccess;
  const unsigned blocks = (unsigned)std::min<int64_t>(8192, ceil_div(total, 256));
  DPRC_LAUNCH(gauss_probe_kernel, dim3(blocks), dim3(256), 0, st, key0, key1, layer, m, k, ld, hi, lo, f32);
  return hipGetLastError();
}

}  // namespace dprc
