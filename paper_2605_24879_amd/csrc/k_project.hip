// Row projection Y = X R (the E_i Z step of the Hutchinson estimator, Algorithm 2;
// also the X' W_S and X [Q | P] steps of Hutch++), bf16 matrix cores.
//
// A workgroup owns 16*RB token rows of one sample and the whole width m; its
// four waves split m into interleaved 64-column sub-chunks (one 128-byte line
// per token row), so every load is a coalesced 16-byte read of a token row and
// X is read from HBM exactly once.  The +-1 probe columns are generated from
// Philox into LDS per workgroup (the probe matrix never exists in HBM) and
// expanded to bf16 in registers; +-1 is exact in bf16 and bf16 x bf16 products
// are exact in fp32, so Y is the fp32 sum of exact terms.  Dense columns
// (Hutch++) arrive pre-split into bf16 hi + lo and take two MFMAs.  The four
// partial Y tiles are summed in LDS and written as bf16 hi/lo pairs in the
// token-contiguous layout that the token-reduction kernel consumes directly.
#include <algorithm>
#include "device.hpp"
#include "kernels.hpp"

namespace dprc {

template <int RB, int NB, bool DENSE, bool FAST>
__global__ __launch_bounds__(kBlock) void project_kernel(ProjectArgs a) {
  extern __shared__ __attribute__((aligned(16))) uint32_t smem[];
  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
  const int g = lane >> 4, l16 = lane & 15;
  const int i = blockIdx.y;
  const int t0 = blockIdx.x * 16 * RB;
  const int wpc = a.words_per_chunk;
  uint32_t* zw = smem;                                            // [nz][wpc + 1]
  float* red = reinterpret_cast<float*>(smem + (a.nz > 0 ? a.nz * (wpc + 1) : 0));
  constexpr int RS = 16 * NB + 4;                                 // padded row of a reduction slot

  if (a.zero_ptr != nullptr && blockIdx.x == 0 && blockIdx.y == 0)
    for (int idx = tid; idx < a.zero_count; idx += kBlock) a.zero_ptr[idx] = 0u;

  const uint16_t* xs = a.X + (int64_t)i * a.x_ss;
  const uint16_t* rowp[RB];
  bool rowok[RB];
#pragma unroll
  for (int rb = 0; rb < RB; ++rb) {
    const int t = t0 + 16 * rb + l16;
    rowok[rb] = t < a.T;
    rowp[rb] = xs + (int64_t)(rowok[rb] ? t : 0) * a.ldx;
  }
  f32x4_t acc[RB][NB];
#pragma unroll
  for (int rb = 0; rb < RB; ++rb)
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) acc[rb][nb] = f32x4_t{0.f, 0.f, 0.f, 0.f};

  const uint16_t* rhi = DENSE ? a.Rhi + (int64_t)i * a.r_ss : nullptr;
  const uint16_t* rlo = DENSE ? a.Rlo + (int64_t)i * a.r_ss : nullptr;

  for (int64_t uc = 0; uc < a.m; uc += 32 * (int64_t)wpc) {
    if (a.nz > 0) {
      __syncthreads();
      const int nblk = wpc >> 2;
      const uint32_t wbase = (uint32_t)(uc >> 5);
      for (int idx = tid; idx < a.nz * nblk; idx += kBlock) {
        const int c = idx / nblk, b = idx - c * nblk;
        const uint32_t w0 = wbase + 4u * (uint32_t)b;
        u32x4 v;
        if (a.probe_kind == kProbeRademacher)
          v = rademacher_block(a.key0, a.key1, a.layer_id, a.stream_id, w0 >> 2, (uint32_t)c);
        else
          v = u32x4{hadamard_word(w0, c), hadamard_word(w0 + 1, c), hadamard_word(w0 + 2, c),
                    hadamard_word(w0 + 3, c)};
        uint32_t* dst = zw + c * (wpc + 1) + 4 * b;     // odd row stride: 16 lanes of 16 columns hit 16 banks
        dst[0] = v.x; dst[1] = v.y; dst[2] = v.z; dst[3] = v.w;
      }
      __syncthreads();
    }
    const int64_t rem = a.m - uc;
    const int nsub = (int)min((int64_t)(wpc >> 1), (rem + 63) >> 6);
    // U sub-chunks per batch: all their loads are issued before the first MFMA
    constexpr int U = RB == 1 ? 8 : (RB == 2 ? 4 : 2);
    for (int qb = wv; qb < nsub; qb += 4 * U) {
      uint4 av[U][RB][2];
#pragma unroll
      for (int uu = 0; uu < U; ++uu) {
        const int q = qb + 4 * uu;
        const int64_t u0 = uc + 64 * (int64_t)(q < nsub ? q : qb);
#pragma unroll
        for (int rb = 0; rb < RB; ++rb)
#pragma unroll
          for (int ks = 0; ks < 2; ++ks)
            av[uu][rb][ks] = load_bf16x8<FAST>(rowp[rb], u0 + 32 * ks + 8 * g, a.m, rowok[rb] && q < nsub, xs);
      }
#pragma unroll
      for (int uu = 0; uu < U; ++uu) {
        const int q = qb + 4 * uu;
        if (q >= nsub) break;                      // wave-uniform
        const int64_t u0 = uc + 64 * (int64_t)q;
#pragma unroll
        for (int ks = 0; ks < 2; ++ks) {
#pragma unroll
          for (int nb = 0; nb < NB; ++nb) {
            const int c = 16 * nb + l16;
            // select, not branch: every lane issues the same loads
            const int cz = c - a.nd;
            const bool isz = cz >= 0 && cz < a.nz;
            const uint32_t word = a.nz > 0 ? zw[(isz ? cz : 0) * (wpc + 1) + 2 * q + ks] : 0u;
            const uint4 zb = signs_to_bf16x8((word >> (8 * g)) & 0xFFu);
            uint4 bh = isz ? zb : uint4{0, 0, 0, 0}, bl = uint4{0, 0, 0, 0};
            if (DENSE && 16 * nb < a.nd) {   // uniform: only column blocks that hold dense columns load them
              const bool isd = c < a.nd;
              const int64_t off = (int64_t)(isd ? c : 0) * a.ld_r + u0 + 32 * ks + 8 * g;
              const uint4 dh = *reinterpret_cast<const uint4*>(rhi + off);
              const uint4 dl = *reinterpret_cast<const uint4*>(rlo + off);
              bh = isd ? dh : bh;
              bl = isd ? dl : bl;
            }
#pragma unroll
            for (int rb = 0; rb < RB; ++rb) {
              acc[rb][nb] = mfma16x16x32(av[uu][rb][ks], bh, acc[rb][nb]);
              if (DENSE) acc[rb][nb] = mfma16x16x32(av[uu][rb][ks], bl, acc[rb][nb]);
            }
          }
        }
      }
    }
  }

  // sum the four waves' partial tiles
  __syncthreads();
  float* slot = red + wv * (16 * RB) * RS;
#pragma unroll
  for (int rb = 0; rb < RB; ++rb)
#pragma unroll
    for (int nb = 0; nb < NB; ++nb)
#pragma unroll
      for (int ii = 0; ii < 4; ++ii) slot[(16 * rb + 4 * g + ii) * RS + 16 * nb + l16] = acc[rb][nb][ii];
  __syncthreads();
  const int rows = 16 * RB;
  uint16_t* yhi = a.Yt + (int64_t)i * a.T_pad + t0;
  uint16_t* ylo = yhi + (int64_t)a.ncols_pad * a.yt_ld;
  for (int idx = tid; idx < rows * 16 * NB; idx += kBlock) {
    const int c = idx / rows, r = idx - c * rows;
    if (c >= a.ncols_pad) continue;
    float y = 0.f;
#pragma unroll
    for (int s = 0; s < 4; ++s) y += red[s * rows * RS + r * RS + c];
    uint32_t h, l;
    split_bf16(y, h, l);
    yhi[(int64_t)c * a.yt_ld + r] = (uint16_t)h;
    ylo[(int64_t)c * a.yt_ld + r] = (uint16_t)l;
  }
}

template <int RB, int NB>
static hipError_t launch_rb_nb(const ProjectArgs& a, hipStream_t st) {
  const size_t zbytes = a.nz > 0 ? (size_t)a.nz * (a.words_per_chunk + 1) * 4 : 0;
  const size_t rbytes = (size_t)4 * 16 * RB * (16 * NB + 4) * 4;
  const size_t lds = zbytes + rbytes;
  dim3 grid((unsigned)(a.T_pad / (16 * RB)), (unsigned)a.B);
  const bool fast = a.vec && a.m % 8 == 0;
  if (a.nd > 0 && fast)
    DPRC_LAUNCH((project_kernel<RB, NB, true, true>), grid, dim3(kBlock), lds, st, a);
  else if (a.nd > 0)
    DPRC_LAUNCH((project_kernel<RB, NB, true, false>), grid, dim3(kBlock), lds, st, a);
  else if (fast)
    DPRC_LAUNCH((project_kernel<RB, NB, false, true>), grid, dim3(kBlock), lds, st, a);
  else
    DPRC_LAUNCH((project_kernel<RB, NB, false, false>), grid, dim3(kBlock), lds, st, a);
  return hipGetLastError();
}

template <int RB>
static hipError_t launch_rb(const ProjectArgs& a, hipStream_t st) {
  switch (a.ncols_pad / 16) {
    case 1: return launch_rb_nb<RB, 1>(a, st);
    case 2: return launch_rb_nb<RB, 2>(a, st);
    case 3: return launch_rb_nb<RB, 3>(a, st);
    case 4: return launch_rb_nb<RB, 4>(a, st);
    case 5: return launch_rb_nb<RB, 5>(a, st);
    case 6: return launch_rb_nb<RB, 6>(a, st);
    case 8: return launch_rb_nb<RB, 8>(a, st);
    case 12: return launch_rb_nb<RB, 12>(a, st);
    case 16: return launch_rb_nb<RB, 16>(a, st);
    default: return hipErrorInvalidValue;
  }
}

hipError_t launch_project(const ProjectArgs& a, int rows_per_wg, hipStream_t st) {
  switch (rows_per_wg) {
    case 16: return launch_rb<1>(a, st);
    case 32: return launch_rb<2>(a, st);
    case 64: return launch_rb<4>(a, st);
    default: return hipErrorInvalidValue;
  }
}

// ---- probe bits (verification export and the fp32 path) -------------------------
__global__ void probe_bits_kernel(int kind, uint32_t key0, uint32_t key1, uint32_t layer,
                                  uint32_t stream_id, int64_t m, int32_t k, uint32_t* out) {
  const int64_t nw = (m + 31) >> 5;
  const int64_t nblk = (nw + 3) >> 2;
  const int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= nblk * k) return;
  const int32_t c = (int32_t)(idx / nblk);
  const int64_t b = idx - (int64_t)c * nblk;
  uint32_t v[4];
  if (kind == kProbeRademacher) {
    const u32x4 r = rademacher_block(key0, key1, layer, stream_id, (uint32_t)b, (uint32_t)c);
    v[0] = r.x; v[1] = r.y; v[2] = r.z; v[3] = r.w;
  } else {
#pragma unroll
    for (int q = 0; q < 4; ++q) v[q] = hadamard_word((uint32_t)(4 * b + q), (uint32_t)c);
  }
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const int64_t w = 4 * b + q;
    if (w < nw) out[(int64_t)c * nw + w] = v[q] & tail_mask(m, w);
  }
}

hipError_t launch_probe_bits(int kind, uint32_t key0, uint32_t key1, uint32_t layer,
                             uint32_t stream_id, int64_t m, int32_t k, uint32_t* out,
                             hipStream_t st) {
  const int64_t nblk = ((m + 31) / 32 + 3) / 4;
  const int64_t total = nblk * k;
  if (total == 0) return hipSuccess;
  DPRC_LAUNCH(probe_bits_kernel, dim3((unsigned)ceil_div(total, 256)), dim3(256), 0, st,
                     kind, key0, key1, layer, stream_id, m, k, out);
  return hipGetLastError();
}

__global__ void fill_u32_kernel(uint32_t* p, int64_t n, uint32_t v) {
  for (int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; idx < n;
       idx += (int64_t)gridDim.x * blockDim.x)
    p[idx] = v;
}

hipError_t launch_fill_u32(uint32_t* p, int64_t n, uint32_t v, hipStream_t st) {
  if (n <= 0) return hipSuccess;
  const unsigned blocks = (unsigned)std::min<int64_t>(1024, ceil_div(n, 256));
  DPRC_LAUNCH(fill_u32_kernel, dim3(blocks), dim3(256), 0, st, p, n, v);
  return hipGetLastError();
}

// ---- fp32 inputs (SIMT) -------------------------------------------------------------
// One thread per (token row, column); plain fp32 sums.  Used for fp32 layers.
__global__ void project_f32_kernel(ProjectF32Args a) {
  const int64_t total = (int64_t)a.B * a.T * a.ncols;
  const int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= total) return;
  const int c = (int)(idx % a.ncols);
  const int64_t row = idx / a.ncols;
  const int i = (int)(row / a.T), t = (int)(row - (int64_t)i * a.T);
  const float* x = a.X + (int64_t)i * a.x_ss + (int64_t)t * a.ldx;
  float s = 0.f;
  if (c < a.nd) {
    const float* r = a.Rd + (int64_t)i * a.r_ss + (int64_t)c * a.ld_r;
    for (int u = 0; u < a.m; ++u) s = fmaf(x[u], r[u], s);
  } else {
    const int64_t nw = (a.m + 31) / 32;
    const uint32_t* zb = a.zbits + (int64_t)(c - a.nd) * nw;
    for (int u = 0; u < a.m; ++u) {
      const uint32_t bit = (zb[u >> 5] >> (u & 31)) & 1u;
      s += bit ? -x[u] : x[u];
    }
  }
  a.Y[row * a.ncols + c] = s;
}

hipError_t launch_project_f32(const ProjectF32Args& a, hipStream_t st) {
  const int64_t total = (int64_t)a.B * a.T * a.ncols;
  DPRC_LAUNCH(project_f32_kernel, dim3((unsigned)ceil_div(total, 256)), dim3(256), 0, st, a);
  return hipGetLastError();
}

}  // namespace dprc
