// Row projection Y = X R (the E_i Z step of the Hutchinson estimator, Algorithm 2;
// also the X' W_S and X [Q | P] steps of Hutch++), bf16 matrix cores.
//
// A workgroup owns 16*RB token rows of one sample and the whole width m, walked
// in stages of 512 columns; in each stage every wave owns a 128-column slice.
// A wave reads its slice four token rows at a time (each row a whole 256-byte
// run, so every load instruction covers full cache lines), keeps P stages in
// flight in registers, and passes each stage through a private LDS tile (XOR
// swizzled, no bank conflicts on either side) to get the MFMA operand layout:
// 16 token rows x 8 consecutive columns per lane.  X is read from HBM exactly
// once.  The +-1 probe columns are generated from Philox into LDS per workgroup
// (the probe matrix never exists in HBM) and expanded to bf16 in registers;
// +-1 is exact in bf16 and bf16 x bf16 products are exact in fp32, so Y is the
// fp32 sum of exact terms.  Dense columns (Hutch++) arrive pre-split into bf16
// hi + lo and take two MFMAs.  The four waves' partial Y tiles are summed in
// LDS and written as bf16 hi/lo pairs in the token-contiguous layout that the
// token-reduction kernel consumes directly.
#include <algorithm>
#include "device.hpp"
#include "kernels.hpp"

namespace dprc {

constexpr int kProjSlice = 128;                 // columns per wave per stage
constexpr int kProjStage = 4 * kProjSlice;      // columns per stage

// Orders a wave's LDS accesses around a hand-off between its lanes (LDS
// operations of one wave execute in issue order; this keeps the compiler from
// moving them across).
__device__ __forceinline__ void wave_lds_fence() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

template <int V>
struct PInt {
  static constexpr int value = V;
};

// NBD: column blocks (of 16) holding dense columns, 0 when all columns are probes.
template <int RB, int NB, int NBD, bool FAST>
__device__ __forceinline__ void project_body(const ProjectArgs& a, int bx, int by) {
  extern __shared__ __attribute__((aligned(16))) uint32_t smem[];
  constexpr bool DENSE = NBD > 0;
  constexpr int P = (RB == 1 && !DENSE) ? 4 : 2;  // stages in flight per wave
  constexpr int NL = 4 * RB;                    // loads per lane per stage
  constexpr int ND = DENSE ? 4 * NBD : 1;       // dense operand fragments (hi and lo) per stage
  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
  const int g = lane >> 4, l16 = lane & 15;
  const int i = by;
  const int t0 = bx * 16 * RB;
  const int wpc = a.words_per_chunk;            // a multiple of 16: chunks are whole stages
  uint32_t* zw = smem;                                            // [nz][wpc + 1]
  uint32_t* region = smem + (a.nz > 0 ? a.nz * (wpc + 1) : 0);
  // X tiles [4 waves][16 RB rows][128 columns], later the reduction slots
  uint16_t* xt = reinterpret_cast<uint16_t*>(region) + wv * (16 * RB * kProjSlice);
  float* red = reinterpret_cast<float*>(region);
  constexpr int RS = 16 * NB + 4;                                 // padded row of a reduction slot

  if (a.zero_ptr != nullptr && bx == 0 && by == 0)
    for (int idx = tid; idx < a.zero_count; idx += kBlock) a.zero_ptr[idx] = 0u;

  // loads: lane -> row 4j + lane/16 of the tile (j = load index), 16-byte piece
  // p = (lane%16) ^ row of its slice, stored at LDS slot lane%16
  const uint16_t* xs = a.X + (int64_t)i * a.x_ss;
  const int vrows = max(0, min(16 * RB, a.T - t0));
  const __amdgpu_buffer_rsrc_t xr = buffer_rsrc(xs + (int64_t)t0 * a.ldx, (uint32_t)(vrows * a.ldx * 2));
  const int lrow = lane >> 4, lslot = lane & 15;
  const uint16_t* rowp[NL];
  uint32_t roff[NL];
  int lpiece[NL];
#pragma unroll
  for (int j = 0; j < NL; ++j) {
    const int rr = 4 * j + lrow;
    lpiece[j] = lslot ^ (rr & 15);
    roff[j] = (uint32_t)(rr * a.ldx) * 2u;
    const int t = t0 + rr;
    rowp[j] = xs + (int64_t)(t < a.T ? t : 0) * a.ldx;
  }

  f32x4_t acc[RB][NB];
#pragma unroll
  for (int rb = 0; rb < RB; ++rb)
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) acc[rb][nb] = f32x4_t{0.f, 0.f, 0.f, 0.f};

  // per column block: probe columns take +-1, others zero (dense columns come from R)
  uint32_t zmask[NB], zone[NB];
  int zrow[NB];
#pragma unroll
  for (int nb = 0; nb < NB; ++nb) {
    const int cz = 16 * nb + l16 - a.nd;
    const bool isz = cz >= 0 && cz < a.nz;
    zmask[nb] = isz ? 0x80008000u : 0u;
    zone[nb] = isz ? 0x3F803F80u : 0u;
    zrow[nb] = (isz ? cz : 0) * (wpc + 1);
  }
  const uint32_t psel = (uint32_t)g * 0x00010001u;               // byte g into both 16-bit halves

  const uint16_t* rhi = DENSE ? a.Rhi + (int64_t)i * a.r_ss : nullptr;
  const uint16_t* rlo = DENSE ? a.Rlo + (int64_t)i * a.r_ss : nullptr;

  // Stage st (absolute) of this wave: columns st*512 + 128*wv .. + 127.  Stages past
  // the chunk are issued too, out of range, so every stage has the same loads and
  // the waits on the in-order load counter count exactly.
  // Dense operand fragments of the stage travel in the same ring: fragment
  // (kb, nbd) of a lane is R[16 nbd + l16][c0 + 32 kb + 8 g .. + 7] (R rows are
  // zero-padded to a multiple of 128 columns); a lane past the dense columns or a
  // slice past the width reads a valid address, and its value is not used.
  auto gload = [&](uint4 (&dst)[NL], uint4 (&dh)[ND], uint4 (&dl)[ND], int st, int col_end)
                   __attribute__((always_inline)) {
    const int c0 = st * kProjStage + kProjSlice * wv;
#pragma unroll
    for (int j = 0; j < NL; ++j) {
      const int col = c0 + 8 * lpiece[j];
      if constexpr (FAST) {
        const bool ok = col < col_end;
        dst[j] = buffer_load16_nt(xr, ok ? roff[j] + 2u * (uint32_t)col : kOobOffset);
      } else {
        dst[j] = load8_elem(rowp[j], col, col_end, t0 + 4 * j + lrow < a.T);
      }
    }
    if constexpr (DENSE) {
      const int cb = c0 < col_end ? c0 : 0;
#pragma unroll
      for (int nbd = 0; nbd < NBD; ++nbd) {
        const int c = 16 * nbd + l16;
        const int64_t rowoff = (int64_t)(c < a.nd ? c : 0) * a.ld_r + cb + 8 * g;
#pragma unroll
        for (int kb = 0; kb < 4; ++kb) {
          dh[4 * nbd + kb] = *reinterpret_cast<const uint4*>(rhi + rowoff + 32 * kb);
          dl[4 * nbd + kb] = *reinterpret_cast<const uint4*>(rlo + rowoff + 32 * kb);
        }
      }
    }
  };
  auto to_lds = [&](const uint4 (&src)[NL]) __attribute__((always_inline)) {
    wave_lds_fence();                              // the previous stage's reads are done
#pragma unroll
    for (int j = 0; j < NL; ++j)
      *reinterpret_cast<uint4*>(&xt[(4 * j + lrow) * kProjSlice + 8 * lslot]) = src[j];
    wave_lds_fence();
  };
  auto mult = [&](int st, int uc, const uint4 (&dh)[ND], const uint4 (&dl)[ND]) __attribute__((always_inline)) {
    const int c0 = st * kProjStage + kProjSlice * wv;
    if (c0 >= a.m) return;                         // wave-uniform: slice past the width
#pragma unroll
    for (int kb = 0; kb < 4; ++kb) {
      const int w = (c0 - uc) / 32 + kb;           // probe word of this k-block within the chunk
#pragma unroll
      for (int nb = 0; nb < NB; ++nb) {
        uint4 bh = uint4{0, 0, 0, 0}, bl = uint4{0, 0, 0, 0};
        if (a.nz > 0) {
          const uint32_t word = zw[zrow[nb] + w];
          bh = expand_signs(__builtin_amdgcn_perm(word, word, psel), zmask[nb], zone[nb]);
        }
        if constexpr (DENSE) {
          if (nb < NBD) {                          // static: column blocks that hold dense columns
            const bool isd = 16 * nb + l16 < a.nd;
            bh = select4(isd, dh[4 * nb + kb], bh);
            bl = select4(isd, dl[4 * nb + kb], bl);
          }
        }
#pragma unroll
        for (int rb = 0; rb < RB; ++rb) {
          const int r = 16 * rb + l16;
          const uint4 av = *reinterpret_cast<const uint4*>(&xt[r * kProjSlice + 8 * ((4 * kb + g) ^ l16)]);
          acc[rb][nb] = mfma16x16x32(av, bh, acc[rb][nb]);
          if (DENSE && nb < NBD) acc[rb][nb] = mfma16x16x32(av, bl, acc[rb][nb]);
        }
      }
    }
  };

  for (int uc = 0; uc < a.m; uc += 32 * wpc) {
    const int col_end = min(a.m, uc + 32 * wpc);
    const int s0 = uc / kProjStage;
    const int nst = (col_end - uc + kProjStage - 1) / kProjStage;
    uint4 ring[P][NL], rdh[P][ND], rdl[P][ND];
#pragma unroll
    for (int q = 0; q < P; ++q) gload(ring[q], rdh[q], rdl[q], s0 + q, q < nst ? col_end : 0);
    if (a.nz > 0) {                                // generated while the first stages are in flight
      __syncthreads();
      const int nblk = wpc >> 2;
      const uint32_t wbase = (uint32_t)(uc >> 5);
      for (int idx = tid; idx < a.nz * nblk; idx += kBlock) {
        const int c = idx / nblk, b = idx - c * nblk;
        const uint32_t w0 = wbase + 4u * (uint32_t)b;
        u32x4 v;
        if (a.probe_kind == kProbeRademacher)
          v = c < a.z_split ? rademacher_block(a.key0, a.key1, a.layer_id, a.stream_id, w0 >> 2, (uint32_t)c)
                            : rademacher_block(a.key0, a.key1, a.layer_id, a.stream_id2, w0 >> 2,
                                               (uint32_t)(c - a.z_split));
        else
          v = u32x4{hadamard_word(w0, c), hadamard_word(w0 + 1, c), hadamard_word(w0 + 2, c),
                    hadamard_word(w0 + 3, c)};
        uint32_t* dst = zw + c * (wpc + 1) + 4 * b;     // odd row stride: 16 lanes of 16 columns hit 16 banks
        dst[0] = v.x; dst[1] = v.y; dst[2] = v.z; dst[3] = v.w;
      }
      __syncthreads();
    }
    auto step = [&](int k, auto ph) __attribute__((always_inline)) {
      constexpr int q = decltype(ph)::value;
      const int st = s0 + k;
      uint4 dh[ND], dl[ND];
#pragma unroll
      for (int e = 0; e < ND; ++e) {
        dh[e] = rdh[q][e];
        dl[e] = rdl[q][e];
      }
      to_lds(ring[q]);
      gload(ring[q], rdh[q], rdl[q], st + P, k + P < nst ? col_end : 0);
      mult(st, uc, dh, dl);
    };
    // whole groups of P stages in the loop (no early exit reaches its back edge,
    // so the compiler's wait counting stays exact), the remainder after it
    int k = 0;
    if constexpr (P == 4) {
      for (; k + 4 <= nst; k += 4) {
        step(k, PInt<0>{});
        step(k + 1, PInt<1>{});
        step(k + 2, PInt<2>{});
        step(k + 3, PInt<3>{});
      }
      if (k < nst) step(k, PInt<0>{});
      if (k + 1 < nst) step(k + 1, PInt<1>{});
      if (k + 2 < nst) step(k + 2, PInt<2>{});
    } else {
      for (; k + 2 <= nst; k += 2) {
        step(k, PInt<0>{});
        step(k + 1, PInt<1>{});
      }
      if (k < nst) step(k, PInt<0>{});
    }
    __syncthreads();                               // zw and the X tiles are reused
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
  uint16_t* ylo = yhi + a.ylo_off;
  for (int idx = tid; idx < rows * 16 * NB; idx += kBlock) {
    const int c = idx / rows, r = idx - c * rows;
    if (c >= a.ncols_write) continue;
    float y = 0.f;
#pragma unroll
    for (int s = 0; s < 4; ++s) y += red[s * rows * RS + r * RS + c];
    uint32_t h, l;
    split_bf16(y, h, l);
    yhi[(int64_t)c * a.yt_ld + r] = (uint16_t)h;
    ylo[(int64_t)c * a.yt_ld + r] = (uint16_t)l;
  }
}

template <int RB, int NB, int NBD, bool FAST>
__global__ __launch_bounds__(kBlock) void project_kernel(ProjectArgs a) {
  project_body<RB, NB, NBD, FAST>(a, blockIdx.x, blockIdx.y);
}

// Projections of several layers in one launch (same instantiation): block (x, sample) of
// job j at blk0[j] + sample * (T_pad / (16 RB)) + x.
template <int RB, int NB, int NBD, bool FAST>
__global__ __launch_bounds__(kBlock) void project_batch_kernel(ProjectBatch bt) {
  int jb = 0;
#pragma unroll
  for (int q = 1; q < kProjMaxJobs; ++q) jb += (q < bt.njobs && (int)blockIdx.x >= bt.blk0[q]) ? 1 : 0;
  const ProjectArgs& a = bt.job[jb];
  const int gx = a.T_pad / (16 * RB);
  const int rel = (int)blockIdx.x - bt.blk0[jb];
  project_body<RB, NB, NBD, FAST>(a, rel % gx, rel / gx);
}

template <int RB, int NB>
static size_t project_lds(const ProjectArgs& a) {
  const size_t zbytes = a.nz > 0 ? (size_t)a.nz * (a.words_per_chunk + 1) * 4 : 0;
  const size_t rbytes = std::max((size_t)4 * 16 * RB * (16 * NB + 4) * 4, (size_t)4 * 16 * RB * kProjSlice * 2);
  return zbytes + rbytes;
}

template <int RB>
static bool project_fast(const ProjectArgs& a) {
  // buffer offsets of one workgroup's rows stay below 2^31
  return a.vec && a.m % 8 == 0 && (int64_t)16 * RB * a.ldx * 2 < ((int64_t)1 << 31);
}

template <int RB, int NB>
static hipError_t launch_batch_rb_nb(const ProjectBatch& bt, hipStream_t st) {
  size_t lds = 0;
  bool fast = true;
  for (int j = 0; j < bt.njobs; ++j) {
    lds = std::max(lds, project_lds<RB, NB>(bt.job[j]));
    fast = fast && project_fast<RB>(bt.job[j]);
  }
  const int nbd = (bt.job[0].nd + 15) / 16;
#define DPRC_PROJECT_BATCH_CASE(NBDV)                                                                    \
  if (nbd == NBDV) {                                                                                      \
    if (fast) DPRC_LAUNCH((project_batch_kernel<RB, NB, NBDV, true>), dim3(bt.blocks), dim3(kBlock), lds, st, bt); \
    else DPRC_LAUNCH((project_batch_kernel<RB, NB, NBDV, false>), dim3(bt.blocks), dim3(kBlock), lds, st, bt);     \
  }
  DPRC_PROJECT_BATCH_CASE(0)
  if constexpr (NB >= 1) { DPRC_PROJECT_BATCH_CASE(1) }
  if constexpr (NB >= 2) { DPRC_PROJECT_BATCH_CASE(2) }
#undef DPRC_PROJECT_BATCH_CASE
  return hipGetLastError();
}

template <int RB>
static hipError_t launch_batch_rb(const ProjectBatch& bt, hipStream_t st) {
  switch (bt.job[0].ncols_pad / 16) {
    case 1: return launch_batch_rb_nb<RB, 1>(bt, st);
    case 2: return launch_batch_rb_nb<RB, 2>(bt, st);
    case 3: return launch_batch_rb_nb<RB, 3>(bt, st);
    case 4: return launch_batch_rb_nb<RB, 4>(bt, st);
    default: return hipErrorInvalidValue;
  }
}

hipError_t launch_project_batch(ProjectBatch bt, int rows_per_wg, hipStream_t st) {
  if (bt.njobs < 1 || bt.njobs > kProjMaxJobs) return hipErrorInvalidValue;
  const int rb = rows_per_wg / 16;
  const int nbd = (bt.job[0].nd + 15) / 16;
  bt.blocks = 0;
  for (int j = 0; j < bt.njobs; ++j) {
    const ProjectArgs& a = bt.job[j];
    // one instantiation serves every job
    if (a.ncols_pad != bt.job[0].ncols_pad || (a.nd + 15) / 16 != nbd || a.words_per_chunk % 16 != 0 ||
        a.nd > 32 || a.nd > a.ncols_pad || a.T_pad % rows_per_wg != 0)
      return hipErrorInvalidValue;
    bt.blk0[j] = bt.blocks;
    bt.blocks += (a.T_pad / rows_per_wg) * a.B;
  }
  switch (rb) {
    case 1: return launch_batch_rb<1>(bt, st);
    case 2: return launch_batch_rb<2>(bt, st);
    case 4: return launch_batch_rb<4>(bt, st);
    default: return hipErrorInvalidValue;
  }
}

template <int RB, int NB>
static hipError_t launch_rb_nb(const ProjectArgs& a, hipStream_t st) {
  const size_t zbytes = a.nz > 0 ? (size_t)a.nz * (a.words_per_chunk + 1) * 4 : 0;
  const size_t rbytes = std::max((size_t)4 * 16 * RB * (16 * NB + 4) * 4, (size_t)4 * 16 * RB * kProjSlice * 2);
  const size_t lds = zbytes + rbytes;
  if (a.words_per_chunk % 16 != 0 || a.nd > 32 || a.nd > 16 * NB) return hipErrorInvalidValue;
  dim3 grid((unsigned)(a.T_pad / (16 * RB)), (unsigned)a.B);
  // buffer offsets of one workgroup's rows stay below 2^31
  const bool fast = a.vec && a.m % 8 == 0 && (int64_t)16 * RB * a.ldx * 2 < ((int64_t)1 << 31);
  const int nbd = (a.nd + 15) / 16;
#define DPRC_PROJECT_CASE(NBD)                                                           \
  if (nbd == NBD) {                                                                      \
    if (fast) DPRC_LAUNCH((project_kernel<RB, NB, NBD, true>), grid, dim3(kBlock), lds, st, a);  \
    else DPRC_LAUNCH((project_kernel<RB, NB, NBD, false>), grid, dim3(kBlock), lds, st, a);      \
  }
  DPRC_PROJECT_CASE(0)
  if constexpr (NB >= 1) { DPRC_PROJECT_CASE(1) }
  if constexpr (NB >= 2) { DPRC_PROJECT_CASE(2) }
#undef DPRC_PROJECT_CASE
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
