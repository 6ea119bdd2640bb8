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
//
// Two bodies share this scheme.  The general one (any column count, dense columns,
// element loads) gives each workgroup one row block.  The row-block body, for sign
// probes with 16-byte loads and at most 64 columns (32 in 32-row blocks), lets a
// workgroup of a narrow layer stream
// several consecutive row blocks (up to 2 MB of X) with its load ring running on
// through probe-chunk and row-block boundaries; wide layers then stream at about
// 6.0 TB/s instead of 5.5.
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

// Sign-probe projection with 16-byte loads, for narrow column counts (RB * NB <= 4).
// The workgroup owns a.rblocks consecutive row blocks (16 RB rows each) of sample by,
// starting at row block bx * a.rblocks.  Its stages (row block r, 512-column stage st)
// run in one sequence, and the load ring runs straight through the boundaries of probe
// chunks and row blocks: at a chunk boundary the probe words are regenerated between two
// barriers while the next stages' loads are in flight, and at a row-block boundary the
// finished block's Y is reduced and written (its probe words are kept when the row is one
// chunk).  Every row block's Y is computed exactly as by a workgroup of its own.
template <int RB, int NB>
__device__ __forceinline__ void project_rows_body(const ProjectArgs& a, int bx, int by) {
  extern __shared__ __attribute__((aligned(16))) uint32_t smem[];
  constexpr int P = RB == 1 ? 4 : 2;            // stages in flight per wave
  constexpr int NL = 4 * RB;                    // loads per lane per stage
  constexpr int ROWS = 16 * RB;
  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
  const int g = lane >> 4, l16 = lane & 15;
  const int i = by;
  const int nrb = a.rblocks;
  const int t_first = bx * nrb * ROWS;
  const int wpc = a.words_per_chunk;            // a multiple of 16: chunks are whole stages
  const int spc = wpc / 16;                     // stages per chunk
  const int srow = (a.m + kProjStage - 1) / kProjStage;   // stages per row block
  const bool multi = srow > spc;                // a row spans several chunks
  const int G = nrb * srow;                     // stages of the workgroup
  uint32_t* zw = smem;                                            // [nz][wpc + 1]
  uint32_t* region = smem + (a.nz > 0 ? a.nz * (wpc + 1) : 0);
  // X tiles [4 waves][16 RB rows][128 columns], later the reduction slots
  uint16_t* xt = reinterpret_cast<uint16_t*>(region) + wv * (ROWS * kProjSlice);
  float* red = reinterpret_cast<float*>(region);
  constexpr int RS = 16 * NB + 4;                                 // padded row of a reduction slot

  if (a.zero_ptr != nullptr && bx == 0 && by == 0)
    for (int idx = tid; idx < a.zero_count; idx += kBlock) a.zero_ptr[idx] = 0u;

  // loads: lane -> row 4j + lane/16 of the block (j = load index), 16-byte piece
  // p = (lane%16) ^ row of its slice, stored at LDS slot lane%16
  const uint16_t* xs = a.X + (int64_t)i * a.x_ss;
  const int vrows = max(0, min(nrb * ROWS, a.T - t_first));
  const __amdgpu_buffer_rsrc_t xr = buffer_rsrc(xs + (int64_t)t_first * a.ldx, (uint32_t)(vrows * a.ldx * 2));
  const uint32_t rbytes = (uint32_t)(ROWS * a.ldx) * 2u;           // one row block
  const int lrow = lane >> 4, lslot = lane & 15;
  uint32_t roff[NL];
  int lpiece[NL];
#pragma unroll
  for (int j = 0; j < NL; ++j) {
    const int rr = 4 * j + lrow;
    lpiece[j] = lslot ^ (rr & 15);
    roff[j] = (uint32_t)(rr * a.ldx) * 2u;
  }

  f32x4_t acc[RB][NB];
#pragma unroll
  for (int rb = 0; rb < RB; ++rb)
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) acc[rb][nb] = f32x4_t{0.f, 0.f, 0.f, 0.f};

  // per column block: probe columns take +-1, padding columns zero
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

  // Stage st of row block r, for this wave: columns st*512 + 128*wv .. + 127.  Stages
  // past the workgroup's last one (ok false) are issued too, out of range, so every
  // step has the same loads and the waits on the in-order load counter count exactly.
  auto gload = [&](uint4 (&dst)[NL], int r, int st, bool ok) __attribute__((always_inline)) {
    const int c0 = st * kProjStage + kProjSlice * wv;
    const int col_end = ok ? a.m : 0;
#pragma unroll
    for (int j = 0; j < NL; ++j) {
      const int col = c0 + 8 * lpiece[j];
      const bool in = col < col_end;
      dst[j] = buffer_load16_nt(xr, in ? (uint32_t)r * rbytes + roff[j] + 2u * (uint32_t)col : kOobOffset);
    }
  };
  auto to_lds = [&](const uint4 (&src)[NL]) __attribute__((always_inline)) {
    wave_lds_fence();                              // the previous stage's reads are done
#pragma unroll
    for (int j = 0; j < NL; ++j)
      *reinterpret_cast<uint4*>(&xt[(4 * j + lrow) * kProjSlice + 8 * lslot]) = src[j];
    wave_lds_fence();
  };
  // uc: first column of the chunk whose probe words are in LDS
  auto mult = [&](int st, int uc) __attribute__((always_inline)) {
    const int c0 = st * kProjStage + kProjSlice * wv;
    if (c0 >= a.m) return;                         // wave-uniform: slice past the width
#pragma unroll
    for (int kb = 0; kb < 4; ++kb) {
      const int w = (c0 - uc) / 32 + kb;           // probe word of this k-block within the chunk
#pragma unroll
      for (int nb = 0; nb < NB; ++nb) {
        const uint32_t word = zw[zrow[nb] + w];
        const uint4 bh = expand_signs(__builtin_amdgcn_perm(word, word, psel), zmask[nb], zone[nb]);
#pragma unroll
        for (int rb = 0; rb < RB; ++rb) {
          const int r = 16 * rb + l16;
          const uint4 av = *reinterpret_cast<const uint4*>(&xt[r * kProjSlice + 8 * ((4 * kb + g) ^ l16)]);
          acc[rb][nb] = mfma16x16x32(av, bh, acc[rb][nb]);
        }
      }
    }
  };
  // probe words of the chunk starting at column uc (callers place the barriers); the
  // key fields are read once, as workgroup-uniform values, so that no per-lane argument
  // load (which would wait for the loads in flight) lands in the generation loop
  const uint32_t key0 = __builtin_amdgcn_readfirstlane(a.key0), key1 = __builtin_amdgcn_readfirstlane(a.key1);
  const uint32_t layer = __builtin_amdgcn_readfirstlane(a.layer_id);
  const uint32_t sid1 = __builtin_amdgcn_readfirstlane(a.stream_id), sid2 = __builtin_amdgcn_readfirstlane(a.stream_id2);
  const int zsplit = __builtin_amdgcn_readfirstlane(a.z_split);
  auto gen_z = [&](int uc) __attribute__((always_inline)) {
    const int nblk = wpc >> 2;
    const uint32_t wbase = (uint32_t)(uc >> 5);
    for (int idx = tid; idx < a.nz * nblk; idx += kBlock) {
      const int c = idx / nblk, b = idx - c * nblk;
      const uint32_t w0 = wbase + 4u * (uint32_t)b;
      u32x4 v;
      if (a.probe_kind == kProbeRademacher) {
        const bool first = c < zsplit;
        v = rademacher_block(key0, key1, layer, first ? sid1 : sid2, w0 >> 2, (uint32_t)(first ? c : c - zsplit));
      } else
        v = u32x4{hadamard_word(w0, c), hadamard_word(w0 + 1, c), hadamard_word(w0 + 2, c),
                  hadamard_word(w0 + 3, c)};
      uint32_t* dst = zw + c * (wpc + 1) + 4 * b;       // odd row stride: 16 lanes of 16 columns hit 16 banks
      dst[0] = v.x; dst[1] = v.y; dst[2] = v.z; dst[3] = v.w;
    }
  };
  // the four waves' partial tiles of row block r into LDS (after a barrier that ends
  // every wave's use of the X tiles), then summed and written as Y; acc restarts at zero
  auto stash = [&]() __attribute__((always_inline)) {
    float* slot = red + wv * ROWS * RS;
#pragma unroll
    for (int rb = 0; rb < RB; ++rb)
#pragma unroll
      for (int nb = 0; nb < NB; ++nb) {
#pragma unroll
        for (int ii = 0; ii < 4; ++ii) slot[(16 * rb + 4 * g + ii) * RS + 16 * nb + l16] = acc[rb][nb][ii];
        acc[rb][nb] = f32x4_t{0.f, 0.f, 0.f, 0.f};
      }
  };
  auto write_y = [&](int r) __attribute__((always_inline)) {
    uint16_t* yhi = a.Yt + (int64_t)i * a.T_pad + t_first + r * ROWS;
    uint16_t* ylo = yhi + a.ylo_off;
    for (int idx = tid; idx < ROWS * 16 * NB; idx += kBlock) {
      const int c = idx / ROWS, rr = idx - c * ROWS;
      if (c >= a.ncols_write) continue;
      float y = 0.f;
#pragma unroll
      for (int s = 0; s < 4; ++s) y += red[s * ROWS * RS + rr * RS + c];
      uint32_t h, l;
      split_bf16(y, h, l);
      yhi[(int64_t)c * a.yt_ld + rr] = (uint16_t)h;
      ylo[(int64_t)c * a.yt_ld + rr] = (uint16_t)l;
    }
  };

  uint4 ring[P][NL];
  // the loading position (row block lr, stage ls) runs P stages ahead of the
  // multiplying one (row block cr, stage cs); uc is the column of the current chunk
  int lr = 0, ls = 0;
  auto advance = [&](int& r, int& st) __attribute__((always_inline)) {
    if (++st == srow) {
      st = 0;
      ++r;
    }
  };
#pragma unroll
  for (int q = 0; q < P; ++q) {
    gload(ring[q], lr, ls, lr < nrb);
    advance(lr, ls);
  }
  gen_z(0);                                        // while the first stages are in flight
  __syncthreads();
  int cr = 0, cs = 0, uc = 0;
  auto step = [&](auto ph) __attribute__((always_inline)) {
    constexpr int q = decltype(ph)::value;
    if (cs == 0 && cr > 0) {                       // a new row block: finish the last one
      __syncthreads();
      stash();
      __syncthreads();
      write_y(cr - 1);
      if (multi) {
        uc = 0;
        gen_z(0);
      }
      __syncthreads();
    } else if (multi && cs * kProjStage == uc + 32 * wpc) {   // the row's next chunk
      uc += 32 * wpc;
      __syncthreads();
      gen_z(uc);
      __syncthreads();
    }
    to_lds(ring[q]);
    gload(ring[q], lr, ls, lr < nrb);
    advance(lr, ls);
    mult(cs, uc);
    advance(cr, cs);
  };
  // whole groups of P stages in the loop (no early exit reaches its back edge,
  // so the compiler's wait counting stays exact), the remainder after it
  int k = 0;
  if constexpr (P == 4) {
    for (; k + 4 <= G; k += 4) {
      step(PInt<0>{});
      step(PInt<1>{});
      step(PInt<2>{});
      step(PInt<3>{});
    }
    if (k < G) step(PInt<0>{});
    if (k + 1 < G) step(PInt<1>{});
    if (k + 2 < G) step(PInt<2>{});
  } else {
    for (; k + 2 <= G; k += 2) {
      step(PInt<0>{});
      step(PInt<1>{});
    }
    if (k < G) step(PInt<0>{});
  }

  // the last row block
  __syncthreads();
  stash();
  __syncthreads();
  write_y(nrb - 1);
}

// The row-block body serves the sign-probe instantiations that fit three workgroups of
// 32 rows in a CU at k = 32 (LDS, and a third of the register file without spills); the
// general body serves the rest, one row block per workgroup.
template <int RB, int NB, int NBD, bool FAST>
constexpr bool kProjRows = NBD == 0 && FAST && RB <= 2 && RB * NB <= 4;

template <int RB, int NB, int NBD, bool FAST>
__device__ __forceinline__ void project_dispatch(const ProjectArgs& a, int bx, int by) {
  if constexpr (kProjRows<RB, NB, NBD, FAST>) project_rows_body<RB, NB>(a, bx, by);
  else project_body<RB, NB, NBD, FAST>(a, bx, by);
}

template <int RB, int NB, int NBD, bool FAST>
__global__ __launch_bounds__(kBlock) __attribute__((amdgpu_waves_per_eu(kProjRows<RB, NB, NBD, FAST> ? 3 : 1)))
void project_kernel(ProjectArgs a) {
  project_dispatch<RB, NB, NBD, FAST>(a, blockIdx.x, blockIdx.y);
}

// Projections of several layers in one launch (same instantiation): block (x, sample) of
// job j at blk0[j] + sample * (T_pad / (16 RB rblocks)) + x.
template <int RB, int NB, int NBD, bool FAST>
__global__ __launch_bounds__(kBlock) __attribute__((amdgpu_waves_per_eu(kProjRows<RB, NB, NBD, FAST> ? 3 : 1)))
void project_batch_kernel(ProjectBatch bt) {
  int jb = 0;
#pragma unroll
  for (int q = 1; q < kProjMaxJobs; ++q) jb += (q < bt.njobs && (int)blockIdx.x >= bt.blk0[q]) ? 1 : 0;
  const ProjectArgs& a = bt.job[jb];
  const int gx = a.T_pad / (16 * RB * a.rblocks);
  const int rel = (int)blockIdx.x - bt.blk0[jb];
  project_dispatch<RB, NB, NBD, FAST>(a, rel % gx, rel / gx);
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
  return a.vec && a.m % 8 == 0 && (int64_t)16 * RB * a.rblocks * a.ldx * 2 < ((int64_t)1 << 31);
}

// Row blocks per workgroup, for the row-block body (the sign-probe instantiations of
// kProjRows with 16-byte loads; every other launch keeps one block per workgroup).  A
// workgroup of a narrow layer streams consecutive row blocks, doubling while it reads at
// most kProjWgBytes of X, and the launch keeps at least kProjMinWgs workgroups (the jobs
// with the most row blocks per workgroup give way first).  Returns whether the launch
// takes 16-byte loads.
constexpr int64_t kProjWgBytes = 2 << 20;
constexpr int kProjMaxRowBlocks = 16;
constexpr int64_t kProjMinWgs = 2048;
template <int RB, int NB>
static bool plan_rblocks(ProjectArgs* jobs, int n) {
  constexpr int rows = 16 * RB;
  bool fast = true, dense = false;
  for (int j = 0; j < n; ++j) {
    jobs[j].rblocks = 1;
    fast = fast && project_fast<RB>(jobs[j]);
    dense = dense || jobs[j].nd > 0;
  }
  if (!kProjRows<RB, NB, 0, true> || !fast || dense) return fast;
  int64_t wgs = 0;
  for (int j = 0; j < n; ++j) {
    ProjectArgs& a = jobs[j];
    const int64_t gx = a.T_pad / rows;
    const int64_t bytes = (int64_t)rows * a.m * 2;
    int r = 1;
    while (r < kProjMaxRowBlocks && bytes * r * 2 <= kProjWgBytes && gx % (2 * r) == 0 &&
           (int64_t)rows * 2 * r * a.ldx * 2 < ((int64_t)1 << 31))
      r *= 2;
    a.rblocks = r;
    wgs += gx / r * a.B;
  }
  while (wgs < kProjMinWgs) {
    int top = 1;
    for (int j = 0; j < n; ++j) top = std::max(top, jobs[j].rblocks);
    if (top == 1) break;
    for (int j = 0; j < n; ++j) {
      ProjectArgs& a = jobs[j];
      if (a.rblocks != top) continue;
      const int64_t gx = a.T_pad / rows;
      wgs += gx / (top / 2) * a.B - gx / top * a.B;
      a.rblocks = top / 2;
    }
  }
  return true;
}

template <int RB, int NB>
static hipError_t launch_batch_rb_nb(ProjectBatch bt, hipStream_t st) {
  const bool fast = plan_rblocks<RB, NB>(bt.job, bt.njobs);
  size_t lds = 0;
  bt.blocks = 0;
  for (int j = 0; j < bt.njobs; ++j) {
    lds = std::max(lds, project_lds<RB, NB>(bt.job[j]));
    bt.blk0[j] = bt.blocks;
    bt.blocks += (bt.job[j].T_pad / (16 * RB * bt.job[j].rblocks)) * bt.job[j].B;
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
  for (int j = 0; j < bt.njobs; ++j) {
    const ProjectArgs& a = bt.job[j];
    // one instantiation serves every job
    if (a.ncols_pad != bt.job[0].ncols_pad || (a.nd + 15) / 16 != nbd || a.words_per_chunk % 16 != 0 ||
        a.nd > 32 || a.nd > a.ncols_pad || a.T_pad % rows_per_wg != 0)
      return hipErrorInvalidValue;
  }
  switch (rb) {
    case 1: return launch_batch_rb<1>(bt, st);
    case 2: return launch_batch_rb<2>(bt, st);
    case 4: return launch_batch_rb<4>(bt, st);
    default: return hipErrorInvalidValue;
  }
}

template <int RB, int NB>
static hipError_t launch_rb_nb(ProjectArgs a, hipStream_t st) {
  if (a.words_per_chunk % 16 != 0 || a.nd > 32 || a.nd > 16 * NB) return hipErrorInvalidValue;
  const bool fast = plan_rblocks<RB, NB>(&a, 1);
  const size_t lds = project_lds<RB, NB>(a);
  dim3 grid((unsigned)(a.T_pad / (16 * RB * a.rblocks)), (unsigned)a.B);
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

hipError_t launch_project(const ProjectArgs& args, int rows_per_wg, hipStream_t st) {
  if (rows_per_wg != 16 && rows_per_wg != 32 && rows_per_wg != 64) return hipErrorInvalidValue;
  if (args.T_pad % rows_per_wg != 0) return hipErrorInvalidValue;
  switch (rows_per_wg) {
    case 16: return launch_rb<1>(args, st);
    case 32: return launch_rb<2>(args, st);
    default: return launch_rb<4>(args, st);
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
