// Token reduction M_i = X_i^T Y_i on bf16 matrix cores (the A_i^T Y_i step of the
// Hutchinson estimator, Algorithm 2; also the W_S, O S and [U | W_P] steps of
// Hutch++), followed by either the squared-norm estimate or a store of M_i.
//
// A workgroup owns one sample, a 128-column tile of X (two adjacent tiles, eight waves,
// in unsplit squared-norm launches) and a contiguous range of tokens.  X tiles (64 tokens x 128 columns, 256 bytes per token row) are
// loaded with coalesced 16-byte reads, double-buffered through LDS and read
// back token-contiguous with the gfx950 LDS transpose read, which is the
// operand layout of the MFMA (the contraction runs over tokens, X is stored
// token-major).  Y (bf16 hi + lo, already token-contiguous) is read directly.
// With several token splits per tile, each split writes its partial tile; a
// second launch sums the splits of a tile in split order and squares (or
// stores) the sum, and a third adds the tile sums of each sample in tile
// order, so the result does not depend on scheduling.
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

// The same sum over each group of four waves of a workgroup of 4 TT waves (red holds
// 4 TT values): every thread gets its own group's total, added as by block_sum_d.
template <int TT>
__device__ __forceinline__ double quad_sum_d(double v, double* red) {
  v = wave_sum(v);
  const int tid = threadIdx.x;
  __syncthreads();
  if ((tid & 63) == 0) red[tid >> 6] = v;
  __syncthreads();
  const double* r4 = red + 4 * (tid >> 8);
  return (r4[0] + r4[1]) + (r4[2] + r4[3]);
}

__device__ __forceinline__ void store4(const TokredArgs& a, int i, int c, int j, const float v[4]) {
  if (c >= a.ncols) return;
  if (a.M && c >= a.m_col0) {
    float* dst = a.M + (int64_t)i * a.m_ss + (int64_t)c * a.m_ld;
#pragma unroll
    for (int q = 0; q < 4; ++q)
      if (j + q < a.n) dst[j + q] = v[q];
  }
  if (a.Mhi && (a.mh_ncols == 0 || c < a.mh_ncols)) {
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

// mode 0: adds a squared entry of column c to its layer's sum (columns past
// ncols, which may hold anything, are left out)
__device__ __forceinline__ void seg_add(const TokredArgs& a, int c, double v, double (&sq)[kMaxGroup]) {
  if (c >= a.ncols) return;
#pragma unroll
  for (int g = 0; g < kMaxGroup; ++g)
    if (c >= g * a.seg && c < (g + 1) * a.seg) sq[g] += v;
}

// Tile sums of a workgroup of TT tiles: the four waves of tile h (tslot0 + h) add their
// squares as a workgroup of one tile does; a tile past the operand's last is not written.
template <int TT>
__device__ __forceinline__ void seg_publish(const TokredArgs& a, int64_t tslot0, int tile0,
                                            double (&sq)[kMaxGroup], double* dred) {
  const int64_t lstride = (int64_t)a.B * a.ntiles;
  const int h = threadIdx.x >> 8;
#pragma unroll
  for (int g = 0; g < kMaxGroup; ++g) {
    if (g >= a.nseg) break;
    const double t = quad_sum_d<TT>(sq[g], dred);
    if ((threadIdx.x & 255) == 0 && tile0 + h < a.ntiles) a.tilesq[g * lstride + tslot0 + h] = t;
  }
}

template <int V>
struct Int {
  static constexpr int value = V;
};

// TT = 2 (unsplit squared-norm launches with an even number of 16-column blocks): a
// workgroup of eight waves reduces two adjacent 128-column tiles, so each Y stage read
// from L2 serves twice the columns.  Waves 4h .. 4h + 3 work on tile h exactly as the
// four waves of a one-tile workgroup do.
template <int NB, bool FAST, int TT = 1>
__device__ __forceinline__ void tokred_body(const TokredArgs& a, int bx, int by) {
  static_assert(TT == 1 || (NB % 2 == 0 && NB <= 4), "two-tile workgroups stage Y through LDS, two halves");
  // Y stages go through LDS with X (one 16-byte load per thread per 16 columns)
  // when they are small; wider Y is read straight from global memory at use.
  constexpr bool YLDS = NB <= 4;
  constexpr int YLd = kStage + 8;                       // padded LDS row of one Y column (144 bytes)
  constexpr int XLd = TT * kTile + 16;                  // padded LDS row of the X stage
  constexpr int YN = YLDS ? NB / TT : 1;                // Y loads per thread per stage
  __shared__ __attribute__((aligned(16))) uint16_t lds[2][kStage * XLd];
  __shared__ __attribute__((aligned(16))) uint16_t ylds[YLDS ? 2 : 1][YLDS ? 2 * 16 * NB * YLd : 8];
  __shared__ double dred[4 * TT];
  constexpr int P = 4;                                  // stages in flight in registers, one more in LDS
  static_assert(P == 4, "the stage loop below is written out for four ring slots");
  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
  const int g = lane >> 4, l16 = lane & 15, r4 = l16 >> 2, c4 = lane & 3;
  const int i = by;
  const int tile = bx / a.S, s = bx - tile * a.S;      // (TT = 2: bx is the tile pair)
  const int j0 = tile * TT * kTile;
  const int tb = s * a.stages_per_split * kStage;
  const int te = min(a.T, tb + a.stages_per_split * kStage);
  const int nst = te > tb ? (te - tb + kStage - 1) / kStage : 0;

  const int lr0 = tid >> (3 + TT), lc = (tid & (16 * TT - 1)) * 8;
  const uint16_t* xs = a.X + (int64_t)i * a.x_ss;
  // FAST: one buffer resource per stage (64 token rows from column j0); rows past
  // the split and columns past n read as zero through out-of-range offsets
  const uint32_t row_bytes = (uint32_t)a.ldx * 2u;
  const uint32_t lane_off = j0 + lc < a.n ? (uint32_t)lr0 * row_bytes + 2u * lc : kOobOffset;
  const uint16_t* ys = a.Yt + (int64_t)i * a.T_pad;
  // Y stage loads: column-half ch = tid / 8 + 32 TT r (h = ch / ncols16, c = ch % ncols16), tokens 8 (tid % 8) ..
  const int ych = tid >> 3, ytk = (tid & 7) * 8;

  struct Stage {
    uint4 x[4];
    uint4 y[YN];
  };
  // Stages past the split (st >= nst) are issued too, with an empty range (X) or
  // clamped to the last stage (Y): the load sequence is the same in every stage,
  // so the waits on the in-order load counter count exactly.
  auto gload = [&](Stage& dst, int st) __attribute__((always_inline)) {
    if constexpr (FAST) {
      const int t0 = tb + st * kStage;
      const int rows = max(0, min(kStage, te - t0));
      const __amdgpu_buffer_rsrc_t xr =
          buffer_rsrc(xs + (int64_t)(rows > 0 ? t0 : 0) * a.ldx + j0, (uint32_t)rows * row_bytes);
#pragma unroll
      for (int q = 0; q < 4; ++q) dst.x[q] = buffer_load16_nt(xr, lane_off + (uint32_t)(16 * q) * row_bytes);
    } else {
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const int t = tb + st * kStage + lr0 + 16 * q;
        const bool ok = st < nst && t < te;
        dst.x[q] = load_bf16x8<false>(xs + (int64_t)(ok ? t : 0) * a.ldx, (int64_t)j0 + lc, a.n, ok, xs);
      }
    }
    if constexpr (YLDS) {
      const int ytok = tb + min(st, nst - 1) * kStage + ytk;
#pragma unroll
      for (int r = 0; r < YN; ++r) {
        const int ch = ych + 32 * TT * r, h = ch / (16 * NB), c = ch - h * 16 * NB;
        dst.y[r] = *reinterpret_cast<const uint4*>(ys + ((int64_t)h * a.ncols_pad + c) * a.yt_ld + ytok);
      }
    }
  };
  auto swrite = [&](const Stage& src, int buf) __attribute__((always_inline)) {
#pragma unroll
    for (int q = 0; q < 4; ++q)
      *reinterpret_cast<uint4*>(&lds[buf][(lr0 + 16 * q) * XLd + lds_swz(lr0 + 16 * q, lc)]) = src.x[q];
    if constexpr (YLDS) {
#pragma unroll
      for (int r = 0; r < YN; ++r)
        *reinterpret_cast<uint4*>(&ylds[buf][(ych + 32 * TT * r) * YLd + ytk]) = src.y[r];
    }
  };

  f32x4_t acc[2][2][NB];
#pragma unroll
  for (int x = 0; x < 2; ++x)
#pragma unroll
    for (int h = 0; h < 2; ++h)
#pragma unroll
      for (int nb = 0; nb < NB; ++nb) acc[x][h][nb] = f32x4_t{0.f, 0.f, 0.f, 0.f};

  auto mult = [&](int buf, int st) __attribute__((always_inline)) {
#pragma unroll
    for (int ks = 0; ks < 2; ++ks) {
      uint4 bop[2][NB];
#pragma unroll
      for (int h = 0; h < 2; ++h)
#pragma unroll
        for (int nb = 0; nb < NB; ++nb) {
          if constexpr (YLDS)
            bop[h][nb] = *reinterpret_cast<const uint4*>(
                &ylds[buf][(h * 16 * NB + 16 * nb + l16) * YLd + 32 * ks + 8 * g]);
          else
            bop[h][nb] = *reinterpret_cast<const uint4*>(
                ys + ((int64_t)h * a.ncols_pad + 16 * nb + l16) * a.yt_ld + tb + st * kStage + 32 * ks + 8 * g);
        }
#pragma unroll
      for (int x = 0; x < 2; ++x) {
        const int mb = 2 * wv + x;
        // rows 32ks + 8g + r4 (+4) all have bit 3 equal to g & 1
        const uint16_t* p = &lds[buf][(32 * ks + 8 * g + r4) * XLd + ((16 * mb + 4 * c4) ^ ((g & 1) << 6))];
        const uint4 av = make_u4(lds_read_tr16(p), lds_read_tr16(p + 4 * XLd));
#pragma unroll
        for (int h = 0; h < 2; ++h)
#pragma unroll
          for (int nb = 0; nb < NB; ++nb) acc[x][h][nb] = mfma16x16x32(av, bop[h][nb], acc[x][h][nb]);
      }
    }
  };

  if (nst > 0) {
    Stage ring[P];
#pragma unroll
    for (int q = 0; q < P; ++q) gload(ring[q], q);
    swrite(ring[0], 0);
    __syncthreads();
    auto step = [&](int st, auto ph) __attribute__((always_inline)) {
      gload(ring[ph.value], st + P);               // ring[ph] held stage st, already in LDS
      mult(ph.value & 1, st);
      // unconditional: after the last stage it stores an unused (empty-range) stage
      swrite(ring[(ph.value + 1) % P], (ph.value + 1) & 1);
      __syncthreads();
    };
    // whole groups of P stages in the loop (no early exit reaches its back edge, so
    // the compiler's wait counting stays exact), the remainder after it
    int st0 = 0;
    for (; st0 + P <= nst; st0 += P) {
      step(st0 + 0, Int<0>{});
      step(st0 + 1, Int<1>{});
      step(st0 + 2, Int<2>{});
      step(st0 + 3, Int<3>{});
    }
    if (st0 + 0 < nst) step(st0 + 0, Int<0>{});
    if (st0 + 1 < nst) step(st0 + 1, Int<1>{});
    if (st0 + 2 < nst) step(st0 + 2, Int<2>{});
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
  if constexpr (TT > 1) {                              // unsplit squared norms only
    double sq[kMaxGroup] = {};
#pragma unroll
    for (int x = 0; x < 2; ++x)
#pragma unroll
      for (int nb = 0; nb < NB; ++nb) {
        const int c = 16 * nb + l16;
#pragma unroll
        for (int q = 0; q < 4; ++q) seg_add(a, c, (double)(w[x][nb][q] * w[x][nb][q]), sq);
      }
    seg_publish<TT>(a, (int64_t)i * a.ntiles + TT * tile, TT * tile, sq, dred);
    return;
  }
  if (a.S == 1) {
    if (a.mode == 0) {
      double sq[kMaxGroup] = {};
#pragma unroll
      for (int x = 0; x < 2; ++x)
#pragma unroll
        for (int nb = 0; nb < NB; ++nb) {
          const int c = 16 * nb + l16;
#pragma unroll
          for (int q = 0; q < 4; ++q) seg_add(a, c, (double)(w[x][nb][q] * w[x][nb][q]), sq);
        }
      seg_publish<1>(a, tslot, tile, sq, dred);
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

template <int NB, bool FAST>
__global__ __launch_bounds__(kBlock) void tokred_kernel(TokredArgs a) {
  tokred_body<NB, FAST>(a, blockIdx.x, blockIdx.y);
}

// Token reductions of several layers in one launch (same instantiation).  Within job j
// the blocks from blk0[j] run sample-major, then split, then tile, so the tiles that read
// the same Y rows (one sample's split) are consecutive.  Workgroup ids are dealt
// round-robin to the 8 XCDs.  When the launch is unsplit (every block reads all of its
// sample's Y rows), each window of 8 kXcdRun ids is read so that XCD x runs blocks
// x kXcdRun .. x kXcdRun + kXcdRun - 1 of the window: such a run of tiles reads its Y rows
// into one L2 instead of eight (the stack's 2048-wide layers reduce 4% faster).  Windows
// follow the block order, so every XCD still gets an even share of each job.  With token
// splits the runs were slower (mlp layers, 5%) and ids map to blocks directly.  The grid
// is padded to whole windows.
constexpr int kXcdRun = 16;
template <int NB, bool FAST, int TT>
__global__ __launch_bounds__(kBlock * TT) void tokred_batch_kernel(TokredBatch bt) {
  constexpr int W = 8 * kXcdRun;
  const int id = (int)blockIdx.x;
  const int b = bt.job[0].S == 1 ? id / W * W + (id & 7) * kXcdRun + (id % W) / 8 : id;
  if (b >= bt.blocks) return;
  int jb = 0;
#pragma unroll
  for (int q = 1; q < kTokMaxJobs; ++q) jb += (q < bt.njobs && b >= bt.blk0[q]) ? 1 : 0;
  const TokredArgs& a = bt.job[jb];
  const int nt = (a.ntiles + TT - 1) / TT;           // tiles, or tile pairs
  const int gx = nt * a.S;
  const int rel = b - bt.blk0[jb], idx = rel % gx;
  const int split = idx / nt, tile = idx - split * nt;
  tokred_body<NB, FAST, TT>(a, tile * a.S + split, rel / gx);
}

// Sum of the token splits of one tile, in split order: its squared norm (mode 0)
// or the stored tile (mode 1).
// Sum of the S split partials of one (sample, tile), in split order.  Each thread
// takes G = 16 / U float4 groups at a time and U splits of each, so 16 loads are
// in flight whatever S is (split indices past S are clamped to S-1 and not added).
template <int U>
__device__ __forceinline__ void tokred_splits_block(const TokredArgs& a, int tile, int i) {
  constexpr int G = 16 / U;
  __shared__ double dred[4];
  const int tid = threadIdx.x;
  const int64_t tslot = (int64_t)i * a.ntiles + tile;
  const float* tp = a.part + tslot * a.S * (int64_t)a.ncols_pad * kTile;
  const int64_t sstride = (int64_t)a.ncols_pad * kTile;
  const int ng = a.ncols_pad * (kTile / 4);
  double sq[kMaxGroup] = {};
  for (int g0 = tid; g0 < ng; g0 += G * kBlock) {
    float v[G][4];
    const float* src[G];
#pragma unroll
    for (int q = 0; q < G; ++q) {
      const int gi = g0 + q * kBlock < ng ? g0 + q * kBlock : g0;
      const int c = gi / (kTile / 4), j4 = (gi - c * (kTile / 4)) * 4;
      src[q] = tp + (int64_t)c * kTile + j4;
      v[q][0] = v[q][1] = v[q][2] = v[q][3] = 0.f;
    }
    for (int s0 = 0; s0 < a.S; s0 += U) {
      float4 pv[G][U];
#pragma unroll
      for (int q = 0; q < G; ++q)
#pragma unroll
        for (int u = 0; u < U; ++u) {
          const int s2 = s0 + u < a.S ? s0 + u : a.S - 1;
          pv[q][u] = *reinterpret_cast<const float4*>(src[q] + s2 * sstride);
        }
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const bool use = s0 + u < a.S;          // adding 0 to a sum leaves it unchanged
#pragma unroll
        for (int q = 0; q < G; ++q) {
          v[q][0] += use ? pv[q][u].x : 0.f; v[q][1] += use ? pv[q][u].y : 0.f;
          v[q][2] += use ? pv[q][u].z : 0.f; v[q][3] += use ? pv[q][u].w : 0.f;
        }
      }
    }
#pragma unroll
    for (int q = 0; q < G; ++q) {
      const int gi = g0 + q * kBlock;
      if (gi >= ng) break;
      const int c = gi / (kTile / 4), j4 = (gi - c * (kTile / 4)) * 4;
      if (a.mode == 0) {
        for (int e = 0; e < 4; ++e) seg_add(a, c, (double)(v[q][e] * v[q][e]), sq);
      } else {
        store4(a, i, c, tile * kTile + j4, v[q]);
      }
    }
  }
  if (a.mode == 0) seg_publish<1>(a, tslot, tile, sq, dred);
}

template <int U>
__global__ __launch_bounds__(kBlock) void tokred_splits_kernel(TokredArgs a) {
  tokred_splits_block<U>(a, blockIdx.x, blockIdx.y);
}

// Split sums of several layers' passes in one launch (block (tile, sample) of job j at
// blk0[j] + sample * ntiles + tile).
template <int U>
__global__ __launch_bounds__(kBlock) void tokred_splits_batch_kernel(TokredBatch bt) {
  int jb = 0;
#pragma unroll
  for (int q = 1; q < kTokMaxJobs; ++q) jb += (q < bt.njobs && (int)blockIdx.x >= bt.blk0[q]) ? 1 : 0;
  const TokredArgs& a = bt.job[jb];
  const int rel = (int)blockIdx.x - bt.blk0[jb];
  tokred_splits_block<U>(a, rel % a.ntiles, rel / a.ntiles);
}

hipError_t launch_tokred_splits_batch(const TokredBatch& bt, hipStream_t st) {
  if (bt.njobs < 1 || bt.njobs > kTokMaxJobs || bt.blocks < 1) return hipErrorInvalidValue;
  int smax = 1;
  for (int j = 0; j < bt.njobs; ++j) smax = std::max(smax, (int)bt.job[j].S);
  const dim3 grid((unsigned)bt.blocks);
  if (smax <= 2) DPRC_LAUNCH(tokred_splits_batch_kernel<2>, grid, dim3(kBlock), 0, st, bt);
  else if (smax <= 4) DPRC_LAUNCH(tokred_splits_batch_kernel<4>, grid, dim3(kBlock), 0, st, bt);
  else DPRC_LAUNCH(tokred_splits_batch_kernel<8>, grid, dim3(kBlock), 0, st, bt);
  return hipGetLastError();
}

// estimate of layer g for sample i = scale * sum over tiles (in tile order);
// n2 gets the layers' estimates added one after another, as separate calls would
__global__ __launch_bounds__(kBlock) void tokred_sample_kernel(TokredArgs a) {
  __shared__ double dred[4];
  const int i = blockIdx.x;
  float n2 = a.accumulate ? a.n2[i] : 0.f;
  for (int g = 0; g < a.nseg; ++g) {
    const double* ts = a.tilesq + ((int64_t)g * a.B + i) * a.ntiles;
    double t = 0.0;
    for (int k = threadIdx.x; k < a.ntiles; k += kBlock) t += ts[k];
    t = block_sum_d(t, dred);
    const float est = (float)(t * (double)a.scale);
    n2 += est;
    if (threadIdx.x == 0 && a.n2_layer) a.n2_layer[(int64_t)g * a.B + i] = est;
  }
  if (threadIdx.x == 0) {
    a.n2[i] = n2;
    if (a.clip_c) a.clip_c[i] = clip_factor(n2, a.clip_C);
  }
}

// Per-sample sums of a whole call's token reductions in one launch (one workgroup of 16
// waves per sample).  The layers' (tile sums, count, estimate slot) are first listed in LDS
// in layer order; wave w then takes the layers w, w + 16, ..., four at a time with all their
// loads issued together, and sums each layer's tile sums exactly as block_sum_d does in
// tokred_sample_kernel (thread t's strided partial, then per wave of 64 such partials, then
// (w0 + w1) + (w2 + w3)), so the estimates are the same bit for bit; the layers' estimates
// then go to n2 in layer order, as a launch per group would add them.
constexpr int kSampleMaxLayers = kSampleMaxGroups * kMaxGroup;
constexpr int kSampleWaves = 16;
__global__ __launch_bounds__(64 * kSampleWaves) void sample_sums_kernel(SampleSumArgs a) {
  __shared__ float est[kSampleMaxLayers];
  __shared__ const double* lts[kSampleMaxLayers];
  __shared__ float* ln2[kSampleMaxLayers];
  __shared__ int lnt[kSampleMaxLayers];
  __shared__ int gseg[kSampleMaxGroups];
  __shared__ int nflat;
  const int i = blockIdx.x, lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
  if ((int)threadIdx.x < a.ngroups) gseg[threadIdx.x] = a.g[threadIdx.x].nseg;
  __syncthreads();
  if ((int)threadIdx.x < a.ngroups) {            // group q lists its layers at its offset
    const int q = threadIdx.x;
    int f = 0;
    for (int u = 0; u < q; ++u) f += gseg[u];
    const SampleGroup& gr = a.g[q];
    for (int s = 0; s < gr.nseg; ++s) {
      lts[f + s] = gr.tilesq + ((int64_t)s * a.B + i) * gr.ntiles;
      ln2[f + s] = gr.n2_layer ? gr.n2_layer + (int64_t)s * a.B + i : nullptr;
      lnt[f + s] = gr.ntiles;
    }
    if (q == a.ngroups - 1) nflat = f + gr.nseg;
  }
  __syncthreads();
  const int nl = nflat;
  constexpr int U = 4;                           // layers of a wave whose loads go out together
  for (int l0 = wv; l0 < nl; l0 += U * kSampleWaves) {
    double v[U][4];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int l = l0 + u * kSampleWaves;
      const int nt = l < nl ? lnt[l] : 0;
      const double* ts = l < nl ? lts[l] : nullptr;
#pragma unroll
      for (int w = 0; w < 4; ++w) v[u][w] = 64 * w + lane < nt ? ts[64 * w + lane] : 0.0;
    }
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int l = l0 + u * kSampleWaves;
      if (l >= nl) break;                          // wave-uniform
      const int nt = lnt[l];
      const double* ts = lts[l];
      double p[4];
#pragma unroll
      for (int w = 0; w < 4; ++w) {
        double t = v[u][w];
        for (int k = 64 * w + lane + kBlock; k < nt; k += kBlock) t += ts[k];   // beyond 256 tiles
        p[w] = wave_sum(t);
      }
      const double t = (p[0] + p[1]) + (p[2] + p[3]);
      const float e = (float)(t * (double)a.scale);
      if (lane == 0) {
        est[l] = e;
        if (ln2[l]) *ln2[l] = e;
      }
    }
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    float n2 = a.accumulate ? a.n2[i] : 0.f;
    for (int l = 0; l < nl; ++l) n2 += est[l];
    a.n2[i] = n2;
    if (a.clip_c) a.clip_c[i] = clip_factor(n2, a.clip_C);
  }
}

hipError_t launch_sample_sums(const SampleSumArgs& a, hipStream_t st) {
  if (a.ngroups < 1 || a.ngroups > kSampleMaxGroups || a.B < 1) return hipErrorInvalidValue;
  for (int q = 0; q < a.ngroups; ++q)
    if (a.g[q].nseg < 1 || a.g[q].nseg > kMaxGroup || a.g[q].ntiles < 1) return hipErrorInvalidValue;
  DPRC_LAUNCH(sample_sums_kernel, dim3((unsigned)a.B), dim3(64 * kSampleWaves), 0, st, a);
  return hipGetLastError();
}


hipError_t launch_tokred_splits(const TokredArgs& a, hipStream_t st) {
  const dim3 grid((unsigned)a.ntiles, (unsigned)a.B);
  if (a.S <= 2) DPRC_LAUNCH(tokred_splits_kernel<2>, grid, dim3(kBlock), 0, st, a);
  else if (a.S <= 4) DPRC_LAUNCH(tokred_splits_kernel<4>, grid, dim3(kBlock), 0, st, a);
  else DPRC_LAUNCH(tokred_splits_kernel<8>, grid, dim3(kBlock), 0, st, a);
  return hipGetLastError();
}

hipError_t launch_tokred_sample(const TokredArgs& a, hipStream_t st) {
  DPRC_LAUNCH(tokred_sample_kernel, dim3((unsigned)a.B), dim3(kBlock), 0, st, a);
  return hipGetLastError();
}

hipError_t launch_tokred_batch(TokredBatch bt, hipStream_t st) {
  if (bt.njobs < 1 || bt.njobs > kTokMaxJobs) return hipErrorInvalidValue;
  bool fast = true, pairs = bt.job[0].ncols_pad % 32 == 0;
  for (int j = 0; j < bt.njobs; ++j) {
    const TokredArgs& a = bt.job[j];
    if (a.ncols_pad != bt.job[0].ncols_pad) return hipErrorInvalidValue;   // one instantiation
    // buffer offsets within one 64-row stage stay below 2^31
    fast = fast && a.vec && a.n % 8 == 0 && (int64_t)kStage * a.ldx * 2 < ((int64_t)1 << 31);
    pairs = pairs && a.S == 1 && a.mode == 0;       // unsplit squared norms: two tiles per workgroup
  }
  const int tt = pairs ? 2 : 1;
  bt.blocks = 0;
  for (int j = 0; j < bt.njobs; ++j) {
    const TokredArgs& a = bt.job[j];
    bt.blk0[j] = bt.blocks;
    bt.blocks += (a.ntiles + tt - 1) / tt * a.S * a.B;
  }
  const dim3 grid((unsigned)round_up(bt.blocks, 8 * kXcdRun));   // whole windows (see the kernel)
#define DPRC_TOKRED_BATCH_LAUNCH(NB, TT)                                                                  \
  if (fast) DPRC_LAUNCH((tokred_batch_kernel<NB, true, TT>), grid, dim3(kBlock * TT), 0, st, bt);        \
  else DPRC_LAUNCH((tokred_batch_kernel<NB, false, TT>), grid, dim3(kBlock * TT), 0, st, bt);
  switch (bt.job[0].ncols_pad / 16) {
    case 1: DPRC_TOKRED_BATCH_LAUNCH(1, 1) break;
    case 2:
      if (tt == 2) { DPRC_TOKRED_BATCH_LAUNCH(2, 2) }
      else { DPRC_TOKRED_BATCH_LAUNCH(2, 1) }
      break;
    case 3: DPRC_TOKRED_BATCH_LAUNCH(3, 1) break;
    case 4:
      if (tt == 2) { DPRC_TOKRED_BATCH_LAUNCH(4, 2) }
      else { DPRC_TOKRED_BATCH_LAUNCH(4, 1) }
      break;
    default: return hipErrorInvalidValue;
  }
#undef DPRC_TOKRED_BATCH_LAUNCH
  return hipGetLastError();
}

hipError_t launch_tokred(const TokredArgs& a, hipStream_t st) {
  dim3 grid((unsigned)(a.ntiles * a.S), (unsigned)a.B);
  // buffer offsets within one 64-row stage stay below 2^31
  const bool fast = a.vec && a.n % 8 == 0 && (int64_t)kStage * a.ldx * 2 < ((int64_t)1 << 31);
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
