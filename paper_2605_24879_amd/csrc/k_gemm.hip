// Clipped accumulation grad = sum_i c_i A_i^T E_i (Algorithm 1, second backward
// pass of a bias-free linear layer) on bf16 matrix cores, fp32 accumulation.
//
// Workgroup tile 256 (d) x 256 (p), eight waves of 128 x 64, each a 4 x 2 grid of
// v_mfma_f32_32x32x16_bf16 (128 fp32 accumulators per lane).  The contraction
// runs over tokens and both operands are token-major, so 32-token slabs of A and E
// (256 columns each, 512-byte rows) are loaded with coalesced 16-byte reads,
// double-buffered through LDS and read back token-contiguous with the LDS
// transpose read.  A 128 x 64 wave tile reads 24 bytes of LDS per 1024 MFMA flops
// (a 64 x 64 tile needs 32), and two waves per SIMD overlap loads with MFMAs.
//
// Per-sample factors scale the fp32 accumulator at sample boundaries
// (acc <- acc * c_prev / c_i, and * c_last at the end), so the result is
// sum_i c_i (A_i^T E_i) without rounding c_i * E to bf16; samples with c_i = 0
// are skipped.  Tiles are ordered so that the workgroups of one XCD (workgroup
// ids are dealt round-robin to the 8 XCDs) share the tiles of the larger operand.
// Splits over the (sample, slab) list write fp32 partials summed in split order.
#include <algorithm>
#include "device.hpp"
#include "kernels.hpp"

namespace dprc {

typedef __attribute__((__vector_size__(16 * sizeof(float)))) float f32x16_t;

constexpr int kGM = 256;            // tile rows (d) and columns (p)
constexpr int kGK = 32;             // tokens per slab
constexpr int kGLd = kGM + 32;      // LDS row: 576 bytes; the 4 rows x 2 column groups of a 32-lane transpose read hit distinct 32-byte bank groups
constexpr int kGThreads = 512;      // 8 waves

__device__ __forceinline__ f32x16_t mfma32x32x16(const uint4& a, const uint4& b, f32x16_t c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8_t, a), __builtin_bit_cast(bf16x8_t, b),
                                                  c, 0, 0, 0);
}

template <bool FAST>
__global__ __launch_bounds__(kGThreads, 1) void gemm_kernel(GemmArgs a) {
  __shared__ __attribute__((aligned(16))) uint16_t la[2][kGK * kGLd];
  __shared__ __attribute__((aligned(16))) uint16_t le[2][kGK * kGLd];
  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
  const int g = lane >> 4, r4 = (lane & 15) >> 2, c4 = lane & 3;
  const int wm = wv >> 2, wn = wv & 3;               // wave tile rows wm*128, columns wn*64

  // tile of this workgroup: consecutive ids of one XCD walk the smaller dimension first
  const int tm_n = (a.d + kGM - 1) / kGM, tn_n = (a.p + kGM - 1) / kGM;
  const int ntiles = tm_n * tn_n;
  const int wg = blockIdx.x;
  // a bijection on [0, ntiles) when ntiles is a multiple of 8; identity otherwise
  const int lin = (ntiles & 7) == 0 ? (wg & 7) * (ntiles >> 3) + (wg >> 3) : wg;
  int tm, tn;
  if (a.d <= a.p) { tm = lin % tm_n; tn = lin / tm_n; } else { tn = lin % tn_n; tm = lin / tn_n; }
  const int d0 = tm * kGM, p0 = tn * kGM, split = blockIdx.y;

  const int sps = a.stages_per_sample;
  const int gs_begin = split * a.stages_per_split;
  const int gs_end = min(a.B * sps, gs_begin + a.stages_per_split);
  const int lr = tid >> 5, lc = (tid & 31) * 8;             // loads: rows lr + 16q, 8 columns at lc
  const int64_t ja = (int64_t)d0 + lc, je = (int64_t)p0 + lc;

  // position in the (sample, slab) list, advanced without divisions; samples with c_i = 0 are skipped
  struct Pos {
    int i, st, gs;
  };
  auto skip_zero = [&](Pos q) __attribute__((always_inline)) {
    while (q.gs < gs_end && a.c[q.i] == 0.f) {
      q.gs += sps - q.st;
      q.i += 1;
      q.st = 0;
    }
    return q;
  };
  auto advance = [&](Pos q) __attribute__((always_inline)) {
    q.gs += 1;
    if (++q.st == sps) {
      q.st = 0;
      q.i += 1;
    }
    return skip_zero(q);
  };
  uint4 ga[2], ge[2];
  auto gload = [&](const Pos& q) __attribute__((always_inline)) {
    const int64_t tok0 = (int64_t)q.st * kGK;
    const uint16_t* as = a.A + (int64_t)q.i * a.a_ss;
    const uint16_t* es = a.E + (int64_t)q.i * a.e_ss;
#pragma unroll
    for (int r = 0; r < 2; ++r) {
      const int64_t t = tok0 + lr + 16 * r;
      const bool ok = t < a.T;
      ga[r] = load_bf16x8<FAST>(as + (ok ? t : 0) * a.lda, ja, a.d, ok, as);
      ge[r] = load_bf16x8<FAST>(es + (ok ? t : 0) * a.lde, je, a.p, ok, es);
    }
  };
  auto swrite = [&](int buf) __attribute__((always_inline)) {
#pragma unroll
    for (int r = 0; r < 2; ++r) {
      *reinterpret_cast<uint4*>(&la[buf][(lr + 16 * r) * kGLd + lc]) = ga[r];
      *reinterpret_cast<uint4*>(&le[buf][(lr + 16 * r) * kGLd + lc]) = ge[r];
    }
  };

  f32x16_t acc[4][2];
#pragma unroll
  for (int x = 0; x < 4; ++x)
#pragma unroll
    for (int y = 0; y < 2; ++y)
#pragma unroll
      for (int q = 0; q < 16; ++q) acc[x][y][q] = 0.f;

  Pos cur = skip_zero(Pos{gs_begin / sps, gs_begin % sps, gs_begin});
  if (cur.gs < gs_end) {
    gload(cur);
    swrite(0);
  }
  Pos nxt = cur.gs < gs_end ? advance(cur) : cur;
  if (nxt.gs < gs_end) gload(nxt);
  __syncthreads();
  int buf = 0, cur_i = -1;
  float cur_c = 0.f;
  // the lane's transpose-read offsets: rows 8*(g/2) + r4 (+4), columns 16*(g%2) + 4*c4
  const int tr_row = 8 * (g >> 1) + r4, tr_col = 16 * (g & 1) + 4 * c4;
  while (cur.gs < gs_end) {
    if (cur.i != cur_i) {
      const float ci = a.c[cur.i];
      if (cur_i >= 0) {
        const float ratio = cur_c / ci;
#pragma unroll
        for (int x = 0; x < 4; ++x)
#pragma unroll
          for (int y = 0; y < 2; ++y) acc[x][y] *= ratio;
      }
      cur_c = ci;
      cur_i = cur.i;
    }
#pragma unroll
    for (int ks = 0; ks < 2; ++ks) {
      uint4 av[4], bv[2];
#pragma unroll
      for (int x = 0; x < 4; ++x) {
        const uint16_t* pa = &la[buf][(16 * ks + tr_row) * kGLd + wm * 128 + 32 * x + tr_col];
        av[x] = make_u4(lds_read_tr16(pa), lds_read_tr16(pa + 4 * kGLd));
      }
#pragma unroll
      for (int y = 0; y < 2; ++y) {
        const uint16_t* pe = &le[buf][(16 * ks + tr_row) * kGLd + wn * 64 + 32 * y + tr_col];
        bv[y] = make_u4(lds_read_tr16(pe), lds_read_tr16(pe + 4 * kGLd));
      }
#pragma unroll
      for (int x = 0; x < 4; ++x)
#pragma unroll
        for (int y = 0; y < 2; ++y) acc[x][y] = mfma32x32x16(av[x], bv[y], acc[x][y]);
    }
    const Pos after = nxt.gs < gs_end ? advance(nxt) : nxt;
    if (nxt.gs < gs_end) swrite(buf ^ 1);
    if (after.gs < gs_end) gload(after);
    __syncthreads();
    buf ^= 1;
    cur = nxt;
    nxt = after;
  }

  // epilogue: lane holds rows 8*(q/4) + 4*(lane/32) + q%4 and column lane%32 of each 32 x 32 block
  float* dst;
  int64_t ld;
  const bool direct = a.S == 1;
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
    for (int y = 0; y < 2; ++y) {
      const int col = p0 + wn * 64 + 32 * y + (lane & 31);
      if (col >= a.p) continue;
#pragma unroll
      for (int q = 0; q < 16; ++q) {
        const int row = d0 + wm * 128 + 32 * x + 8 * (q >> 2) + 4 * (lane >> 5) + (q & 3);
        if (row >= a.d) continue;
        const float v = acc[x][y][q] * cur_c;
        float* o = dst + (int64_t)row * ld + col;
        if (direct && a.accumulate) *o += v;
        else *o = v;
      }
    }
}

GemmPlan gemm_plan_v2(int64_t B, int64_t T, int64_t d, int64_t p) {
  GemmPlan g;
  g.sps = (int32_t)ceil_div(T, kGK);
  const int64_t total = B * g.sps;
  const int64_t tiles = ceil_div(d, kGM) * ceil_div(p, kGM);
  int64_t S = 1;
  if (tiles < 256) S = std::min<int64_t>(ceil_div(256, tiles), std::max<int64_t>(1, total / 16));
  g.spl = (int32_t)ceil_div(total, S);
  g.S = (int32_t)ceil_div(total, g.spl);
  g.tiles = (int32_t)tiles;
  return g;
}

hipError_t launch_gemm(const GemmArgs& a, hipStream_t st) {
  const int tiles = (int)(ceil_div(a.d, kGM) * ceil_div(a.p, kGM));
  dim3 grid((unsigned)tiles, (unsigned)a.S);
  if (a.vec_a && a.vec_e && a.d % 8 == 0 && a.p % 8 == 0)
    DPRC_LAUNCH(gemm_kernel<true>, grid, dim3(kGThreads), 0, st, a);
  else
    DPRC_LAUNCH(gemm_kernel<false>, grid, dim3(kGThreads), 0, st, a);
  return hipGetLastError();
}

}  // namespace dprc
