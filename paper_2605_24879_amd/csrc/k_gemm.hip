// Clipped accumulation grad = sum_i c_i A_i^T E_i (Algorithm 1, second backward
// pass of a bias-free linear layer) on bf16 matrix cores, fp32 accumulation.
//
// Workgroup tile 256 (d) x 256 (p), eight waves of 128 x 64 (two per SIMD), each a
// 4 x 2 grid of v_mfma_f32_32x32x16_bf16 (128 fp32 accumulators per lane).  The
// contraction runs over tokens and both operands are token-major, so 32-token
// slabs of A and E (256 columns each, 512-byte rows) are loaded with coalesced
// 16-byte buffer reads, two slabs ahead in registers, double-buffered through LDS
// and read back token-contiguous with the LDS transpose read.  Each step is
// software-pipelined over the two 16-token halves of a slab, and the two waves of
// a SIMD cover each other's waits (one wave of 128 x 128 per SIMD with the same
// pipeline, or with LDS reads, writes and loads placed between the MFMAs by
// scheduling barriers, was 7 to 10 percent slower).
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
constexpr int kGK = 32;             // tokens per slab (64-token slabs measured 5 to 15 percent slower)
constexpr int kGLd = kGM + 32;      // LDS row: 576 bytes; the 4 rows x 2 column groups of a 32-lane transpose read hit distinct 32-byte bank groups

__device__ __forceinline__ f32x16_t mfma32x32x16(const uint4& a, const uint4& b, f32x16_t c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8_t, a), __builtin_bit_cast(bf16x8_t, b),
                                                  c, 0, 0, 0);
}

// NW = 8: waves of 128 x 64 (2 x 4 of them); NW = 4: waves of 128 x 128 (2 x 2).
template <int V>
struct GInt {
  static constexpr int value = V;
};

// wg: the tile (before the XCD reordering), split: the token split.
template <int NW, int NS, bool FAST>
__device__ __forceinline__ void gemm_body(const GemmArgs& a, int wg, int split) {
  constexpr int kThreads = 64 * NW;
  constexpr int WN = NW == 8 ? 64 : 128;             // wave tile columns
  constexpr int YB = WN / 32;                        // 32-column MFMA blocks per wave
  constexpr int RP = kThreads / 32;                  // slab rows per load pass
  constexpr int RQ = kGK / RP;                       // load passes per slab
  __shared__ __attribute__((aligned(16))) uint16_t la[2][kGK * kGLd];
  __shared__ __attribute__((aligned(16))) uint16_t le[2][kGK * kGLd];
  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
  const int g = lane >> 4, r4 = (lane & 15) >> 2, c4 = lane & 3;
  const int wm = wv / (kGM / WN), wn = wv % (kGM / WN);   // wave tile rows wm*128, columns wn*WN

  // tile of this workgroup: consecutive ids of one XCD walk the smaller dimension first
  const int tm_n = (a.d + kGM - 1) / kGM, tn_n = (a.p + kGM - 1) / kGM;
  const int ntiles = tm_n * tn_n;
  // a bijection on [0, ntiles) when ntiles is a multiple of 8; identity otherwise
  const int lin = (ntiles & 7) == 0 ? (wg & 7) * (ntiles >> 3) + (wg >> 3) : wg;
  int tm, tn;
  if (a.d <= a.p) { tm = lin % tm_n; tn = lin / tm_n; } else { tn = lin % tn_n; tm = lin / tn_n; }
  const int d0 = tm * kGM, p0 = tn * kGM;

  const int sps = a.stages_per_sample;
  const int gs_begin = split * a.stages_per_split;
  const int gs_end = min(a.B * sps, gs_begin + a.stages_per_split);
  const int lr = tid >> 5, lc = (tid & 31) * 8;             // loads: rows lr + RP q, 8 columns at lc
  const int64_t ja = (int64_t)d0 + lc, je = (int64_t)p0 + lc;

  uint4 ga[NS][RQ], ge[NS][RQ];                   // slabs in flight
  // FAST: per slab one buffer resource per operand over its (up to) 32 token rows,
  // starting at the tile's first column; rows past T and columns past d / p read
  // as zero through out-of-range offsets, and a slab past the sample's last one has
  // an empty range.  Element loads otherwise.
  const uint32_t arow = (uint32_t)a.lda * 2u, erow = (uint32_t)a.lde * 2u;
  const uint32_t aoff = d0 + lc < a.d ? (uint32_t)lr * arow + 2u * lc : kOobOffset;
  const uint32_t eoff = p0 + lc < a.p ? (uint32_t)lr * erow + 2u * lc : kOobOffset;
  auto gload = [&](int sl, int i, int st, int st_end) __attribute__((always_inline)) {
    const int tok0 = st * kGK;
    const uint16_t* as = a.A + (int64_t)i * a.a_ss;
    const uint16_t* es = a.E + (int64_t)i * a.e_ss;
    if constexpr (FAST) {
      const int rows = st < st_end ? min(kGK, a.T - tok0) : 0;
      const int64_t t0 = rows > 0 ? tok0 : 0;
      const __amdgpu_buffer_rsrc_t ar = buffer_rsrc(as + t0 * a.lda + d0, (uint32_t)rows * arow);
      const __amdgpu_buffer_rsrc_t er = buffer_rsrc(es + t0 * a.lde + p0, (uint32_t)rows * erow);
#pragma unroll
      for (int r = 0; r < RQ; ++r) {
        ga[sl][r] = buffer_load16(ar, aoff + (uint32_t)(RP * r) * arow);
        ge[sl][r] = buffer_load16(er, eoff + (uint32_t)(RP * r) * erow);
      }
    } else {
#pragma unroll
      for (int r = 0; r < RQ; ++r) {
        const int t = tok0 + lr + RP * r;
        const bool ok = st < st_end && t < a.T;
        ga[sl][r] = load8_elem(as + (int64_t)(ok ? t : 0) * a.lda, ja, a.d, ok);
        ge[sl][r] = load8_elem(es + (int64_t)(ok ? t : 0) * a.lde, je, a.p, ok);
      }
    }
  };
  auto swrite = [&](int sl, int buf) __attribute__((always_inline)) {
#pragma unroll
    for (int r = 0; r < RQ; ++r) {
      *reinterpret_cast<uint4*>(&la[buf][(lr + RP * r) * kGLd + lc]) = ga[sl][r];
      *reinterpret_cast<uint4*>(&le[buf][(lr + RP * r) * kGLd + lc]) = ge[sl][r];
    }
  };

  f32x16_t acc[4][YB];
#pragma unroll
  for (int x = 0; x < 4; ++x)
#pragma unroll
    for (int y = 0; y < YB; ++y)
#pragma unroll
      for (int q = 0; q < 16; ++q) acc[x][y][q] = 0.f;

  // the lane's transpose-read offsets: rows 8*(g/2) + r4 (+4), columns 16*(g%2) + 4*c4
  const int tr_row = 8 * (g >> 1) + r4, tr_col = 16 * (g & 1) + 4 * c4;
  // The two 16-token halves of a slab are separate register fragment sets (f0, f1):
  // a step multiplies half 0 while reading half 1 and writing the next slab to the
  // other LDS buffer, then (after the step's one barrier) multiplies half 1 while
  // reading half 0 of the next slab, so a wave always has MFMAs whose operands are
  // already in registers.
  uint4 f0a[4], f0b[YB], f1a[4], f1b[YB];
  auto frag = [&](uint4 (&av)[4], uint4 (&bv)[YB], int buf, int ks) __attribute__((always_inline)) {
#pragma unroll
    for (int x = 0; x < 4; ++x) {
      const uint16_t* pa = &la[buf][(16 * ks + tr_row) * kGLd + wm * 128 + 32 * x + tr_col];
      av[x] = make_u4(lds_read_tr16(pa), lds_read_tr16(pa + 4 * kGLd));
    }
#pragma unroll
    for (int y = 0; y < YB; ++y) {
      const uint16_t* pe = &le[buf][(16 * ks + tr_row) * kGLd + wn * WN + 32 * y + tr_col];
      bv[y] = make_u4(lds_read_tr16(pe), lds_read_tr16(pe + 4 * kGLd));
    }
  };
  auto mm = [&](const uint4 (&av)[4], const uint4 (&bv)[YB]) __attribute__((always_inline)) {
#pragma unroll
    for (int x = 0; x < 4; ++x)
#pragma unroll
      for (int y = 0; y < YB; ++y) acc[x][y] = mfma32x32x16(av[x], bv[y], acc[x][y]);
  };

  // samples of this split in order; the accumulator is rescaled between samples
  // (outside the slab loop), samples with c_i = 0 are skipped
  float cur_c = 0.f;
  bool started = false;
  const int i_first = gs_begin / sps, i_last = gs_end > gs_begin ? (gs_end - 1) / sps : i_first - 1;
  for (int i = i_first; i <= i_last; ++i) {
    const float ci = a.c[i];
    if (ci == 0.f) continue;
    const int st_lo = max(0, gs_begin - i * sps), st_hi = min(sps, gs_end - i * sps);
    if (started) {
      const float ratio = cur_c / ci;
#pragma unroll
      for (int x = 0; x < 4; ++x)
#pragma unroll
        for (int y = 0; y < YB; ++y) acc[x][y] *= ratio;
    }
    started = true;
    cur_c = ci;
    __syncthreads();                               // the previous sample's last slab is consumed
    // slab k sits in LDS buffer k % 2 while it is multiplied; register slot k % NS
    // receives slab k + NS at the start of that step, and slot (k + 1) % NS (slab
    // k + 1, issued NS - 1 steps earlier) goes to the other buffer at its end.
    // Slabs past the sample's last load empty ranges (zeros).
#pragma unroll
    for (int q = 0; q < NS; ++q) gload(q, i, st_lo + q, st_hi);
    swrite(0, 0);
    __syncthreads();
    frag(f0a, f0b, 0, 0);
    constexpr int NQ = kGK / 16;                 // 16-token quarters of a slab (even)
    auto step = [&](int st, auto u) __attribute__((always_inline)) {
      constexpr int k = decltype(u)::value;      // step index modulo 2 NS
      // loads of slab k + NS (register slot k % NS, free since slab k went to LDS);
      // then the MFMAs of each 16-token part of slab k while reading the next part;
      // slab k + 1 (slot (k + 1) % NS) goes to the other buffer before the barrier,
      // after which the last part is multiplied while part 0 of slab k + 1 is read
      gload(k % NS, i, st + NS, st_hi);
#pragma unroll
      for (int qq = 0; qq + 1 < NQ; ++qq) {
        if (qq % 2 == 0) {
          frag(f1a, f1b, k % 2, qq + 1);
          mm(f0a, f0b);
        } else {
          frag(f0a, f0b, k % 2, qq + 1);
          mm(f1a, f1b);
        }
      }
      swrite((k + 1) % NS, (k + 1) % 2);
      __syncthreads();
      frag(f0a, f0b, (k + 1) % 2, 0);
      mm(f1a, f1b);
    };
    // whole groups of 2 NS steps in the loop (no early exit reaches its back edge,
    // so the compiler's wait counting stays exact), the remainder after it
    int st = st_lo;
    for (; st + 2 * NS <= st_hi; st += 2 * NS) {
      step(st, GInt<0>{});
      step(st + 1, GInt<1>{});
      if constexpr (NS > 1) {
        step(st + 2, GInt<2>{});
        step(st + 3, GInt<3>{});
      }
      if constexpr (NS > 2) {
        step(st + 4, GInt<4>{});
        step(st + 5, GInt<5>{});
      }
    }
    if (st < st_hi) step(st, GInt<0>{});
    if constexpr (NS > 1) {
      if (st + 1 < st_hi) step(st + 1, GInt<1>{});
      if (st + 2 < st_hi) step(st + 2, GInt<2>{});
    }
    if constexpr (NS > 2) {
      if (st + 3 < st_hi) step(st + 3, GInt<3>{});
      if (st + 4 < st_hi) step(st + 4, GInt<4>{});
    }
    __syncthreads();                               // the last reads of both buffers are done
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
    for (int y = 0; y < YB; ++y) {
      const int col = p0 + wn * WN + 32 * y + (lane & 31);
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

template <int NW, int NS, bool FAST>
__global__ __launch_bounds__(64 * NW, 1) void gemm_kernel(GemmArgs a) {
  gemm_body<NW, NS, FAST>(a, blockIdx.x, blockIdx.y);
}

// Several layers in one launch, each unsplit (S = 1): job j owns blocks blk0[j] ..
// blk0[j] + ntiles_j - 1, and blk0[j] is a multiple of 8, so that a job's blocks are
// dealt to the XCDs as those of a launch of its own; blocks up to the next multiple of
// 8 are idle.
template <int NW, int NS, bool FAST>
__global__ __launch_bounds__(64 * NW, 1) void gemm_batch_kernel(GemmBatch bt) {
  int jb = 0;
#pragma unroll 8
  for (int q = 1; q < kGemmMaxJobs; ++q) jb += (q < bt.njobs && (int)blockIdx.x >= bt.blk0[q]) ? 1 : 0;
  const GemmArgs& a = bt.job[jb];
  const int wg = (int)blockIdx.x - bt.blk0[jb];
  if (wg >= (int)(((int64_t)a.d + kGM - 1) / kGM * (((int64_t)a.p + kGM - 1) / kGM))) return;
  gemm_body<NW, NS, FAST>(a, wg, 0);
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
  constexpr int NW = 8, NS = 2;
  // buffer offsets within one 32-row slab stay below 2^31
  if (a.vec_a && a.vec_e && a.d % 8 == 0 && a.p % 8 == 0 &&
      (int64_t)kGK * std::max(a.lda, a.lde) * 2 < ((int64_t)1 << 31))
    DPRC_LAUNCH((gemm_kernel<NW, NS, true>), grid, dim3(64 * NW), 0, st, a);
  else
    DPRC_LAUNCH((gemm_kernel<NW, NS, false>), grid, dim3(64 * NW), 0, st, a);
  return hipGetLastError();
}

hipError_t launch_gemm_batch(GemmBatch bt, hipStream_t st) {
  if (bt.njobs < 1 || bt.njobs > kGemmMaxJobs) return hipErrorInvalidValue;
  constexpr int NW = 8, NS = 2;
  bool fast = true;
  int64_t blocks = 0;
  for (int j = 0; j < bt.njobs; ++j) {
    const GemmArgs& a = bt.job[j];
    if (a.S != 1) return hipErrorInvalidValue;
    fast = fast && a.vec_a && a.vec_e && a.d % 8 == 0 && a.p % 8 == 0 &&
           (int64_t)kGK * std::max(a.lda, a.lde) * 2 < ((int64_t)1 << 31);
    bt.blk0[j] = (int32_t)blocks;
    blocks += round_up(ceil_div(a.d, kGM) * ceil_div(a.p, kGM), 8);
  }
  if (blocks >= ((int64_t)1 << 31)) return hipErrorInvalidValue;
  const dim3 grid((unsigned)blocks);
  if (fast) DPRC_LAUNCH((gemm_batch_kernel<NW, NS, true>), grid, dim3(64 * NW), 0, st, bt);
  else DPRC_LAUNCH((gemm_batch_kernel<NW, NS, false>), grid, dim3(64 * NW), 0, st, bt);
  return hipGetLastError();
}

}  // namespace dprc
