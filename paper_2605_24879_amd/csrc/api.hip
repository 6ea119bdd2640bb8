// C-ABI entry points of libdprc (declared in include/dprc.h): argument
// validation, side resolution, workspace planning and the launch sequence of
// each call.  Nothing here allocates device memory or synchronises the stream.
#include <algorithm>
#include <cmath>
#include <cstring>
#include <mutex>

#include "../../include/dprc.h"
#include "kernels.hpp"

using namespace dprc;

namespace {

constexpr size_t kAlign = 256;

struct Arena {  // carves 256-byte aligned regions out of the caller's workspace
  char* base;
  size_t off = 0;
  explicit Arena(void* b) : base(static_cast<char*>(b)) {}
  template <class T>
  T* take(size_t count) {
    off = (off + kAlign - 1) / kAlign * kAlign;
    T* p = base ? reinterpret_cast<T*>(base + off) : nullptr;
    off += count * sizeof(T);
    return p;
  }
};

// A layer after side resolution: X is sketched (m columns = probe rows), Xo is the other operand.
struct View {
  const void* X;
  int64_t ldx, m;
  const void* Xo;
  int64_t ldo, n;
  int64_t B, T;
  dprc_dtype dtype;
  uint32_t layer_id;
};

dprc_side resolve(const dprc_layer& L, dprc_side side) {
  if (side == DPRC_SIDE_AUTO) return L.d > L.p ? DPRC_SIDE_IN : DPRC_SIDE_OUT;
  return side;
}

View view_of(const dprc_layer& L, dprc_side side) {
  View v;
  if (resolve(L, side) == DPRC_SIDE_OUT) {
    v.X = L.E; v.ldx = L.lde; v.m = L.p;
    v.Xo = L.A; v.ldo = L.lda; v.n = L.d;
  } else {
    v.X = L.A; v.ldx = L.lda; v.m = L.d;
    v.Xo = L.E; v.ldo = L.lde; v.n = L.p;
  }
  v.B = L.B; v.T = L.T; v.dtype = L.dtype; v.layer_id = L.layer_id;
  return v;
}

bool aligned(const void* p, size_t a) { return (reinterpret_cast<uintptr_t>(p) % a) == 0; }

// bf16 token rows starting on 16-byte boundaries take the 16-byte load path
int rows16(const void* p, int64_t ld) { return aligned(p, 16) && ld % 8 == 0; }

dprc_status check_layer(const dprc_layer& L) {
  if (!L.A || !L.E) return DPRC_ERROR_INVALID_VALUE;
  if (L.B < 1 || L.T < 1 || L.d < 1 || L.p < 1) return DPRC_ERROR_INVALID_VALUE;
  if (L.lda < L.d || L.lde < L.p) return DPRC_ERROR_INVALID_VALUE;
  if (L.dtype != DPRC_F32 && L.dtype != DPRC_BF16) return DPRC_ERROR_INVALID_VALUE;
  if (L.B > 65535 || L.T > (1LL << 30) || L.d > (1LL << 30) || L.p > (1LL << 30))
    return DPRC_ERROR_NOT_SUPPORTED;
  if (L.B * L.T > (1LL << 31)) return DPRC_ERROR_NOT_SUPPORTED;
  const size_t elem = L.dtype == DPRC_BF16 ? 2 : 4;
  if (!aligned(L.A, elem) || !aligned(L.E, elem)) return DPRC_ERROR_NOT_SUPPORTED;
  return DPRC_SUCCESS;
}

dprc_status check_layers(const dprc_layer* layers, int32_t num, dprc_side side) {
  if (!layers || num < 1) return DPRC_ERROR_INVALID_VALUE;
  if (side != DPRC_SIDE_OUT && side != DPRC_SIDE_IN && side != DPRC_SIDE_AUTO) return DPRC_ERROR_INVALID_VALUE;
  for (int32_t l = 0; l < num; ++l) {
    dprc_status s = check_layer(layers[l]);
    if (s != DPRC_SUCCESS) return s;
    if (layers[l].B != layers[0].B) return DPRC_ERROR_INVALID_VALUE;
  }
  return DPRC_SUCCESS;
}

void key_of(uint64_t seed, uint32_t& k0, uint32_t& k1) {
  k0 = (uint32_t)(seed & 0xFFFFFFFFu);
  k1 = (uint32_t)(seed >> 32);
}

// column blocks of 16 the kernels are instantiated for
int pad_cols(int ncols) {
  static const int nbs[] = {1, 2, 3, 4, 5, 6, 8, 12, 16};
  const int need = (ncols + 15) / 16;
  for (int nb : nbs)
    if (nb >= need) return 16 * nb;
  return -1;
}

int rows_per_wg(int64_t rows, int ncols_pad, bool dense = false) {
  const int nb = ncols_pad / 16;
  // 32-row workgroups while that still gives 256 or more of them (fixed per-workgroup
  // costs such as the probe generation are spread over twice the data).  With dense
  // columns every workgroup reads the whole dense operand from L2 (as many bytes as its
  // rows for 32 rows and 16 dense columns), so 64-row workgroups halve that traffic.
  if (dense && rows >= 64 * 256 && nb <= 4) return 64;
  // 48 sign columns stay in 16-row blocks, where the projection's row-block body takes
  // them (it serves at most 64 columns per 16 rows, 32 per 32): 10% faster on Hutch++
  // pass 1 of a decoder layer at 32768 tokens
  int rb = 1;
  if (rows >= 8 * 1024 && (dense || nb != 3)) rb = 2;
  while (rb > 1 && rb * nb > 8) rb >>= 1;
  return 16 * rb;
}

int words_per_chunk(int64_t m, int nz) {
  // whole 512-column stages of the projection kernel per chunk; at most 4096 probe words
  // (16 KB of LDS), so that three 32-row workgroups fit in a CU's 160 KB even at k = 32
  const int64_t all = round_up(ceil_div(m, 32), 16);
  if (nz <= 0) return (int)all;
  return (int)std::min<int64_t>(all, std::max(16, (4096 / nz) & ~15));
}

// Token-reduction geometry for one (operand width n, columns) pass.
struct TokPlan {
  int32_t ntiles, S, sps, T_pad;
};
TokPlan tok_plan(int64_t B, int64_t T, int64_t n) {
  TokPlan p;
  p.T_pad = (int32_t)round_up(T, kStage);
  p.ntiles = (int32_t)ceil_div(n, kTile);
  const int64_t stages = p.T_pad / kStage;
  const int64_t base = B * p.ntiles;
  int64_t S = std::max<int64_t>(1, ceil_div(256, base));
  S = std::min<int64_t>(S, std::max<int64_t>(1, stages / 4));  // >= 4 stages (256 tokens) per split
  p.sps = (int32_t)ceil_div(stages, S);
  p.S = (int32_t)ceil_div(stages, p.sps);
  return p;
}

struct TokBufs {
  float* part;
  double* tilesq;
  uint16_t* Y = nullptr;     // a group's own Y (batched launches)
};

TokBufs take_tok(Arena& ar, int64_t B, const TokPlan& tp, int ncols_pad, int nseg = 1) {
  TokBufs b;
  b.part = tp.S > 1 ? ar.take<float>((size_t)B * tp.ntiles * tp.S * ncols_pad * kTile) : nullptr;
  b.tilesq = ar.take<double>((size_t)nseg * B * tp.ntiles);
  return b;
}

dprc_status hip_status(hipError_t e) { return e == hipSuccess ? DPRC_SUCCESS : DPRC_ERROR_HIP; }

// Per-launch timing for diagnostics (dprc_trace_launches): host-thread state only.
struct Trace {
  hipEvent_t* events = nullptr;
  int32_t* kinds = nullptr;
  int32_t capacity = 0;
  int32_t* count = nullptr;
};
thread_local Trace g_trace;
thread_local LaunchEvents g_next_events;

// The start/stop events ride on the launch itself (hipExtLaunchKernelGGL in DPRC_LAUNCH).
template <class F>
hipError_t traced(int kind, hipStream_t, F&& launch) {
  Trace& t = g_trace;
  const bool on = t.events && t.count && *t.count < t.capacity;
  if (on) g_next_events = LaunchEvents{t.events[2 * *t.count], t.events[2 * *t.count + 1]};
  const hipError_t e = launch();
  g_next_events = LaunchEvents{};
  if (on && e == hipSuccess) {
    if (t.kinds) t.kinds[*t.count] = kind;
    ++*t.count;
  }
  return e;
}

// ---- one projection + token-reduction pass (bf16) --------------------------------------------
struct PassSpec {
  const uint16_t* X; int64_t ldx, m;      // projected operand
  const uint16_t* Xo; int64_t ldo, n;     // reduced operand
  int32_t nd; const uint16_t* Rhi; const uint16_t* Rlo; int64_t ld_r;   // dense columns
  bool shared_r;                                                        // one R for all samples
  int32_t nz; uint32_t stream_id; int probe_kind;                       // generated columns
  int32_t z_split; uint32_t stream_id2;    // columns from z_split on: stream_id2 (0: none)
  int mode; float scale; float* n2; float* n2_layer; int accumulate;    // mode 0
  float* M; int64_t m_ld; uint16_t* Mhi; uint16_t* Mlo; int64_t mh_ld;  // mode 1
  int32_t m_col0, mh_ncols;                // M takes columns >= m_col0, Mhi/Mlo < mh_ncols (0: all)
  int64_t m_ss, mh_ss;                     // per-sample strides (0: columns x leading dimension)
};

size_t pass_ws(Arena& ar, int64_t B, int64_t T, int64_t n, int ncols_pad, uint16_t** Yt, TokBufs* tb,
               TokPlan* tpo, int nseg = 1) {
  const TokPlan tp = tok_plan(B, T, n);
  uint16_t* y = ar.take<uint16_t>((size_t)2 * ncols_pad * B * tp.T_pad);
  TokBufs t = take_tok(ar, B, tp, ncols_pad, nseg);
  if (Yt) *Yt = y;
  if (tb) *tb = t;
  if (tpo) *tpo = tp;
  return ar.off;
}

// One projection + token-reduction pass.  With `part`, the token-split partials go there
// instead of the pass scratch; with `defer` (store mode), the split sums are not launched
// and the token-reduction arguments are returned for a batched launch (defer->S tells
// whether one is needed).
// Kernel arguments of one pass over the given Y and token-reduction buffers.
void pass_args(const PassSpec& ps, int64_t B, int64_t T, uint32_t k0, uint32_t k1, uint32_t layer, uint16_t* Yt,
               const TokBufs& tb, const TokPlan& tp, ProjectArgs& pa, TokredArgs& ta) {
  const int ncols = ps.nd + ps.nz;
  const int ncols_pad = pad_cols(ncols);
  pa.X = ps.X; pa.ldx = ps.ldx; pa.x_ss = T * ps.ldx;
  pa.B = (int32_t)B; pa.T = (int32_t)T; pa.m = (int32_t)ps.m; pa.T_pad = tp.T_pad;
  pa.nd = ps.nd; pa.nz = ps.nz; pa.ncols_pad = ncols_pad;
  pa.Rhi = ps.Rhi; pa.Rlo = ps.Rlo; pa.ld_r = ps.ld_r; pa.r_ss = ps.shared_r ? 0 : (int64_t)ps.nd * ps.ld_r;
  pa.probe_kind = ps.probe_kind; pa.key0 = k0; pa.key1 = k1; pa.layer_id = layer; pa.stream_id = ps.stream_id;
  pa.z_split = ps.z_split > 0 ? ps.z_split : ps.nz; pa.stream_id2 = ps.stream_id2;
  pa.words_per_chunk = words_per_chunk(ps.m, ps.nz);
  pa.Yt = Yt; pa.yt_ld = B * tp.T_pad;
  pa.ylo_off = (int64_t)ncols_pad * pa.yt_ld; pa.ncols_write = ncols_pad;
  pa.zero_ptr = nullptr; pa.zero_count = 0;
  pa.vec = rows16(ps.X, ps.ldx);

  ta.X = ps.Xo; ta.ldx = ps.ldo; ta.x_ss = T * ps.ldo;
  ta.B = (int32_t)B; ta.T = (int32_t)T; ta.n = (int32_t)ps.n;
  ta.Yt = Yt; ta.yt_ld = B * tp.T_pad; ta.T_pad = tp.T_pad; ta.ncols = ncols; ta.ncols_pad = ncols_pad;
  ta.ntiles = tp.ntiles; ta.S = tp.S; ta.stages_per_split = tp.sps;
  ta.mode = ps.mode; ta.seg = ncols; ta.nseg = 1;
  ta.clip_C = 0.f; ta.clip_c = nullptr;
  ta.part = tb.part; ta.tilesq = tb.tilesq;
  ta.scale = ps.scale; ta.n2 = ps.n2; ta.n2_layer = ps.n2_layer; ta.accumulate = ps.accumulate;
  ta.M = ps.M; ta.m_ld = ps.m_ld; ta.m_ss = ps.m_ss > 0 ? ps.m_ss : (int64_t)ncols * ps.m_ld;
  ta.Mhi = ps.Mhi; ta.Mlo = ps.Mlo; ta.mh_ld = ps.mh_ld; ta.mh_ss = ps.mh_ss > 0 ? ps.mh_ss : (int64_t)ncols * ps.mh_ld;
  ta.m_col0 = ps.m_col0; ta.mh_ncols = ps.mh_ncols;
  ta.vec = rows16(ps.Xo, ps.ldo);
}

dprc_status run_pass(const PassSpec& ps, int64_t B, int64_t T, uint32_t k0, uint32_t k1, uint32_t layer,
                     void* ws, hipStream_t st, float* part = nullptr, TokredArgs* defer = nullptr) {
  const int ncols_pad = pad_cols(ps.nd + ps.nz);
  Arena ar(ws);
  uint16_t* Yt;
  TokBufs tb;
  TokPlan tp;
  pass_ws(ar, B, T, ps.n, ncols_pad, &Yt, &tb, &tp);
  if (part && tp.S > 1) tb.part = part;
  ProjectArgs pa;
  TokredArgs ta;
  pass_args(ps, B, T, k0, k1, layer, Yt, tb, tp, pa, ta);
  hipError_t e = traced(DPRC_KERNEL_PROJECT, st, [&] { return launch_project(pa, rows_per_wg(B * tp.T_pad, ncols_pad, pa.nd > 0), st); });
  if (e != hipSuccess) return DPRC_ERROR_HIP;
  e = traced(DPRC_KERNEL_TOKEN_REDUCE, st, [&] { return launch_tokred(ta, st); });
  if (e != hipSuccess) return DPRC_ERROR_HIP;
  if (defer && ps.mode == 1) {
    *defer = ta;
    return DPRC_SUCCESS;
  }
  if (tp.S > 1) {
    e = traced(DPRC_KERNEL_TOKEN_SPLITS, st, [&] { return launch_tokred_splits(ta, st); });
    if (e != hipSuccess) return DPRC_ERROR_HIP;
  }
  if (ps.mode == 0) return hip_status(traced(DPRC_KERNEL_SAMPLE_SUM, st, [&] { return launch_tokred_sample(ta, st); }));
  return DPRC_SUCCESS;
}

// Token-split partial floats of a pass (0 without splits).
int64_t part_floats(int64_t B, int64_t T, int64_t n, int ncols) {
  const TokPlan tp = tok_plan(B, T, n);
  return tp.S > 1 ? B * tp.ntiles * tp.S * pad_cols(ncols) * kTile : 0;
}

// Split sums of deferred passes (those with token splits), up to kTokMaxJobs per launch.
dprc_status run_splits_batch(const TokredArgs* ta, int n, hipStream_t st) {
  TokredBatch bt{};
  auto flush = [&]() -> bool {
    if (bt.njobs == 0) return true;
    const hipError_t e = traced(DPRC_KERNEL_TOKEN_SPLITS, st, [&] { return launch_tokred_splits_batch(bt, st); });
    bt.njobs = 0; bt.blocks = 0;
    return e == hipSuccess;
  };
  for (int j = 0; j < n; ++j) {
    if (ta[j].S <= 1) continue;
    bt.blk0[bt.njobs] = bt.blocks;
    bt.job[bt.njobs++] = ta[j];
    bt.blocks += ta[j].ntiles * ta[j].B;
    if (bt.njobs == kTokMaxJobs && !flush()) return DPRC_ERROR_HIP;
  }
  return flush() ? DPRC_SUCCESS : DPRC_ERROR_HIP;
}

size_t pass_ws_bytes(int64_t B, int64_t T, int64_t n, int ncols) {
  Arena ar(nullptr);
  return pass_ws(ar, B, T, n, pad_cols(ncols), nullptr, nullptr, nullptr);
}

// ---- Hutchinson ---------------------------------------------------------------------------------
constexpr int32_t kMaxGaussK = 32;   // Gaussian probes travel as dense columns (at most 32)

// Gaussian probe columns, generated at the front of the workspace: bf16 hi + lo
// pairs with rows padded to a multiple of 128 (the projection reads whole
// 128-column slices), or fp32 for fp32 layers.
struct GaussBufs { uint16_t *hi, *lo; float* f32; int64_t ld; };

GaussBufs take_gauss(Arena& ar, const View& v, int32_t k) {
  GaussBufs g{};
  if (v.dtype == DPRC_BF16) {
    g.ld = round_up(v.m, kTile);
    g.hi = ar.take<uint16_t>((size_t)k * g.ld);
    g.lo = ar.take<uint16_t>((size_t)k * g.ld);
  } else {
    g.ld = v.m;
    g.f32 = ar.take<float>((size_t)k * g.ld);
  }
  return g;
}

// Consecutive bf16 layers that read the same activations (same A, shape and row
// stride) and sketch the output side share one token reduction over A: each
// layer's Y = E Z fills k columns of one Y, and the reduction squares each
// layer's columns separately (q, k, v of an attention block; gate and up).
int32_t group_end(const dprc_layer* layers, int32_t l0, int32_t num_layers, int32_t k, dprc_side side) {
  const dprc_layer& L = layers[l0];
  if (L.dtype != DPRC_BF16 || resolve(L, side) != DPRC_SIDE_OUT) return l0 + 1;
  int32_t l = l0 + 1;
  while (l < num_layers && l - l0 < kMaxGroup && (int64_t)(l - l0 + 1) * k <= 256) {
    const dprc_layer& M = layers[l];
    if (M.A != L.A || M.lda != L.lda || M.d != L.d || M.B != L.B || M.T != L.T || M.dtype != L.dtype ||
        resolve(M, side) != DPRC_SIDE_OUT)
      break;
    ++l;
  }
  return l;
}

int64_t max_m(const View* v, int G) {
  int64_t m = 0;
  for (int l = 0; l < G; ++l) m = std::max(m, v[l].m);
  return m;
}

size_t hutch_group_ws(const View* v, int G, int32_t k, int probe) {
  Arena ar(nullptr);
  View vm = v[0];
  vm.m = max_m(v, G);
  if (probe == DPRC_PROBE_GAUSSIAN) take_gauss(ar, vm, k);
  if (v[0].dtype == DPRC_BF16) {
    pass_ws(ar, v[0].B, v[0].T, v[0].n, pad_cols(G * k), nullptr, nullptr, nullptr, G);
    return ar.off;
  }
  if (probe != DPRC_PROBE_GAUSSIAN) ar.take<uint32_t>((size_t)k * ceil_div(v[0].m, 32));
  ar.take<float>((size_t)v[0].B * v[0].T * k);
  ar.take<float>((size_t)v[0].B * k * v[0].n);
  return ar.off;
}

dprc_status hutch_f32(const View& v, int32_t k, int probe, uint32_t k0, uint32_t k1, float* n2,
                      float* n2_layer, int accumulate, void* ws, hipStream_t st) {
  const bool gauss = probe == DPRC_PROBE_GAUSSIAN;
  Arena ar(ws);
  GaussBufs g{};
  hipError_t e = hipSuccess;
  if (gauss) {
    g = take_gauss(ar, v, k);
    if ((e = traced(DPRC_KERNEL_PROBE_GAUSS, st, [&] {
           return launch_gauss_probe(k0, k1, v.layer_id, v.m, k, g.ld, nullptr, nullptr, g.f32, st); })) != hipSuccess)
      return DPRC_ERROR_HIP;
  }
  uint32_t* zb = gauss ? nullptr : ar.take<uint32_t>((size_t)k * ceil_div(v.m, 32));
  float* Y = ar.take<float>((size_t)v.B * v.T * k);
  float* M = ar.take<float>((size_t)v.B * k * v.n);
  if (!gauss && (e = traced(DPRC_KERNEL_PROBE_BITS, st, [&] { return launch_probe_bits(probe, k0, k1, v.layer_id, 0, v.m, k, zb, st); })) != hipSuccess)
    return DPRC_ERROR_HIP;
  ProjectF32Args pa = gauss
      ? ProjectF32Args{(const float*)v.X, v.ldx, v.T * v.ldx, (int32_t)v.B, (int32_t)v.T, (int32_t)v.m,
                       k, 0, k, g.f32, g.ld, 0, nullptr, Y}
      : ProjectF32Args{(const float*)v.X, v.ldx, v.T * v.ldx, (int32_t)v.B, (int32_t)v.T, (int32_t)v.m,
                       0, k, k, nullptr, 0, 0, zb, Y};
  if ((e = traced(DPRC_KERNEL_PROJECT_F32, st, [&] { return launch_project_f32(pa, st); })) != hipSuccess) return DPRC_ERROR_HIP;
  TokredF32Args ta{(const float*)v.Xo, v.ldo, v.T * v.ldo, (int32_t)v.B, (int32_t)v.T, (int32_t)v.n, Y, k,
                   M, v.n, (int64_t)k * v.n};
  if ((e = traced(DPRC_KERNEL_TOKEN_REDUCE_F32, st, [&] { return launch_tokred_f32(ta, st); })) != hipSuccess) return DPRC_ERROR_HIP;
  return hip_status(traced(DPRC_KERNEL_SAMPLE_SQ, st, [&] { return launch_sample_sq(M, v.n, (int64_t)k * v.n, (int32_t)v.B, k, (int32_t)v.n,
                                     1.0f / (float)k, n2, n2_layer, accumulate, st); }));
}

// G layers (G = 1, or a shared-activation group of bf16 OUT layers): one projection
// per layer into its columns of a shared Y, then one token reduction.
// With `defer` (bf16 layers), the split sums and the estimate are not launched: the
// token-reduction arguments are returned for a batched launch, and the group's token-split
// partials and tile sums go to `own` instead of the scratch.
dprc_status hutch_group(const View* v, int G, int32_t k, int probe, uint32_t k0, uint32_t k1, float* n2,
                        float* n2_layers, int accumulate, void* ws, hipStream_t st, float clipC = 0.f,
                        float* clip_c = nullptr, TokredArgs* defer = nullptr, const TokBufs* own = nullptr,
                        ProjectArgs* pjobs = nullptr, int* npj = nullptr) {
  if (v[0].dtype != DPRC_BF16) {
    dprc_status s = hutch_f32(v[0], k, probe, k0, k1, n2, n2_layers, accumulate, ws, st);
    if (s != DPRC_SUCCESS || !clip_c) return s;
    return hip_status(traced(DPRC_KERNEL_CLIP_SCALE, st, [&] { return launch_clip_scale(n2, v[0].B, clipC, clip_c, st); }));
  }
  const bool gauss = probe == DPRC_PROBE_GAUSSIAN;
  const int64_t B = v[0].B, T = v[0].T;
  Arena ar(ws);
  View vm = v[0];
  vm.m = max_m(v, G);
  GaussBufs gz = gauss ? take_gauss(ar, vm, k) : GaussBufs{};
  const int ncols = G * k, ncols_pad = pad_cols(ncols);
  uint16_t* Yt;
  TokBufs tb;
  TokPlan tp;
  pass_ws(ar, B, T, v[0].n, ncols_pad, &Yt, &tb, &tp, G);
  if (own && own->Y) Yt = own->Y;
  const int64_t yt_ld = B * tp.T_pad;
  hipError_t e = hipSuccess;
  for (int l = 0; l < G; ++l) {
    const View& w = v[l];
    const int64_t ldz = round_up(w.m, kTile);
    if (gauss && (e = traced(DPRC_KERNEL_PROBE_GAUSS, st, [&] {
                    return launch_gauss_probe(k0, k1, w.layer_id, w.m, k, ldz, gz.hi, gz.lo, nullptr, st); })) != hipSuccess)
      return DPRC_ERROR_HIP;
    ProjectArgs pa;
    pa.X = (const uint16_t*)w.X; pa.ldx = w.ldx; pa.x_ss = T * w.ldx;
    pa.B = (int32_t)B; pa.T = (int32_t)T; pa.m = (int32_t)w.m; pa.T_pad = tp.T_pad;
    pa.nd = gauss ? k : 0; pa.nz = gauss ? 0 : k; pa.ncols_pad = pad_cols(k);
    pa.Rhi = gz.hi; pa.Rlo = gz.lo; pa.ld_r = gauss ? ldz : 0; pa.r_ss = 0;
    pa.probe_kind = probe; pa.key0 = k0; pa.key1 = k1; pa.layer_id = w.layer_id; pa.stream_id = 0;
    pa.z_split = pa.nz; pa.stream_id2 = 0;
    pa.words_per_chunk = words_per_chunk(w.m, pa.nz);
    pa.Yt = Yt + (int64_t)l * k * yt_ld; pa.yt_ld = yt_ld;
    pa.ylo_off = (int64_t)ncols_pad * yt_ld;
    pa.ncols_write = G == 1 ? pa.ncols_pad : k;   // inside a shared Y only the layer's own columns
    pa.zero_ptr = nullptr; pa.zero_count = 0;
    pa.vec = rows16(w.X, w.ldx);
    if (pjobs) {                                   // collected: the caller launches them in batches
      pjobs[(*npj)++] = pa;
      continue;
    }
    if ((e = traced(DPRC_KERNEL_PROJECT, st, [&] { return launch_project(pa, rows_per_wg(B * tp.T_pad, pa.ncols_pad, pa.nd > 0), st); })) != hipSuccess)
      return DPRC_ERROR_HIP;
  }
  TokredArgs ta{};
  ta.X = (const uint16_t*)v[0].Xo; ta.ldx = v[0].ldo; ta.x_ss = T * v[0].ldo;
  ta.B = (int32_t)B; ta.T = (int32_t)T; ta.n = (int32_t)v[0].n;
  ta.Yt = Yt; ta.yt_ld = yt_ld; ta.T_pad = tp.T_pad; ta.ncols = ncols; ta.ncols_pad = ncols_pad;
  ta.ntiles = tp.ntiles; ta.S = tp.S; ta.stages_per_split = tp.sps;
  ta.mode = 0; ta.seg = k; ta.nseg = G;
  ta.part = tb.part; ta.tilesq = tb.tilesq;
  ta.scale = 1.0f / (float)k; ta.n2 = n2; ta.n2_layer = n2_layers; ta.accumulate = accumulate;
  ta.clip_C = clipC; ta.clip_c = clip_c;
  ta.vec = rows16(v[0].Xo, v[0].ldo);
  if (own) {
    ta.part = own->part;
    ta.tilesq = own->tilesq;
  }
  if (pjobs) {
    *defer = ta;
    return DPRC_SUCCESS;
  }
  if ((e = traced(DPRC_KERNEL_TOKEN_REDUCE, st, [&] { return launch_tokred(ta, st); })) != hipSuccess) return DPRC_ERROR_HIP;
  if (defer) {
    *defer = ta;
    return DPRC_SUCCESS;
  }
  if (tp.S > 1 && (e = traced(DPRC_KERNEL_TOKEN_SPLITS, st, [&] { return launch_tokred_splits(ta, st); })) != hipSuccess)
    return DPRC_ERROR_HIP;
  return hip_status(traced(DPRC_KERNEL_SAMPLE_SUM, st, [&] { return launch_tokred_sample(ta, st); }));
}

// ---- Hutch++ -------------------------------------------------------------------------------------
struct PPBufs {
  uint16_t *WShi, *WSlo; int64_t ld_ws;   // pass-1 result, dense operand of pass 2 (bf16)
  float* WS32;                             // same, fp32 path
  float* OS;                               // [B][s][m]
  QrArgs qr;                               // QR scratch (s > 0)
  FinalArgs fin;                           // finalize scratch (s > 0)
  float* Q;                                // [B][s][m]
  uint16_t *Qhi, *Qlo; int64_t ld_q;       // bf16 path
  float* UW;                               // [B][s+r][n]
  uint32_t* zb;                            // fp32 path: probe bits (s or r columns)
  float* Y32;                              // fp32 path
  void* pass_ws;                           // bf16 path: scratch of one pass
  float* part;                             // grouped layers: the layer's own token-split partials
  uint16_t* Y;                             // grouped layers: the layer's own Y (batched passes)
};

// Bytes of the bf16 pass scratch of one layer (the Y buffer and token-split partials).
size_t hpp_pass_bytes(const View& v, int32_t s, int32_t r) {
  size_t need = std::max(pass_ws_bytes(v.B, v.T, v.n, std::max(s, 1)), pass_ws_bytes(v.B, v.T, v.m, std::max(s, 1)));
  return std::max(need, pass_ws_bytes(v.B, v.T, v.n, s + r));
}

// Buffers of one layer carved from ws.  With own_pass false the bf16 pass scratch is
// not reserved (layers of one call then share one, given by the caller).
size_t hutchpp_layout(const View& v, int32_t s, int32_t r, void* ws, PPBufs* out, bool own_pass = true) {
  Arena ar(ws);
  PPBufs b{};
  const int64_t B = v.B;
  if (s > 0) {
    if (v.dtype == DPRC_BF16) {
      b.ld_ws = ceil_div(v.n, kTile) * kTile;
      b.WShi = ar.take<uint16_t>((size_t)B * s * b.ld_ws);
      b.WSlo = ar.take<uint16_t>((size_t)B * s * b.ld_ws);
      b.ld_q = ceil_div(v.m, kTile) * kTile;
      b.Qhi = ar.take<uint16_t>((size_t)B * s * b.ld_q);
      b.Qlo = ar.take<uint16_t>((size_t)B * s * b.ld_q);
    } else {
      b.WS32 = ar.take<float>((size_t)B * s * v.n);
    }
    b.OS = ar.take<float>((size_t)B * s * v.m);
    b.Q = ar.take<float>((size_t)B * s * v.m);
    b.UW = ar.take<float>((size_t)B * (s + r) * v.n);
    int32_t rows[kQrMaxLevels], nblk[kQrMaxLevels];
    int64_t dbl = 0;
    const int32_t nlev = qr_levels(v.m, s, rows, nblk, &dbl);
    b.qr.B = (int32_t)B; b.qr.m = (int32_t)v.m; b.qr.s = s; b.qr.r = r; b.qr.nlev = nlev;
    for (int l = 0; l < nlev; ++l) {
      QrLevel& L = b.qr.lev[l];
      L.rows = rows[l]; L.nblk = nblk[l];
      L.V = ar.take<double>((size_t)B * nblk[l] * s * kQrRows);
      L.tau = ar.take<double>((size_t)B * nblk[l] * s);
      L.M = l > 0 ? ar.take<double>((size_t)B * s * rows[l]) : nullptr;
      L.Q = l > 0 ? ar.take<double>((size_t)B * s * rows[l]) : nullptr;
    }
    b.qr.Cpart = ar.take<double>((size_t)B * (nlev > 0 ? nblk[0] : 1) * s * r);
    b.fin.nchunk = final_chunks(v.n);
    b.fin.Fpart = ar.take<double>((size_t)B * b.fin.nchunk * 2);
    b.fin.C = ar.take<double>((size_t)B * s * r);
  }
  if (v.dtype == DPRC_BF16) {
    if (own_pass) {
      b.pass_ws = ar.base ? ar.base + ((ar.off + kAlign - 1) / kAlign) * kAlign : nullptr;
      ar.off = (ar.off + kAlign - 1) / kAlign * kAlign;
      ar.off += hpp_pass_bytes(v, s, r);
    }
  } else {
    b.zb = ar.take<uint32_t>((size_t)std::max(s, r) * ceil_div(std::max(v.m, v.n), 32));
    b.Y32 = ar.take<float>((size_t)B * v.T * (s + r));
    if (s == 0) b.UW = ar.take<float>((size_t)B * r * v.n);
  }
  if (out) *out = b;
  return ar.off;
}

// The QR job of one layer at one tree level.
QrJob qr_job(const PPBufs& b, const View& v, int level, uint32_t k0, uint32_t k1, bool bf16_out) {
  const QrArgs& q = b.qr;
  QrJob j{};
  j.level = level; j.nlev = q.nlev;
  j.B = q.B; j.m = q.m; j.s = q.s; j.r = q.r;
  j.L = q.lev[level];
  j.X = level + 1 < q.nlev ? q.lev[level + 1] : QrLevel{};
  j.OS = b.OS; j.os_ld = v.m; j.os_ss = (int64_t)q.s * v.m;
  j.Cpart = q.Cpart;
  j.key0 = k0; j.key1 = k1; j.layer = v.layer_id;
  j.Q = b.Q; j.q_ld = v.m; j.q_ss = (int64_t)q.s * v.m;
  j.Qhi = bf16_out ? b.Qhi : nullptr; j.Qlo = bf16_out ? b.Qlo : nullptr;
  j.qh_ld = bf16_out ? b.ld_q : 0; j.qh_ss = (int64_t)q.s * j.qh_ld;
  return j;
}

// Q = orth(O S) of n layers (TSQR trees: factor launches up, expansion launches down),
// with C = Q^T P formed alongside by each layer's last expansion.  The layers' trees are
// independent, so one launch takes a level of up to kQrMaxJobs layers: the whole step
// costs (levels of the tallest tree) x 2 launches instead of that many per layer.
dprc_status run_qr(PPBufs* const* bs, const View* vs, int n, uint32_t k0, uint32_t k1, bool bf16_out,
                   hipStream_t st) {
  int maxlev = 0;
  for (int l = 0; l < n; ++l) {
    if (bs[l]->qr.nlev < 1) return DPRC_ERROR_NOT_SUPPORTED;
    maxlev = std::max(maxlev, (int)bs[l]->qr.nlev);
  }
  for (int pass = 0; pass < 2; ++pass) {              // 0: factor levels bottom-up, 1: expansions top-down
    for (int e = 0; e < maxlev; ++e) {
      QrBatch bt{};
      bt.s = bs[0]->qr.s; bt.r = bs[0]->qr.r;
      auto flush = [&]() -> bool {
        if (bt.njobs == 0) return true;
        const int kind = pass == 1 ? DPRC_KERNEL_QR_EXPAND : (e == 0 ? DPRC_KERNEL_QR : DPRC_KERNEL_QR_COMBINE);
        const hipError_t h = traced(kind, st, [&] {
          return pass == 0 ? launch_qr_factor(bt, st) : launch_qr_expand(bt, st); });
        bt.njobs = 0; bt.blocks = 0;
        return h == hipSuccess;
      };
      for (int l = 0; l < n; ++l) {
        const int nlev = bs[l]->qr.nlev;
        if (e >= nlev) continue;
        const int level = pass == 0 ? e : nlev - 1 - e;
        QrJob j = qr_job(*bs[l], vs[l], level, k0, k1, bf16_out);
        j.blk0 = bt.blocks;
        bt.job[bt.njobs++] = j;
        bt.blocks += j.L.nblk * j.B;
        if (bt.njobs == kQrMaxJobs && !flush()) return DPRC_ERROR_HIP;
      }
      if (!flush()) return DPRC_ERROR_HIP;
    }
  }
  return DPRC_SUCCESS;
}

dprc_status hpp_pass(int which, const View& v, int32_t s, int32_t r, uint32_t k0, uint32_t k1, const PPBufs& b,
                     hipStream_t st, TokredArgs* defer);
dprc_status hutchpp_f32(const View& v, int32_t s, int32_t r, uint32_t k0, uint32_t k1, PPBufs& b, float* n2,
                        float* n2_layer, int accumulate, hipStream_t st);
dprc_status hpp_final(const View& v, int32_t s, int32_t r, const PPBufs& b, float* n2, float* n2_layer,
                      int accumulate, hipStream_t st);

// One layer on its own: passes 1 and 2, its QR, pass 3 and the estimate.
dprc_status hutchpp_layer(const View& v, int32_t s, int32_t r, uint32_t k0, uint32_t k1, float* n2,
                          float* n2_layer, int accumulate, void* ws, hipStream_t st) {
  PPBufs b;
  hutchpp_layout(v, s, r, ws, &b);
  const int64_t B = v.B, T = v.T;
  if (v.dtype == DPRC_BF16) {
    const uint16_t* X = (const uint16_t*)v.X;
    const uint16_t* Xo = (const uint16_t*)v.Xo;
    if (s == 0) {  // Hutchinson with the r residual probes
      PassSpec ps{};
      ps.X = X; ps.ldx = v.ldx; ps.m = v.m; ps.Xo = Xo; ps.ldo = v.ldo; ps.n = v.n;
      ps.nz = r; ps.stream_id = 0; ps.probe_kind = 0;
      ps.mode = 0; ps.scale = 1.0f / (float)r; ps.n2 = n2; ps.n2_layer = n2_layer; ps.accumulate = accumulate;
      return run_pass(ps, B, T, k0, k1, v.layer_id, b.pass_ws, st);
    }
    dprc_status stt;
    if ((stt = hpp_pass(1, v, s, r, k0, k1, b, st, nullptr)) != DPRC_SUCCESS) return stt;
    if ((stt = hpp_pass(2, v, s, r, k0, k1, b, st, nullptr)) != DPRC_SUCCESS) return stt;
    PPBufs* bp = &b;
    if ((stt = run_qr(&bp, &v, 1, k0, k1, true, st)) != DPRC_SUCCESS) return stt;
    if ((stt = hpp_pass(3, v, s, r, k0, k1, b, st, nullptr)) != DPRC_SUCCESS) return stt;
    return hpp_final(v, s, r, b, n2, n2_layer, accumulate, st);
  } else {
    return hutchpp_f32(v, s, r, k0, k1, b, n2, n2_layer, accumulate, st);
  }
}

// Hutch++ pass `which` of a bf16 layer:
//   1: [W_S | W_P] = Xo^T (X [S | P]);  2: O S = X^T (Xo W_S);  3: U = Xo^T (X Q).
// The residual probes P do not depend on Q, so they ride along with the sketch S in
// pass 1 (W_S goes to the bf16 operand of pass 2, W_P to its columns of [U | W_P]);
// pass 3 then projects Q alone.  Each column's arithmetic is what it would be in pass 3.
PassSpec hpp_spec(int which, const View& v, int32_t s, int32_t r, const PPBufs& b) {
  const uint16_t* X = (const uint16_t*)v.X;
  const uint16_t* Xo = (const uint16_t*)v.Xo;
  PassSpec p{};
  if (which == 2) {
    p.X = Xo; p.ldx = v.ldo; p.m = v.n; p.Xo = X; p.ldo = v.ldx; p.n = v.m;
    p.nd = s; p.Rhi = b.WShi; p.Rlo = b.WSlo; p.ld_r = b.ld_ws;
    p.mode = 1; p.M = b.OS; p.m_ld = v.m;
  } else {
    p.X = X; p.ldx = v.ldx; p.m = v.m; p.Xo = Xo; p.ldo = v.ldo; p.n = v.n;
    p.mode = 1; p.probe_kind = 0;
    p.M = b.UW; p.m_ld = v.n; p.m_ss = (int64_t)(s + r) * v.n;     // [U | W_P], [B][s + r][n]
    if (which == 1) {
      p.nz = s + r; p.stream_id = 1; p.z_split = s; p.stream_id2 = 0;
      p.Mhi = b.WShi; p.Mlo = b.WSlo; p.mh_ld = b.ld_ws; p.mh_ncols = s; p.mh_ss = (int64_t)s * b.ld_ws;
      p.m_col0 = s;
    } else {
      p.nd = s; p.Rhi = b.Qhi; p.Rlo = b.Qlo; p.ld_r = b.ld_q;
    }
  }
  return p;
}

dprc_status hpp_pass(int which, const View& v, int32_t s, int32_t r, uint32_t k0, uint32_t k1, const PPBufs& b,
                     hipStream_t st, TokredArgs* defer = nullptr) {
  return run_pass(hpp_spec(which, v, s, r, b), v.B, v.T, k0, k1, v.layer_id, b.pass_ws, st, b.part, defer);
}

// Pass `which` of a group of layers: one projection launch and one token-reduction launch
// for all of them (each layer has its own Y and partials), the split sums deferred to the
// caller.  Passes wider than 64 columns take a launch pair per layer.
dprc_status hpp_pass_group(int which, const View* vs, PPBufs* bufs, int ng, int32_t s, int32_t r, uint32_t k0,
                           uint32_t k1, hipStream_t st, TokredArgs* def) {
  const PassSpec p0 = hpp_spec(which, vs[0], s, r, bufs[0]);
  const int ncols_pad = pad_cols(p0.nd + p0.nz);
  if (ncols_pad > 64 || ng > kProjMaxJobs || !bufs[0].Y) {
    for (int q = 0; q < ng; ++q) {
      const dprc_status stt = hpp_pass(which, vs[q], s, r, k0, k1, bufs[q], st, &def[q]);
      if (stt != DPRC_SUCCESS) return stt;
    }
    return DPRC_SUCCESS;
  }
  ProjectArgs pas[kProjMaxJobs];
  int64_t rows = 0;
  for (int q = 0; q < ng; ++q) {
    const PassSpec p = hpp_spec(which, vs[q], s, r, bufs[q]);
    const TokPlan tp = tok_plan(vs[q].B, vs[q].T, p.n);
    TokBufs own{tp.S > 1 ? bufs[q].part : nullptr, nullptr};
    pass_args(p, vs[q].B, vs[q].T, k0, k1, vs[q].layer_id, bufs[q].Y, own, tp, pas[q], def[q]);
    rows = vs[q].B * tp.T_pad;
  }
  // widest layers first, so that the narrow ones fill the tail of each launch
  int op[kProjMaxJobs], ot[kProjMaxJobs];
  for (int q = 0; q < ng; ++q) op[q] = ot[q] = q;
  std::stable_sort(op, op + ng, [&](int a, int b) { return pas[a].m > pas[b].m; });
  std::stable_sort(ot, ot + ng, [&](int a, int b) { return def[a].n > def[b].n; });
  ProjectBatch pb{};
  TokredBatch tb{};
  for (int q = 0; q < ng; ++q) {
    pb.job[pb.njobs++] = pas[op[q]];
    tb.job[tb.njobs++] = def[ot[q]];
  }
  const int rpw = rows_per_wg(rows, ncols_pad, p0.nd > 0);
  if (traced(DPRC_KERNEL_PROJECT, st, [&] { return launch_project_batch(pb, rpw, st); }) != hipSuccess ||
      traced(DPRC_KERNEL_TOKEN_REDUCE, st, [&] { return launch_tokred_batch(tb, st); }) != hipSuccess)
    return DPRC_ERROR_HIP;
  return DPRC_SUCCESS;
}

// The fp32 Hutch++ path (the tiny workload): SIMT passes, the same QR and finalize.
dprc_status hutchpp_f32(const View& v, int32_t s, int32_t r, uint32_t k0, uint32_t k1, PPBufs& b, float* n2,
                        float* n2_layer, int accumulate, hipStream_t st) {
  const int64_t B = v.B, T = v.T;
  hipError_t e;
  {
    const float* X = (const float*)v.X;
    const float* Xo = (const float*)v.Xo;
    if (s > 0) {
      if ((e = traced(DPRC_KERNEL_PROBE_BITS, st, [&] { return launch_probe_bits(0, k0, k1, v.layer_id, 1, v.m, s, b.zb, st); })) != hipSuccess) return DPRC_ERROR_HIP;
      ProjectF32Args a1{X, v.ldx, T * v.ldx, (int32_t)B, (int32_t)T, (int32_t)v.m, 0, s, s, nullptr, 0, 0, b.zb, b.Y32};
      if ((e = traced(DPRC_KERNEL_PROJECT_F32, st, [&] { return launch_project_f32(a1, st); })) != hipSuccess) return DPRC_ERROR_HIP;
      TokredF32Args t1{Xo, v.ldo, T * v.ldo, (int32_t)B, (int32_t)T, (int32_t)v.n, b.Y32, s, b.WS32, v.n, (int64_t)s * v.n};
      if ((e = traced(DPRC_KERNEL_TOKEN_REDUCE_F32, st, [&] { return launch_tokred_f32(t1, st); })) != hipSuccess) return DPRC_ERROR_HIP;
      ProjectF32Args a2{Xo, v.ldo, T * v.ldo, (int32_t)B, (int32_t)T, (int32_t)v.n, s, 0, s, b.WS32, v.n,
                        (int64_t)s * v.n, nullptr, b.Y32};
      if ((e = traced(DPRC_KERNEL_PROJECT_F32, st, [&] { return launch_project_f32(a2, st); })) != hipSuccess) return DPRC_ERROR_HIP;
      TokredF32Args t2{X, v.ldx, T * v.ldx, (int32_t)B, (int32_t)T, (int32_t)v.m, b.Y32, s, b.OS, v.m, (int64_t)s * v.m};
      if ((e = traced(DPRC_KERNEL_TOKEN_REDUCE_F32, st, [&] { return launch_tokred_f32(t2, st); })) != hipSuccess) return DPRC_ERROR_HIP;
      PPBufs* bp = &b;
      const dprc_status sq = run_qr(&bp, &v, 1, k0, k1, false, st);
      if (sq != DPRC_SUCCESS) return sq;
    }
    if ((e = traced(DPRC_KERNEL_PROBE_BITS, st, [&] { return launch_probe_bits(0, k0, k1, v.layer_id, 0, v.m, r, b.zb, st); })) != hipSuccess) return DPRC_ERROR_HIP;
    ProjectF32Args a3{X, v.ldx, T * v.ldx, (int32_t)B, (int32_t)T, (int32_t)v.m, s, r, s + r, b.Q, v.m,
                      (int64_t)s * v.m, b.zb, b.Y32};
    if ((e = traced(DPRC_KERNEL_PROJECT_F32, st, [&] { return launch_project_f32(a3, st); })) != hipSuccess) return DPRC_ERROR_HIP;
    TokredF32Args t3{Xo, v.ldo, T * v.ldo, (int32_t)B, (int32_t)T, (int32_t)v.n, b.Y32, s + r, b.UW, v.n,
                     (int64_t)(s + r) * v.n};
    if ((e = traced(DPRC_KERNEL_TOKEN_REDUCE_F32, st, [&] { return launch_tokred_f32(t3, st); })) != hipSuccess) return DPRC_ERROR_HIP;
    if (s == 0)
      return hip_status(traced(DPRC_KERNEL_SAMPLE_SQ, st, [&] { return launch_sample_sq(b.UW, v.n, (int64_t)r * v.n, (int32_t)B, r, (int32_t)v.n,
                                         1.0f / (float)r, n2, n2_layer, accumulate, st); }));
  }
  return hpp_final(v, s, r, b, n2, n2_layer, accumulate, st);
}

// C = sum of the block partials of Q^T P, the row pass, and the per-sample estimate.
FinalArgs final_args(const View& v, int32_t s, int32_t r, const PPBufs& b, float* n2, float* n2_layer,
                     int accumulate) {
  FinalArgs fa = b.fin;
  fa.UW = b.UW; fa.uw_ld = v.n; fa.uw_ss = (int64_t)(s + r) * v.n;
  fa.B = (int32_t)v.B; fa.n = (int32_t)v.n; fa.s = s; fa.r = r; fa.nblk = b.qr.nlev > 0 ? b.qr.lev[0].nblk : 0;
  fa.Cpart = b.qr.Cpart; fa.n2 = n2; fa.n2_layer = n2_layer; fa.accumulate = accumulate;
  return fa;
}

dprc_status hpp_final(const View& v, int32_t s, int32_t r, const PPBufs& b, float* n2, float* n2_layer,
                      int accumulate, hipStream_t st) {
  hipError_t e;
  const FinalArgs fa = final_args(v, s, r, b, n2, n2_layer, accumulate);
  if ((e = traced(DPRC_KERNEL_QR_EXPAND, st, [&] { return launch_hpp_csum(fa, st); })) != hipSuccess)
    return DPRC_ERROR_HIP;
  if ((e = traced(DPRC_KERNEL_HUTCHPP_FINAL, st, [&] { return launch_hpp_rows(fa, st); })) != hipSuccess)
    return DPRC_ERROR_HIP;
  return hip_status(traced(DPRC_KERNEL_HUTCHPP_SUM, st, [&] { return launch_hpp_sum(fa, st); }));
}

// ---- clipped accumulation ----------------------------------------------------------------------------
GemmPlan gemm_plan(const dprc_layer& L) { return gemm_plan_v2(L.B, L.T, L.d, L.p); }

// n-point Gauss-Legendre nodes and weights on [-1, 1]: Newton iteration on the
// roots of P_n, started from the Chebyshev-like guesses cos(pi (q + 3/4) / (n + 1/2)),
// with P_n and P_n' from the three-term recurrence; w = 2 / ((1 - x^2) P_n'(x)^2).
void gauss_legendre(int n, double* x, double* w) {
  for (int q = 0; q < (n + 1) / 2; ++q) {
    double z = std::cos(M_PI * (q + 0.75) / (n + 0.5)), dp = 1.0;
    for (int it = 0; it < 100; ++it) {
      double p0 = 1.0, p1 = 0.0;
      for (int j = 1; j <= n; ++j) {
        const double p2 = p1;
        p1 = p0;
        p0 = ((2.0 * j - 1.0) * z * p1 - (j - 1.0) * p2) / j;
      }
      dp = n * (z * p0 - p1) / (z * z - 1.0);
      const double dz = p0 / dp;
      z -= dz;
      if (std::fabs(dz) < 1e-15) break;
    }
    x[q] = -z;
    x[n - 1 - q] = z;
    w[q] = w[n - 1 - q] = 2.0 / ((1.0 - z * z) * dp * dp);
  }
}

// Scratch of dprc_norm_hutch_clip_static: one array on every device the library runs
// on, held until the process ends.  In host code the name `scratch` is a host-side
// stand-in, not a device address: the address comes from hipGetSymbolAddress, taken
// once per device (with that device current) on the entry point's first call there,
// and only that pointer reaches kernels.  Nothing in it has to start at zero: every
// kernel of the Hutchinson path writes the scratch it later reads, as it does with a
// caller's uninitialised workspace.
static __device__ __align__(256) uint8_t scratch[DPRC_STATIC_SCRATCH_BYTES];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};

dprc_status static_scratch(hipStream_t stream, void** out) {
  int cur = -1;
  hipDevice_t sdev = -1;
  if (hipGetDevice(&cur) != hipSuccess || hipStreamGetDevice(stream, &sdev) != hipSuccess) return DPRC_ERROR_HIP;
  if (sdev != cur) return DPRC_ERROR_INVALID_VALUE;            // the stream's device must be current
  if (cur < 0 || cur >= kMaxDevices) return DPRC_ERROR_NOT_SUPPORTED;
  std::lock_guard<std::mutex> lk(g_scratch_mu);
  if (!g_scratch_ptr[cur]) {
    void* p = nullptr;
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) return DPRC_ERROR_HIP;
    if (!aligned(p, kAlign)) return DPRC_ERROR_HIP;
    g_scratch_ptr[cur] = p;
  }
  *out = g_scratch_ptr[cur];
  return DPRC_SUCCESS;
}

}  // namespace

namespace dprc {
LaunchEvents& next_launch_events() { return g_next_events; }
}  // namespace dprc

extern "C" {

const char* dprc_status_string(dprc_status s) {
  switch (s) {
    case DPRC_SUCCESS: return "DPRC_SUCCESS";
    case DPRC_ERROR_INVALID_VALUE: return "DPRC_ERROR_INVALID_VALUE: invalid argument";
    case DPRC_ERROR_NOT_SUPPORTED: return "DPRC_ERROR_NOT_SUPPORTED: unsupported alignment, stride or size";
    case DPRC_ERROR_WORKSPACE_TOO_SMALL: return "DPRC_ERROR_WORKSPACE_TOO_SMALL: workspace smaller than the query";
    case DPRC_ERROR_HIP: return "DPRC_ERROR_HIP: a HIP runtime call or kernel launch failed";
    case DPRC_ERROR_SCRATCH_LIMIT:
      return "DPRC_ERROR_SCRATCH_LIMIT: the call needs more scratch than the library's static buffer "
             "(DPRC_STATIC_SCRATCH_BYTES per device)";
  }
  return "unknown dprc_status";
}

const char* dprc_version(void) { return "dprc 0.1.0 (gfx950)"; }

dprc_status dprc_trace_launches(hipEvent_t* events, int32_t* kinds, int32_t capacity, int32_t* count) {
  if (events && (capacity < 0 || !count)) return DPRC_ERROR_INVALID_VALUE;
  g_trace.events = events;
  g_trace.kinds = kinds;
  g_trace.capacity = events ? capacity : 0;
  g_trace.count = events ? count : nullptr;
  if (count) *count = 0;
  return DPRC_SUCCESS;
}

// Calls whose layers are all bf16 finish up to kTokMaxJobs activation groups at once: the
// projections and token reductions of every group, then one split-sum launch.  Each group
// keeps its own token-split partials (the rest of the per-batch scratch is shared) and its
// tile sums, which stay until the end of the call: one launch there adds every layer's
// estimate to n2 in layer order and writes the clip factors.
bool hutch_batched(const dprc_layer* layers, int32_t n) {
  if (n < 2) return false;
  for (int32_t l = 0; l < n; ++l)
    if (layers[l].dtype != DPRC_BF16) return false;
  return true;
}

// The collected projections (widest first, up to kProjMaxJobs per launch) and token
// reductions (one launch per column count) of a batch of activation groups; work over
// more than 64 columns takes one launch per layer or group.
dprc_status hutch_launch_batched(ProjectArgs* pj, int npj, const TokredBatch& groups, hipStream_t st) {
  std::stable_sort(pj, pj + npj, [](const ProjectArgs& a, const ProjectArgs& b) { return a.m > b.m; });
  for (int c = 0; c < npj && pj[c].ncols_pad > 64; ++c)    // batched launches take up to 64 columns
    if (traced(DPRC_KERNEL_PROJECT, st, [&] {
          return launch_project(pj[c], rows_per_wg((int64_t)pj[c].B * pj[c].T_pad, pj[c].ncols_pad, false), st); }) !=
        hipSuccess)
      return DPRC_ERROR_HIP;
  for (int c = 0; c < npj && pj[0].ncols_pad <= 64; c += kProjMaxJobs) {
    ProjectBatch pb{};
    for (int q = c; q < std::min(npj, c + kProjMaxJobs); ++q) pb.job[pb.njobs++] = pj[q];
    const int rpw = rows_per_wg((int64_t)pb.job[0].B * pb.job[0].T_pad, pb.job[0].ncols_pad, false);
    if (traced(DPRC_KERNEL_PROJECT, st, [&] { return launch_project_batch(pb, rpw, st); }) != hipSuccess)
      return DPRC_ERROR_HIP;
  }
  TokredArgs tj[kTokMaxJobs];
  for (int q = 0; q < groups.njobs; ++q) tj[q] = groups.job[q];
  std::stable_sort(tj, tj + groups.njobs, [](const TokredArgs& a, const TokredArgs& b) {
    return a.ncols_pad != b.ncols_pad ? a.ncols_pad < b.ncols_pad : a.n > b.n; });
  for (int q = 0; q < groups.njobs;) {
    if (tj[q].ncols_pad > 64) {
      if (traced(DPRC_KERNEL_TOKEN_REDUCE, st, [&] { return launch_tokred(tj[q], st); }) != hipSuccess)
        return DPRC_ERROR_HIP;
      ++q;
      continue;
    }
    TokredBatch tb{};
    const int np = tj[q].ncols_pad;
    while (q < groups.njobs && tj[q].ncols_pad == np) tb.job[tb.njobs++] = tj[q++];
    if (traced(DPRC_KERNEL_TOKEN_REDUCE, st, [&] { return launch_tokred_batch(tb, st); }) != hipSuccess)
      return DPRC_ERROR_HIP;
  }
  return DPRC_SUCCESS;
}

// A batch whose token reductions have at least kUnsplitPairs (sample, tile) pairs fills the
// GPU without token splits: every job then runs unsplit (one workgroup per pair over all
// tokens, writing its tile sum directly), which halves the per-workgroup start and finish
// costs of two-way splits and drops the split-sum launch.  The batch layout reserves no
// split partials for such a batch.
constexpr int64_t kUnsplitPairs = 1024;
void unsplit_large_batch(TokredBatch& bt) {
  int64_t pairs = 0;
  for (int q = 0; q < bt.njobs; ++q) pairs += (int64_t)bt.job[q].B * bt.job[q].ntiles;
  if (pairs < kUnsplitPairs) return;
  for (int q = 0; q < bt.njobs; ++q) {
    TokredArgs& a = bt.job[q];
    if (a.mode != 0) continue;
    a.stages_per_split = a.S * a.stages_per_split;
    a.S = 1;
    a.part = nullptr;
  }
}

// The tile sums of an activation group (layers l .. le - 1) of a batched call,
// [nseg][B][ntiles] doubles, kept until the per-sample sums at the end of the call: the
// bytes of its slice, and of all groups' slices in order.
size_t group_tilesq_bytes(const dprc_layer* layers, int32_t l, int32_t le, dprc_side side) {
  const View v0 = view_of(layers[l], side);
  const TokPlan tp = tok_plan(v0.B, v0.T, v0.n);
  return ((size_t)(le - l) * v0.B * tp.ntiles * sizeof(double) + kAlign - 1) / kAlign * kAlign;
}

size_t hutch_tilesq_bytes(const dprc_layer* layers, int32_t n, int32_t k, dprc_side side) {
  size_t off = 0;
  for (int32_t l = 0; l < n;) {
    const int32_t le = group_end(layers, l, n, k, side);
    off += group_tilesq_bytes(layers, l, le, side);
    l = le;
  }
  return off;
}

// Up to kTokMaxJobs consecutive activation groups starting at layer l0: their bounds in
// ends[], their own buffers (token-split partials and Y; the tile sums are the call's)
// carved from ws (own may be null) after the shared scratch.  Returns the bytes used.
size_t hutch_batch_layout(const dprc_layer* layers, int32_t l0, int32_t n, int32_t k, int probe, dprc_side side,
                          void* ws, int32_t* ends, int* ngroups, TokBufs* own) {
  View v[kMaxGroup];
  size_t shared = 0;
  int ng = 0;
  int32_t l = l0;
  while (l < n && ng < kTokMaxJobs) {
    const int32_t le = group_end(layers, l, n, k, side);
    for (int32_t j = l; j < le; ++j) v[j - l] = view_of(layers[j], side);
    shared = std::max(shared, hutch_group_ws(v, le - l, k, probe));
    ends[ng++] = le;
    l = le;
  }
  // a batch whose launches are batched and unsplit (unsplit_large_batch) needs no partials
  int64_t pairs = 0;
  for (int q = 0, lq = l0; q < ng; lq = ends[q++]) {
    const View v0 = view_of(layers[lq], side);
    pairs += v0.B * tok_plan(v0.B, v0.T, v0.n).ntiles;
  }
  const bool unsplit = probe != DPRC_PROBE_GAUSSIAN && pairs >= kUnsplitPairs;
  char* base = static_cast<char*>(ws);
  size_t off = (shared + kAlign - 1) / kAlign * kAlign;
  l = l0;
  for (int q = 0; q < ng; ++q) {
    const View v0 = view_of(layers[l], side);
    const int G = ends[q] - l;
    const TokPlan tp = tok_plan(v0.B, v0.T, v0.n);
    const size_t pf = !unsplit && tp.S > 1 ? (size_t)v0.B * tp.ntiles * tp.S * pad_cols(G * k) * kTile : 0;
    if (own) own[q].part = base && pf ? reinterpret_cast<float*>(base + off) : nullptr;
    off = (off + pf * sizeof(float) + kAlign - 1) / kAlign * kAlign;
    if (probe != DPRC_PROBE_GAUSSIAN) {          // its own Y: the groups' launches are batched
      if (own) own[q].Y = base ? reinterpret_cast<uint16_t*>(base + off) : nullptr;
      off = (off + (size_t)2 * pad_cols(G * k) * v0.B * tp.T_pad * sizeof(uint16_t) + kAlign - 1) / kAlign * kAlign;
    } else if (own) {
      own[q].Y = nullptr;
    }
    l = ends[q];
  }
  *ngroups = ng;
  return off;
}

size_t dprc_norm_hutch_workspace(const dprc_layer* layers, int32_t num_layers, int32_t k, dprc_probe probe,
                                 dprc_side side) {
  if (check_layers(layers, num_layers, side) != DPRC_SUCCESS || k < 1 || k > 256) return 0;
  if (probe != DPRC_PROBE_RADEMACHER && probe != DPRC_PROBE_HADAMARD && probe != DPRC_PROBE_GAUSSIAN) return 0;
  if (probe == DPRC_PROBE_GAUSSIAN && k > kMaxGaussK) return 0;
  size_t need = 0;
  View v[kMaxGroup];
  for (int32_t l = 0; l < num_layers;) {
    const int32_t le = group_end(layers, l, num_layers, k, side);
    for (int32_t j = l; j < le; ++j) v[j - l] = view_of(layers[j], side);
    need = std::max(need, hutch_group_ws(v, le - l, k, (int)probe));
    l = le;
  }
  if (hutch_batched(layers, num_layers)) {
    int32_t ends[kTokMaxJobs];
    int ng = 0;
    for (int32_t l = 0; l < num_layers;) {
      need = std::max(need, hutch_batch_layout(layers, l, num_layers, k, (int)probe, side, nullptr, ends, &ng, nullptr));
      l = ends[ng - 1];
    }
    need += hutch_tilesq_bytes(layers, num_layers, k, side);   // the call's tile sums come first
  }
  return need;
}

static dprc_status norm_hutch(const dprc_layer* layers, int32_t num_layers, int32_t k, dprc_probe probe,
                              uint64_t seed, dprc_side side, float* n2, float* n2_layers, int32_t accumulate,
                              void* ws, size_t ws_bytes, hipStream_t stream, float clipC, float* clip_c) {
  dprc_status s = check_layers(layers, num_layers, side);
  if (s != DPRC_SUCCESS) return s;
  if (k < 1 || k > 256 || !n2) return DPRC_ERROR_INVALID_VALUE;
  if (probe != DPRC_PROBE_RADEMACHER && probe != DPRC_PROBE_HADAMARD && probe != DPRC_PROBE_GAUSSIAN)
    return DPRC_ERROR_INVALID_VALUE;
  if (probe == DPRC_PROBE_GAUSSIAN && k > kMaxGaussK) return DPRC_ERROR_NOT_SUPPORTED;
  const size_t need = dprc_norm_hutch_workspace(layers, num_layers, k, probe, side);
  if (ws_bytes < need) return DPRC_ERROR_WORKSPACE_TOO_SMALL;
  if (!ws || !aligned(ws, kAlign)) return DPRC_ERROR_INVALID_VALUE;
  uint32_t k0, k1;
  key_of(seed, k0, k1);
  const int64_t B = layers[0].B;
  View v[kMaxGroup];
  if (hutch_batched(layers, num_layers)) {
    // every group's tile sums for the whole call at the front, then the batches' scratch;
    // the per-sample sums run once at the end over all groups (kSampleMaxGroups per launch)
    char* tq = static_cast<char*>(ws);
    ws = tq + hutch_tilesq_bytes(layers, num_layers, k, side);
    SampleSumArgs ss{};
    int launched = 0;
    auto flush = [&](bool last) -> dprc_status {
      if (ss.ngroups == 0) return DPRC_SUCCESS;
      ss.B = (int32_t)B;
      ss.n2 = n2;
      ss.accumulate = (accumulate || launched > 0) ? 1 : 0;
      ss.clip_C = clipC;
      ss.clip_c = last ? clip_c : nullptr;
      if (traced(DPRC_KERNEL_SAMPLE_SUM, stream, [&] { return launch_sample_sums(ss, stream); }) != hipSuccess)
        return DPRC_ERROR_HIP;
      ++launched;
      ss.ngroups = 0;
      return DPRC_SUCCESS;
    };
    for (int32_t l = 0; l < num_layers;) {
      int32_t ends[kTokMaxJobs];
      int ng = 0;
      TokBufs own[kTokMaxJobs];
      hutch_batch_layout(layers, l, num_layers, k, (int)probe, side, ws, ends, &ng, own);
      for (int q = 0, lq = l; q < ng; lq = ends[q++]) {
        own[q].tilesq = reinterpret_cast<double*>(tq);
        tq += group_tilesq_bytes(layers, lq, ends[q], side);
      }
      TokredBatch bt{};
      const bool batched = own[0].Y != nullptr;
      ProjectArgs pj[kTokMaxJobs * kMaxGroup];
      int npj = 0;
      for (int q = 0; q < ng; ++q) {
        const int32_t le = ends[q];
        for (int32_t j = l; j < le; ++j) v[j - l] = view_of(layers[j], side);
        TokredArgs ta{};
        s = hutch_group(v, le - l, k, (int)probe, k0, k1, n2, n2_layers ? n2_layers + (int64_t)l * B : nullptr,
                        (accumulate || l > 0) ? 1 : 0, ws, stream, 0.f, nullptr, &ta, &own[q],
                        batched ? pj : nullptr, batched ? &npj : nullptr);
        if (s != DPRC_SUCCESS) return s;
        bt.blk0[bt.njobs] = bt.blocks;
        bt.job[bt.njobs++] = ta;
        l = le;
      }
      if (batched) unsplit_large_batch(bt);       // (unbatched groups launched theirs already)
      if (batched && (s = hutch_launch_batched(pj, npj, bt, stream)) != DPRC_SUCCESS) return s;
      if ((s = run_splits_batch(bt.job, bt.njobs, stream)) != DPRC_SUCCESS) return s;
      for (int q = 0; q < bt.njobs; ++q) {
        if (ss.ngroups == kSampleMaxGroups && (s = flush(false)) != DPRC_SUCCESS) return s;
        const TokredArgs& a = bt.job[q];
        ss.scale = a.scale;                        // 1/k for every group of the call
        ss.g[ss.ngroups++] = SampleGroup{a.tilesq, a.n2_layer, a.ntiles, a.nseg};
      }
    }
    return flush(true);
  }
  for (int32_t l = 0; l < num_layers;) {
    const int32_t le = group_end(layers, l, num_layers, k, side);
    for (int32_t j = l; j < le; ++j) v[j - l] = view_of(layers[j], side);
    const bool last = le == num_layers;
    s = hutch_group(v, le - l, k, (int)probe, k0, k1, n2, n2_layers ? n2_layers + (int64_t)l * B : nullptr,
                    (accumulate || l > 0) ? 1 : 0, ws, stream, clipC, last ? clip_c : nullptr);
    if (s != DPRC_SUCCESS) return s;
    l = le;
  }
  return DPRC_SUCCESS;
}

dprc_status dprc_norm_hutch(const dprc_layer* layers, int32_t num_layers, int32_t k, dprc_probe probe,
                            uint64_t seed, dprc_side side, float* n2, float* n2_layers, int32_t accumulate,
                            void* ws, size_t ws_bytes, hipStream_t stream) {
  return norm_hutch(layers, num_layers, k, probe, seed, side, n2, n2_layers, accumulate, ws, ws_bytes, stream, 0.f,
                    nullptr);
}

dprc_status dprc_norm_hutch_clip(const dprc_layer* layers, int32_t num_layers, int32_t k, dprc_probe probe,
                                 uint64_t seed, dprc_side side, float C, float* n2, float* c, float* n2_layers,
                                 int32_t accumulate, void* ws, size_t ws_bytes, hipStream_t stream) {
  if (!c || !(C > 0.f) || std::isinf(C)) return DPRC_ERROR_INVALID_VALUE;
  return norm_hutch(layers, num_layers, k, probe, seed, side, n2, n2_layers, accumulate, ws, ws_bytes, stream, C, c);
}

dprc_status dprc_norm_hutch_clip_static(const dprc_layer* layers, int32_t num_layers, int32_t k, dprc_probe probe,
                                        uint64_t seed, dprc_side side, float C, float* n2, float* c,
                                        float* n2_layers, int32_t accumulate, hipStream_t stream) {
  if (!c || !(C > 0.f) || std::isinf(C)) return DPRC_ERROR_INVALID_VALUE;
  dprc_status s = check_layers(layers, num_layers, side);
  if (s != DPRC_SUCCESS) return s;
  const size_t need = dprc_norm_hutch_workspace(layers, num_layers, k, probe, side);
  if (need > (size_t)DPRC_STATIC_SCRATCH_BYTES) return DPRC_ERROR_SCRATCH_LIMIT;
  void* ws = nullptr;
  if ((s = static_scratch(stream, &ws)) != DPRC_SUCCESS) return s;
  return norm_hutch(layers, num_layers, k, probe, seed, side, n2, n2_layers, accumulate, ws,
                    (size_t)DPRC_STATIC_SCRATCH_BYTES, stream, C, c);
}

// Calls with several bf16 layers and a sketch run them in groups of up to kQrMaxJobs:
// passes 1 and 2 of every layer of the group, one batched QR per tree level, then pass 3
// and the estimate in layer order (so n2 adds the layers' estimates in the same order).
// Each layer of a group keeps its own buffers; the pass scratch is shared.
bool hpp_grouped(const dprc_layer* layers, int32_t n, int32_t s) {
  if (s <= 0 || n < 2) return false;
  for (int32_t l = 0; l < n; ++l)
    if (layers[l].dtype != DPRC_BF16) return false;
  return true;
}

// Buffers of layers [l0, l1) carved from ws (bufs may be null); returns the bytes used.
size_t hpp_group_layout(const dprc_layer* layers, int32_t l0, int32_t l1, int32_t s, int32_t r, dprc_side side,
                        void* ws, PPBufs* bufs) {
  char* base = static_cast<char*>(ws);
  size_t off = 0, pass = 0;
  for (int32_t l = l0; l < l1; ++l) {
    const View v = view_of(layers[l], side);
    off += hutchpp_layout(v, s, r, base ? base + off : nullptr, bufs ? &bufs[l - l0] : nullptr, false);
    off = (off + kAlign - 1) / kAlign * kAlign;
    // the layer's own token-split partials (its passes' split sums are launched for the group)
    const int64_t pf = std::max({part_floats(v.B, v.T, v.n, s), part_floats(v.B, v.T, v.m, s),
                                 part_floats(v.B, v.T, v.n, s + r)});
    if (bufs) bufs[l - l0].part = base && pf > 0 ? reinterpret_cast<float*>(base + off) : nullptr;
    off += (size_t)pf * sizeof(float);
    off = (off + kAlign - 1) / kAlign * kAlign;
    // and its own Y (the group's passes run as one projection launch and one reduction launch)
    const size_t ny = (size_t)2 * pad_cols(s + r) * v.B * round_up(v.T, kStage);
    if (bufs) bufs[l - l0].Y = base ? reinterpret_cast<uint16_t*>(base + off) : nullptr;
    off += ny * sizeof(uint16_t);
    off = (off + kAlign - 1) / kAlign * kAlign;
    pass = std::max(pass, hpp_pass_bytes(v, s, r));
  }
  if (bufs)
    for (int32_t l = l0; l < l1; ++l) bufs[l - l0].pass_ws = base ? base + off : nullptr;
  return off + pass;
}

size_t dprc_norm_hutchpp_workspace(const dprc_layer* layers, int32_t num_layers, int32_t s, int32_t r,
                                   dprc_side side) {
  if (check_layers(layers, num_layers, side) != DPRC_SUCCESS) return 0;
  if (s < 0 || s > 32 || r < 1 || r > 256 || s + r > 256) return 0;
  size_t need = 0;
  for (int32_t l = 0; l < num_layers; ++l) {
    const View v = view_of(layers[l], side);
    if (s > v.m) return 0;
    need = std::max(need, hutchpp_layout(v, s, r, nullptr, nullptr));
  }
  if (hpp_grouped(layers, num_layers, s))
    for (int32_t g0 = 0; g0 < num_layers; g0 += kQrMaxJobs)
      need = std::max(need, hpp_group_layout(layers, g0, std::min(num_layers, g0 + kQrMaxJobs), s, r, side,
                                             nullptr, nullptr));
  return need;
}

dprc_status dprc_norm_hutchpp(const dprc_layer* layers, int32_t num_layers, int32_t s, int32_t r, uint64_t seed,
                              dprc_side side, float* n2, float* n2_layers, int32_t accumulate, void* ws,
                              size_t ws_bytes, hipStream_t stream) {
  dprc_status st = check_layers(layers, num_layers, side);
  if (st != DPRC_SUCCESS) return st;
  if (s < 0 || s > 32 || r < 1 || r > 256 || s + r > 256 || !n2) return DPRC_ERROR_INVALID_VALUE;
  for (int32_t l = 0; l < num_layers; ++l) {
    const View v = view_of(layers[l], side);
    if (s > v.m) return DPRC_ERROR_INVALID_VALUE;
    int32_t rows[kQrMaxLevels], nblk[kQrMaxLevels];
    if (s > 0 && qr_levels(v.m, s, rows, nblk, nullptr) == 0) return DPRC_ERROR_NOT_SUPPORTED;
  }
  const size_t need = dprc_norm_hutchpp_workspace(layers, num_layers, s, r, side);
  if (ws_bytes < need) return DPRC_ERROR_WORKSPACE_TOO_SMALL;
  if (!ws || !aligned(ws, kAlign)) return DPRC_ERROR_INVALID_VALUE;
  uint32_t k0, k1;
  key_of(seed, k0, k1);
  const int64_t B = layers[0].B;
  if (hpp_grouped(layers, num_layers, s)) {
    for (int32_t g0 = 0; g0 < num_layers; g0 += kQrMaxJobs) {
      const int32_t g1 = std::min(num_layers, g0 + kQrMaxJobs), ng = g1 - g0;
      PPBufs bufs[kQrMaxJobs];
      View views[kQrMaxJobs];
      PPBufs* bp[kQrMaxJobs];
      hpp_group_layout(layers, g0, g1, s, r, side, ws, bufs);
      for (int32_t q = 0; q < ng; ++q) {
        views[q] = view_of(layers[g0 + q], side);
        bp[q] = &bufs[q];
      }
      TokredArgs def[kQrMaxJobs];
      // one pass of layers [q0, q1), followed by one split-sum launch for them
      auto pass = [&](int which, int q0, int q1) {
        dprc_status e = hpp_pass_group(which, views + q0, bufs + q0, q1 - q0, s, r, k0, k1, stream, def + q0);
        return e != DPRC_SUCCESS ? e : run_splits_batch(def + q0, q1 - q0, stream);
      };
      if ((st = pass(1, 0, ng)) != DPRC_SUCCESS || (st = pass(2, 0, ng)) != DPRC_SUCCESS) return st;
      if ((st = run_qr(bp, views, ng, k0, k1, true, stream)) != DPRC_SUCCESS) return st;
      if ((st = pass(3, 0, ng)) != DPRC_SUCCESS) return st;
      // the estimates, added to n2 in layer order
      FinalBatch fb{};
      for (int32_t q = 0; q < ng; ++q) {
        const int32_t l = g0 + q;
        fb.job[fb.njobs++] = final_args(views[q], s, r, bufs[q], n2, n2_layers ? n2_layers + (int64_t)l * B : nullptr,
                                        (accumulate || l > 0) ? 1 : 0);
      }
      if (traced(DPRC_KERNEL_QR_EXPAND, stream, [&] { return launch_hpp_csum_batch(fb, stream); }) != hipSuccess ||
          traced(DPRC_KERNEL_HUTCHPP_FINAL, stream, [&] { return launch_hpp_rows_batch(fb, stream); }) != hipSuccess ||
          traced(DPRC_KERNEL_HUTCHPP_SUM, stream, [&] { return launch_hpp_sum_batch(fb, stream); }) != hipSuccess)
        return DPRC_ERROR_HIP;
    }
    return DPRC_SUCCESS;
  }
  for (int32_t l = 0; l < num_layers; ++l) {
    st = hutchpp_layer(view_of(layers[l], side), s, r, k0, k1, n2, n2_layers ? n2_layers + (int64_t)l * B : nullptr,
                       (accumulate || l > 0) ? 1 : 0, ws, stream);
    if (st != DPRC_SUCCESS) return st;
  }
  return DPRC_SUCCESS;
}

dprc_status dprc_clip_scale(const float* n2, int64_t B, float C, float* c, hipStream_t stream) {
  if (!n2 || !c || B < 1 || !(C > 0.f) || std::isinf(C)) return DPRC_ERROR_INVALID_VALUE;
  return hip_status(traced(DPRC_KERNEL_CLIP_SCALE, stream, [&] { return launch_clip_scale(n2, B, C, c, stream); }));
}

size_t dprc_clip_accumulate_workspace(const dprc_layer* L) {
  if (!L || check_layer(*L) != DPRC_SUCCESS) return 0;
  if (L->dtype == DPRC_F32) return 0;
  const GemmPlan g = gemm_plan(*L);
  return g.S > 1 ? (size_t)g.S * L->d * L->p * sizeof(float) : 0;
}

dprc_status dprc_clip_accumulate(const dprc_layer* L, const float* c, float* grad, int64_t ldg, int32_t accumulate,
                                 void* ws, size_t ws_bytes, hipStream_t stream) {
  if (!L) return DPRC_ERROR_INVALID_VALUE;
  dprc_status s = check_layer(*L);
  if (s != DPRC_SUCCESS) return s;
  if (!c || !grad || ldg < L->p) return DPRC_ERROR_INVALID_VALUE;
  if (L->d * L->p > (1LL << 40)) return DPRC_ERROR_NOT_SUPPORTED;
  const size_t need = dprc_clip_accumulate_workspace(L);
  if (ws_bytes < need) return DPRC_ERROR_WORKSPACE_TOO_SMALL;
  if (need && (!ws || !aligned(ws, kAlign))) return DPRC_ERROR_INVALID_VALUE;
  if (L->dtype == DPRC_F32)
    return hip_status(traced(DPRC_KERNEL_ACCUMULATE_F32, stream, [&] { return launch_gemm_f32((const float*)L->A, L->lda, L->T * L->lda, (const float*)L->E, L->lde,
                                      L->T * L->lde, (int32_t)L->B, (int32_t)L->T, (int32_t)L->d, (int32_t)L->p, c,
                                      grad, ldg, accumulate, stream); }));
  const GemmPlan g = gemm_plan(*L);
  GemmArgs a;
  a.A = (const uint16_t*)L->A; a.lda = L->lda; a.a_ss = L->T * L->lda;
  a.E = (const uint16_t*)L->E; a.lde = L->lde; a.e_ss = L->T * L->lde;
  a.B = (int32_t)L->B; a.T = (int32_t)L->T; a.d = (int32_t)L->d; a.p = (int32_t)L->p;
  a.c = c; a.out = grad; a.ldo = ldg; a.accumulate = accumulate;
  a.S = g.S; a.stages_per_sample = g.sps; a.stages_per_split = g.spl;
  a.part = (float*)ws;
  a.vec_a = rows16(L->A, L->lda);
  a.vec_e = rows16(L->E, L->lde);
  hipError_t e = traced(DPRC_KERNEL_ACCUMULATE, stream, [&] { return launch_gemm(a, stream); });
  if (e != hipSuccess) return DPRC_ERROR_HIP;
  if (g.S > 1) return hip_status(traced(DPRC_KERNEL_SPLITK_REDUCE, stream, [&] { return launch_splitk_reduce(a.part, g.S, a.d, a.p, grad, ldg, accumulate, stream); }));
  return DPRC_SUCCESS;
}

dprc_status dprc_clip_accumulate_layers(const dprc_layer* layers, int32_t num_layers, const float* c,
                                        float* const* grads, const int64_t* ldg, int32_t accumulate,
                                        hipStream_t stream) {
  if (num_layers < 0 || (num_layers > 0 && (!layers || !grads || !ldg || !c))) return DPRC_ERROR_INVALID_VALUE;
  for (int32_t l = 0; l < num_layers; ++l) {
    const dprc_layer& L = layers[l];
    const dprc_status s = check_layer(L);
    if (s != DPRC_SUCCESS) return s;
    if (L.B != layers[0].B || !grads[l] || ldg[l] < L.p) return DPRC_ERROR_INVALID_VALUE;
    if (L.dtype != DPRC_BF16 || L.d * L.p > (1LL << 40)) return DPRC_ERROR_NOT_SUPPORTED;
  }
  auto args_of = [&](int32_t l) {
    const dprc_layer& L = layers[l];
    const GemmPlan g = gemm_plan(L);
    GemmArgs a;
    a.A = (const uint16_t*)L.A; a.lda = L.lda; a.a_ss = L.T * L.lda;
    a.E = (const uint16_t*)L.E; a.lde = L.lde; a.e_ss = L.T * L.lde;
    a.B = (int32_t)L.B; a.T = (int32_t)L.T; a.d = (int32_t)L.d; a.p = (int32_t)L.p;
    a.c = c; a.out = grads[l]; a.ldo = ldg[l]; a.accumulate = accumulate;
    a.S = 1; a.stages_per_sample = g.sps; a.stages_per_split = (int32_t)(L.B * g.sps);
    a.part = nullptr;
    a.vec_a = rows16(L.A, L.lda);
    a.vec_e = rows16(L.E, L.lde);
    return a;
  };
  // A layer with a whole round of tiles (one per CU) runs in a launch of its own, all its
  // tiles in step through the tokens (they share operand slabs in L2); the smaller ones
  // share launches, up to kGemmMaxJobs at a time, instead of splitting over tokens.
  GemmBatch bt{};
  auto flush = [&]() -> dprc_status {
    if (bt.njobs == 0) return DPRC_SUCCESS;
    std::stable_sort(bt.job, bt.job + bt.njobs, [](const GemmArgs& x, const GemmArgs& y) {
      return ceil_div(x.d, 256) * ceil_div(x.p, 256) > ceil_div(y.d, 256) * ceil_div(y.p, 256); });
    const hipError_t e = traced(DPRC_KERNEL_ACCUMULATE, stream, [&] { return launch_gemm_batch(bt, stream); });
    bt.njobs = 0;
    return e == hipSuccess ? DPRC_SUCCESS : DPRC_ERROR_HIP;
  };
  for (int32_t l = 0; l < num_layers; ++l) {
    const GemmArgs a = args_of(l);
    if (ceil_div(a.d, 256) * ceil_div(a.p, 256) >= kGemmRoundTiles) {
      if (traced(DPRC_KERNEL_ACCUMULATE, stream, [&] { return launch_gemm(a, stream); }) != hipSuccess)
        return DPRC_ERROR_HIP;
      continue;
    }
    bt.job[bt.njobs++] = a;
    if (bt.njobs == kGemmMaxJobs) {
      const dprc_status s = flush();
      if (s != DPRC_SUCCESS) return s;
    }
  }
  return flush();
}

dprc_status dprc_add_noise(float* grad, int64_t numel, float sigma, float C, uint64_t seed, uint32_t tensor_id,
                           hipStream_t stream) {
  if (numel < 0 || (numel > 0 && !grad)) return DPRC_ERROR_INVALID_VALUE;
  if (!(sigma >= 0.f) || std::isinf(sigma) || !(C > 0.f) || std::isinf(C)) return DPRC_ERROR_INVALID_VALUE;
  if (!aligned(grad, 4)) return DPRC_ERROR_NOT_SUPPORTED;
  if (numel == 0) return DPRC_SUCCESS;
  uint32_t k0, k1;
  key_of(seed, k0, k1);
  return hip_status(traced(DPRC_KERNEL_NOISE, stream, [&] { return launch_noise(grad, numel, sigma * C, k0, k1, tensor_id, stream); }));
}

dprc_status dprc_probe_bits(dprc_probe probe, uint64_t seed, uint32_t layer_id, uint32_t stream_id, int64_t m,
                            int32_t k, uint32_t* out, hipStream_t stream) {
  if (!out || m < 1 || k < 1 || m > (1LL << 36)) return DPRC_ERROR_INVALID_VALUE;
  if (probe != DPRC_PROBE_RADEMACHER && probe != DPRC_PROBE_HADAMARD) return DPRC_ERROR_INVALID_VALUE;
  uint32_t k0, k1;
  key_of(seed, k0, k1);
  return hip_status(traced(DPRC_KERNEL_PROBE_BITS, stream, [&] { return launch_probe_bits((int)probe, k0, k1, layer_id, stream_id, m, k, out, stream); }));
}

dprc_status dprc_private_adamw(float* theta, float* m, float* v, int64_t ldt, const float* G, int64_t ldg,
                               int64_t d, int64_t p, float sigma, float C, uint64_t seed, uint32_t tensor_id,
                               float inv_batch, const dprc_adamw_params* hp, uint16_t* w, int64_t ldw,
                               hipStream_t stream) {
  if (!theta || !m || !v || !G || !hp || d < 0 || p < 0 || ldt < p || ldg < p) return DPRC_ERROR_INVALID_VALUE;
  if (w && ldw < d) return DPRC_ERROR_INVALID_VALUE;
  if (!(sigma >= 0.f) || !std::isfinite(sigma) || !(C > 0.f) || !std::isfinite(C) || !std::isfinite(inv_batch))
    return DPRC_ERROR_INVALID_VALUE;
  const dprc_adamw_params& h = *hp;
  if (!(h.lr >= 0.f) || !std::isfinite(h.lr) || !(h.beta1 >= 0.f && h.beta1 < 1.f) ||
      !(h.beta2 >= 0.f && h.beta2 < 1.f) || !(h.eps > 0.f) || !std::isfinite(h.eps) ||
      !std::isfinite(h.weight_decay) || h.step < 1)
    return DPRC_ERROR_INVALID_VALUE;
  if (!aligned(theta, 4) || !aligned(m, 4) || !aligned(v, 4) || !aligned(G, 4) || (w && !aligned(w, 2)))
    return DPRC_ERROR_INVALID_VALUE;
  if (d == 0 || p == 0) return DPRC_SUCCESS;
  AdamArgs a;
  a.theta = theta; a.m = m; a.v = v; a.ldt = ldt; a.G = G; a.ldg = ldg; a.d = d; a.p = p;
  a.noise_scale = sigma * C;
  key_of(seed, a.key0, a.key1);
  a.tensor = tensor_id; a.inv_batch = inv_batch;
  a.decay = (float)(1.0 - (double)h.lr * h.weight_decay);
  a.beta1 = h.beta1; a.beta2 = h.beta2;
  a.one_minus_beta1 = (float)(1.0 - (double)h.beta1); a.one_minus_beta2 = (float)(1.0 - (double)h.beta2);
  const double bc1 = 1.0 - std::pow((double)h.beta1, h.step), bc2 = 1.0 - std::pow((double)h.beta2, h.step);
  a.step_size = (float)(h.lr / bc1);
  a.inv_sqrt_bc2 = (float)(1.0 / std::sqrt(bc2));
  a.eps = h.eps;
  a.w = w; a.ldw = ldw;
  a.vec = p % 4 == 0 && ldt % 4 == 0 && ldg % 4 == 0 && aligned(theta, 16) && aligned(m, 16) && aligned(v, 16) &&
          aligned(G, 16);
  a.wvec = w && ldw % 8 == 0 && aligned(w, 16);
  return hip_status(traced(DPRC_KERNEL_ADAMW, stream, [&] { return launch_private_adamw(a, stream); }));
}

size_t dprc_envelope_middle_workspace(int32_t nx, int32_t d, int32_t n_lambda) {
  if (nx < 1 || nx > 65535 || d < 2 || n_lambda < 1 || n_lambda > 4096) return 0;
  const int64_t ncand = (int64_t)d * (d - 1) / 2 * n_lambda;
  Arena ar(nullptr);
  ar.take<double>((size_t)nx * env_blocks(ncand));
  ar.take<int64_t>((size_t)nx * env_blocks(ncand));
  return ar.off;
}

dprc_status dprc_envelope_middle(const double* x, int32_t nx, int32_t k, int32_t d, int32_t n_lambda,
                                 double* best, int32_t* arg, void* ws, size_t ws_bytes, hipStream_t stream) {
  if (!x || !best || nx < 1 || nx > 65535 || k < 1 || d < 2 || (int64_t)k * d >= ((int64_t)1 << 31) ||
      n_lambda < 1 || n_lambda > 4096)
    return DPRC_ERROR_INVALID_VALUE;
  const size_t need = dprc_envelope_middle_workspace(nx, d, n_lambda);
  if (ws_bytes < need) return DPRC_ERROR_WORKSPACE_TOO_SMALL;
  if (!ws || !aligned(ws, kAlign) || !aligned(x, 8) || !aligned(best, 8) || (arg && !aligned(arg, 4)))
    return DPRC_ERROR_INVALID_VALUE;
  EnvArgs a;
  a.x = x; a.nx = nx; a.k = k; a.d = d; a.n_lambda = n_lambda;
  a.ncand = (int64_t)d * (d - 1) / 2 * n_lambda;
  a.panels = 16;
  gauss_legendre(kEnvNodes, a.gx, a.gw);
  Arena ar(ws);
  const int nblk = env_blocks(a.ncand);
  a.part_v = ar.take<double>((size_t)nx * nblk);
  a.part_c = ar.take<int64_t>((size_t)nx * nblk);
  a.best = best; a.arg = arg;
  return hip_status(traced(DPRC_KERNEL_ENVELOPE, stream, [&] { return launch_env_middle(a, stream); }));
}

dprc_status dprc_chi2_cdf(const double* x, int64_t n, double dof, double scale, double* out, hipStream_t stream) {
  if (!x || !out || n < 0 || !(dof > 0.0) || !std::isfinite(dof) || !(scale > 0.0) || !std::isfinite(scale))
    return DPRC_ERROR_INVALID_VALUE;
  if (!aligned(x, 8) || !aligned(out, 8)) return DPRC_ERROR_INVALID_VALUE;
  return hip_status(traced(DPRC_KERNEL_CHI2_CDF, stream, [&] { return launch_chi2_cdf(x, n, dof, scale, out, stream); }));
}

dprc_status dprc_envelope_bins(const double* F, int32_t n_bins, double y_min, double y_max, double* ybar, double* w,
                               hipStream_t stream) {
  if (!F || !ybar || !w || n_bins < 1 || !std::isfinite(y_min) || !std::isfinite(y_max) || !(y_max > y_min))
    return DPRC_ERROR_INVALID_VALUE;
  if (!aligned(F, 8) || !aligned(ybar, 8) || !aligned(w, 8)) return DPRC_ERROR_INVALID_VALUE;
  return hip_status(traced(DPRC_KERNEL_PLD, stream, [&] {
    return launch_envelope_bins(F, n_bins, y_min, y_max, ybar, w, stream); }));
}

size_t dprc_pld_step_workspace(int64_t n_half) {
  if (n_half < 1 || n_half > (1LL << 30)) return 0;
  return (size_t)round_up(2 * n_half * (int64_t)sizeof(double), kAlign);
}

dprc_status dprc_pld_step(double sigma, double p, double h, int64_t n_half, const double* ybar, const double* w,
                          int32_t n_bins, double* q, double* q_inf, void* ws, size_t ws_bytes, hipStream_t stream) {
  if (!(sigma > 0.0) || !std::isfinite(sigma) || !(p > 0.0 && p <= 1.0) || !(h > 0.0) || !std::isfinite(h) ||
      n_half < 1 || n_half > (1LL << 30) || n_bins < 0 || !q || !q_inf)
    return DPRC_ERROR_INVALID_VALUE;
  if (n_bins > 0 && (!ybar || !w || !aligned(ybar, 8) || !aligned(w, 8))) return DPRC_ERROR_INVALID_VALUE;
  const size_t need = dprc_pld_step_workspace(n_half);
  if (ws_bytes < need) return DPRC_ERROR_WORKSPACE_TOO_SMALL;
  if (!ws || !aligned(ws, kAlign) || !aligned(q, 8) || !aligned(q_inf, 8)) return DPRC_ERROR_INVALID_VALUE;
  PldArgs a;
  a.sigma = sigma; a.p = p; a.h = h;
  a.t_min = p < 1.0 ? std::log1p(-p) : -INFINITY;
  a.n = n_half; a.ybar = n_bins > 0 ? ybar : nullptr; a.w = n_bins > 0 ? w : nullptr; a.n_bins = n_bins;
  a.S = static_cast<double*>(ws); a.q = q; a.q_inf = q_inf;
  return hip_status(traced(DPRC_KERNEL_PLD, stream, [&] { return launch_pld_step(a, stream); }));
}

dprc_status dprc_pld_fold(const double* r, int64_t L, const double* ainf, const double* binf, double* q,
                          double* q_inf, hipStream_t stream) {
  if (!r || !ainf || !binf || !q || !q_inf || L < 1 || L % 2 == 0 || L > (1LL << 30)) return DPRC_ERROR_INVALID_VALUE;
  if (!aligned(r, 8) || !aligned(ainf, 8) || !aligned(binf, 8) || !aligned(q, 8) || !aligned(q_inf, 8))
    return DPRC_ERROR_INVALID_VALUE;
  return hip_status(traced(DPRC_KERNEL_PLD, stream, [&] { return launch_pld_fold(r, L, ainf, binf, q, q_inf, stream); }));
}

dprc_status dprc_pld_delta(const double* q, int64_t L, double h, const double* q_inf, const double* eps, int32_t n_eps,
                           double* delta, hipStream_t stream) {
  if (!q || !q_inf || !eps || !delta || L < 1 || L % 2 == 0 || !(h > 0.0) || !std::isfinite(h) || n_eps < 1 ||
      n_eps > 65535)
    return DPRC_ERROR_INVALID_VALUE;
  if (!aligned(q, 8) || !aligned(q_inf, 8) || !aligned(eps, 8) || !aligned(delta, 8)) return DPRC_ERROR_INVALID_VALUE;
  return hip_status(traced(DPRC_KERNEL_PLD, stream, [&] {
    return launch_pld_delta(q, L, h, q_inf, eps, n_eps, delta, stream); }));
}

dprc_status dprc_probe_gaussian(uint64_t seed, uint32_t layer_id, int64_t m, int32_t k, float* out,
                                hipStream_t stream) {
  if (!out || m < 1 || k < 1 || k > 256 || m > (1LL << 36)) return DPRC_ERROR_INVALID_VALUE;
  if (!aligned(out, 4)) return DPRC_ERROR_INVALID_VALUE;
  uint32_t k0, k1;
  key_of(seed, k0, k1);
  return hip_status(traced(DPRC_KERNEL_PROBE_GAUSS, stream, [&] {
    return launch_gauss_probe(k0, k1, layer_id, m, k, m, nullptr, nullptr, out, stream); }));
}

}  // extern "C"
