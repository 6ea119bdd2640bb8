// Kernel argument blocks and launch wrappers (host <-> device interface inside
// the library).  Every launch wrapper enqueues on the given stream and returns
// hipGetLastError().
#pragma once
#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace dprc {

// Start/stop events for the next launch on this host thread, set by the
// launch-trace hook of the C ABI (null otherwise).  With events, the kernel is
// launched through hipExtLaunchKernelGGL, which stamps them from the dispatch
// itself (no extra packets, so no timing overhead is added to the kernel).
struct LaunchEvents {
  hipEvent_t start = nullptr, stop = nullptr;
};
LaunchEvents& next_launch_events();

#define DPRC_LAUNCH(kernel, grid, block, lds, st, ...)                                            \
  do {                                                                                             \
    ::dprc::LaunchEvents& ev_ = ::dprc::next_launch_events();                                      \
    if (ev_.start)                                                                                 \
      hipExtLaunchKernelGGL(kernel, grid, block, lds, st, ev_.start, ev_.stop, 0u, __VA_ARGS__);   \
    else                                                                                           \
      hipLaunchKernelGGL(kernel, grid, block, lds, st, __VA_ARGS__);                               \
  } while (0)

constexpr int kWave = 64;
constexpr int kBlock = 256;        // threads per workgroup of the streaming kernels
constexpr int kStage = 64;         // tokens per pipeline stage of the token reduction
constexpr int kMaxGroup = 4;       // layers sharing one token reduction (same activations)
constexpr int kTile = 128;         // result rows per token-reduction workgroup
// Padded LDS row (elements) of a staged 64 x 128 bf16 tile: 288 bytes, so the four
// rows of one 16-lane transpose read start 32 bytes apart; rows with bit 3 set are
// stored with their 64-column halves swapped, so the rows 8 apart that neighbouring
// lane groups read land in the other half of the banks.
constexpr int kLdsLd = kTile + 16;
__host__ __device__ constexpr int lds_swz(int row, int col) { return col ^ (((row >> 3) & 1) << 6); }

inline int64_t ceil_div(int64_t a, int64_t b) { return (a + b - 1) / b; }
inline int64_t round_up(int64_t a, int64_t b) { return ceil_div(a, b) * b; }

// Y = X R on matrix cores.  X: bf16 token rows [B][T][ldx] (width m).  R has
// `nd` dense columns per sample (bf16 hi/lo pairs, Rhi/Rlo[i][c][ld_r]) followed
// by `nz` generated +-1 columns.  Output Yt: bf16 hi/lo, column-major per
// sample: Yt[h][c][i*T_pad + t], h = 0 hi, 1 lo; zero for t >= T and for
// columns >= nd + nz.
struct ProjectArgs {
  const uint16_t* X;
  int64_t ldx, x_ss;
  int32_t B, T, m, T_pad;
  int32_t nd, nz, ncols_pad;
  const uint16_t* Rhi;
  const uint16_t* Rlo;
  int64_t ld_r, r_ss;
  int32_t probe_kind;
  uint32_t key0, key1, layer_id, stream_id;
  int32_t z_split;          // generated columns c >= z_split come from stream_id2, as its column c - z_split
  uint32_t stream_id2;
  int32_t words_per_chunk;  // probe words per column staged in LDS at a time
  uint16_t* Yt;             // hi plane: Yt[c*yt_ld + i*T_pad + t]; lo plane at Yt + ylo_off
  int64_t yt_ld;            // B * T_pad
  int64_t ylo_off;
  int32_t ncols_write;      // columns written (ncols_pad, or only the real ones inside a shared Y)
  uint32_t* zero_ptr;       // counters cleared by workgroup (0,0) (may be null)
  int32_t zero_count;
  int32_t vec;              // token rows of X are 16-byte aligned: 16-byte loads
  int32_t rblocks;          // row blocks per workgroup (set by the launcher)
};

// Projections of several layers in one launch (one kernel instantiation: same columns,
// same dense-column count, same rows per workgroup).
constexpr int kProjMaxJobs = 32;      // 5.5 KB of kernel arguments
struct ProjectBatch {
  int32_t njobs, blocks;         // blocks and blk0 are set by the launcher
  int32_t blk0[kProjMaxJobs];
  ProjectArgs job[kProjMaxJobs];
};

// M_i = X_i^T Y_i per sample (result rows = the n columns of X; result
// columns = the ncols columns of Y), reduced over tokens in splits.
// mode 0: squared-norm estimate -> n2; mode 1: store M (fp32 and/or bf16 hi/lo).
struct TokredArgs {
  const uint16_t* X;
  int64_t ldx, x_ss;
  int32_t B, T, n;
  const uint16_t* Yt;
  int64_t yt_ld;
  int32_t T_pad, ncols, ncols_pad;
  int32_t ntiles, S, stages_per_split;
  int32_t mode;
  int32_t seg, nseg;      // mode 0: columns [g*seg, (g+1)*seg) are layer g of nseg (<= kMaxGroup)
  float* part;            // [B][ntiles][S][ncols_pad][kTile] (S > 1)
  double* tilesq;         // [nseg][B][ntiles] (mode 0)
  float scale;            // estimate = scale * ||M_i||^2
  float* n2;
  float* n2_layer;        // [nseg][B] (may be null)
  int32_t accumulate;
  float clip_C;           // with clip_c: clip_c[i] = clip factor of the final n2[i]
  float* clip_c;
  float* M;               // M[i*m_ss + c*m_ld + j]
  int64_t m_ld, m_ss;
  uint16_t* Mhi;          // Mhi/Mlo[i*mh_ss + c*mh_ld + j]
  uint16_t* Mlo;
  int64_t mh_ld, mh_ss;
  int32_t m_col0;         // M takes the columns c >= m_col0
  int32_t mh_ncols;       // Mhi/Mlo take the columns c < mh_ncols (0: all)
  int32_t vec;            // token rows of X are 16-byte aligned
};

// Token-split sums of several layers' passes in one launch.
constexpr int kTokMaxJobs = 32;       // 7.3 KB of kernel arguments
struct TokredBatch {
  int32_t njobs, blocks;
  int32_t blk0[kTokMaxJobs];     // first block of each job (ntiles * B blocks each)
  TokredArgs job[kTokMaxJobs];   // S > 1
};

// Per-sample sums of a call's token reductions (mode 0), up to kSampleMaxGroups groups in
// one launch: sample i walks the groups in order, each group's layers in order, adding each
// layer's estimate (its tile sums summed in the order of tokred_sample_kernel) to n2.
constexpr int kSampleMaxGroups = 128;
struct SampleGroup {
  const double* tilesq;   // [nseg][B][ntiles]
  float* n2_layer;        // [nseg][B] estimates per layer (may be null)
  int32_t ntiles, nseg;
};
struct SampleSumArgs {
  int32_t ngroups, B;
  float scale;            // estimate = scale * sum of the layer's tile sums
  float clip_C;
  float* n2;              // [B]
  float* clip_c;          // [B] clip factors from the final n2 (may be null)
  int32_t accumulate;     // add to n2 (else start from zero)
  SampleGroup g[kSampleMaxGroups];
};

struct GemmArgs {
  const uint16_t* A;
  int64_t lda, a_ss;
  const uint16_t* E;
  int64_t lde, e_ss;
  int32_t B, T, d, p;
  const float* c;
  float* out;
  int64_t ldo;
  int32_t accumulate;
  int32_t S, stages_per_sample, stages_per_split;
  float* part;            // [S][d][p] (S > 1)
  int32_t vec_a, vec_e;   // token rows 16-byte aligned
};
// Unsplit accumulations of several layers in one launch (the launcher sets blk0).
constexpr int kGemmMaxJobs = 64;     // 8.7 KB of kernel arguments
constexpr int64_t kGemmRoundTiles = 256;   // 256 x 256 tiles that occupy every CU once
struct GemmBatch {
  int32_t njobs;
  int32_t blk0[kGemmMaxJobs];
  GemmArgs job[kGemmMaxJobs];
};
struct GemmPlan {
  int32_t S, sps, spl, tiles;   // splits, slabs per sample, slabs per split, output tiles
};
GemmPlan gemm_plan_v2(int64_t B, int64_t T, int64_t d, int64_t p);

// fp32 (SIMT) variants, used for fp32 inputs.
struct ProjectF32Args {
  const float* X;
  int64_t ldx, x_ss;
  int32_t B, T, m;
  int32_t nd, nz, ncols;
  const float* Rd;        // dense columns [i][c][ld_r]
  int64_t ld_r, r_ss;
  const uint32_t* zbits;  // generated columns, packed [c][ceil(m/32)]
  float* Y;               // [B][T][ncols]
};

struct TokredF32Args {
  const float* X;
  int64_t ldx, x_ss;
  int32_t B, T, n;
  const float* Y;         // [B][T][ncols]
  int32_t ncols;
  float* M;               // M[i*m_ss + c*m_ld + j]
  int64_t m_ld, m_ss;
};

// Tall-skinny QR of O S (m x s per sample, s <= 32) and C = Q^T P (Hutch++), as a
// tree of 128-row Householder block factorizations (one wavefront per block).
// Level 1 factors 128-row blocks of O S; level l + 1 factors the stacked s x s R
// factors of level l, until one block remains.  The expansion runs back down:
// block b of level l starts from rows b*s .. b*s+s-1 of level l+1's Q (the identity
// at the top) and applies its reflectors.
constexpr int kQrRows = 128;   // rows per block (two per lane)
constexpr int kQrMaxLevels = 8;
struct QrLevel {
  int32_t rows, nblk;            // input rows, blocks (= ceil(rows / 128))
  double* V;                     // [B][nblk][s][128] reflectors, zero above the diagonal
  double* tau;                   // [B][nblk][s]
  double* M;                     // [B][s][rows] fp64 input (levels >= 2); level 1 reads O S
  double* Q;                     // [B][s][rows] explicit Q of this level (levels >= 2)
};
struct QrArgs {                  // one layer's tree (host side): level geometry and scratch
  int32_t B, m, s, r;
  int32_t nlev;
  QrLevel lev[kQrMaxLevels];
  double* Cpart;                 // [B][nblk1][s][r]
};
// Level geometry for m rows and s columns; doubles of workspace per sample in *dbl.
int32_t qr_levels(int64_t m, int s, int32_t rows[kQrMaxLevels], int32_t nblk[kQrMaxLevels], int64_t* dbl);

// One layer's share of a QR launch: one tree level of that layer.  Launches take up
// to kQrMaxJobs layers at once (their trees are independent), so a whole level of
// every layer's tree costs one launch.  Blocks blk0 .. blk0 + L.nblk * B - 1 of the
// launch belong to the job (block b of sample i at blk0 + i * L.nblk + b).
struct QrJob {
  int32_t blk0;
  int32_t level, nlev;           // tree level worked on; levels of the layer's tree
  int32_t B, m, s, r;
  QrLevel L;                     // level `level`
  QrLevel X;                     // level `level` + 1 when it exists (factor: its input M; expand: its Q)
  const float* OS;               // level 0 input: OS[i*os_ss + c*os_ld + j]
  int64_t os_ld, os_ss;
  double* Cpart;                 // [B][nblk1][s][r]
  uint32_t key0, key1, layer;
  float* Q;                      // Q[i*q_ss + c*q_ld + j] (may be null)
  int64_t q_ld, q_ss;
  uint16_t* Qhi;                 // bf16 hi/lo pairs, zero for rows m .. qh_ld-1 (may be null)
  uint16_t* Qlo;
  int64_t qh_ld, qh_ss;
};
constexpr int kQrMaxJobs = 8;
struct QrBatch {
  int32_t njobs, blocks;         // jobs, total blocks of the launch
  int32_t s, r;                  // shared by every job
  QrJob job[kQrMaxJobs];
};

// Hutch++ estimate from U | W_P (UW[i*uw_ss + c*uw_ld + j], c < s + r) and C.
struct FinalArgs {
  const float* UW;
  int64_t uw_ld, uw_ss;
  int32_t B, n, s, r, nblk, nchunk;
  const double* Cpart;    // [B][nblk][s][r]
  double* C;              // [B][s][r]: C = Q^T P, the block partials summed in block order
  double* Fpart;          // [B][nchunk][2]
  float* n2;
  float* n2_layer;
  int32_t accumulate;
};
int32_t final_chunks(int64_t n);
// The finalize of several layers (same s, r and B): one launch per step for all of them.
constexpr int kFinMaxJobs = 8;
struct FinalBatch {
  int32_t njobs;
  int32_t blk0[kFinMaxJobs];     // set by the launchers
  FinalArgs job[kFinMaxJobs];
};

hipError_t launch_probe_bits(int probe_kind, uint32_t key0, uint32_t key1, uint32_t layer,
                             uint32_t stream_id, int64_t m, int32_t k, uint32_t* out,
                             hipStream_t st);
// MiddleRegionCDF over a batch of points (see dprc_envelope_middle).
constexpr int kEnvNodes = 16;
struct EnvArgs {
  const double* x;
  int32_t nx, k, d, n_lambda;
  int64_t ncand;          // d (d - 1) / 2 * n_lambda
  int32_t panels;
  double gx[kEnvNodes], gw[kEnvNodes];   // Gauss-Legendre nodes and weights on [-1, 1]
  double* part_v;         // [nx][blocks]
  int64_t* part_c;
  double* best;           // [nx]
  int32_t* arg;           // [nx][3] or null
};
int env_blocks(int64_t ncand);
hipError_t launch_env_middle(const EnvArgs& a, hipStream_t st);
hipError_t launch_chi2_cdf(const double* x, int64_t n, double dof, double scale, double* out, hipStream_t st);

// Privacy accounting (see dprc_pld_step and the others): one subsampled step's
// survival function at 2n cut points into S, then its 2n - 1 cell masses and atom.
struct PldArgs {
  double sigma, p, h, t_min;   // t_min = log(1 - p) (-inf for p = 1)
  int64_t n;                   // cut points per side
  const double* ybar;          // envelope bins (null with n_bins = 0: a = 1)
  const double* w;
  int32_t n_bins;
  double* S;                   // [2n] scratch
  double* q;                   // [2n - 1]
  double* q_inf;               // [1]
};
hipError_t launch_envelope_bins(const double* F, int32_t M, double y_min, double y_max, double* ybar, double* w,
                                hipStream_t st);
hipError_t launch_pld_step(const PldArgs& a, hipStream_t st);
hipError_t launch_pld_fold(const double* r, int64_t L, const double* ainf, const double* binf, double* q,
                           double* q_inf, hipStream_t st);
hipError_t launch_pld_delta(const double* q, int64_t L, double h, const double* q_inf, const double* eps,
                            int32_t n_eps, double* delta, hipStream_t st);

// One private AdamW step on a [d, p] fp32 master (see dprc_private_adamw).
struct AdamArgs {
  float* theta;
  float* m;
  float* v;
  int64_t ldt;
  const float* G;
  int64_t ldg;
  int64_t d, p;
  float noise_scale;       // sigma * C (0: no noise)
  uint32_t key0, key1, tensor;
  float inv_batch;
  float decay;             // 1 - lr * weight_decay
  float beta1, beta2, one_minus_beta1, one_minus_beta2;
  float step_size;         // lr / (1 - beta1^t)
  float inv_sqrt_bc2;      // 1 / sqrt(1 - beta2^t)
  float eps;
  uint16_t* w;             // bf16 [p, d] copy (may be null)
  int64_t ldw;
  int32_t vec, wvec;
};
hipError_t launch_private_adamw(const AdamArgs& a, hipStream_t st);

// Gaussian probe columns, column j at [j*ld .. j*ld + ld) (rows >= m zero);
// any of hi/lo (both or neither) and f32 may be null.
hipError_t launch_gauss_probe(uint32_t key0, uint32_t key1, uint32_t layer, int64_t m, int32_t k, int64_t ld,
                              uint16_t* hi, uint16_t* lo, float* f32, hipStream_t st);
hipError_t launch_fill_u32(uint32_t* p, int64_t n, uint32_t v, hipStream_t st);
hipError_t launch_project(const ProjectArgs& a, int rows_per_wg, hipStream_t st);
hipError_t launch_project_batch(ProjectBatch bt, int rows_per_wg, hipStream_t st);   // <= 64 columns
hipError_t launch_tokred_batch(TokredBatch bt, hipStream_t st);                      // <= 64 columns
hipError_t launch_tokred(const TokredArgs& a, hipStream_t st);
hipError_t launch_tokred_splits(const TokredArgs& a, hipStream_t st);   // S > 1
hipError_t launch_tokred_splits_batch(const TokredBatch& bt, hipStream_t st);
// mode 0: the estimates of the jobs' layers added to n2 in order, then the clip factor (clip_c may be null)
hipError_t launch_sample_sums(const SampleSumArgs& a, hipStream_t st);
hipError_t launch_tokred_sample(const TokredArgs& a, hipStream_t st);   // mode 0
hipError_t launch_project_f32(const ProjectF32Args& a, hipStream_t st);
hipError_t launch_tokred_f32(const TokredF32Args& a, hipStream_t st);
// n2 (=|+=) scale * sum_{c<ncols, j<n} M[i][c][j]^2 (+ optional per-layer copy)
hipError_t launch_sample_sq(const float* M, int64_t m_ld, int64_t m_ss, int32_t B, int32_t ncols,
                            int32_t n, float scale, float* n2, float* n2_layer, int accumulate,
                            hipStream_t st);
hipError_t launch_qr_factor(const QrBatch& bt, hipStream_t st);   // a level-0 job reads O S
hipError_t launch_qr_expand(const QrBatch& bt, hipStream_t st);   // a level-0 job writes Q and C
hipError_t launch_hpp_csum(const FinalArgs& a, hipStream_t st);
hipError_t launch_hpp_rows(const FinalArgs& a, hipStream_t st);
hipError_t launch_hpp_sum(const FinalArgs& a, hipStream_t st);
// the finalize of a group of layers (same s, r, B): C sums, row chunks, per-sample sums in layer order
hipError_t launch_hpp_csum_batch(const FinalBatch& bt, hipStream_t st);
hipError_t launch_hpp_rows_batch(const FinalBatch& bt, hipStream_t st);
hipError_t launch_hpp_sum_batch(const FinalBatch& bt, hipStream_t st);
hipError_t launch_clip_scale(const float* n2, int64_t B, float C, float* c, hipStream_t st);
hipError_t launch_gemm(const GemmArgs& a, hipStream_t st);
hipError_t launch_gemm_batch(GemmBatch bt, hipStream_t st);
hipError_t launch_gemm_f32(const float* A, int64_t lda, int64_t a_ss, const float* E, int64_t lde,
                           int64_t e_ss, int32_t B, int32_t T, int32_t d, int32_t p,
                           const float* c, float* out, int64_t ldo, int accumulate,
                           hipStream_t st);
hipError_t launch_splitk_reduce(const float* part, int32_t S, int32_t d, int32_t p, float* out,
                                int64_t ldo, int accumulate, hipStream_t st);
hipError_t launch_noise(float* g, int64_t numel, float scale, uint32_t key0, uint32_t key1,
                        uint32_t tensor_id, hipStream_t st);

}  // namespace dprc
