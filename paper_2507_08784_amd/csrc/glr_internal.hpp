// Internal interface between the host runtime and the kernel launchers.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "greedylore.h"

namespace glr {

constexpr int kJB = 16;   // rows per Jacobi block

// The fp64 Gram A = W W^T of a refresh is kept packed by 16 x 16 blocks:
// block (a, b), a <= b, row-major, at pk_off(a, b, nb) doubles.
__host__ __device__ inline int64_t pk_off(int a, int b, int nb) {
  return ((int64_t)a * nb - (int64_t)a * (a - 1) / 2 + (b - a)) * (kJB * kJB);
}
__host__ __device__ inline int64_t pk_doubles(int nb) { return (int64_t)nb * (nb + 1) / 2 * (kJB * kJB); }

// Per-refresh control words of the block Jacobi (device memory).
constexpr int kInfoInts = 64;   // per-matrix info block in the state
constexpr int kHistory = 60;    // sweeps whose off-norm is recorded

struct JacCtl {
  uint32_t converged;
  uint32_t sweeps;
  uint32_t sweep_max_bits;     // float bits of the largest pair off-norm this sweep
  uint32_t pad;
  uint64_t rowmax2_bits;       // double bits of the largest squared row norm seen
  uint32_t history[kHistory];  // float bits of each sweep's largest off-norm
};

// Bits of the device status word (first word of the state blob), latched by
// kernels and read and cleared by glr_sync_status.
constexpr uint32_t kStatusNonfinite = 1u;       // a gradient held NaN or Inf
constexpr uint32_t kStatusNotConverged = 2u;    // Jacobi sweeps ended above tol
constexpr uint32_t kStatusBreakdown = 4u;       // an orthonormalisation still broke down after its repair pass
constexpr uint32_t kStatusSubNotConverged = 8u; // tau = 1 block iteration above its tolerance after its budget
constexpr uint32_t kStatusRepaired = 16u;       // dependent rows of an orthonormalisation were replaced

// Info block of a matrix (kInfoInts ints in the state): [0] Jacobi sweeps of
// the last refresh, [1] its converged flag, [2 + s] sweep s's largest pair
// off-norm (float bits); for the tau = 1 refresh also:
constexpr int kInfoSubIters = 62;    // block iterations run (fewer than the budget: the leading r rows met the tolerance)
constexpr int kInfoSubGain = 63;     // float bits: relative gain of the block's captured energy over the last iteration

// Control words of the subspace iteration (device memory).
struct SubCtl {
  int iters;
  int converged;               // the leading r rows moved by less than the tolerance
  double change2;              // squared Frobenius norm of the last change of the leading r rows
  int gate_iter;               // nonzero: the current iteration is skipped (converged before it)
  int gate_pass;               // nonzero: the current orthonormalisation pass is skipped
  int gate_rest;               // nonzero: the rest of the pass is skipped (gated, or its rows are
                               // orthonormal already)
  int repaired;                // rows replaced by the last orthonormalisation pass
  int reuse_z;                 // nonzero: a warm iteration met the tolerance; P keeps the basis it
                               // started from and Z = P^T Mo of that basis serves the Rayleigh-Ritz
                               // step (no product of its own)
  int stop;                    // no further iteration: converged, at its cap, or past 2 with a closed gap
  double e_in;                 // ||P Mo||^2 of the K-row block entering the last iteration run
  double e_out;                // ||P Mo||^2 of the final block
  uint32_t history[kHistory];  // float bits of each iteration's change / sqrt(r)
};

// A CholeskyQR pivot of the diagonally scaled Gram (1 for a row independent of
// the rows before it, 0 for a dependent one) at or below this marks its row
// as dependent: the fp32 rows and their fp32-summed products resolve the
// pivots only to about 1e-6.
constexpr double kPivotFloor = 1e-5;
// A CholeskyQR pass after the first is skipped when the Gram of its rows is
// the identity to within this (largest |cosine| between two rows and largest
// |squared norm - 1|): about the resolution of the fp32-product Gram itself.
constexpr double kOrthSkip = 4e-6;
// partial sums of a block's captured energy (fp64), before their in-order sum
constexpr int kEnergyParts = 256;
// tau = 1 block iterations: at least kSubMinIters, then more (up to the cap)
// while the leading r rows still move by more than the tolerance and the
// previous refresh's Ritz values show an open eigengap at r,
// (sigma_r^2 - sigma_{r+1}^2) / sigma_1^2 >= kSubGapOpen (below it the top-r
// subspace is not determined by the data and only the captured energy is)
constexpr int kSubMinIters = 2;
constexpr int kSubCapWarm = 4;
constexpr int kSubCapCold = 8;
constexpr double kSubGapOpen = 1e-3;

constexpr int kMaxSubK = 256;   // largest rank the subspace-iteration refresh takes
constexpr int kCholTile = 64;   // tile of the K x K Cholesky factorisation
inline int chol_pad(int K) { return (K + kCholTile - 1) / kCholTile * kCholTile; }

// The tau = 1 refresh needs only span(U[:, :r]): subspace iteration then, on
// an oversampled block of sub_block(r, d) directions.
inline bool use_subspace(int tau, int r, int64_t d) { return tau == 1 && r < d && r <= kMaxSubK; }
// rows of a subspace GEMM tile for an M-row product, and its tile count
inline int gemm_rows(int M) { return M % 128 != 0 ? 64 : 128; }
inline int gemm_blocks(int M, int N) { return ((N + 127) / 128) * ((M + gemm_rows(M) - 1) / gemm_rows(M)); }
// oversampling: r / 4 extra directions, at least 32
inline int sub_block(int r, int64_t d) {
  const int64_t k = (int64_t)r + (r / 4 > 32 ? r / 4 : 32);
  return (int)(k < d ? k : d);
}

// One matrix of the current step, as the kernels see it.
struct MatView {
  int64_t m, n, d, D;
  bool right;                // m > n
  int r;                     // effective rank
  int N;                     // workers
  int mat;                   // matrix index (RNG counter)
  bool st16;                 // G^(i) and E^(i) are bf16 (GLR_STORE_BF16), else fp32
  // state (E: N x m x n elements of the storage type)
  void* E;       float* Ebar;  float* Ut;   float* sigma;  int* J;
  float* score;  float* S1;    float* S2;   float* Rbar;   int* info;
  uint32_t* status;
  // caller buffers (G: N x m x n elements of the storage type)
  float* X;      const void* G;
  // workspace
  float* Mbar;   float* Q;     float* Qpart; float* lam_part;
  float* W;      float* Utw;   double* Apk;  double* Apk2; float* Vrot;   double* V64;   int* skip;
  double* gpart;   // split-contraction partials of the Gram (or null)
  JacCtl* ctl;   float* sigma_w; int* perm;
  // subspace iteration
  float* sub_P;  float* sub_Pn; float* sub_Z;  float* sub_Zt; float* sub_R; float* sub_part;
  double* sub_S; double* sub_L; double* sub_Dinv; double* sub_Li; double* sub_T;
  float* sub_Linv; float* sub_C; double* sub_sums; SubCtl* sub_ctl;
  int* sub_bad;    // rows marked dependent by the current CholeskyQR pass (K ints)
  // Rayleigh-Ritz: Jacobi on the fp64 Gram of the K x D projection
  float* rr_Utw; float* rr_Y; double* rr_Apk; float* rr_V; double* rr_V64; int* rr_skip;
  JacCtl* rr_ctl; float* rr_sigw; int* rr_perm; double* rr_gpart;
};

// Optional timing brackets around launch groups (glr_prof_group ids); a
// no-op unless the host runtime installs a callback.
struct ProfHook {
  void* ctx = nullptr;
  void (*fn)(void* ctx, int group, int begin) = nullptr;
  void begin(int g) const { if (fn) fn(ctx, g, 1); }
  void end(int g) const { if (fn) fn(ctx, g, 0); }
};

// Slices of the d contraction of the projection.  Above rank 64 one tile
// covers all r rows (r <= 128: 128 x 64 tiles, above: 256 x 64) and
// accumulates 1024 terms in fp32 per slice; the slices are added in fp64 by
// the reduction (1024 rather than 512 terms halves the partial products
// written and read back: 0.94 instead of 1.88 GB on the 8192 x 28672 matrix
// with four workers).  Up to rank 64 slices (of at least 256) are only made
// to fill the chip, and the kernel itself adds fp32 partial sums of 512
// terms into fp64.
constexpr int kProjWideRank = 128;
constexpr int kProjSlice = 1024;
constexpr int kProjFlushRank = 64;
// fp32 terms per slice of the tiers above kProjFlushRank (0: a flushing tier)
inline int proj_slice(int r) { return r > kProjFlushRank ? kProjSlice : 0; }
inline int proj_splits(int64_t d, int64_t D, int r, int N) {
  if (const int sl = proj_slice(r)) return (int)((d + sl - 1) / sl);
  const int64_t tiles = ((D + 63) / 64) * N;
  if (tiles >= 2048) return 1;
  int64_t sp = (2048 + tiles - 1) / tiles;
  const int64_t mx = d / 256;
  if (sp > mx) sp = mx;
  return sp < 1 ? 1 : (int)sp;
}
// the slice length a projection launch uses
inline int proj_kslice(int64_t d, int64_t D, int r, int N) {
  if (const int sl = proj_slice(r)) return sl;
  const int sp = proj_splits(d, D, r, N);
  return (int)(((d + sp - 1) / sp + 31) / 32 * 32);
}

// above this rank the residuals come first from a wider-tile kernel
constexpr int kResidWideRank = 128;

struct OptParams {
  int opt;                   // 0 MSGD, 1 Adam, 2 plain step X -= lr Ghat (GaLore: Ghat = P Rhat)
  float lr, beta1, beta2, eps;
  int ef = 1;                // error feedback: write E^(i) and Ebar = Mbar - Ghat (0: both stay zero)
};

// launchers (return the first launch error)
hipError_t launch_fill_zero(void* p, size_t bytes, hipStream_t s);
hipError_t launch_eye(float* Ut, int64_t d, hipStream_t s);
hipError_t launch_ef_mean(const MatView& v, bool check_finite, hipStream_t s);
hipError_t launch_sel_scores(const MatView& v, bool approx, bool bf16, uint64_t seed, int64_t t, hipStream_t s);
hipError_t launch_topr(const MatView& v, hipStream_t s);
hipError_t launch_iota_J(const MatView& v, hipStream_t s);
hipError_t launch_proj(const MatView& v, hipStream_t s);
hipError_t launch_rbar(const MatView& v, hipStream_t s);
hipError_t launch_resid_opt(const MatView& v, const OptParams& o, hipStream_t s);
hipError_t launch_full_refresh(const MatView& v, const OptParams& o, hipStream_t s);
// Algorithm 5 (GaLore Adam in the r x D subspace): S1, S2 <- the moments of
// Rbar (from zero when `reset`), Rbar <- S1 / (sqrt(S2) + eps)
hipError_t launch_galore_adam(const MatView& v, const OptParams& o, bool reset, hipStream_t s);

// One matrix of a grouped selection step (device memory, rewritten every such
// step: the view carries that step's X and G) and its projection slicing.
struct GroupMat {
  MatView v;
  int splits, kslice;
};
// the kernels of a grouped selection step, each one launch over all matrices
enum { kGrpEfMean = 0, kGrpSelScores, kGrpSelFinish, kGrpProj, kGrpRbar, kGrpResid, kGrpKinds };
struct GroupPlan {
  const GroupMat* gm = nullptr;   // num entries
  const int* first = nullptr;     // kGrpKinds tables of num + 1 first blocks
  int num = 0;
  bool right = false;             // every matrix of the group has the same side, rank and kernel variants
  bool st16 = false;              // storage type of G and E (the handle's)
  int r = 0;
  size_t topr_lds = 0;            // the largest matrix's top-r sort keys
  int total[kGrpKinds] = {};
};
// the slicing of one matrix's projection and its block count in every grouped launch
void group_fill(GroupMat& g, int (&blocks)[kGrpKinds]);
size_t topr_lds_bytes(int64_t d);
// one selection step of every matrix of the plan: M-bar, the Approx-Top-r (or
// exact) scores and their top r, the projection and its mean, the residual
// and the optimizer update, seven launches in all (part 1: M-bar only; part
// 2: the launches after it; 0: all)
hipError_t launch_group_select(const GroupPlan& gp, bool check_finite, bool approx, bool bf16, uint64_t seed,
                               int64_t t, const OptParams& o, int part, hipStream_t s);

// One matrix of a joint refresh (device memory): its views for the two buffer
// parities of the per-sweep reordering (v[1] is v[0] with Apk <-> Apk2 and
// Utw <-> W) and the sizes of its tournament.
struct JointMat {
  MatView v[2];
  int nb, seats, groups, rounds, chunks, width;
};
// Block-offset tables of the joint launches (each num + 1 ints; entry m is the
// first block of matrix m, entry num the grid size)
enum { kJointSolve = 0, kJointSolveApply, kJointUpdate, kJointDiag, kJointPermute, kJointGather, kJointKinds };
// A joint refresh as the host sees it: device tables, and the grid sizes
struct JointPlan {
  const JointMat* jm = nullptr;
  const int* first = nullptr;   // kJointKinds tables of num + 1 ints
  int* flags = nullptr;         // num ints: converged flags for the host
  int num = 0, ng = 0, rounds_max = 0, npad_max = 2;
  int total[kJointKinds] = {};
};
// the sizes of matrix J.v[0]'s tournament and its block counts per launch kind
void joint_fill(JointMat& J, int (&blocks)[kJointKinds]);
hipError_t launch_joint_sort(const JointPlan& jp, int par, hipStream_t s);
hipError_t launch_joint_solve(const JointPlan& jp, int par, int round, float tol, int max_inner, double floor_rel2,
                              hipStream_t s);
hipError_t launch_joint_solve_apply(const JointPlan& jp, int par, int round, float tol, int max_inner,
                                    double floor_rel2, hipStream_t s);
hipError_t launch_joint_update(const JointPlan& jp, int par, int round, hipStream_t s);
hipError_t launch_joint_check(const JointPlan& jp, float tol, hipStream_t s);

// Jacobi on the fp64 Gram of the rows of W
int jac_blocks(int64_t d);
int jac_seats(int64_t d);
int jac_group_blocks(int64_t d);
int jac_groups(int64_t d);
int jac_rounds(int64_t d);
int64_t jac_vbuf(int64_t d);   // entries of one round's group rotations
hipError_t launch_jac_reset(const MatView& v, hipStream_t s);
hipError_t launch_jac_init(const MatView& v, bool warm, hipStream_t s);
// one round = update(round) after solve(round); the rotation of U^T rows by
// round k runs inside solve_apply(k + 1), or apply(k) after the last round
hipError_t launch_jac_update(const MatView& v, int round, hipStream_t s);
hipError_t launch_jac_solve_apply(const MatView& v, int round, float tol, int max_inner, double floor_rel2,
                                  hipStream_t s);
hipError_t launch_jac_apply(const MatView& v, int round, hipStream_t s);
// reorders the rows by descending diag(A): A (into Apk2) and U^T (into W);
// the caller then swaps Apk <-> Apk2 and Utw <-> W
hipError_t launch_jac_sort(const MatView& v, hipStream_t s);
hipError_t launch_jac_solve(const MatView& v, int round, float tol, int max_inner, double floor_rel2,
                            hipStream_t s);
hipError_t launch_jac_check(const MatView& v, float tol, hipStream_t s);
hipError_t launch_jac_finish(const MatView& v, int max_sweeps, hipStream_t s);
hipError_t launch_reorth(const MatView& v, hipStream_t s);

// A (packed fp64 blocks, zero padded) = W W^T for n rows of length Kc (ld)
int gram_splits(int64_t n, int64_t Kc);
hipError_t launch_gram_packed(const float* W, int64_t ld, int64_t n, int64_t Kc, double* Apk, double* part64,
                              hipStream_t s);

// subspace iteration (tau = 1)
size_t sub_part_floats(int K, int64_t d, int64_t D);
hipError_t launch_sub_start(const MatView& v, bool warm, uint64_t seed, int64_t t, hipStream_t s);
hipError_t launch_sub_iter(const MatView& v, float tol, uint64_t seed, int64_t t, int it, bool cold, int cap,
                           const ProfHook& prof, hipStream_t s);
hipError_t launch_sub_rr_begin(const MatView& v, MatView* rr, hipStream_t s);
hipError_t launch_sub_rr_end(const MatView& v, float tol, int cap, hipStream_t s);

}  // namespace glr
