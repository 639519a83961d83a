// Refresh step: complete left singular basis U of Mbar (d x D) by block
// Jacobi on the fp64 Gram A = W W^T of the rows of W = U_0^T Mo (U_0 the
// previous basis, or I): the eigenvectors of A are the left singular vectors.
//
// A is formed once per refresh (fp64-accumulated products of the fp32 rows)
// and kept packed by 16 x 16 blocks.  Rows are grouped in blocks of kJB; a
// round splits the blocks into groups of NG (two or four, NR = 16 NG rows),
// and each group is treated as a whole:
//   solve  : one cyclic two-sided Jacobi sweep on the group's NR x NR
//            diagonal block of A in LDS (fp64) gives the rotation V
//   update : A <- J^T A J with J = diag(V_group), block by block: the NR x NR
//            block (g, h) of two groups becomes V_g^T A_gh V_h (fp64 MFMA)
//   apply  : rows of U^T <- V^T rows, in place, as u + (V - I)^T u
//            (fp32 MFMA), in the same launch as the next round's solves
// A sweep meets every pair of blocks once: S - 1 rounds of pairs (circle
// method on S seats), or (S - 1) / 3 rounds of groups of four for S = 4^j
// seats, so that A and U^T are streamed a third as often; pairs serve small
// d, where the rounds are bound by the latency of the solves, and block
// counts far from a power of 4.  Padding seats hold empty blocks.  The
// sweeps stop when every group solved in a sweep passes the measure of the
// solve.  The singular values are sqrt(diag A), sorted descending (ties keep
// the lower row first); U^T rows follow the sort.
#include "glr_device.hpp"
#include "glr_internal.hpp"

namespace glr {

int jac_blocks(int64_t d) { return (int)((d + kJB - 1) / kJB); }
static int pow4_at_least(int n) {
  int s = 4;
  while (s < n) s *= 4;
  return s;
}
// Blocks per group: four when the 16-row blocks nearly fill a power of 4 of
// at least 64 seats (the rounds then stream A and U^T a third as often as
// pairs do), two otherwise (fewer seats wasted on padding, and for small d a
// round is bound by the latency of its solves, which is shorter for pairs).
int jac_group_blocks(int64_t d) {
  const int nb = jac_blocks(d);
  return (nb >= 64 && 4 * nb >= 3 * pow4_at_least(nb)) ? 4 : 2;
}
int jac_seats(int64_t d) {
  const int nb = jac_blocks(d);
  if (jac_group_blocks(d) == 4) return pow4_at_least(nb);
  return nb + (nb & 1) < 2 ? 2 : nb + (nb & 1);
}
int jac_groups(int64_t d) { return jac_seats(d) / jac_group_blocks(d); }
int jac_rounds(int64_t d) {
  return jac_group_blocks(d) == 4 ? (jac_seats(d) - 1) / 3 : jac_seats(d) - 1;
}
int64_t jac_vbuf(int64_t d) {
  const int64_t nr = (int64_t)jac_group_blocks(d) * kJB;
  return (int64_t)jac_groups(d) * nr * nr;
}

// Block indices are vectors over F_2 (S = 2^k seats, k even), read as
// vectors of k/2 digits over F_4 = {0, 1, w, w^2}, a digit being two bits
// (1 = 01, w = 10, w^2 = 11).  Multiplication by w, digit by digit:
// (h, l) -> (h ^ l, h).
__device__ __forceinline__ uint32_t f4_times_w(uint32_t x) {
  const uint32_t h = (x >> 1) & 0x55555555u, l = x & 0x55555555u;
  return ((h ^ l) << 1) | h;
}
// Blocks of group g in round t.
// Groups of four: the rounds are the (S - 1) / 3 lines {0, v, w v, w^2 v}
// through the origin (v with leading digit 1), which cover every non-zero
// vector exactly once.  The groups of a round are the cosets x0 + line, so
// two blocks a, b share a group exactly in the round whose line holds a ^ b.
// Member m of a group is the block whose digit p (the leading digit of v)
// equals m; x0 is g with a zero digit inserted at p.
// Pairs: the circle method on the seats (seat S - 1 fixed, the others turn).
template <int NG>
__device__ __forceinline__ void group_blocks(int t, int g, int seats, int (&blk)[NG]) {
  if constexpr (NG == 4) {
    int p = 0, base = 0;
    while (t >= base + (1 << (2 * p))) {
      base += 1 << (2 * p);
      ++p;
    }
    const uint32_t v = (1u << (2 * p)) | (uint32_t)(t - base);
    const uint32_t v2 = f4_times_w(v), v3 = v ^ v2;
    const uint32_t low = (1u << (2 * p)) - 1u;
    const uint32_t x0 = (((uint32_t)g & ~low) << 2) | ((uint32_t)g & low);
    blk[0] = (int)x0;
    blk[1] = (int)(x0 ^ v);
    blk[2] = (int)(x0 ^ v2);
    blk[3] = (int)(x0 ^ v3);
  } else {
    const int last = seats - 1;
    if (g == 0) {
      blk[0] = t;
      blk[1] = last;
    } else {
      blk[0] = (t + g) % last;
      blk[1] = (t - g + last) % last;
    }
  }
}

// ---------------------------------------------------------------------------
// initialisation: cold (W = Mo, Utw = I) or warm (Utw = Ut, W = Ut Mo)
// ---------------------------------------------------------------------------
__global__ void k_jac_copy_cold(const float* __restrict__ Mbar, float* __restrict__ W, int64_t d,
                                int64_t D, int right) {
  // W[a][b] = Mo[a][b]: a straight copy (left) or a transpose (right)
  __shared__ float tile[32][33];
  const int64_t a0 = (int64_t)blockIdx.y * 32, b0 = (int64_t)blockIdx.x * 32;
  const int tx = threadIdx.x & 31, ty = threadIdx.x >> 5;   // 32 x 8
  if (!right) {
    for (int k = ty; k < 32; k += 8) {
      int64_t a = a0 + k, b = b0 + tx;
      if (a < d && b < D) W[a * D + b] = Mbar[a * D + b];
    }
    return;
  }
  // Mbar is D x d (row b, column a)
  for (int k = ty; k < 32; k += 8) {
    int64_t b = b0 + k, a = a0 + tx;
    tile[k][tx] = (b < D && a < d) ? Mbar[b * d + a] : 0.f;
  }
  __syncthreads();
  for (int k = ty; k < 32; k += 8) {
    int64_t a = a0 + k, b = b0 + tx;
    if (a < d && b < D) W[a * D + b] = tile[tx][k];
  }
}

__global__ void k_copy(const float* __restrict__ src, float* __restrict__ dst, int64_t n) {
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < n; i += stride) dst[i] = src[i];
}

__global__ void k_ctl_reset(JacCtl* ctl) {
  if (threadIdx.x == 0) {
    ctl->converged = 0;
    ctl->sweeps = 0;
    ctl->sweep_max_bits = 0;
    ctl->rowmax2_bits = 0;
  }
}

// W (d x D) = Ut (d x d) Mo (d x D), MFMA tiles 128 x 128
template <bool RIGHT>
__global__ void __launch_bounds__(256)
k_jac_warm(const float* __restrict__ Mbar, const float* __restrict__ Ut, float* __restrict__ W,
           int64_t d, int64_t D) {
  using T = MfmaTile<128, 128, 2, 2>;
  __shared__ __align__(16) float smem[T::LDS_FLOATS];
  const int n0 = blockIdx.x * 128;  // b
  const int m0 = blockIdx.y * 128;  // j
  T tile;
  LoadK<128, 32, false, false> la(Ut, nullptr, d, m0, (int)d, (int)d, nullptr);
  if (RIGHT) {
    LoadK<128, 32, false, false> lb(Mbar, nullptr, d, n0, (int)D, (int)d, nullptr);
    tile.run(la, lb, (int)d, smem);
  } else {
    LoadR<128, 32, false> lb(Mbar, nullptr, D, n0, (int)D, (int)d);
    tile.run(la, lb, (int)d, smem);
  }
#pragma unroll
  for (int tm = 0; tm < T::TM; ++tm)
#pragma unroll
    for (int tn = 0; tn < T::TN; ++tn) {
      const int b = n0 + tile.col(tn);
      if (b >= D) continue;
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        const int j = m0 + tile.row(tm, v);
        if (j < d) W[(int64_t)j * D + b] = tile.acc[tm][tn][v];
      }
    }
}

static inline int grid1(int64_t n) {
  int64_t g = (n + 1023) / 1024;
  if (g < 1) g = 1;
  if (g > 8192) g = 8192;
  return (int)g;
}

hipError_t launch_jac_reset(const MatView& v, hipStream_t s) {
  hipLaunchKernelGGL(k_ctl_reset, dim3(1), dim3(64), 0, s, v.ctl);
  return hipGetLastError();
}

hipError_t launch_jac_init(const MatView& v, bool warm, hipStream_t s) {
  hipLaunchKernelGGL(k_ctl_reset, dim3(1), dim3(64), 0, s, v.ctl);
  if (warm) {
    hipLaunchKernelGGL(k_copy, dim3(grid1(v.d * v.d)), dim3(256), 0, s, v.Ut, v.Utw, v.d * v.d);
    dim3 grid((unsigned)((v.D + 127) / 128), (unsigned)((v.d + 127) / 128));
    if (v.right)
      hipLaunchKernelGGL(k_jac_warm<true>, grid, dim3(256), 0, s, v.Mbar, v.Ut, v.W, v.d, v.D);
    else
      hipLaunchKernelGGL(k_jac_warm<false>, grid, dim3(256), 0, s, v.Mbar, v.Ut, v.W, v.d, v.D);
  } else {
    hipError_t e = launch_eye(v.Utw, v.d, s);
    if (e != hipSuccess) return e;
    dim3 grid((unsigned)((v.D + 31) / 32), (unsigned)((v.d + 31) / 32));
    hipLaunchKernelGGL(k_jac_copy_cold, grid, dim3(256), 0, s, v.Mbar, v.W, v.d, v.D, v.right ? 1 : 0);
  }
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  return launch_gram_packed(v.W, v.D, v.d, v.D, v.Apk, v.gpart, s);
}

// ---------------------------------------------------------------------------
// one round: solve (one block per pair), update (one block per two pairs),
// apply (column chunks of every pair's rows of U^T)
// ---------------------------------------------------------------------------
// entry (x, y) of the 32 x 32 block of A whose rows are the blocks (bx0, bx1)
// and columns (by0, by1); zero for padding blocks
__device__ __forceinline__ double pk_get(const double* __restrict__ Apk, int nb, int bx, int by, int lx,
                                         int ly) {
  if (bx >= nb || by >= nb) return 0.0;
  return bx <= by ? Apk[pk_off(bx, by, nb) + lx * kJB + ly] : Apk[pk_off(by, bx, nb) + ly * kJB + lx];
}


// Rotation V of a group's Gram by one cyclic two-sided Jacobi sweep in LDS
// (fp64).  Convergence measure of a pair of rows (p, q):
//   |w_p . w_q| / max(|w_p| |w_q|,  | |w_p|^2 - |w_q|^2 |,  f^2),
//   f = 2^-10 max_k |w_k|.
// Below tol it bounds both the cosine of the two rows and the angle of the
// rotation that would still separate them, so that a converged basis is
// accurate for every singular-vector subspace whose gap in sigma^2 is above
// f^2 = 2^-20 sigma_1^2 -- far below what the fp32 data resolves -- without
// chasing orthogonality between tiny rows that fp32 rounding re-creates.
//
// A sweep of the NR x NR eigenproblem (NR = 16 NG rows) is NR - 1 steps of
// NR / 2 disjoint rotations (circle method); when the rows inside each block
// already meet the measure, only the steps between blocks are taken (16 per
// pairing of the blocks: one pairing for NG = 2, three for NG = 4).  In a
// step, a thread owns one 2 x 2 block rows {p_a, q_a} x columns {p_b, q_b}
// (a <= b) of the upper triangle of G and one 2 x 2 block of V, so that the
// update G <- J^T G J, V <- V J is in place and private to the thread; the
// rotations are computed by one wave from the diagonal 2 x 2 blocks while
// the other waves apply the previous step's rotations to V.
// Rotation J = [[c, s], [-s, c]] that diagonalises [[gpp, gpq], [gpq, gqq]]:
// t = tan(theta) = sign(d h) |h| / (|d| + sqrt(d^2 + h^2)), d = gqq - gpp,
// h = 2 gpq, c = 1 / sqrt(1 + t^2), s = c t.  t comes from the hardware fp64
// square root and reciprocal (approximations: an inexact angle only leaves a
// small share of the entry it removes for the next sweeps); c from the
// hardware reciprocal square root refined by one Newton step, so that
// c^2 + s^2 = 1 to ~1e-15 for the t used.  Gram entries of fp32 data stay far
// inside the fp64 range, so d^2 + h^2 needs no scaling.  No rotation (c = 1,
// s = 0) when gpq is zero or negligible against sqrt(gpp gqq); the choice is
// a select, so that a wave forming rotations does not branch.
__device__ __forceinline__ void jac_rotation(double gpp, double gqq, double gpq, double& c, double& s) {
  const double d = gqq - gpp, h = 2.0 * gpq;
  const double r = __builtin_amdgcn_sqrt(fma(d, d, h * h));
  const double tm = fabs(h) * __builtin_amdgcn_rcp(fabs(d) + r);
  const double t = ((d < 0.0) != (h < 0.0)) ? -tm : tm;
  const double z = fma(t, t, 1.0);
  double y = __builtin_amdgcn_rsq(z);
  y = y * fma(-0.5 * z, y * y, 1.5);                     // 1 / sqrt(z)
  const bool none = gpq == 0.0 || gpq * gpq <= 1e-34 * (gpp * gqq);
  c = none ? 1.0 : y;
  s = none ? 0.0 : y * t;
}

template <int NG>
struct JacShape {
  static constexpr int NR = NG * kJB;        // rows of a group
  static constexpr int NP = NR / 2;          // rotations per step
  static constexpr int NT = NG == 4 ? 512 : 256;   // solve threads
  static constexpr int NW = NT / 64;
  static constexpr int CROSS = (NG == 2 ? 1 : 3) * kJB;   // steps between blocks
};

// rotation j of step `step` of the circle method on NR rows (p and q in
// either order: the rotation diagonalises the 2 x 2 block either way)
template <int NR>
__host__ __device__ constexpr void full_pair(int step, int j, int& p, int& q) {
  constexpr int last = NR - 1;
  if (j == 0) { p = step; q = last; }
  else { p = (step + j) % last; q = (step - j + last) % last; }
}

// rotation j of step `step` of the steps between blocks: for NG = 4 the
// block pairings (0,1)(2,3), (0,2)(1,3), (0,3)(1,2) in turn, for NG = 2 the
// pairing (0,1); each for the 16 steps that pair row k of one block with row
// (k + step) mod 16 of the other
template <int NG>
__host__ __device__ constexpr void cross_pair(int step, int j, int& p, int& q) {
  const int rho = step >> 4, k = step & (kJB - 1), half = j >> 4, kk = j & (kJB - 1);
  int ma = 0, mb = 1;
  if (NG == 2 || rho == 0) { ma = half ? 2 : 0; mb = half ? 3 : 1; }
  else if (rho == 1) { ma = half ? 1 : 0; mb = half ? 3 : 2; }
  else { ma = half ? 1 : 0; mb = half ? 2 : 3; }
  p = kJB * ma + kk;
  q = kJB * mb + ((kk + k) & (kJB - 1));
}

template <int NG>
__host__ __device__ constexpr void step_pair(bool cross, int step, int j, int& p, int& q) {
  if (cross) cross_pair<NG>(step, j, p, q);
  else full_pair<JacShape<NG>::NR>(step, j, p, q);
}

template <int NG>
__device__ __forceinline__ bool group_empty(const int (&blk)[NG], int nb) {
  bool e = true;
#pragma unroll
  for (int m = 0; m < NG; ++m) e = e && blk[m] >= nb;
  return e;
}

// The group solve keeps G in "slot" coordinates: at every step the rows of
// rotation j sit in slots 2j (p) and 2j + 1 (q), so the data of a step moves
// to the next step's slots by a fixed permutation.  Rotation j of the next
// step is formed from slot 2 X + sx (its p) and slot 2 Y + sy (its q) of this
// step.  Circle: the rows of rotation j at step s + 1 are p_{j+1}(s) and
// q_{j-1}(s), with the ends adjusted; steps between blocks: p_j(s) and
// q_{j+1}(s), j + 1 taken within the 16 rotations of a half.
template <int NP>
__host__ __device__ constexpr void next_source(bool cross, int j, int& X, int& sx, int& Y, int& sy) {
  if (cross) {
    X = j; sx = 0; Y = (j & ~(kJB - 1)) | ((j + 1) & (kJB - 1)); sy = 1;
  } else if (j == 0) {
    X = 1; sx = 0; Y = 0; sy = 1;
  } else if (j == 1) {
    X = 2; sx = 0; Y = 0; sy = 0;
  } else if (j < NP - 1) {
    X = j + 1; sx = 0; Y = j - 1; sy = 1;
  } else {
    X = NP - 1; sx = 1; Y = NP - 2; sy = 1;
  }
}

// Tables of a group solve, fixed by the group size and the schedule (full
// circle or steps between blocks), formed at compile time:
//   pq[st][j]   rows p | q << 8 of rotation j at step st
//   pos0[row]   slot of each row at step 0
//   sig[c][P]   next slot of slot P: c = 0 a regular step; c = 1..3 the
//               changes of block pairing after steps 15, 31, 47 (four-block
//               groups, steps between blocks; the last back to step 0)
//   blk[i]      off-diagonal 2 x 2 block (a | b << 8, a < b) of work item i:
//               first the NP blocks that hold the next step's rotations (item
//               j makes rotation j), then the others in triangular order
//   dsel[j]     which source of rotation j (0: X, 1: Y) has its diagonal 2 x 2
//               block updated by item j (each diagonal block by one item)
template <int NG, bool CROSS>
struct alignas(16) JacTab {
  static constexpr int NR = JacShape<NG>::NR, NP = NR / 2, NOFF = NP * (NP - 1) / 2;
  static constexpr int STEPS = CROSS ? JacShape<NG>::CROSS : NR - 1;
  uint16_t pq[STEPS][NP];
  uint16_t blk[NOFF];
  uint8_t sig[4][NR];
  uint8_t pos0[NR];
  uint8_t dsel[NP];
};

// augmenting path for the matching of rotations j to their source pairs
template <int NP>
__host__ __device__ constexpr bool jt_augment(bool cross, int j, int* match, bool* seen) {
  int X = 0, sx = 0, Y = 0, sy = 0;
  next_source<NP>(cross, j, X, sx, Y, sy);
  const int cand[2] = {X, Y};
  for (int c = 0; c < 2; ++c) {
    const int a = cand[c];
    if (seen[a]) continue;
    seen[a] = true;
    if (match[a] < 0 || jt_augment<NP>(cross, match[a], match, seen)) {
      match[a] = j;
      return true;
    }
  }
  return false;
}

template <int NG, bool CROSS>
__host__ __device__ constexpr JacTab<NG, CROSS> make_jac_tab() {
  using T = JacTab<NG, CROSS>;
  constexpr int NP = T::NP, STEPS = T::STEPS;
  T t{};
  for (int st = 0; st < STEPS; ++st)
    for (int j = 0; j < NP; ++j) {
      int p = 0, q = 0;
      step_pair<NG>(CROSS, st, j, p, q);
      t.pq[st][j] = (uint16_t)(p | (q << 8));
    }
  for (int j = 0; j < NP; ++j) {
    t.pos0[t.pq[0][j] & 0xFF] = (uint8_t)(2 * j);
    t.pos0[t.pq[0][j] >> 8] = (uint8_t)(2 * j + 1);
    int X = 0, sx = 0, Y = 0, sy = 0;
    next_source<NP>(CROSS, j, X, sx, Y, sy);
    t.sig[0][2 * X + sx] = (uint8_t)(2 * j);
    t.sig[0][2 * Y + sy] = (uint8_t)(2 * j + 1);
  }
  if (NG == 4 && CROSS) {
    for (int c = 0; c < 3; ++c) {
      const int st = kJB * c + kJB - 1, sn = (st + 1) % STEPS;
      for (int j = 0; j < NP; ++j) {
        const int pn = t.pq[sn][j] & 0xFF, qn = t.pq[sn][j] >> 8;
        for (int i = 0; i < NP; ++i) {
          const int po = t.pq[st][i] & 0xFF, qo = t.pq[st][i] >> 8;
          if (po == pn) t.sig[1 + c][2 * i] = (uint8_t)(2 * j);
          if (qo == pn) t.sig[1 + c][2 * i + 1] = (uint8_t)(2 * j);
          if (po == qn) t.sig[1 + c][2 * i] = (uint8_t)(2 * j + 1);
          if (qo == qn) t.sig[1 + c][2 * i + 1] = (uint8_t)(2 * j + 1);
        }
      }
    }
  }
  int next = NP;
  for (int a = 0; a < NP; ++a)
    for (int b = a + 1; b < NP; ++b) {
      int slot = -1;
      for (int j = 0; j < NP; ++j) {
        int X = 0, sx = 0, Y = 0, sy = 0;
        next_source<NP>(CROSS, j, X, sx, Y, sy);
        if ((X < Y ? X : Y) == a && (X < Y ? Y : X) == b) slot = j;
      }
      if (slot < 0) slot = next++;
      t.blk[slot] = (uint16_t)(a | (b << 8));
    }
  // every pair is a source of exactly two rotations: a perfect matching of
  // rotations to pairs exists (the sources form even cycles)
  int match[NP] = {};
  for (int a = 0; a < NP; ++a) match[a] = -1;
  for (int j = 0; j < NP; ++j) {
    bool seen[NP] = {};
    jt_augment<NP>(CROSS, j, match, seen);
  }
  for (int a = 0; a < NP; ++a) {
    const int j = match[a];
    int X = 0, sx = 0, Y = 0, sy = 0;
    next_source<NP>(CROSS, j, X, sx, Y, sy);
    t.dsel[j] = (uint8_t)(a == X ? 0 : 1);
  }
  return t;
}

__constant__ JacTab<2, false> kJacTab2f = make_jac_tab<2, false>();
__constant__ JacTab<2, true> kJacTab2c = make_jac_tab<2, true>();
__constant__ JacTab<4, false> kJacTab4f = make_jac_tab<4, false>();
__constant__ JacTab<4, true> kJacTab4c = make_jac_tab<4, true>();

template <int NG, bool CROSS>
__device__ __forceinline__ const JacTab<NG, CROSS>& jac_tab();
template <>
__device__ __forceinline__ const JacTab<2, false>& jac_tab<2, false>() { return kJacTab2f; }
template <>
__device__ __forceinline__ const JacTab<2, true>& jac_tab<2, true>() { return kJacTab2c; }
template <>
__device__ __forceinline__ const JacTab<4, false>& jac_tab<4, false>() { return kJacTab4f; }
template <>
__device__ __forceinline__ const JacTab<4, true>& jac_tab<4, true>() { return kJacTab4c; }

// LDS of a group solve; the rotation of U^T reuses it for V - I (fp32).
// Only the upper triangle of G is kept (two copies, read one / write the
// other by step parity); rows have an even stride, so that the two entries
// of a 2 x 2 block row are one 16-byte load.
template <int NR>
__device__ __forceinline__ int gat(int P, int Q) {
  return P * (NR + 2) + Q;
}
template <int NG>
struct SolveLds {
  static constexpr int NR = JacShape<NG>::NR, NP = NR / 2, NPK = NR * (NR + 2);
  // past the matrix: a place for the stores of lanes without a block
  static constexpr int NDUM = 4 * (JacShape<NG>::NT - NP * (NP - 1) / 2 + 64);
  double Gp[2][NPK + NDUM];
  double V[NR][NR + 1];              // row coordinates
  double2 rot[2][64];                // (c, s) of the rotations of two consecutive steps (lanes
                                     // NP.. of wave 0 store theirs past the real ones)
  double red[JacShape<NG>::NW], redw[JacShape<NG>::NW];
  uint32_t pq[NR * NP / 2];          // the step table (uint16 pairs)
};
template <int NG>
union JacLds {
  SolveLds<NG> s;
  float Va[JacShape<NG>::NR][JacShape<NG>::NR + 1];
};

// One cyclic sweep over the rotations of the group, on G in slot
// coordinates (see JacTab), V <- V J in row coordinates.  Work items: the
// NP (NP + 1) / 2 upper 2 x 2 blocks of G and the NR / 2 x NP 2 x 2 blocks
// of V (rows 2 i, 2 i + 1; columns of rotation j), spread over 256 threads
// (a few per thread: four waves keep the per-step scalar work of the loop
// small).  One barrier per step: the items that produce the entry G[p'][q']
// of a next-step rotation (all in wave 0) also form its new diagonal entries
// from the old diagonal blocks of its two source rotations and compute it.
template <int NG, bool CROSS>
__device__ __forceinline__ void sweep_group(SolveLds<NG>& L, int max_inner) {
  using SH = JacShape<NG>;
  using TB = JacTab<NG, CROSS>;
  constexpr int NR = SH::NR, NT = SH::NT, NP = NR / 2, NOFF = NP * (NP - 1) / 2, STEPS = TB::STEPS;
  constexpr int NPK = SolveLds<NG>::NPK;
  constexpr int VB = (NR / 2) * NP / NT;            // V items per thread
  static_assert(NOFF <= NT && VB * NT == (NR / 2) * NP, "one G item, whole V items per thread");
  const TB& tab = jac_tab<NG, CROSS>();
  const int tid = threadIdx.x, lane = lane_id(), w = wave_id();
  // this thread's off-diagonal 2 x 2 block (a, b), a < b, of G: the LDS
  // offsets of its two rows now and of its four entries at the next step
  // (threads without a block read block 0 and store into the dummy slots)
  const bool has = tid < NOFF;
  const uint32_t be = tab.blk[has ? tid : 0];
  const int ua = be & 0xFF, ub = be >> 8;
  const int rd0 = gat<NR>(2 * ua, 2 * ub), rd1 = gat<NR>(2 * ua + 1, 2 * ub);
  auto dest4 = [&](const uint8_t* sg, int (&wo)[4]) {
#pragma unroll
    for (int x = 0; x < 2; ++x)
#pragma unroll
      for (int y = 0; y < 2; ++y) {
        const int Pn = sg[2 * ua + x], Qn = sg[2 * ub + y];
        wo[2 * x + y] = has ? gat<NR>(min(Pn, Qn), max(Pn, Qn)) : NPK + 4 * (tid - NOFF) + 2 * x + y;
      }
  };
  int wr[4];
  dest4(tab.sig[0], wr);
  // wave 0: lane j < NP forms rotation j of the next step from entry (2 X +
  // sx, 2 Y + sy) of its block and the diagonal blocks of X and Y, and
  // stores the new diagonal block of one of them (dsel); the other lanes
  // repeat lane 0's work into the dummy slots
  const int oj = lane < NP ? lane : 0;
  int ox = 0, osx = 0, oy = 0, osy = 0;
  next_source<NP>(CROSS, oj, ox, osx, oy, osy);
  const int osel = ox == ua ? 2 * osx + osy : 2 * osy + osx;
  const int odx = gat<NR>(2 * ox, 2 * ox), ody = gat<NR>(2 * oy, 2 * oy);
  const int dsel = tab.dsel[oj], dp = dsel == 0 ? ox : oy;
  const bool ownr = w == 0 && lane < NP;
  auto dest3 = [&](const uint8_t* sg, int (&wo)[3]) {
    const int Pn = sg[2 * dp], Qn = sg[2 * dp + 1];
    wo[0] = ownr ? gat<NR>(Pn, Pn) : NPK + 4 * (NT - NOFF + lane);
    wo[1] = ownr ? gat<NR>(min(Pn, Qn), max(Pn, Qn)) : NPK + 4 * (NT - NOFF + lane) + 1;
    wo[2] = ownr ? gat<NR>(Qn, Qn) : NPK + 4 * (NT - NOFF + lane) + 2;
  };
  int wd[3];
  dest3(tab.sig[0], wd);
  const int vb = tid % NP, vr0 = 2 * (tid / NP);
  // J^T B J of a diagonal 2 x 2 block (g00, g01, g11) by its own rotation
  auto diag_update = [](double g00, double g01, double g11, double c, double sn, double& n00, double& n01,
                        double& n11) {
    const double t00 = g00 * c - g01 * sn, t01 = g00 * sn + g01 * c;
    const double t10 = g01 * c - g11 * sn, t11 = g01 * sn + g11 * c;
    n00 = c * t00 - sn * t10;
    n01 = c * t01 - sn * t11;
    n11 = sn * t01 + c * t11;
  };
  // the rotations of a step from its copy of G (slots 2j, 2j + 1): step 0
  // and the steps after a change of pairing
  auto rotations_from_g = [&](int buf) {
    if (w == 0 && lane < NP) {
      const double* Gc = L.Gp[buf];
      const int o = gat<NR>(2 * lane, 2 * lane);
      double c, sn;
      jac_rotation(Gc[o], Gc[o + NR + 3], Gc[o + 1], c, sn);
      L.rot[buf][lane] = double2{c, sn};
    }
  };
  rotations_from_g(0);
  __syncthreads();
  const uint16_t* pq16 = reinterpret_cast<const uint16_t*>(L.pq);
  for (int inner = 0; inner < max_inner; ++inner) {
    for (int st = 0; st < STEPS; ++st) {
      const int pcur = (inner * STEPS + st) & 1, pnxt = pcur ^ 1;
      const bool more = st + 1 < STEPS || inner + 1 < max_inner;
      const bool change = NG == 4 && CROSS && (st & (kJB - 1)) == kJB - 1;
      const double* Gc = L.Gp[pcur];
      double* Gn = L.Gp[pnxt];
      const double2* rc = L.rot[pcur];
      // every load of the step first (the stores go to the other copy of G
      // and to this thread's own entries of V), then the arithmetic, then the
      // stores: one LDS round trip per step
      const double2 ra = rc[ua], rb = rc[ub];
      const double2 g0 = *reinterpret_cast<const double2*>(Gc + rd0);
      const double2 g1 = *reinterpret_cast<const double2*>(Gc + rd1);
      double dx0 = 0.0, dx1 = 0.0, dx2 = 0.0, dy0 = 0.0, dy1 = 0.0, dy2 = 0.0;
      if (w == 0) {
        dx0 = Gc[odx]; dx1 = Gc[odx + 1]; dx2 = Gc[odx + NR + 3];
        dy0 = Gc[ody]; dy1 = Gc[ody + 1]; dy2 = Gc[ody + NR + 3];
      }
      const uint32_t e = pq16[st * NP + vb];
      const int pv = e & 0xFF, qv = e >> 8;
      const double2 rv = rc[vb];
      double vv[VB][4];
#pragma unroll
      for (int k = 0; k < VB; ++k) {
        const int vr = vr0 + k * (2 * NT / NP);
        vv[k][0] = L.V[vr][pv]; vv[k][1] = L.V[vr][qv];
        vv[k][2] = L.V[vr + 1][pv]; vv[k][3] = L.V[vr + 1][qv];
      }
      if (change) {
        const uint8_t* sg = tab.sig[1 + (st >> 4)];
        dest4(sg, wr);
        dest3(sg, wd);
      }
      // off-diagonal block: G <- J_a^T G J_b
      const double ca = ra.x, sa = ra.y, cb = rb.x, sb = rb.y;
      const double t00 = g0.x * cb - g0.y * sb, t01 = g0.x * sb + g0.y * cb;
      const double t10 = g1.x * cb - g1.y * sb, t11 = g1.x * sb + g1.y * cb;
      const double n00 = ca * t00 - sa * t10, n01 = ca * t01 - sa * t11;
      const double n10 = sa * t00 + ca * t10, n11 = sa * t01 + ca * t11;
      if (w == 0) {
        const double2 rx = ox == ua ? ra : rb, ry = ox == ua ? rb : ra;
        double x00, x01, x11, y00, y01, y11;
        diag_update(dx0, dx1, dx2, rx.x, rx.y, x00, x01, x11);
        diag_update(dy0, dy1, dy2, ry.x, ry.y, y00, y01, y11);
        if (more && !change) {
          const double gpq = osel == 0 ? n00 : (osel == 1 ? n01 : (osel == 2 ? n10 : n11));
          double c, sn;
          jac_rotation(osx == 0 ? x00 : x11, osy == 0 ? y00 : y11, gpq, c, sn);
          L.rot[pnxt][lane] = double2{c, sn};
        }
        Gn[wd[0]] = dsel == 0 ? x00 : y00;
        Gn[wd[1]] = dsel == 0 ? x01 : y01;
        Gn[wd[2]] = dsel == 0 ? x11 : y11;
      }
      Gn[wr[0]] = n00;
      Gn[wr[1]] = n01;
      Gn[wr[2]] = n10;
      Gn[wr[3]] = n11;
      {
        // V <- V J on rows (row coordinates): columns p, q of rotation vb
        const double cv = rv.x, sv = rv.y;
#pragma unroll
        for (int k = 0; k < VB; ++k) {
          const int vr = vr0 + k * (2 * NT / NP);
          L.V[vr][pv] = vv[k][0] * cv - vv[k][1] * sv;
          L.V[vr][qv] = vv[k][0] * sv + vv[k][1] * cv;
          L.V[vr + 1][pv] = vv[k][2] * cv - vv[k][3] * sv;
          L.V[vr + 1][qv] = vv[k][2] * sv + vv[k][3] * cv;
        }
      }
      __syncthreads();
      if (more && change) {
        rotations_from_g(pnxt);
        __syncthreads();
        dest4(tab.sig[0], wr);
        dest3(tab.sig[0], wd);
      }
    }
  }
}

template <int NG>
__device__ __forceinline__ void solve_group(const double* __restrict__ Apk, JacCtl* __restrict__ ctl, int round,
                                            int seats, int nb, float tol, int max_inner, double floor_rel2,
                                            float* __restrict__ Vout, double* __restrict__ V64,
                                            int* __restrict__ skip, int grp, SolveLds<NG>& L) {
  using SH = JacShape<NG>;
  constexpr int NR = SH::NR, NT = SH::NT, NW = SH::NW;
  int blk[NG];
  group_blocks<NG>(round, grp, seats, blk);
  const int tid = threadIdx.x, lane = lane_id(), w = wave_id();
  if (group_empty<NG>(blk, nb)) {
    if (tid == 0) skip[grp] = 1;
    return;
  }
  double* red = L.red;
  double* redw = L.redw;
  constexpr int NE = NR * NR / NT;
  const double rm_prev = __longlong_as_double((long long)ctl->rowmax2_bits);
  // the group's diagonal NR x NR block of A; element k of this thread is
  // (x, y) = (tid / NR + k (NT / NR), tid % NR)
  double g[NE];
#pragma unroll
  for (int k = 0; k < NE; ++k) {
    const int e = tid + NT * k, x = e / NR, y = e % NR;
    g[k] = pk_get(Apk, nb, blk[x / kJB], blk[y / kJB], x % kJB, y % kJB);
  }
  // the diagonal goes through V's storage (overwritten by V = I below)
  double* dg = &L.V[0][0];
  double dmax = 0.0;
#pragma unroll
  for (int k = 0; k < NE; ++k) {
    const int e = tid + NT * k, x = e / NR, y = e % NR;
    if (x == y) {
      dg[x] = g[k];
      dmax = fmax(dmax, g[k]);
    }
  }
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) dmax = fmax(dmax, __shfl_xor(dmax, o, 64));
  if (lane == 0) red[w] = dmax;
  __syncthreads();
  dmax = 0.0;
#pragma unroll
  for (int i = 0; i < NW; ++i) dmax = fmax(dmax, red[i]);
  __syncthreads();
  if (tid == 0 && dmax > 0.0)
    atomicMax((unsigned long long*)&ctl->rowmax2_bits, (unsigned long long)__double_as_longlong(dmax));
  const double rowmax2 = fmax(dmax, rm_prev);
  const double floor2 = floor_rel2 * rowmax2;
  double m2 = 0.0, mw2 = 0.0;   // all pairs / pairs inside one block
#pragma unroll
  for (int k = 0; k < NE; ++k) {
    const int e = tid + NT * k, x = e / NR, y = e % NR;
    if (x < y) {
      // (g / max(sqrt(gxx gyy), |gxx - gyy|, floor))^2, all terms squared
      const double gxx = dg[x], gyy = dg[y], df = gxx - gyy;
      const double den2 = fmax(fmax(gxx * gyy, df * df), floor2 * floor2);
      if (den2 > 0.0) {
        const double q2 = g[k] * g[k] / den2;
        m2 = fmax(m2, q2);
        if (x / kJB == y / kJB) mw2 = fmax(mw2, q2);
      }
    }
  }
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    m2 = fmax(m2, __shfl_xor(m2, o, 64));
    mw2 = fmax(mw2, __shfl_xor(mw2, o, 64));
  }
  if (lane == 0) { red[w] = m2; redw[w] = mw2; }
  __syncthreads();
  m2 = 0.0;
  mw2 = 0.0;
#pragma unroll
  for (int i = 0; i < NW; ++i) {
    m2 = fmax(m2, red[i]);
    mw2 = fmax(mw2, redw[i]);
  }
  const double m = sqrt(m2);
  // rows inside each block already orthogonal: only the steps between blocks
  const bool cross = sqrt(mw2) <= (double)tol;
  if (tid == 0) atomicMax(&ctl->sweep_max_bits, __float_as_uint((float)m));
  if (m <= (double)tol) {
    if (tid == 0) skip[grp] = 1;
    return;
  }
  // the step table into LDS; G (slot coordinates, upper, copy 0); V = I
  {
    const uint8_t* pos0 = cross ? jac_tab<NG, true>().pos0 : jac_tab<NG, false>().pos0;
    const uint32_t* src = cross ? reinterpret_cast<const uint32_t*>(jac_tab<NG, true>().pq)
                                : reinterpret_cast<const uint32_t*>(jac_tab<NG, false>().pq);
    const int words = (cross ? JacTab<NG, true>::STEPS : JacTab<NG, false>::STEPS) * (NR / 2) / 2;
    for (int i = tid; i < words; i += NT) L.pq[i] = src[i];
    __syncthreads();   // dg (in V's storage) is read above by every thread
#pragma unroll
    for (int k = 0; k < NE; ++k) {
      const int e = tid + NT * k, x = e / NR, y = e % NR;
      const int P = pos0[x], Q = pos0[y];
      if (P <= Q) L.Gp[0][gat<NR>(P, Q)] = g[k];
      L.V[x][y] = x == y ? 1.0 : 0.0;
    }
    __syncthreads();
  }
  if (cross) sweep_group<NG, true>(L, max_inner);
  else sweep_group<NG, false>(L, max_inner);
  float* vo = Vout + (int64_t)grp * NR * NR;
  double* vd = V64 + (int64_t)grp * NR * NR;
#pragma unroll
  for (int k = 0; k < NE; ++k) {
    const int e = tid + NT * k;
    vo[e] = (float)L.V[e / NR][e % NR];
    vd[e] = L.V[e / NR][e % NR];
  }
  if (tid == 0) skip[grp] = 0;
}

// columns of U^T rotated by one workgroup of 256 threads (in proportion for
// the larger workgroups beside the solves of four-block groups)
constexpr int JAC_CHUNK = 512;

// rows of the group in U^T <- V^T rows on this block's chunk, computed as
// w + (V - I)^T w (fp32 MFMA, NR / 32 output tiles of 32 rows, K = NR).  The
// k index is permuted so that the B operand held by each lane is exactly the
// set of rows that lane outputs: k slot 16 h + kk of a lane is physical row
// 32 h + mfma32_row(kk, lane), which is register kk of output tile h.
template <int NG>
__device__ __forceinline__ void apply_chunk(float* __restrict__ Utw, int64_t d, const float* __restrict__ Vin,
                                            const int* __restrict__ skip, int round, int seats, int nb,
                                            int grp, int chunk, int width,
                                            float (*Va)[JacShape<NG>::NR + 1]) {
  constexpr int NR = JacShape<NG>::NR;
  if (skip[grp]) return;
  int blk[NG];
  group_blocks<NG>(round, grp, seats, blk);
  if (group_empty<NG>(blk, nb)) return;
  const int lane = lane_id(), w = wave_id();
  const int l32 = lane & 31, lh4 = 4 * (lane >> 5);
  const float* V = Vin + (int64_t)grp * NR * NR;
  constexpr int KS = NR / 2;   // k slots of the two-row MFMA steps
  for (int e = threadIdx.x; e < NR * NR; e += blockDim.x) {
    const int i = e / NR, j = e % NR;
    Va[i][j] = V[e] - (i == j ? 1.0f : 0.0f);
  }
  __syncthreads();
  // slot kk is row blk[m] * 16 + r of U^T with m = slot_block(kk) and
  // r = slot_row(kk) + 4 (lane / 32)
  auto slot_block = [](int kk) { return 2 * (kk >> 4) + ((kk & 15) >= 8 ? 1 : 0); };
  auto slot_row = [](int kk) { return 8 * (((kk & 15) >> 2) & 1) + (kk & 3); };
  // d <= 8192: element offsets of U^T fit 32 bits, so every access is the
  // uniform base plus a 32-bit lane offset
  const int dd = (int)d;
  int first[NG];   // row index of r = 4 (lane / 32) in each member block, -1 if padding
#pragma unroll
  for (int m = 0; m < NG; ++m) first[m] = blk[m] < nb ? blk[m] * kJB + lh4 : -1;
  auto at = [&](int row, int col) -> float* {
    return reinterpret_cast<float*>(reinterpret_cast<char*>(Utw) + ((uint32_t)(row * dd + col) << 2));
  };
  const int c0 = chunk * width;
  const int span = 32 * (int)(blockDim.x >> 6);   // columns per pass, 32 per wave
  for (int it = 0; it < width; it += span) {
    const int cb = c0 + it + w * 32;
    if (cb >= dd) break;
    const int cc = cb + l32;
    const bool cok = cc < dd;
    float b[KS];
#pragma unroll
    for (int kk = 0; kk < KS; ++kk) {
      const int f = first[slot_block(kk)], row = f + slot_row(kk);
      b[kk] = (cok && f >= 0 && row < dd) ? *at(row, cc) : 0.f;
    }
    // output tile h: rows 32 h + mfma32_row(v, lane), held by slot 16 h + v
#pragma unroll
    for (int h = 0; h < NR / 32; ++h) {
      f32x16 acc;
#pragma unroll
      for (int v = 0; v < 16; ++v) acc[v] = 0.f;
#pragma unroll
      for (int kk = 0; kk < KS; ++kk) {
        const int pr = 32 * (kk >> 4) + mfma32_row(kk & 15, lane);
        acc = mfma32(Va[pr][32 * h + l32], b[kk], acc);
      }
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        const int kk = 16 * h + v;
        const int f = first[slot_block(kk)], row = f + slot_row(kk);
        if (cok && f >= 0 && row < dd) *at(row, cc) = b[kk] + acc[v];
      }
    }
  }
}

// A <- J^T A J: the NR x NR block of rows of group g and columns of group h
// (g <= h) becomes V_g^T A_gh V_h (fp64 MFMA 16x16x4; wave w computes the
// (NR / 2) x (NR / 2) quadrant (w / 2, w % 2) of each product).  The 16 x 16
// blocks of A are read and written whole (coalesced) through one LDS tile;
// blocks below the diagonal are not stored, so each stored block is written
// by exactly one workgroup.  A group whose V is the identity skips its
// product.
template <int NG>
__device__ __forceinline__ void update_pair(double* __restrict__ Apk, const double* __restrict__ V64,
                                            const int* __restrict__ skip, int round, int seats, int nb, int groups,
                                            int bid, double (*S)[JacShape<NG>::NR + 1]) {
  constexpr int NR = JacShape<NG>::NR, TW = NR / 32;   // 16 x 16 tiles per quadrant side
  int g = 0, rem = bid;
  while (rem >= groups - g) {
    rem -= groups - g;
    ++g;
  }
  const int h = g + rem;
  const bool sg = skip[g] != 0, sh = skip[h] != 0;
  if (sg && sh) return;
  int bg[NG], bh[NG];
  group_blocks<NG>(round, g, seats, bg);
  group_blocks<NG>(round, h, seats, bh);
  const int tid = threadIdx.x, lane = lane_id(), w = wave_id();
  const int er = tid / kJB, ec = tid % kJB;
  const int R0 = (w >> 1) * (NR / 2), C0 = (w & 1) * (NR / 2), li = lane & 15, lk = lane >> 4;
  double sv[NG * NG];
#pragma unroll
  for (int mb = 0; mb < NG * NG; ++mb) {
    const int bx = bg[mb / NG], by = bh[mb % NG];
    sv[mb] = (bx < nb && by < nb) ? Apk[(bx <= by ? pk_off(bx, by, nb) : pk_off(by, bx, nb)) + tid] : 0.0;
  }
  // B operand of T = A_gh V_h, fetched while the blocks land in LDS
  double vb[NR / 4][TW];
  if (!sh) {
    const double* vh = V64 + (int64_t)h * NR * NR;
#pragma unroll
    for (int k = 0; k < NR / 4; ++k)
#pragma unroll
      for (int j = 0; j < TW; ++j) vb[k][j] = vh[(4 * k + lk) * NR + C0 + 16 * j + li];
  }
#pragma unroll
  for (int mb = 0; mb < NG * NG; ++mb) {
    const int mx = mb / NG, my = mb % NG;
    if (bg[mx] <= bh[my]) S[kJB * mx + er][kJB * my + ec] = sv[mb];
    else S[kJB * mx + ec][kJB * my + er] = sv[mb];
  }
  __syncthreads();
  f64x4 acc[TW][TW];
  if (!sh) {
#pragma unroll
    for (int i = 0; i < TW; ++i)
#pragma unroll
      for (int j = 0; j < TW; ++j) acc[i][j] = f64x4{0.0, 0.0, 0.0, 0.0};
#pragma unroll
    for (int k = 0; k < NR / 4; ++k)
#pragma unroll
      for (int i = 0; i < TW; ++i) {
        const double x = S[R0 + 16 * i + li][4 * k + lk];
#pragma unroll
        for (int j = 0; j < TW; ++j) acc[i][j] = mfma64(x, vb[k][j], acc[i][j]);
      }
    __syncthreads();
#pragma unroll
    for (int i = 0; i < TW; ++i)
#pragma unroll
      for (int j = 0; j < TW; ++j)
#pragma unroll
        for (int v = 0; v < 4; ++v) S[R0 + 16 * i + 4 * v + lk][C0 + 16 * j + li] = acc[i][j][v];
    __syncthreads();
  }
  if (!sg) {
    const double* vg = V64 + (int64_t)g * NR * NR;
    double va[NR / 4][TW];
#pragma unroll
    for (int k = 0; k < NR / 4; ++k)
#pragma unroll
      for (int i = 0; i < TW; ++i) va[k][i] = vg[(4 * k + lk) * NR + R0 + 16 * i + li];
#pragma unroll
    for (int i = 0; i < TW; ++i)
#pragma unroll
      for (int j = 0; j < TW; ++j) acc[i][j] = f64x4{0.0, 0.0, 0.0, 0.0};
#pragma unroll
    for (int k = 0; k < NR / 4; ++k)
#pragma unroll
      for (int j = 0; j < TW; ++j) {
        const double y = S[4 * k + lk][C0 + 16 * j + li];
#pragma unroll
        for (int i = 0; i < TW; ++i) acc[i][j] = mfma64(va[k][i], y, acc[i][j]);
      }
    __syncthreads();
#pragma unroll
    for (int i = 0; i < TW; ++i)
#pragma unroll
      for (int j = 0; j < TW; ++j)
#pragma unroll
        for (int v = 0; v < 4; ++v) S[R0 + 16 * i + 4 * v + lk][C0 + 16 * j + li] = acc[i][j][v];
    __syncthreads();
  }
#pragma unroll
  for (int mb = 0; mb < NG * NG; ++mb) {
    const int mx = mb / NG, my = mb % NG;
    const int bx = bg[mx], by = bh[my];
    if (bx >= nb || by >= nb) continue;
    if (bx <= by) Apk[pk_off(bx, by, nb) + tid] = S[kJB * mx + er][kJB * my + ec];
    else if (g != h) Apk[pk_off(by, bx, nb) + tid] = S[kJB * mx + ec][kJB * my + er];
  }
}

// the group solves of one round
template <int NG>
__global__ void __launch_bounds__(JacShape<NG>::NT)
k_jac_solve(const double* __restrict__ Apk, JacCtl* __restrict__ ctl, int round, int seats, int nb, float tol,
            int max_inner, double floor_rel2, float* __restrict__ Vout, double* __restrict__ V64,
            int* __restrict__ skip) {
  if (ctl->converged) return;
  __shared__ SolveLds<NG> lds;
  solve_group<NG>(Apk, ctl, round, seats, nb, tol, max_inner, floor_rel2, Vout, V64, skip, blockIdx.x, lds);
}

// A <- J^T A J over all pairs of groups
template <int NG>
__global__ void __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(4, 4)))
k_jac_update(double* __restrict__ Apk, const double* __restrict__ V64, const int* __restrict__ skip,
             const JacCtl* __restrict__ ctl, int round, int seats, int nb, int groups) {
  if (ctl->converged) return;
  __shared__ double S[JacShape<NG>::NR][JacShape<NG>::NR + 1];
  update_pair<NG>(Apk, V64, skip, round, seats, nb, groups, blockIdx.x, S);
}

// the group solves of round `round` (workgroups [0, groups)) together with
// the rotation of U^T rows by the previous round's V (the rest): the rotation
// does not depend on the new solves, and the solves leave most of the chip idle
template <int NG>
__global__ void __launch_bounds__(JacShape<NG>::NT)
k_jac_solve_apply(const double* __restrict__ Apk, JacCtl* __restrict__ ctl, int round, int seats, int nb,
                  float tol, int max_inner, double floor_rel2, float* __restrict__ Vout,
                  double* __restrict__ V64, int* __restrict__ skip, float* __restrict__ Utw, int64_t d,
                  const float* __restrict__ Vprev, const int* __restrict__ skip_prev, int groups, int chunks,
                  int width) {
  if (ctl->converged) return;
  __shared__ JacLds<NG> lds;
  const int b = blockIdx.x;
  if (b < groups) {
    solve_group<NG>(Apk, ctl, round, seats, nb, tol, max_inner, floor_rel2, Vout, V64, skip, b, lds.s);
  } else {
    const int idx = b - groups;
    apply_chunk<NG>(Utw, d, Vprev, skip_prev, round - 1, seats, nb, idx / chunks, idx % chunks, width, lds.Va);
  }
}

// U^T rows of the last round of a sweep
template <int NG>
__global__ void __launch_bounds__(256)
k_jac_apply(float* __restrict__ Utw, int64_t d, const float* __restrict__ V32, const int* __restrict__ skip,
            const JacCtl* __restrict__ ctl, int round, int seats, int nb, int chunks) {
  if (ctl->converged) return;
  __shared__ float Va[JacShape<NG>::NR][JacShape<NG>::NR + 1];
  apply_chunk<NG>(Utw, d, V32, skip, round, seats, nb, blockIdx.x / chunks, blockIdx.x % chunks, JAC_CHUNK, Va);
}

// per-round buffers alternate between two copies (round parity), so that a
// round's solves can run while the previous round's rotations are applied
struct RoundBufs {
  float* V32;
  double* V64;
  int* skip;
};
static RoundBufs round_bufs(const MatView& v, int round) {
  const int64_t vb = jac_vbuf(v.d), groups = jac_groups(v.d), par = round & 1;
  return {v.Vrot + par * vb, v.V64 + par * vb, v.skip + par * groups};
}

template <int NG>
static hipError_t update_ng(const MatView& v, int round, hipStream_t s) {
  const int nb = jac_blocks(v.d), groups = jac_groups(v.d), seats = jac_seats(v.d);
  const RoundBufs rb = round_bufs(v, round);
  hipLaunchKernelGGL(k_jac_update<NG>, dim3((unsigned)(groups * (groups + 1) / 2)), dim3(256), 0, s, v.Apk,
                     rb.V64, rb.skip, v.ctl, round, seats, nb, groups);
  return hipGetLastError();
}
hipError_t launch_jac_update(const MatView& v, int round, hipStream_t s) {
  return jac_group_blocks(v.d) == 4 ? update_ng<4>(v, round, s) : update_ng<2>(v, round, s);
}

template <int NG>
static hipError_t solve_apply_ng(const MatView& v, int round, float tol, int max_inner, double floor_rel2,
                                 hipStream_t s) {
  const int nb = jac_blocks(v.d), groups = jac_groups(v.d), seats = jac_seats(v.d);
  const int width = JAC_CHUNK * JacShape<NG>::NT / 256;
  const int chunks = (int)((v.d + width - 1) / width);
  const RoundBufs rb = round_bufs(v, round), pb = round_bufs(v, round - 1);
  hipLaunchKernelGGL(k_jac_solve_apply<NG>, dim3((unsigned)(groups + groups * chunks)), dim3(JacShape<NG>::NT),
                     0, s, v.Apk, v.ctl, round, seats, nb, tol, max_inner, floor_rel2, rb.V32, rb.V64, rb.skip,
                     v.Utw, v.d, pb.V32, pb.skip, groups, chunks, width);
  return hipGetLastError();
}
hipError_t launch_jac_solve_apply(const MatView& v, int round, float tol, int max_inner, double floor_rel2,
                                  hipStream_t s) {
  return jac_group_blocks(v.d) == 4 ? solve_apply_ng<4>(v, round, tol, max_inner, floor_rel2, s)
                                    : solve_apply_ng<2>(v, round, tol, max_inner, floor_rel2, s);
}

template <int NG>
static hipError_t apply_ng(const MatView& v, int round, hipStream_t s) {
  const int nb = jac_blocks(v.d), groups = jac_groups(v.d), seats = jac_seats(v.d);
  const int chunks = (int)((v.d + JAC_CHUNK - 1) / JAC_CHUNK);
  const RoundBufs rb = round_bufs(v, round);
  hipLaunchKernelGGL(k_jac_apply<NG>, dim3((unsigned)(groups * chunks)), dim3(256), 0, s, v.Utw, v.d, rb.V32,
                     rb.skip, v.ctl, round, seats, nb, chunks);
  return hipGetLastError();
}
hipError_t launch_jac_apply(const MatView& v, int round, hipStream_t s) {
  return jac_group_blocks(v.d) == 4 ? apply_ng<4>(v, round, s) : apply_ng<2>(v, round, s);
}

template <int NG>
static hipError_t solve_ng(const MatView& v, int round, float tol, int max_inner, double floor_rel2,
                           hipStream_t s) {
  const int nb = jac_blocks(v.d), groups = jac_groups(v.d), seats = jac_seats(v.d);
  const RoundBufs rb = round_bufs(v, round);
  hipLaunchKernelGGL(k_jac_solve<NG>, dim3(groups), dim3(JacShape<NG>::NT), 0, s, v.Apk, v.ctl, round, seats, nb,
                     tol, max_inner, floor_rel2, rb.V32, rb.V64, rb.skip);
  return hipGetLastError();
}
hipError_t launch_jac_solve(const MatView& v, int round, float tol, int max_inner, double floor_rel2,
                            hipStream_t s) {
  return jac_group_blocks(v.d) == 4 ? solve_ng<4>(v, round, tol, max_inner, floor_rel2, s)
                                    : solve_ng<2>(v, round, tol, max_inner, floor_rel2, s);
}

__global__ void k_jac_check(JacCtl* ctl, float tol) {
  if (threadIdx.x != 0 || ctl->converged) return;
  if (ctl->sweeps < (uint32_t)kHistory) ctl->history[ctl->sweeps] = ctl->sweep_max_bits;
  ctl->sweeps += 1;
  if (__uint_as_float(ctl->sweep_max_bits) <= tol) ctl->converged = 1;
  ctl->sweep_max_bits = 0;
}

hipError_t launch_jac_check(const MatView& v, float tol, hipStream_t s) {
  hipLaunchKernelGGL(k_jac_check, dim3(1), dim3(64), 0, s, v.ctl, tol);
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// finish: sigma_j = sqrt(A_jj), sort descending, permute U^T rows
// ---------------------------------------------------------------------------
__device__ __forceinline__ void diag_sqrt_at(const double* __restrict__ Apk, int64_t d, int nb,
                                             float* __restrict__ sig, int64_t j) {
  if (j >= d) return;
  const int b = (int)(j / kJB), l = (int)(j % kJB);
  sig[j] = (float)sqrt(fmax(Apk[pk_off(b, b, nb) + l * (kJB + 1)], 0.0));
}
__global__ void k_diag_sqrt(const double* __restrict__ Apk, int64_t d, int nb, float* __restrict__ sig) {
  diag_sqrt_at(Apk, d, nb, sig, blockIdx.x * (int64_t)blockDim.x + threadIdx.x);
}

// the descending order of sigma (ties to the smaller index) by one block, in
// n_pad keys of LDS; the identity when `identity` (a sweep enqueued after the
// refresh converged: the reordering then only moves the data to the other
// buffer of the pair, so that every enqueued sweep leaves its result in the
// same buffer whether it ran or not)
__device__ __forceinline__ void sort_desc_block(const float* __restrict__ sig, int d, int n_pad,
                                                int* __restrict__ perm, uint64_t* keys, bool identity = false) {
  if (identity) {
    for (int i = threadIdx.x; i < d; i += blockDim.x) perm[i] = i;
    return;
  }
  for (int i = threadIdx.x; i < n_pad; i += blockDim.x) {
    if (i < d) keys[i] = ((uint64_t)(~float_order(sig[i])) << 32) | (uint32_t)i;
    else keys[i] = ~0ull;
  }
  __syncthreads();
  bitonic_sort(keys, n_pad);
  for (int i = threadIdx.x; i < d; i += blockDim.x) perm[i] = (int)(keys[i] & 0xFFFFFFFFu);
}
__global__ void __launch_bounds__(1024)
k_sort_desc(const float* __restrict__ sig, int d, int n_pad, int* __restrict__ perm,
            const JacCtl* __restrict__ ctl) {
  extern __shared__ __align__(16) unsigned char dyn[];
  sort_desc_block(sig, d, n_pad, perm, reinterpret_cast<uint64_t*>(dyn), ctl && ctl->converged);
}

__global__ void k_permute(const float* __restrict__ Utw, const float* __restrict__ sig_w,
                          const int* __restrict__ perm, int64_t d, float* __restrict__ Ut,
                          float* __restrict__ sigma, int* __restrict__ J, int r,
                          const JacCtl* __restrict__ ctl, int* __restrict__ info,
                          uint32_t* __restrict__ status, int max_sweeps) {
  const int64_t k = blockIdx.x;
  const int64_t src = perm[k];
  for (int64_t a = threadIdx.x; a < d; a += blockDim.x) Ut[k * d + a] = Utw[src * d + a];
  if (threadIdx.x == 0) {
    sigma[k] = sig_w[src];
    if (k < r) J[k] = (int)k;
    if (k == 0) {
      info[0] = (int)ctl->sweeps;
      info[1] = (int)ctl->converged;
      for (int i = 0; i < kHistory; ++i)
        info[2 + i] = i < (int)ctl->sweeps ? (int)ctl->history[i] : 0;
      if (!ctl->converged) atomicOr(status, 2u);
    }
  }
}

// A' = P A P^T (packed) for the row permutation perm, and U^T' = P U^T.
// A random gather of 8-byte entries: each thread takes the same entry of
// kPermBlocks consecutive stored blocks, issuing all its loads before its
// stores, so that many loads are in flight per thread.
constexpr int kPermBlocks = 8;
// the kPermBlocks stored blocks from `bid * kPermBlocks` of B = A with rows and
// columns reordered by perm
__device__ __forceinline__ void pk_permute_blocks(const double* __restrict__ A, double* __restrict__ B,
                                                  const int* __restrict__ perm, int64_t d, int nb, int64_t bid) {
  const int64_t nblk = (int64_t)nb * (nb + 1) / 2;
  const int r = threadIdx.x / kJB, c = threadIdx.x % kJB;
  const int64_t first = bid * kPermBlocks;
  // (a, b) of the first block, then walk along the packed order
  int64_t blk = first;
  int a = 0;
  while (a < nb && blk >= nb - a) { blk -= nb - a; ++a; }
  int b = a + (int)blk;
  double x[kPermBlocks];
#pragma unroll
  for (int q = 0; q < kPermBlocks; ++q) {
    x[q] = 0.0;
    if (first + q < nblk) {
      const int64_t i = (int64_t)a * kJB + r, j = (int64_t)b * kJB + c;
      if (i < d && j < d) {
        const int pi = perm[i], pj = perm[j];
        x[q] = pk_get(A, nb, pi / kJB, pj / kJB, pi % kJB, pj % kJB);
      }
      if (++b == nb) { ++a; b = a; }
    }
  }
#pragma unroll
  for (int q = 0; q < kPermBlocks; ++q)
    if (first + q < nblk) B[(first + q) * (kJB * kJB) + threadIdx.x] = x[q];
}
__global__ void __launch_bounds__(256)
k_pk_permute(const double* __restrict__ A, double* __restrict__ B, const int* __restrict__ perm, int64_t d,
             int nb) {
  pk_permute_blocks(A, B, perm, d, nb, blockIdx.x);
}

__device__ __forceinline__ void row_gather_row(const float* __restrict__ src, float* __restrict__ dst,
                                               const int* __restrict__ perm, int64_t d, int64_t k) {
  const int64_t p = perm[k];
  for (int64_t a = threadIdx.x; a < d; a += blockDim.x) dst[k * d + a] = src[p * d + a];
}
__global__ void k_row_gather(const float* __restrict__ src, float* __restrict__ dst, const int* __restrict__ perm,
                             int64_t d) {
  row_gather_row(src, dst, perm, d, blockIdx.x);
}

hipError_t launch_jac_sort(const MatView& v, hipStream_t s) {
  const int nb = jac_blocks(v.d);
  hipLaunchKernelGGL(k_diag_sqrt, dim3((unsigned)((v.d + 255) / 256)), dim3(256), 0, s, v.Apk, v.d, nb,
                     v.sigma_w);
  int n_pad = 2;
  while (n_pad < v.d) n_pad <<= 1;
  hipLaunchKernelGGL(k_sort_desc, dim3(1), dim3(1024), (size_t)n_pad * 8, s, v.sigma_w, (int)v.d, n_pad, v.perm,
                     (const JacCtl*)v.ctl);
  const int64_t nblk = (int64_t)nb * (nb + 1) / 2;
  hipLaunchKernelGGL(k_pk_permute, dim3((unsigned)((nblk + kPermBlocks - 1) / kPermBlocks)), dim3(256), 0, s, v.Apk,
                     v.Apk2, v.perm, v.d, nb);
  hipLaunchKernelGGL(k_row_gather, dim3((unsigned)v.d), dim3(256), 0, s, v.Utw, v.W, v.perm, v.d);
  return hipGetLastError();
}

hipError_t launch_jac_finish(const MatView& v, int max_sweeps, hipStream_t s) {
  hipLaunchKernelGGL(k_diag_sqrt, dim3((unsigned)((v.d + 255) / 256)), dim3(256), 0, s, v.Apk, v.d,
                     jac_blocks(v.d), v.sigma_w);
  int n_pad = 2;
  while (n_pad < v.d) n_pad <<= 1;
  hipLaunchKernelGGL(k_sort_desc, dim3(1), dim3(1024), (size_t)n_pad * 8, s, v.sigma_w, (int)v.d,
                     n_pad, v.perm, (const JacCtl*)nullptr);
  hipLaunchKernelGGL(k_permute, dim3((unsigned)v.d), dim3(256), 0, s, v.Utw, v.sigma_w, v.perm, v.d,
                     v.Ut, v.sigma, v.J, v.r, v.ctl, v.info, v.status, max_sweeps);
  return hipGetLastError();
}


// ---------------------------------------------------------------------------
// Joint refresh: the sweeps of several matrices (one group size NG) in the
// same launches.  Every matrix owns a range of blocks of each launch (tables
// of first blocks); a block finds its matrix and runs the per-matrix code on
// that matrix's buffers, so each matrix computes exactly what its own
// launches compute.  A matrix past its last round, or converged, leaves.
// ---------------------------------------------------------------------------
__device__ __forceinline__ int joint_find(const int* __restrict__ first, int num, int b) {
  int lo = 0, hi = num - 1;   // the last m with first[m] <= b
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (first[mid] <= b) lo = mid;
    else hi = mid - 1;
  }
  return lo;
}

__global__ void k_joint_diag_sqrt(const JointMat* __restrict__ jm, const int* __restrict__ first, int num, int par) {
  const int m = joint_find(first, num, blockIdx.x);
  const MatView& v = jm[m].v[par];
  if (v.ctl->converged) return;
  diag_sqrt_at(v.Apk, v.d, jm[m].nb, v.sigma_w, (int64_t)(blockIdx.x - first[m]) * blockDim.x + threadIdx.x);
}

// a converged matrix takes the identity order: its data only moves to the
// other buffer (see sort_desc_block), so every matrix ends in the buffer of
// the last enqueued sweep
__global__ void __launch_bounds__(1024) k_joint_sort_desc(const JointMat* __restrict__ jm, int par) {
  const MatView& v = jm[blockIdx.x].v[par];
  extern __shared__ __align__(16) unsigned char dyn[];
  int n_pad = 2;
  while (n_pad < v.d) n_pad <<= 1;
  sort_desc_block(v.sigma_w, (int)v.d, n_pad, v.perm, reinterpret_cast<uint64_t*>(dyn), v.ctl->converged != 0);
}

__global__ void __launch_bounds__(256)
k_joint_pk_permute(const JointMat* __restrict__ jm, const int* __restrict__ first, int num, int par) {
  const int m = joint_find(first, num, blockIdx.x);
  const MatView& v = jm[m].v[par];
  pk_permute_blocks(v.Apk, v.Apk2, v.perm, v.d, jm[m].nb, blockIdx.x - first[m]);
}

__global__ void k_joint_row_gather(const JointMat* __restrict__ jm, const int* __restrict__ first, int num, int par) {
  const int m = joint_find(first, num, blockIdx.x);
  const MatView& v = jm[m].v[par];
  row_gather_row(v.Utw, v.W, v.perm, v.d, blockIdx.x - first[m]);
}

template <int NG>
__global__ void __launch_bounds__(JacShape<NG>::NT)
k_joint_solve(const JointMat* __restrict__ jm, const int* __restrict__ first, int num, int par, int round,
              float tol, int max_inner, double floor_rel2) {
  const int m = joint_find(first, num, blockIdx.x);
  const JointMat& J = jm[m];
  const MatView& v = J.v[par];
  if (v.ctl->converged || round >= J.rounds) return;
  __shared__ SolveLds<NG> lds;
  const int64_t vb = (int64_t)J.groups * JacShape<NG>::NR * JacShape<NG>::NR, p = round & 1;
  solve_group<NG>(v.Apk, v.ctl, round, J.seats, J.nb, tol, max_inner, floor_rel2, v.Vrot + p * vb, v.V64 + p * vb,
                  v.skip + p * J.groups, blockIdx.x - first[m], lds);
}

// the solves of `round` (matrices with more rounds) beside the rotation of U^T
// rows by round - 1 (matrices whose sweep reached it)
template <int NG>
__global__ void __launch_bounds__(JacShape<NG>::NT)
k_joint_solve_apply(const JointMat* __restrict__ jm, const int* __restrict__ first, int num, int par, int round,
                    float tol, int max_inner, double floor_rel2) {
  const int m = joint_find(first, num, blockIdx.x);
  const JointMat& J = jm[m];
  const MatView& v = J.v[par];
  if (v.ctl->converged || round > J.rounds) return;
  __shared__ JacLds<NG> lds;
  const int64_t vb = (int64_t)J.groups * JacShape<NG>::NR * JacShape<NG>::NR;
  const int b = blockIdx.x - first[m];
  if (b < J.groups) {
    if (round < J.rounds) {
      const int64_t p = round & 1;
      solve_group<NG>(v.Apk, v.ctl, round, J.seats, J.nb, tol, max_inner, floor_rel2, v.Vrot + p * vb,
                      v.V64 + p * vb, v.skip + p * J.groups, b, lds.s);
    }
  } else {
    const int idx = b - J.groups;
    const int64_t q = (round - 1) & 1;
    apply_chunk<NG>(v.Utw, v.d, v.Vrot + q * vb, v.skip + q * J.groups, round - 1, J.seats, J.nb, idx / J.chunks,
                    idx % J.chunks, J.width, lds.Va);
  }
}

template <int NG>
__global__ void __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(4, 4)))
k_joint_update(const JointMat* __restrict__ jm, const int* __restrict__ first, int num, int par, int round) {
  const int m = joint_find(first, num, blockIdx.x);
  const JointMat& J = jm[m];
  const MatView& v = J.v[par];
  if (v.ctl->converged || round >= J.rounds) return;
  __shared__ double S[JacShape<NG>::NR][JacShape<NG>::NR + 1];
  const int64_t vb = (int64_t)J.groups * JacShape<NG>::NR * JacShape<NG>::NR, p = round & 1;
  update_pair<NG>(v.Apk, v.V64 + p * vb, v.skip + p * J.groups, round, J.seats, J.nb, J.groups,
                  blockIdx.x - first[m], S);
}

// the sweep's check of every matrix, and its converged flag for the host
__global__ void k_joint_check(const JointMat* __restrict__ jm, float tol, int* __restrict__ flags) {
  JacCtl* ctl = jm[blockIdx.x].v[0].ctl;
  if (threadIdx.x != 0) return;
  if (!ctl->converged) {
    if (ctl->sweeps < (uint32_t)kHistory) ctl->history[ctl->sweeps] = ctl->sweep_max_bits;
    ctl->sweeps += 1;
    if (__uint_as_float(ctl->sweep_max_bits) <= tol) ctl->converged = 1;
    ctl->sweep_max_bits = 0;
  }
  flags[blockIdx.x] = (int)ctl->converged;
}

void joint_fill(JointMat& J, int (&blocks)[kJointKinds]) {
  const int64_t d = J.v[0].d;
  const int ng = jac_group_blocks(d);
  J.nb = jac_blocks(d);
  J.seats = jac_seats(d);
  J.groups = jac_groups(d);
  J.rounds = jac_rounds(d);
  J.width = JAC_CHUNK * (ng == 4 ? JacShape<4>::NT : JacShape<2>::NT) / 256;
  J.chunks = (int)((d + J.width - 1) / J.width);
  const int64_t nblk = (int64_t)J.nb * (J.nb + 1) / 2;
  blocks[kJointSolve] = J.groups;
  blocks[kJointSolveApply] = J.groups + J.groups * J.chunks;
  blocks[kJointUpdate] = J.groups * (J.groups + 1) / 2;
  blocks[kJointDiag] = (int)((d + 255) / 256);
  blocks[kJointPermute] = (int)((nblk + kPermBlocks - 1) / kPermBlocks);
  blocks[kJointGather] = (int)d;
}

static const int* joint_table(const JointPlan& jp, int kind) { return jp.first + (int64_t)kind * (jp.num + 1); }

hipError_t launch_joint_sort(const JointPlan& jp, int par, hipStream_t s) {
  hipLaunchKernelGGL(k_joint_diag_sqrt, dim3((unsigned)jp.total[kJointDiag]), dim3(256), 0, s, jp.jm,
                     joint_table(jp, kJointDiag), jp.num, par);
  hipLaunchKernelGGL(k_joint_sort_desc, dim3((unsigned)jp.num), dim3(1024), (size_t)jp.npad_max * 8, s, jp.jm, par);
  hipLaunchKernelGGL(k_joint_pk_permute, dim3((unsigned)jp.total[kJointPermute]), dim3(256), 0, s, jp.jm,
                     joint_table(jp, kJointPermute), jp.num, par);
  hipLaunchKernelGGL(k_joint_row_gather, dim3((unsigned)jp.total[kJointGather]), dim3(256), 0, s, jp.jm,
                     joint_table(jp, kJointGather), jp.num, par);
  return hipGetLastError();
}

hipError_t launch_joint_solve(const JointPlan& jp, int par, int round, float tol, int max_inner, double floor_rel2,
                              hipStream_t s) {
  const int* f = joint_table(jp, kJointSolve);
  if (jp.ng == 4)
    hipLaunchKernelGGL(k_joint_solve<4>, dim3((unsigned)jp.total[kJointSolve]), dim3(JacShape<4>::NT), 0, s, jp.jm,
                       f, jp.num, par, round, tol, max_inner, floor_rel2);
  else
    hipLaunchKernelGGL(k_joint_solve<2>, dim3((unsigned)jp.total[kJointSolve]), dim3(JacShape<2>::NT), 0, s, jp.jm,
                       f, jp.num, par, round, tol, max_inner, floor_rel2);
  return hipGetLastError();
}

hipError_t launch_joint_solve_apply(const JointPlan& jp, int par, int round, float tol, int max_inner,
                                    double floor_rel2, hipStream_t s) {
  const int* f = joint_table(jp, kJointSolveApply);
  const dim3 grid((unsigned)jp.total[kJointSolveApply]);
  if (jp.ng == 4)
    hipLaunchKernelGGL(k_joint_solve_apply<4>, grid, dim3(JacShape<4>::NT), 0, s, jp.jm, f, jp.num, par, round, tol,
                       max_inner, floor_rel2);
  else
    hipLaunchKernelGGL(k_joint_solve_apply<2>, grid, dim3(JacShape<2>::NT), 0, s, jp.jm, f, jp.num, par, round, tol,
                       max_inner, floor_rel2);
  return hipGetLastError();
}

hipError_t launch_joint_update(const JointPlan& jp, int par, int round, hipStream_t s) {
  const int* f = joint_table(jp, kJointUpdate);
  const dim3 grid((unsigned)jp.total[kJointUpdate]);
  if (jp.ng == 4) hipLaunchKernelGGL(k_joint_update<4>, grid, dim3(256), 0, s, jp.jm, f, jp.num, par, round);
  else hipLaunchKernelGGL(k_joint_update<2>, grid, dim3(256), 0, s, jp.jm, f, jp.num, par, round);
  return hipGetLastError();
}

hipError_t launch_joint_check(const JointPlan& jp, float tol, hipStream_t s) {
  hipLaunchKernelGGL(k_joint_check, dim3((unsigned)jp.num), dim3(64), 0, s, jp.jm, tol, jp.flags);
  return hipGetLastError();
}

}  // namespace glr
