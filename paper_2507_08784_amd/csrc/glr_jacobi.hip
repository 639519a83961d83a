// Refresh step: complete left singular basis U of Mbar (d x D) by block
// Jacobi on the fp64 Gram A = W W^T of the rows of W = U_0^T Mo (U_0 the
// previous basis, or I): the eigenvectors of A are the left singular vectors.
//
// A is formed once per refresh (fp64-accumulated products of the fp32 rows)
// and kept packed by 16 x 16 blocks.  Rows are grouped in blocks of kJB; a
// round splits the blocks into groups of four (kJR = 64 rows), and each group
// is treated as a whole:
//   solve  : one cyclic two-sided Jacobi sweep on the group's 64 x 64
//            diagonal block of A in LDS (fp64) gives the rotation V
//   update : A <- J^T A J with J = diag(V_group), block by block: the 64 x 64
//            block (g, h) of two groups becomes V_g^T A_gh V_h (fp64 MFMA)
//   apply  : rows of U^T <- V^T rows, in place, as u + (V - I)^T u
//            (fp32 MFMA), in the same launch as the next round's solves
// A sweep is (S - 1) / 3 rounds for S = 4^j seats (blocks and empty padding
// blocks): every two blocks share a group in exactly one round, so a sweep
// meets every pair of blocks once while A and U^T are streamed only once per
// round.  The sweeps stop when every group solved in a sweep passes the
// measure of the solve.  The singular values are sqrt(diag A), sorted
// descending (ties keep the lower row first); U^T rows follow the sort.
#include "glr_device.hpp"
#include "glr_internal.hpp"

namespace glr {

int jac_blocks(int64_t d) { return (int)((d + kJB - 1) / kJB); }
int jac_seats(int64_t d) {
  const int nb = jac_blocks(d);
  int s = kJG;
  while (s < nb) s *= 4;
  return s;
}
int jac_groups(int64_t d) { return jac_seats(d) / kJG; }
int jac_rounds(int64_t d) { return (jac_seats(d) - 1) / 3; }

// Block indices are vectors over F_2 (S = 2^k seats, k even), read as
// vectors of k/2 digits over F_4 = {0, 1, w, w^2}, a digit being two bits
// (1 = 01, w = 10, w^2 = 11).  Multiplication by w, digit by digit:
// (h, l) -> (h ^ l, h).
__device__ __forceinline__ uint32_t f4_times_w(uint32_t x) {
  const uint32_t h = (x >> 1) & 0x55555555u, l = x & 0x55555555u;
  return ((h ^ l) << 1) | h;
}
// Blocks of group g in round t.  The rounds are the (S - 1) / 3 lines
// {0, v, w v, w^2 v} through the origin (v with leading digit 1): they cover
// every non-zero vector exactly once.  The groups of a round are the cosets
// x0 + line, so two blocks a, b share a group exactly in the round whose line
// holds a ^ b.  Member m of a group is the block whose digit p (the leading
// digit of v) equals m; x0 is g with a zero digit inserted at p.
__device__ __forceinline__ void group_blocks(int t, int g, int (&blk)[kJG]) {
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

// columns of U^T rotated by one workgroup: 512 for 256 threads; the
// 1024-thread workgroups beside the solves take 1024, so that the solves and
// all the rotation workgroups of a round are resident together
constexpr int JAC_CHUNK = 512;
constexpr int JAC_CHUNK_WIDE = 1024;

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
// A sweep of the 64 x 64 eigenproblem is 63 steps of 32 disjoint rotations
// (circle method); when the rows inside each of the four blocks already meet
// the measure, only the 48 steps between blocks are taken (three pairings of
// the blocks, 16 steps each).  In a step, each thread owns one 2 x 2 block
// rows {p_a, q_a} x columns {p_b, q_b} of G and of V, so that the update
// G <- J^T G J, V <- V J is in place and private to the thread; the thread
// owning (a, a) first computes rotation a from that diagonal block.
// Rotation J = [[c, s], [-s, c]] that diagonalises [[gpp, gpq], [gpq, gqq]]:
// t = tan(theta) = sign(d h) |h| / (|d| + sqrt(d^2 + h^2)), d = gqq - gpp,
// h = 2 gpq, c = 1 / sqrt(1 + t^2), s = c t.  d and h are first scaled by a
// power of two (exact) so that t can be formed in fp32; c then comes from an
// fp32 estimate of 1 / sqrt(1 + t^2) refined by one Newton step in fp64, so
// that c^2 + s^2 = 1 to ~1e-14 for the t used.  An fp32 angle leaves an
// off-diagonal entry ~1e-7 of the one it removes, which the next sweeps take.
__device__ __forceinline__ void jac_rotation(double gpp, double gqq, double gpq, double& c, double& s) {
  c = 1.0;
  s = 0.0;
  if (gpq == 0.0 || gpq * gpq <= 1e-34 * (gpp * gqq)) return;
  const double d0 = gqq - gpp, h0 = 2.0 * gpq;
  int ex;
  (void)frexp(fmax(fabs(d0), fabs(h0)), &ex);
  const float dd = (float)ldexp(d0, -ex), h = (float)ldexp(h0, -ex);   // max(|dd|, |h|) in [0.5, 1)
  const float r = __builtin_amdgcn_sqrtf(dd * dd + h * h);
  const float tf = fabsf(h) * __builtin_amdgcn_rcpf(fabsf(dd) + r);
  const double t = ((dd < 0.0f) != (h < 0.0f)) ? -(double)tf : (double)tf;
  const double z = 1.0 + t * t;
  double y = (double)__builtin_amdgcn_rsqf((float)z);
  y = y * (1.5 - 0.5 * z * y * y);                        // 1 / sqrt(z)
  c = y;
  s = y * t;
}

// rotation j of step `step` of the circle method on 64 rows (p and q in
// either order: the rotation diagonalises the 2 x 2 block either way)
__device__ __forceinline__ void full_pair(int step, int j, int& p, int& q) {
  constexpr int last = kJR - 1;
  if (j == 0) { p = step; q = last; }
  else { p = (step + j) % last; q = (step - j + last) % last; }
}

// rotation j of step `step` of the 48 steps between blocks: block pairings
// (0,1)(2,3), (0,2)(1,3), (0,3)(1,2) in turn, each for the 16 steps that
// pair row k of one block with row (k + step) mod 16 of the other
__device__ __forceinline__ void cross_pair(int step, int j, int& p, int& q) {
  const int rho = step >> 4, k = step & (kJB - 1), half = j >> 4, kk = j & (kJB - 1);
  int ma, mb;
  if (rho == 0) { ma = half ? 2 : 0; mb = half ? 3 : 1; }
  else if (rho == 1) { ma = half ? 1 : 0; mb = half ? 3 : 2; }
  else { ma = half ? 1 : 0; mb = half ? 2 : 3; }
  p = kJB * ma + kk;
  q = kJB * mb + ((kk + k) & (kJB - 1));
}

__device__ __forceinline__ void step_pair(bool cross, int step, int j, int& p, int& q) {
  if (cross) cross_pair(step, j, p, q);
  else full_pair(step, j, p, q);
}

__device__ __forceinline__ bool group_empty(const int (&blk)[kJG], int nb) {
  return blk[0] >= nb && blk[1] >= nb && blk[2] >= nb && blk[3] >= nb;
}

// A group solve runs 1024 threads (16 waves): thread (a, b) owns the 2 x 2
// block {p_a, q_a} x {p_b, q_b} of G and V, a = t / 32, b = t % 32.  With
// four waves per SIMD the LDS latency of one wave hides behind the others.
constexpr int kSolveThreads = kJR * kJR / 4;
constexpr int kSolveWaves = kSolveThreads / 64;

// LDS of a group solve; the rotation of U^T reuses it for V - I (fp32)
struct SolveLds {
  double G[kJR][kJR + 1];
  double V[kJR][kJR + 1];
  double rc[kJR / 2], rs[kJR / 2];
  double red[kSolveWaves], redw[kSolveWaves];
};
union JacLds {
  SolveLds s;
  float Va[kJR][kJR + 1];
};

__device__ __forceinline__ void solve_group(const double* __restrict__ Apk, JacCtl* __restrict__ ctl, int round,
                                            int nb, float tol, int max_inner, double floor_rel2,
                                            float* __restrict__ Vout, double* __restrict__ V64,
                                            int* __restrict__ skip, int grp, SolveLds& L) {
  int blk[kJG];
  group_blocks(round, grp, blk);
  const int tid = threadIdx.x, lane = lane_id(), w = wave_id();
  if (group_empty(blk, nb)) {
    if (tid == 0) skip[grp] = 1;
    return;
  }
  double (*G)[kJR + 1] = L.G;
  double (*V)[kJR + 1] = L.V;
  double* rc = L.rc;
  double* rs = L.rs;
  double* red = L.red;
  double* redw = L.redw;
  constexpr int NE = kJR * kJR / kSolveThreads;
  const double rm_prev = __longlong_as_double((long long)ctl->rowmax2_bits);
  // the group's diagonal 64 x 64 block of A
  double g[NE];
#pragma unroll
  for (int k = 0; k < NE; ++k) {
    const int e = tid + kSolveThreads * k, x = e / kJR, y = e % kJR;
    g[k] = pk_get(Apk, nb, blk[x / kJB], blk[y / kJB], x % kJB, y % kJB);
  }
  double dmax = 0.0;
#pragma unroll
  for (int k = 0; k < NE; ++k) {
    const int e = tid + kSolveThreads * k, x = e / kJR, y = e % kJR;
    G[x][y] = g[k];
    V[x][y] = x == y ? 1.0 : 0.0;
    if (x == y) dmax = fmax(dmax, g[k]);
  }
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) dmax = fmax(dmax, __shfl_xor(dmax, o, 64));
  if (lane == 0) red[w] = dmax;
  __syncthreads();
  dmax = 0.0;
#pragma unroll
  for (int i = 0; i < kSolveWaves; ++i) dmax = fmax(dmax, red[i]);
  __syncthreads();
  if (tid == 0 && dmax > 0.0)
    atomicMax((unsigned long long*)&ctl->rowmax2_bits, (unsigned long long)__double_as_longlong(dmax));
  const double rowmax2 = fmax(dmax, rm_prev);
  const double floor2 = floor_rel2 * rowmax2;
  double m2 = 0.0, mw2 = 0.0;   // all pairs / pairs inside one block
#pragma unroll
  for (int k = 0; k < NE; ++k) {
    const int e = tid + kSolveThreads * k, x = e / kJR, y = e % kJR;
    if (x < y) {
      const double gxx = G[x][x], gyy = G[y][y];
      const double den = fmax(fmax(sqrt(gxx * gyy), fabs(gxx - gyy)), floor2);
      if (den > 0.0) {
        const double q2 = (g[k] / den) * (g[k] / den);
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
  for (int i = 0; i < kSolveWaves; ++i) {
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
  // the 16 lanes of an LDS access share the row pair a and take 16
  // consecutive column pairs b, whose rows are (up to the wrap of the
  // circle) distinct modulo 16: few bank conflicts
  const int a = tid >> 5, bb = tid & 31;
  const int steps = cross ? 3 * kJB : kJR - 1;
  for (int sweep = 0; sweep < max_inner; ++sweep) {
    int pa = 0, qa = 0, pb = 0, qb = 0;
    for (int st = 0; st < steps; ++st) {
      // the pairs move by one place per step: p + 1, q + 1 on the circle of
      // 63 (q = 63 stays), or q + 1 within its block between blocks
      if (st == 0 || (cross && (st & (kJB - 1)) == 0)) {
        step_pair(cross, st, a, pa, qa);
        step_pair(cross, st, bb, pb, qb);
      } else if (cross) {
        qa = (qa & ~(kJB - 1)) | ((qa + 1) & (kJB - 1));
        qb = (qb & ~(kJB - 1)) | ((qb + 1) & (kJB - 1));
      } else {
        pa = pa == kJR - 2 ? 0 : pa + 1;
        pb = pb == kJR - 2 ? 0 : pb + 1;
        qa = qa == kJR - 1 ? qa : (qa == kJR - 2 ? 0 : qa + 1);
        qb = qb == kJR - 1 ? qb : (qb == kJR - 2 ? 0 : qb + 1);
      }
      if (a == bb) {
        double c, sn;
        jac_rotation(G[pa][pa], G[qa][qa], G[pa][qa], c, sn);
        rc[a] = c;
        rs[a] = sn;
      }
      __syncthreads();
      // J restricted to a pair (p, q) is [[c, s], [-s, c]]; every entry
      // belongs to the 2 x 2 block of exactly one thread
      const double ca = rc[a], sa = rs[a], cb = rc[bb], sb = rs[bb];
      const double g00 = G[pa][pb], g01 = G[pa][qb], g10 = G[qa][pb], g11 = G[qa][qb];
      const double v00 = V[pa][pb], v01 = V[pa][qb], v10 = V[qa][pb], v11 = V[qa][qb];
      const double t00 = g00 * cb - g01 * sb, t01 = g00 * sb + g01 * cb;
      const double t10 = g10 * cb - g11 * sb, t11 = g10 * sb + g11 * cb;
      G[pa][pb] = ca * t00 - sa * t10;
      G[pa][qb] = ca * t01 - sa * t11;
      G[qa][pb] = sa * t00 + ca * t10;
      G[qa][qb] = sa * t01 + ca * t11;
      V[pa][pb] = v00 * cb - v01 * sb;
      V[pa][qb] = v00 * sb + v01 * cb;
      V[qa][pb] = v10 * cb - v11 * sb;
      V[qa][qb] = v10 * sb + v11 * cb;
      __syncthreads();
    }
  }
  float* vo = Vout + (int64_t)grp * kJR * kJR;
  double* vd = V64 + (int64_t)grp * kJR * kJR;
#pragma unroll
  for (int k = 0; k < NE; ++k) {
    const int e = tid + kSolveThreads * k;
    vo[e] = (float)V[e / kJR][e % kJR];
    vd[e] = V[e / kJR][e % kJR];
  }
  if (tid == 0) skip[grp] = 0;
}

// rows of the group in U^T <- V^T rows on this block's chunk, computed as
// w + (V - I)^T w (fp32 MFMA, two 32-row output tiles, K = 64).  The k index
// is permuted so that the B operand held by each lane is exactly the set of
// rows that lane outputs: k slot kk < 16 of a lane is physical row
// mfma32_row(kk, lane) (output tile 0, register kk) and slot 16 + kk is
// 32 + mfma32_row(kk, lane) (output tile 1, register kk).
__device__ __forceinline__ void apply_chunk(float* __restrict__ Utw, int64_t d, const float* __restrict__ Vin,
                                            const int* __restrict__ skip, int round, int nb, int grp,
                                            int chunk, int width, float (*Va)[kJR + 1]) {
  if (skip[grp]) return;
  int blk[kJG];
  group_blocks(round, grp, blk);
  if (group_empty(blk, nb)) return;
  const int lane = lane_id(), w = wave_id();
  const int l32 = lane & 31, lh4 = 4 * (lane >> 5);
  const float* V = Vin + (int64_t)grp * kJR * kJR;
  constexpr int KS = kJR / 2;   // k slots of the two-row MFMA steps
  for (int e = threadIdx.x; e < kJR * kJR; e += blockDim.x) {
    const int i = e / kJR, j = e % kJR;
    Va[i][j] = V[e] - (i == j ? 1.0f : 0.0f);
  }
  __syncthreads();
  // slot kk is row blk[m] * 16 + r of U^T with m = slot_block(kk) and
  // r = slot_row(kk) + 4 (lane / 32)
  auto slot_block = [](int kk) { return (kk < 16 ? 0 : 2) + ((kk & 15) >= 8 ? 1 : 0); };
  auto slot_row = [](int kk) { return 8 * (((kk & 15) >> 2) & 1) + (kk & 3); };
  int64_t first[kJG];   // row index of r = 4 (lane / 32) in each member block, -1 if padding
#pragma unroll
  for (int m = 0; m < kJG; ++m) first[m] = blk[m] < nb ? (int64_t)blk[m] * kJB + lh4 : -1;
  const int64_t c0 = (int64_t)chunk * width;
  const int span = 32 * (int)(blockDim.x >> 6);   // columns per pass, 32 per wave
  for (int it = 0; it < width; it += span) {
    const int64_t cb = c0 + it + w * 32;
    if (cb >= d) break;
    const int64_t cc = cb + l32;
    const bool cok = cc < d;
    float b[KS];
#pragma unroll
    for (int kk = 0; kk < KS; ++kk) {
      const int64_t f = first[slot_block(kk)], row = f + slot_row(kk);
      b[kk] = (cok && f >= 0 && row < d) ? Utw[row * d + cc] : 0.f;
    }
    // output tile h: rows 32 h + mfma32_row(v, lane), held by slot 16 h + v
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      f32x16 acc;
#pragma unroll
      for (int v = 0; v < 16; ++v) acc[v] = 0.f;
#pragma unroll
      for (int kk = 0; kk < KS; ++kk) {
        const int pr = (kk < 16 ? 0 : 32) + mfma32_row(kk & 15, lane);
        acc = mfma32(Va[pr][32 * h + l32], b[kk], acc);
      }
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        const int kk = 16 * h + v;
        const int64_t f = first[slot_block(kk)], row = f + slot_row(kk);
        if (cok && f >= 0 && row < d) Utw[row * d + cc] = b[kk] + acc[v];
      }
    }
  }
}

// A <- J^T A J: the 64 x 64 block of rows of group g and columns of group h
// (g <= h) becomes V_g^T A_gh V_h (fp64 MFMA 16x16x4; wave w computes the
// 32 x 32 quadrant (w / 2, w % 2) of each product).  The 16 x 16 blocks of A
// are read and written whole (coalesced) through one LDS tile; blocks below
// the diagonal are not stored, so each stored block is written by exactly
// one workgroup.  A group whose V is the identity skips its product.
__global__ void __launch_bounds__(256)
k_jac_update(double* __restrict__ Apk, const double* __restrict__ V64, const int* __restrict__ skip,
             const JacCtl* __restrict__ ctl, int round, int nb, int groups) {
  if (ctl->converged) return;
  int g = 0, rem = blockIdx.x;
  while (rem >= groups - g) {
    rem -= groups - g;
    ++g;
  }
  const int h = g + rem;
  const bool sg = skip[g] != 0, sh = skip[h] != 0;
  if (sg && sh) return;
  int bg[kJG], bh[kJG];
  group_blocks(round, g, bg);
  group_blocks(round, h, bh);
  __shared__ double S[kJR][kJR + 1];
  const int tid = threadIdx.x, lane = lane_id(), w = wave_id();
  const int er = tid / kJB, ec = tid % kJB;
  const int R0 = (w >> 1) * 32, C0 = (w & 1) * 32, li = lane & 15, lk = lane >> 4;
  double sv[kJG * kJG];
#pragma unroll
  for (int mb = 0; mb < kJG * kJG; ++mb) {
    const int bx = bg[mb >> 2], by = bh[mb & 3];
    sv[mb] = (bx < nb && by < nb) ? Apk[(bx <= by ? pk_off(bx, by, nb) : pk_off(by, bx, nb)) + tid] : 0.0;
  }
  // B operand of T = A_gh V_h, fetched while the blocks land in LDS
  double vb[kJR / 4][2];
  if (!sh) {
    const double* vh = V64 + (int64_t)h * kJR * kJR;
#pragma unroll
    for (int k = 0; k < kJR / 4; ++k) {
      const int kr = 4 * k + lk;
      vb[k][0] = vh[kr * kJR + C0 + li];
      vb[k][1] = vh[kr * kJR + C0 + 16 + li];
    }
  }
#pragma unroll
  for (int mb = 0; mb < kJG * kJG; ++mb) {
    const int mx = mb >> 2, my = mb & 3;
    if (bg[mx] <= bh[my]) S[kJB * mx + er][kJB * my + ec] = sv[mb];
    else S[kJB * mx + ec][kJB * my + er] = sv[mb];
  }
  __syncthreads();
  f64x4 acc[2][2];
  if (!sh) {
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
      for (int j = 0; j < 2; ++j) acc[i][j] = f64x4{0.0, 0.0, 0.0, 0.0};
#pragma unroll
    for (int k = 0; k < kJR / 4; ++k) {
      const double x0 = S[R0 + li][4 * k + lk], x1 = S[R0 + 16 + li][4 * k + lk];
      acc[0][0] = mfma64(x0, vb[k][0], acc[0][0]);
      acc[0][1] = mfma64(x0, vb[k][1], acc[0][1]);
      acc[1][0] = mfma64(x1, vb[k][0], acc[1][0]);
      acc[1][1] = mfma64(x1, vb[k][1], acc[1][1]);
    }
    __syncthreads();
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
      for (int j = 0; j < 2; ++j)
#pragma unroll
        for (int v = 0; v < 4; ++v) S[R0 + 16 * i + 4 * v + lk][C0 + 16 * j + li] = acc[i][j][v];
    __syncthreads();
  }
  if (!sg) {
    const double* vg = V64 + (int64_t)g * kJR * kJR;
    double va[kJR / 4][2];
#pragma unroll
    for (int k = 0; k < kJR / 4; ++k) {
      const int kr = 4 * k + lk;
      va[k][0] = vg[kr * kJR + R0 + li];
      va[k][1] = vg[kr * kJR + R0 + 16 + li];
    }
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
      for (int j = 0; j < 2; ++j) acc[i][j] = f64x4{0.0, 0.0, 0.0, 0.0};
#pragma unroll
    for (int k = 0; k < kJR / 4; ++k) {
      const double y0 = S[4 * k + lk][C0 + li], y1 = S[4 * k + lk][C0 + 16 + li];
      acc[0][0] = mfma64(va[k][0], y0, acc[0][0]);
      acc[0][1] = mfma64(va[k][0], y1, acc[0][1]);
      acc[1][0] = mfma64(va[k][1], y0, acc[1][0]);
      acc[1][1] = mfma64(va[k][1], y1, acc[1][1]);
    }
    __syncthreads();
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
      for (int j = 0; j < 2; ++j)
#pragma unroll
        for (int v = 0; v < 4; ++v) S[R0 + 16 * i + 4 * v + lk][C0 + 16 * j + li] = acc[i][j][v];
    __syncthreads();
  }
#pragma unroll
  for (int mb = 0; mb < kJG * kJG; ++mb) {
    const int mx = mb >> 2, my = mb & 3;
    const int bx = bg[mx], by = bh[my];
    if (bx >= nb || by >= nb) continue;
    if (bx <= by) Apk[pk_off(bx, by, nb) + tid] = S[kJB * mx + er][kJB * my + ec];
    else if (g != h) Apk[pk_off(by, bx, nb) + tid] = S[kJB * mx + ec][kJB * my + er];
  }
}

// the group solves of one round
__global__ void __launch_bounds__(kSolveThreads)
k_jac_solve(const double* __restrict__ Apk, JacCtl* __restrict__ ctl, int round, int nb, float tol,
            int max_inner, double floor_rel2, float* __restrict__ Vout, double* __restrict__ V64,
            int* __restrict__ skip) {
  if (ctl->converged) return;
  __shared__ SolveLds lds;
  solve_group(Apk, ctl, round, nb, tol, max_inner, floor_rel2, Vout, V64, skip, blockIdx.x, lds);
}

// the group solves of round `round` (workgroups [0, groups)) together with
// the rotation of U^T rows by the previous round's V (the rest): the rotation
// does not depend on the new solves, and the solves leave most of the chip idle
__global__ void __launch_bounds__(kSolveThreads)
k_jac_solve_apply(const double* __restrict__ Apk, JacCtl* __restrict__ ctl, int round, int nb, float tol,
                  int max_inner, double floor_rel2, float* __restrict__ Vout, double* __restrict__ V64,
                  int* __restrict__ skip, float* __restrict__ Utw, int64_t d, const float* __restrict__ Vprev,
                  const int* __restrict__ skip_prev, int groups, int chunks) {
  if (ctl->converged) return;
  __shared__ JacLds lds;
  const int b = blockIdx.x;
  if (b < groups) {
    solve_group(Apk, ctl, round, nb, tol, max_inner, floor_rel2, Vout, V64, skip, b, lds.s);
  } else {
    const int idx = b - groups;
    apply_chunk(Utw, d, Vprev, skip_prev, round - 1, nb, idx / chunks, idx % chunks, JAC_CHUNK_WIDE, lds.Va);
  }
}

// U^T rows of the last round of a sweep
__global__ void __launch_bounds__(256)
k_jac_apply(float* __restrict__ Utw, int64_t d, const float* __restrict__ V32, const int* __restrict__ skip,
            const JacCtl* __restrict__ ctl, int round, int nb, int chunks) {
  if (ctl->converged) return;
  __shared__ float Va[kJR][kJR + 1];
  apply_chunk(Utw, d, V32, skip, round, nb, blockIdx.x / chunks, blockIdx.x % chunks, JAC_CHUNK, Va);
}

// per-round buffers alternate between two copies (round parity), so that a
// round's solves can run while the previous round's rotations are applied
struct RoundBufs {
  float* V32;
  double* V64;
  int* skip;
};
static RoundBufs round_bufs(const MatView& v, int round) {
  const int64_t groups = jac_groups(v.d), par = round & 1;
  return {v.Vrot + par * groups * kJR * kJR, v.V64 + par * groups * kJR * kJR, v.skip + par * groups};
}

hipError_t launch_jac_update(const MatView& v, int round, hipStream_t s) {
  const int nb = jac_blocks(v.d), groups = jac_groups(v.d);
  const RoundBufs rb = round_bufs(v, round);
  hipLaunchKernelGGL(k_jac_update, dim3((unsigned)(groups * (groups + 1) / 2)), dim3(256), 0, s, v.Apk, rb.V64,
                     rb.skip, v.ctl, round, nb, groups);
  return hipGetLastError();
}

hipError_t launch_jac_solve_apply(const MatView& v, int round, float tol, int max_inner, double floor_rel2,
                                  hipStream_t s) {
  const int nb = jac_blocks(v.d), groups = jac_groups(v.d);
  const int chunks = (int)((v.d + JAC_CHUNK_WIDE - 1) / JAC_CHUNK_WIDE);
  const RoundBufs rb = round_bufs(v, round), pb = round_bufs(v, round - 1);
  hipLaunchKernelGGL(k_jac_solve_apply, dim3((unsigned)(groups + groups * chunks)), dim3(kSolveThreads), 0, s, v.Apk,
                     v.ctl, round, nb, tol, max_inner, floor_rel2, rb.V32, rb.V64, rb.skip, v.Utw, v.d, pb.V32,
                     pb.skip, groups, chunks);
  return hipGetLastError();
}

hipError_t launch_jac_apply(const MatView& v, int round, hipStream_t s) {
  const int nb = jac_blocks(v.d), groups = jac_groups(v.d);
  const int chunks = (int)((v.d + JAC_CHUNK - 1) / JAC_CHUNK);
  const RoundBufs rb = round_bufs(v, round);
  hipLaunchKernelGGL(k_jac_apply, dim3((unsigned)(groups * chunks)), dim3(256), 0, s, v.Utw, v.d, rb.V32,
                     rb.skip, v.ctl, round, nb, chunks);
  return hipGetLastError();
}

hipError_t launch_jac_solve(const MatView& v, int round, float tol, int max_inner, double floor_rel2,
                            hipStream_t s) {
  const int nb = jac_blocks(v.d), groups = jac_groups(v.d);
  const RoundBufs rb = round_bufs(v, round);
  hipLaunchKernelGGL(k_jac_solve, dim3(groups), dim3(kSolveThreads), 0, s, v.Apk, v.ctl, round, nb, tol, max_inner,
                     floor_rel2, rb.V32, rb.V64, rb.skip);
  return hipGetLastError();
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
__global__ void k_diag_sqrt(const double* __restrict__ Apk, int64_t d, int nb, float* __restrict__ sig) {
  const int64_t j = blockIdx.x * (int64_t)blockDim.x + threadIdx.x;
  if (j >= d) return;
  const int b = (int)(j / kJB), l = (int)(j % kJB);
  sig[j] = (float)sqrt(fmax(Apk[pk_off(b, b, nb) + l * (kJB + 1)], 0.0));
}

__global__ void __launch_bounds__(1024)
k_sort_desc(const float* __restrict__ sig, int d, int n_pad, int* __restrict__ perm) {
  extern __shared__ __align__(16) unsigned char dyn[];
  uint64_t* keys = reinterpret_cast<uint64_t*>(dyn);
  for (int i = threadIdx.x; i < n_pad; i += blockDim.x) {
    if (i < d) keys[i] = ((uint64_t)(~float_order(sig[i])) << 32) | (uint32_t)i;
    else keys[i] = ~0ull;
  }
  __syncthreads();
  bitonic_sort(keys, n_pad);
  for (int i = threadIdx.x; i < d; i += blockDim.x) perm[i] = (int)(keys[i] & 0xFFFFFFFFu);
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

// A' = P A P^T (packed) for the row permutation perm, and U^T' = P U^T
__global__ void __launch_bounds__(256)
k_pk_permute(const double* __restrict__ A, double* __restrict__ B, const int* __restrict__ perm, int64_t d,
             int nb) {
  // one workgroup per stored block (a, b), a <= b; one thread per entry
  int64_t blk = blockIdx.x;
  int a = 0;
  while (blk >= nb - a) { blk -= nb - a; ++a; }
  const int b = a + (int)blk;
  const int r = threadIdx.x / kJB, c = threadIdx.x % kJB;
  const int64_t i = (int64_t)a * kJB + r, j = (int64_t)b * kJB + c;
  double x = 0.0;
  if (i < d && j < d) {
    const int pi = perm[i], pj = perm[j];
    x = pk_get(A, nb, pi / kJB, pj / kJB, pi % kJB, pj % kJB);
  }
  B[pk_off(a, b, nb) + threadIdx.x] = x;
}

__global__ void k_row_gather(const float* __restrict__ src, float* __restrict__ dst, const int* __restrict__ perm,
                             int64_t d) {
  const int64_t k = blockIdx.x;
  const int64_t p = perm[k];
  for (int64_t a = threadIdx.x; a < d; a += blockDim.x) dst[k * d + a] = src[p * d + a];
}

hipError_t launch_jac_sort(const MatView& v, hipStream_t s) {
  const int nb = jac_blocks(v.d);
  hipLaunchKernelGGL(k_diag_sqrt, dim3((unsigned)((v.d + 255) / 256)), dim3(256), 0, s, v.Apk, v.d, nb,
                     v.sigma_w);
  int n_pad = 2;
  while (n_pad < v.d) n_pad <<= 1;
  hipLaunchKernelGGL(k_sort_desc, dim3(1), dim3(1024), (size_t)n_pad * 8, s, v.sigma_w, (int)v.d, n_pad, v.perm);
  hipLaunchKernelGGL(k_pk_permute, dim3((unsigned)(nb * (nb + 1) / 2)), dim3(256), 0, s, v.Apk, v.Apk2, v.perm,
                     v.d, nb);
  hipLaunchKernelGGL(k_row_gather, dim3((unsigned)v.d), dim3(256), 0, s, v.Utw, v.W, v.perm, v.d);
  return hipGetLastError();
}

hipError_t launch_jac_finish(const MatView& v, int max_sweeps, hipStream_t s) {
  hipLaunchKernelGGL(k_diag_sqrt, dim3((unsigned)((v.d + 255) / 256)), dim3(256), 0, s, v.Apk, v.d,
                     jac_blocks(v.d), v.sigma_w);
  int n_pad = 2;
  while (n_pad < v.d) n_pad <<= 1;
  hipLaunchKernelGGL(k_sort_desc, dim3(1), dim3(1024), (size_t)n_pad * 8, s, v.sigma_w, (int)v.d,
                     n_pad, v.perm);
  hipLaunchKernelGGL(k_permute, dim3((unsigned)v.d), dim3(256), 0, s, v.Utw, v.sigma_w, v.perm, v.d,
                     v.Ut, v.sigma, v.J, v.r, v.ctl, v.info, v.status, max_sweeps);
  return hipGetLastError();
}

}  // namespace glr
