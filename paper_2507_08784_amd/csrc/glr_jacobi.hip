// Refresh step: complete left singular basis U of Mbar (d x D) by block
// Jacobi on the fp64 Gram A = W W^T of the rows of W = U_0^T Mo (U_0 the
// previous basis, or I): the eigenvectors of A are the left singular vectors.
//
// A is formed once per refresh (fp64-accumulated products of the fp32 rows)
// and kept packed by 16 x 16 blocks.  Rows are grouped in blocks of kJB; a
// round of the round-robin tournament pairs the blocks two by two, and each
// pair (2 kJB rows) is treated as a whole:
//   solve  : cyclic two-sided Jacobi on the pair's 32 x 32 diagonal block of
//            A in LDS (fp64) gives its eigenvectors V
//   update : A <- J^T A J with J = diag(V_pair), block by block: the 32 x 32
//            block (P, Q) of two pairs becomes V_P^T A_PQ V_Q (fp64 MFMA)
//   apply  : rows of U^T <- V^T rows, in place, as u + (V - I)^T u
//            (fp32 MFMA), in the same launch as the next round's solves
// A sweep is one tournament (every pair of blocks meets once).  The sweeps
// stop when every pair met in a sweep passes the measure of k_jac_solve.
// The singular values are sqrt(diag A), sorted descending (ties keep the
// lower row first); U^T rows follow the sort.
#include "glr_device.hpp"
#include "glr_internal.hpp"

namespace glr {

int jac_blocks(int64_t d) { return (int)((d + kJB - 1) / kJB); }
int jac_seats(int64_t d) {
  int nb = jac_blocks(d);
  return nb + (nb & 1) < 2 ? 2 : nb + (nb & 1);
}
// blocks met by `pair` in `round` of the circle-method tournament on `seats`
__device__ __forceinline__ void pair_blocks(int round, int pair, int seats, int& bi, int& bj) {
  const int last = seats - 1;
  if (pair == 0) {
    bi = round;
    bj = last;
  } else {
    bi = (round + pair) % last;
    bj = (round - pair + last) % last;
  }
}

__device__ __forceinline__ int64_t pair_row(int lr, int bi, int bj) {
  return lr < kJB ? (int64_t)bi * kJB + lr : (int64_t)bj * kJB + (lr - kJB);
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

constexpr int JAC_CHUNK = 512;   // columns of U^T rotated by one block

// Eigenvectors V of the pair Gram by cyclic two-sided Jacobi in LDS (fp64).
// Convergence measure of a pair of rows (p, q):
//   |w_p . w_q| / max(|w_p| |w_q|,  | |w_p|^2 - |w_q|^2 |,  f^2),
//   f = 2^-10 max_k |w_k|.
// Below tol it bounds both the cosine of the two rows and the angle of the
// rotation that would still separate them, so that a converged basis is
// accurate for every singular-vector subspace whose gap in sigma^2 is above
// f^2 = 2^-20 sigma_1^2 -- far below what the fp32 data resolves -- without
// chasing orthogonality between tiny rows that fp32 rounding re-creates.
//
// A sweep of the 32 x 32 eigenproblem is 31 steps of 16 disjoint rotations
// (circle method); when the rows inside each of the two blocks already meet
// the measure, only the 16 steps between the blocks are taken.  In a step,
// thread (a, b) of the 256 owns the 2 x 2 block rows {p_a, q_a} x columns
// {p_b, q_b} of G and of V, so that the update G <- J^T G J, V <- V J is in
// place and private to the thread; thread (a, a) first computes rotation a
// from its own diagonal block.
// Rotation J = [[c, s], [-s, c]] that diagonalises [[gpp, gpq], [gpq, gqq]]:
// t = tan(theta) = sign(d h) |h| / (|d| + sqrt(d^2 + h^2)), d = gqq - gpp,
// h = 2 gpq, c = 1 / sqrt(1 + t^2), s = c t.  d and h are first scaled by a
// power of two (exact) so that the square root, the reciprocal and the
// reciprocal square root can start from fp32 estimates, each refined by one
// Newton step in fp64 (relative error ~1e-14, far below what the iteration
// needs; c^2 + s^2 = 1 to the same level).
__device__ __forceinline__ void jac_rotation(double gpp, double gqq, double gpq, double& c, double& s) {
  c = 1.0;
  s = 0.0;
  if (gpq == 0.0 || gpq * gpq <= 1e-34 * (gpp * gqq)) return;
  const double d0 = gqq - gpp, h0 = 2.0 * gpq;
  int ex;
  (void)frexp(fmax(fabs(d0), fabs(h0)), &ex);
  const double dd = ldexp(d0, -ex), h = ldexp(h0, -ex);   // max(|dd|, |h|) in [0.5, 1)
  const double x = dd * dd + h * h;
  const double yr = (double)rsqrtf((float)x);
  double r = x * yr;
  r = r + 0.5 * yr * (x - r * r);                         // sqrt(x)
  const double den = fabs(dd) + r;
  double q = (double)(1.0f / (float)den);
  q = q * (2.0 - den * q);                                // 1 / den
  double t = fabs(h) * q;
  if ((dd < 0.0) != (h < 0.0)) t = -t;
  const double z = 1.0 + t * t;
  double y = (double)rsqrtf((float)z);
  y = y * (1.5 - 0.5 * z * y * y);                        // 1 / sqrt(z)
  c = y;
  s = y * t;
}

// step k of the 16 steps that pair each row of one block with each row of
// the other: rows (k, 16 + (k + step) mod 16)
__device__ __forceinline__ void cross_pair(int step, int k, int& p, int& q) {
  p = k;
  q = kJB + ((k + step) & (kJB - 1));
}

__device__ __forceinline__ void inner_pair(int rd, int k, int& p, int& q) {
  constexpr int last = kJP - 1;
  if (k == 0) { p = rd; q = last; }
  else { p = (rd + k) % last; q = (rd - k + last) % last; }
  if (p > q) { const int t = p; p = q; q = t; }
}

__device__ __forceinline__ void solve_pair(const double* __restrict__ Apk, JacCtl* __restrict__ ctl, int round,
                                           int seats, int nb, float tol, int max_inner, double floor_rel2,
                                           float* __restrict__ Vout, double* __restrict__ V64,
                                           int* __restrict__ skip, int pair) {
  int bi, bj;
  pair_blocks(round, pair, seats, bi, bj);
  if (bi >= nb && bj >= nb) return;
  __shared__ double G[kJP][kJP + 1];
  __shared__ double V[kJP][kJP + 1];
  __shared__ double rc[kJP / 2], rs[kJP / 2];
  __shared__ double red[4], redw[4];
  const int tid = threadIdx.x, lane = lane_id(), w = wave_id();
  const double rm_prev = __longlong_as_double((long long)ctl->rowmax2_bits);
  // the pair's diagonal 32 x 32 block of A
  double g[4];
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    const int e = tid + 256 * k, x = e / kJP, y = e % kJP;
    g[k] = pk_get(Apk, nb, x < kJB ? bi : bj, y < kJB ? bi : bj, x % kJB, y % kJB);
  }
  double dmax = 0.0;
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    const int e = tid + 256 * k, x = e / kJP, y = e % kJP;
    G[x][y] = g[k];
    V[x][y] = x == y ? 1.0 : 0.0;
    if (x == y) dmax = fmax(dmax, g[k]);
  }
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) dmax = fmax(dmax, __shfl_xor(dmax, o, 64));
  if (lane == 0) red[w] = dmax;
  __syncthreads();
  dmax = fmax(fmax(red[0], red[1]), fmax(red[2], red[3]));
  __syncthreads();
  if (tid == 0 && dmax > 0.0)
    atomicMax((unsigned long long*)&ctl->rowmax2_bits, (unsigned long long)__double_as_longlong(dmax));
  const double rowmax2 = fmax(dmax, rm_prev);
  const double floor2 = floor_rel2 * rowmax2;
  double m2 = 0.0, mw2 = 0.0;   // all pairs / pairs inside one block
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    const int e = tid + 256 * k, x = e / kJP, y = e % kJP;
    if (x < y) {
      const double gxx = G[x][x], gyy = G[y][y];
      const double den = fmax(fmax(sqrt(gxx * gyy), fabs(gxx - gyy)), floor2);
      if (den > 0.0) {
        const double q2 = (g[k] / den) * (g[k] / den);
        m2 = fmax(m2, q2);
        if ((x < kJB) == (y < kJB)) mw2 = fmax(mw2, q2);
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
  const double m = sqrt(fmax(fmax(red[0], red[1]), fmax(red[2], red[3])));
  // rows inside each block already orthogonal: only the 16 cross steps
  const bool cross_only = sqrt(fmax(fmax(redw[0], redw[1]), fmax(redw[2], redw[3]))) <= (double)tol;
  if (tid == 0) atomicMax(&ctl->sweep_max_bits, __float_as_uint((float)m));
  if (m <= (double)tol) {
    if (tid == 0) skip[pair] = 1;
    return;
  }
  const int a = tid >> 4, b = tid & 15;
  const int steps = cross_only ? kJB : kJP - 1;
  for (int sweep = 0; sweep < max_inner; ++sweep) {
    for (int rd = 0; rd < steps; ++rd) {
      int pa, qa, pb, qb;
      if (cross_only) {
        cross_pair(rd, a, pa, qa);
        cross_pair(rd, b, pb, qb);
      } else {
        inner_pair(rd, a, pa, qa);
        inner_pair(rd, b, pb, qb);
      }
      if (a == b) {
        double c, s;
        jac_rotation(G[pa][pa], G[qa][qa], G[pa][qa], c, s);
        rc[a] = c;
        rs[a] = s;
      }
      __syncthreads();
      // J restricted to a pair (p, q) is [[c, s], [-s, c]]
      const double ca = rc[a], sa = rs[a], cb = rc[b], sb = rs[b];
      const double g00 = G[pa][pb], g01 = G[pa][qb], g10 = G[qa][pb], g11 = G[qa][qb];
      const double t00 = g00 * cb - g01 * sb, t01 = g00 * sb + g01 * cb;
      const double t10 = g10 * cb - g11 * sb, t11 = g10 * sb + g11 * cb;
      G[pa][pb] = ca * t00 - sa * t10;
      G[pa][qb] = ca * t01 - sa * t11;
      G[qa][pb] = sa * t00 + ca * t10;
      G[qa][qb] = sa * t01 + ca * t11;
      const double v00 = V[pa][pb], v01 = V[pa][qb], v10 = V[qa][pb], v11 = V[qa][qb];
      V[pa][pb] = v00 * cb - v01 * sb;
      V[pa][qb] = v00 * sb + v01 * cb;
      V[qa][pb] = v10 * cb - v11 * sb;
      V[qa][qb] = v10 * sb + v11 * cb;
      __syncthreads();
    }
  }
  float* vo = Vout + (int64_t)pair * kJP * kJP;
  double* vd = V64 + (int64_t)pair * kJP * kJP;
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    const int e = tid + 256 * k;
    vo[e] = (float)V[e / kJP][e % kJP];
    vd[e] = V[e / kJP][e % kJP];
  }
  if (tid == 0) skip[pair] = 0;
}

// rows of the pair in U^T <- V^T rows on this block's chunk, computed
// as w + (V - I)^T w (fp32 MFMA).  The k index is permuted so that the B
// operand held by each lane is exactly the set of rows that lane outputs:
// physical row of k = 2kk + h is mfma32_row(kk, 32h), and B register kk is
// output register kk.
__device__ __forceinline__ void apply_chunk(float* __restrict__ Utw, int64_t d, const float* __restrict__ Vin,
                                            const int* __restrict__ skip, int round, int seats, int nb,
                                            int pair, int chunk) {
  if (skip[pair]) return;
  int bi, bj;
  pair_blocks(round, pair, seats, bi, bj);
  if (bi >= nb && bj >= nb) return;
  const int lane = lane_id(), w = wave_id();
  const int l32 = lane & 31;
  const float* V = Vin + (int64_t)pair * kJP * kJP;
  float a[kJP / 2];
  int64_t rows[kJP / 2];
#pragma unroll
  for (int kk = 0; kk < kJP / 2; ++kk) {
    const int pr = mfma32_row(kk, lane);
    a[kk] = V[pr * kJP + l32] - (pr == l32 ? 1.0f : 0.0f);
    rows[kk] = pair_row(pr, bi, bj);
  }
  const int64_t c0 = (int64_t)chunk * JAC_CHUNK;
  for (int it = 0; it < JAC_CHUNK / 128; ++it) {
    const int64_t cb = c0 + it * 128 + w * 32;
    if (cb >= d) break;
    const int64_t cc = cb + l32;
    const bool cok = cc < d;
    float b[kJP / 2];
#pragma unroll
    for (int kk = 0; kk < kJP / 2; ++kk) b[kk] = (cok && rows[kk] < d) ? Utw[rows[kk] * d + cc] : 0.f;
    f32x16 acc;
#pragma unroll
    for (int v = 0; v < 16; ++v) acc[v] = 0.f;
#pragma unroll
    for (int kk = 0; kk < kJP / 2; ++kk) acc = mfma32(a[kk], b[kk], acc);
#pragma unroll
    for (int v = 0; v < 16; ++v)
      if (cok && rows[v] < d) Utw[rows[v] * d + cc] = b[v] + acc[v];
  }
}

// A <- J^T A J: the 32 x 32 block of rows of pair P and columns of pair Q
// (P <= Q) becomes V_P^T A_PQ V_Q (fp64 MFMA; V_P held in registers as the
// A operand of the second product, V_Q read as the B operand of the first).
// A workgroup takes one P and up to kUpdQ consecutive Q.  The 16 x 16 blocks
// of A are read and written whole (coalesced) through one LDS tile; blocks
// below the diagonal are not stored, so each stored block is written by
// exactly one workgroup.
constexpr int kUpdQ = 2;

__device__ __forceinline__ void update_group(double* __restrict__ Apk, const double* __restrict__ V64,
                                             const int* __restrict__ skip, int round, int seats, int nb,
                                             int pairs, int P, int Q0, double (*S)[kJP + 1]) {
  int pi, pj;
  pair_blocks(round, P, seats, pi, pj);
  if (pi >= nb && pj >= nb) return;
  const int tid = threadIdx.x, lane = lane_id(), w = wave_id();
  const int wi = (w >> 1) * 16, wj = (w & 1) * 16;   // wave w: result block (w >> 1, w & 1)
  const int li = lane & 15, lk = lane >> 4;
  const int er = tid / kJB, ec = tid % kJB;             // element of a 16 x 16 block
  const bool sp = skip[P] != 0;
  const double* vp = V64 + (int64_t)P * kJP * kJP;
  double vpo[kJP / 4];
#pragma unroll
  for (int k = 0; k < kJP / 4; ++k) {
    const int kk = 4 * k + lk;
    vpo[k] = sp ? (kk == wi + li ? 1.0 : 0.0) : vp[kk * kJP + wi + li];
  }
  for (int q = 0; q < kUpdQ; ++q) {
    const int Q = Q0 + q;
    if (Q >= pairs) break;
    int qi, qj;
    pair_blocks(round, Q, seats, qi, qj);
    if (qi >= nb && qj >= nb) continue;
    const bool sq = skip[Q] != 0;
    if (sp && sq) continue;
    const double* vq = V64 + (int64_t)Q * kJP * kJP;
    double sv[4], vqo[kJP / 4];
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      const int bx = (k >> 1) ? pj : pi, by = (k & 1) ? qj : qi;
      sv[k] = (bx < nb && by < nb) ? Apk[(bx <= by ? pk_off(bx, by, nb) : pk_off(by, bx, nb)) + tid] : 0.0;
    }
#pragma unroll
    for (int k = 0; k < kJP / 4; ++k) {
      const int kk = 4 * k + lk;
      vqo[k] = sq ? (kk == wj + li ? 1.0 : 0.0) : vq[kk * kJP + wj + li];
    }
    __syncthreads();   // the previous Q is done with S
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      const int h = k >> 1, g = k & 1;
      const int bx = h ? pj : pi, by = g ? qj : qi;
      if (bx <= by) S[h * kJB + er][g * kJB + ec] = sv[k];
      else S[h * kJB + ec][g * kJB + er] = sv[k];
    }
    __syncthreads();
    // a pair that met the stopping rule this round has V = I: its product is skipped
    if (!sq) {
      f64x4 acc = {0.0, 0.0, 0.0, 0.0};
#pragma unroll
      for (int k = 0; k < kJP / 4; ++k) acc = mfma64(S[wi + li][4 * k + lk], vqo[k], acc);   // T = A_PQ V_Q
      __syncthreads();
#pragma unroll
      for (int v = 0; v < 4; ++v) S[wi + 4 * v + lk][wj + li] = acc[v];
      __syncthreads();
    }
    if (!sp) {
      f64x4 acc = {0.0, 0.0, 0.0, 0.0};
#pragma unroll
      for (int k = 0; k < kJP / 4; ++k) acc = mfma64(vpo[k], S[4 * k + lk][wj + li], acc);  // V_P^T T
      __syncthreads();
#pragma unroll
      for (int v = 0; v < 4; ++v) S[wi + 4 * v + lk][wj + li] = acc[v];
      __syncthreads();
    }
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      const int h = k >> 1, g = k & 1;
      if (P == Q && h == 1 && g == 0) continue;   // the transpose of block (0, 1)
      const int bx = h ? pj : pi, by = g ? qj : qi;
      if (bx >= nb || by >= nb) continue;
      if (bx <= by) Apk[pk_off(bx, by, nb) + tid] = S[h * kJB + er][g * kJB + ec];
      else Apk[pk_off(by, bx, nb) + tid] = S[h * kJB + ec][g * kJB + er];
    }
  }
}

// A <- J^T A J for one round (one P and up to kUpdQ consecutive Q per workgroup)
__global__ void __launch_bounds__(256)
k_jac_update(double* __restrict__ Apk, const double* __restrict__ V64, const int* __restrict__ skip,
             const JacCtl* __restrict__ ctl, int round, int seats, int nb, int pairs) {
  if (ctl->converged) return;
  __shared__ double S[kJP][kJP + 1];
  int P = 0, rem = blockIdx.x;
  for (;;) {
    const int cnt = (pairs - P + kUpdQ - 1) / kUpdQ;
    if (rem < cnt) break;
    rem -= cnt;
    ++P;
  }
  update_group(Apk, V64, skip, round, seats, nb, pairs, P, P + rem * kUpdQ, S);
}

// the pair eigensolves of one round
__global__ void __launch_bounds__(256)
k_jac_solve(const double* __restrict__ Apk, JacCtl* __restrict__ ctl, int round, int seats, int nb, float tol,
            int max_inner, double floor_rel2, float* __restrict__ Vout, double* __restrict__ V64,
            int* __restrict__ skip) {
  if (ctl->converged) return;
  solve_pair(Apk, ctl, round, seats, nb, tol, max_inner, floor_rel2, Vout, V64, skip, blockIdx.x);
}

// the pair eigensolves of round `round` (workgroups [0, pairs)) together with
// the rotation of U^T rows by the previous round's V (the rest): the rotation
// does not depend on the new solves, and the solves leave most of the chip idle
__global__ void __launch_bounds__(256)
k_jac_solve_apply(const double* __restrict__ Apk, JacCtl* __restrict__ ctl, int round, int seats, int nb,
                  float tol, int max_inner, double floor_rel2, float* __restrict__ Vout,
                  double* __restrict__ V64, int* __restrict__ skip, float* __restrict__ Utw, int64_t d,
                  const float* __restrict__ Vprev, const int* __restrict__ skip_prev, int pairs, int chunks) {
  if (ctl->converged) return;
  const int b = blockIdx.x;
  if (b < pairs) {
    solve_pair(Apk, ctl, round, seats, nb, tol, max_inner, floor_rel2, Vout, V64, skip, b);
  } else {
    const int idx = b - pairs;
    apply_chunk(Utw, d, Vprev, skip_prev, round - 1, seats, nb, idx / chunks, idx % chunks);
  }
}

// U^T rows of the last round of a sweep
__global__ void __launch_bounds__(256)
k_jac_apply(float* __restrict__ Utw, int64_t d, const float* __restrict__ V32, const int* __restrict__ skip,
            const JacCtl* __restrict__ ctl, int round, int seats, int nb, int chunks) {
  if (ctl->converged) return;
  apply_chunk(Utw, d, V32, skip, round, seats, nb, blockIdx.x / chunks, blockIdx.x % chunks);
}

// per-round buffers alternate between two copies (round parity), so that a
// round's solves can run while the previous round's rotations are applied
struct RoundBufs {
  float* V32;
  double* V64;
  int* skip;
};
static RoundBufs round_bufs(const MatView& v, int round) {
  const int pairs = jac_seats(v.d) / 2, par = round & 1;
  return {v.Vrot + (int64_t)par * pairs * kJP * kJP, v.V64 + (int64_t)par * pairs * kJP * kJP,
          v.skip + (int64_t)par * pairs};
}

hipError_t launch_jac_update(const MatView& v, int round, hipStream_t s) {
  const int nb = jac_blocks(v.d), seats = jac_seats(v.d), pairs = seats / 2;
  int n_upd = 0;
  for (int P = 0; P < pairs; ++P) n_upd += (pairs - P + kUpdQ - 1) / kUpdQ;
  const RoundBufs rb = round_bufs(v, round);
  hipLaunchKernelGGL(k_jac_update, dim3((unsigned)n_upd), dim3(256), 0, s, v.Apk, rb.V64, rb.skip, v.ctl, round,
                     seats, nb, pairs);
  return hipGetLastError();
}

hipError_t launch_jac_solve_apply(const MatView& v, int round, float tol, int max_inner, double floor_rel2,
                                  hipStream_t s) {
  const int nb = jac_blocks(v.d), seats = jac_seats(v.d), pairs = seats / 2;
  const int chunks = (int)((v.d + JAC_CHUNK - 1) / JAC_CHUNK);
  const RoundBufs rb = round_bufs(v, round), pb = round_bufs(v, round - 1);
  hipLaunchKernelGGL(k_jac_solve_apply, dim3((unsigned)(pairs + pairs * chunks)), dim3(256), 0, s, v.Apk, v.ctl,
                     round, seats, nb, tol, max_inner, floor_rel2, rb.V32, rb.V64, rb.skip, v.Utw, v.d, pb.V32,
                     pb.skip, pairs, chunks);
  return hipGetLastError();
}

hipError_t launch_jac_apply(const MatView& v, int round, hipStream_t s) {
  const int nb = jac_blocks(v.d), seats = jac_seats(v.d), pairs = seats / 2;
  const int chunks = (int)((v.d + JAC_CHUNK - 1) / JAC_CHUNK);
  const RoundBufs rb = round_bufs(v, round);
  hipLaunchKernelGGL(k_jac_apply, dim3((unsigned)(pairs * chunks)), dim3(256), 0, s, v.Utw, v.d, rb.V32, rb.skip,
                     v.ctl, round, seats, nb, chunks);
  return hipGetLastError();
}

hipError_t launch_jac_solve(const MatView& v, int round, float tol, int max_inner, double floor_rel2,
                            hipStream_t s) {
  const int nb = jac_blocks(v.d), seats = jac_seats(v.d), pairs = seats / 2;
  const RoundBufs rb = round_bufs(v, round);
  hipLaunchKernelGGL(k_jac_solve, dim3(pairs), dim3(256), 0, s, v.Apk, v.ctl, round, seats, nb, tol,
                     max_inner, floor_rel2, rb.V32, rb.V64, rb.skip);
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
