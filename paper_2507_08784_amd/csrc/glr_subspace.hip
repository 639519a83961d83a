// Refresh step when only the top-r block of U is consumed (tau = 1: every
// step is a refresh and J = {0..r-1}, so only span(U[:, :r]) matters).
//
// Block subspace iteration on K = min(d, 2r) directions, orthonormalised
// after each half step:
//     Z  = orth(P^T Mo)        (K x D)
//     P^T = orth(Z Mo^T)       (K x d)
// The top-r directions converge at the rate (sigma_{K+1} / sigma_r)^2 per
// iteration whatever the gap at r (error feedback often closes that gap),
// and the half-step orthonormalisation does not square the conditioning the
// way iterating with Mo Mo^T would.  orth() is CholeskyQR2: S = Y Y^T (fp32
// MFMA products, partial sums reduced in fp64), S = L L^T (fp64, one block),
// Y <- L^-1 Y (fp32 MFMA), twice.  The iteration stops when the subspace
// change ||P_new - (P_new P^T) P|| / sqrt(K) is below its tolerance or after
// its iteration budget; Rayleigh-Ritz then takes the exact SVD of the small
// projection B = P^T Mo (K x D) with the block Jacobi kernels and keeps the
// Ritz vectors in descending order of Ritz value.
#include "glr_device.hpp"
#include "glr_internal.hpp"

namespace glr {

// ---------------------------------------------------------------------------
// generic MFMA GEMM  C = A B  with A (M x Kc) contiguous along k (lda), B
// either contiguous along k (B_KC: element (k, j) at B[j ldb + k]) or along
// j (element (k, j) at B[k ldb + j]).  grid.z splits the contraction into
// slices of `kslice`; slice z writes C + z * cstride.
//   EPI 0: C = acc
//   EPI 1: C = X - acc, and per block the sum of squares of C (fp64) in sums
// ---------------------------------------------------------------------------
template <int BM, int BN, int WM, int WN, bool B_KC, int EPI>
__global__ void __launch_bounds__(256)
k_gemm(const float* __restrict__ A, int64_t lda, const float* __restrict__ B, int64_t ldb,
       float* __restrict__ C, int64_t ldc, int M, int N, int Kc, int kslice, int64_t cstride,
       const float* __restrict__ X, double* __restrict__ sums) {
  using T = MfmaTile<BM, BN, WM, WN>;
  __shared__ __align__(16) float smem[T::LDS_FLOATS];
  const int n0 = blockIdx.x * BN, m0 = blockIdx.y * BM;
  const int k0 = blockIdx.z * kslice;
  const int klen = (Kc - k0 < kslice) ? Kc - k0 : kslice;
  T tile;
  if (klen > 0) {
    LoadK<BM, 32, false, false> la(A + k0, nullptr, lda, m0, M, klen, nullptr);
    if (B_KC) {
      LoadK<BN, 32, false, false> lb(B + k0, nullptr, ldb, n0, N, klen, nullptr);
      tile.run(la, lb, klen, smem);
    } else {
      LoadR<BN, 32, false> lb(B + (int64_t)k0 * ldb, nullptr, ldb, n0, N, klen);
      tile.run(la, lb, klen, smem);
    }
  }
  float* Cz = C + (int64_t)blockIdx.z * cstride;
  double ss = 0.0;
#pragma unroll
  for (int tm = 0; tm < T::TM; ++tm)
#pragma unroll
    for (int tn = 0; tn < T::TN; ++tn) {
      const int j = n0 + tile.col(tn);
      if (j >= N) continue;
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        const int i = m0 + tile.row(tm, v);
        if (i >= M) continue;
        if (EPI == 0) {
          Cz[(int64_t)i * ldc + j] = tile.acc[tm][tn][v];
        } else {
          const float o = X[(int64_t)i * ldc + j] - tile.acc[tm][tn][v];
          Cz[(int64_t)i * ldc + j] = o;
          ss += (double)o * (double)o;
        }
      }
    }
  if (EPI == 1) {
    __shared__ double red[4];
    ss = wave_sum(ss);
    if (lane_id() == 0) red[wave_id()] = ss;
    __syncthreads();
    if (threadIdx.x == 0)
      sums[(int64_t)blockIdx.y * gridDim.x + blockIdx.x] = red[0] + red[1] + red[2] + red[3];
  }
}

struct GemmPlan {
  int splits, kslice;
};

GemmPlan plan_splits(int M, int N, int Kc, int want_blocks = 1024);
GemmPlan plan_splits(int M, int N, int Kc, int want_blocks) {
  const int tiles = ((M + 127) / 128) * ((N + 127) / 128);
  int splits = (want_blocks + tiles - 1) / tiles;
  const int maxs = (Kc + 127) / 128;
  if (splits > maxs) splits = maxs;
  if (splits < 1) splits = 1;
  int kslice = ((Kc + splits - 1) / splits + 31) / 32 * 32;
  splits = (Kc + kslice - 1) / kslice;
  return {splits, kslice};
}

template <bool B_KC, int EPI>
static void gemm_launch(const float* A, int64_t lda, const float* B, int64_t ldb, float* C,
                        int64_t ldc, int M, int N, int Kc, GemmPlan p, int64_t cstride,
                        const float* X, double* sums, hipStream_t s) {
  dim3 grid((N + 127) / 128, (M + 127) / 128, p.splits);
  hipLaunchKernelGGL((k_gemm<128, 128, 2, 2, B_KC, EPI>), grid, dim3(256), 0, s, A, lda, B, ldb, C,
                     ldc, M, N, Kc, p.kslice, cstride, X, sums);
}

// out[i] = sum over splits of part[s * count + i], in a fixed order, fp64
__global__ void k_reduce_splits(const float* __restrict__ part, int splits, int64_t count,
                                float* __restrict__ out32, double* __restrict__ out64) {
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < count; i += stride) {
    // partials summed in split order; loads issued 8 at a time
    double s = 0.0;
    for (int z0 = 0; z0 < splits; z0 += 8) {
      float t[8];
#pragma unroll
      for (int j = 0; j < 8; ++j) t[j] = z0 + j < splits ? part[(int64_t)(z0 + j) * count + i] : 0.f;
#pragma unroll
      for (int j = 0; j < 8; ++j) s += (double)t[j];
    }
    if (out32) out32[i] = (float)s;
    if (out64) out64[i] = s;
  }
}

static int grid_n(int64_t n) {
  int64_t g = (n + 255) / 256;
  if (g < 1) g = 1;
  if (g > 8192) g = 8192;
  return (int)g;
}

// ---------------------------------------------------------------------------
// Cholesky S = L L^T and the inverse L^-1 of a K x K (K <= kMaxSubK) matrix,
// fp64, one block of 4 waves, 32 x 32 tiles (Kp = K rounded up to 32; the
// padding is the identity).  Lm, Dinv, Li are fp64 scratch in global memory
// (L2-resident); the result is written as fp32 Linv (Kp x Kp, zero above the
// diagonal).  A non-positive pivot sets status bit 4 and is replaced by a
// tiny positive value so that the sweep can continue.
// ---------------------------------------------------------------------------
constexpr int kTile = 32;

__device__ __forceinline__ void wave_lds_sync() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup");
}

// C (32x32) = / -= / = -(A B), one wave.  A tile row-major (lda); B given as
// B[k][j] at Bp[k * ldb + j], or as rows B[j][k] at Bp[j * ldb + k] (b_rows).
// mode 0: C = A B;  1: C -= A B;  2: C = -(A B).
__device__ __forceinline__ void tile_mm(const double* A, int lda, const double* Bp, int ldb, bool b_rows, double* Cp,
                        int ldc, int mode, double (*Bs)[kTile + 1]) {
  const int lane = lane_id();
  const int i = lane & 31, half = lane >> 5;
  for (int e = lane; e < kTile * kTile; e += 64) {
    const int j = e / kTile, k = e % kTile;   // Bs[j][k] = B(k, j)
    Bs[j][k] = b_rows ? Bp[j * ldb + k] : Bp[k * ldb + j];
  }
  double a[kTile];
#pragma unroll
  for (int k = 0; k < kTile; ++k) a[k] = A[i * lda + k];
  wave_lds_sync();
  double acc[16];
#pragma unroll
  for (int jj = 0; jj < 16; ++jj) {
    const int j = half * 16 + jj;
    double s = 0.0;
#pragma unroll
    for (int k = 0; k < kTile; ++k) s += a[k] * Bs[j][k];
    acc[jj] = s;
  }
#pragma unroll
  for (int jj = 0; jj < 16; ++jj) {
    const int j = half * 16 + jj;
    double* c = Cp + i * ldc + j;
    if (mode == 0) *c = acc[jj];
    else if (mode == 1) *c -= acc[jj];
    else *c = -acc[jj];
  }
  wave_lds_sync();
}

__global__ void __launch_bounds__(256)
k_chol_inv(const double* __restrict__ S, int K, int Kp, double* __restrict__ Lm,
           double* __restrict__ Dinv, double* __restrict__ Li, double* __restrict__ Tw,
           float* __restrict__ Linv, uint32_t* __restrict__ status) {
  __shared__ double Bs[4][kTile][kTile + 1];
  const int tid = threadIdx.x, lane = lane_id(), w = wave_id();
  const int nt = Kp / kTile;
  for (int e = tid; e < Kp * Kp; e += 256) {
    const int i = e / Kp, j = e % Kp;
    double x;
    if (i < K && j < K) x = S[(int64_t)i * K + j];
    else x = (i == j) ? 1.0 : 0.0;
    Lm[e] = x;
    Li[e] = 0.0;
  }
  __syncthreads();
  for (int J = 0; J < nt; ++J) {
    double* TJJ = Lm + (J * kTile) * Kp + J * kTile;
    double* DJ = Dinv + J * kTile * kTile;
    if (w == 0) {
      // factor the diagonal tile in this wave's LDS tile (right-looking)
      double (*Tl)[kTile + 1] = Bs[0];
      for (int e = lane; e < kTile * kTile; e += 64) Tl[e / kTile][e % kTile] = TJJ[(e / kTile) * Kp + e % kTile];
      wave_lds_sync();
      bool bad = false;
      for (int j = 0; j < kTile; ++j) {
        double piv = Tl[j][j];
        if (!(piv > 0.0)) { bad = true; piv = 1e-300; }
        const double ljj = sqrt(piv);
        wave_lds_sync();
        if (lane < kTile) {
          if (lane > j) Tl[lane][j] = Tl[lane][j] / ljj;
          else if (lane == j) Tl[j][j] = ljj;
        }
        wave_lds_sync();
        for (int e = lane; e < kTile * kTile; e += 64) {
          const int i = e / kTile, k = e % kTile;
          if (k > j && k <= i) Tl[i][k] -= Tl[i][j] * Tl[k][j];
        }
        wave_lds_sync();
      }
      if (bad && lane == 0) atomicOr(status, 4u);
      for (int e = lane; e < kTile * kTile; e += 64) {
        const int i = e / kTile, k = e % kTile;
        TJJ[i * Kp + k] = (k <= i) ? Tl[i][k] : 0.0;
      }
      // inverse of the lower-triangular tile: lane c solves L x = e_c
      if (lane < kTile) {
        const int c = lane;
        double x[kTile];
#pragma unroll
        for (int ii = 0; ii < kTile; ++ii) {
          double sacc = (ii == c) ? 1.0 : 0.0;
#pragma unroll
          for (int k = 0; k < ii; ++k) sacc -= Tl[ii][k] * x[k];
          x[ii] = sacc / Tl[ii][ii];
        }
#pragma unroll
        for (int ii = 0; ii < kTile; ++ii) DJ[ii * kTile + c] = x[ii];
      }
      wave_lds_sync();
    }
    __syncthreads();
    // panel: L_IJ = A_IJ inv(L_JJ)^T
    for (int I = J + 1 + w; I < nt; I += 4) {
      double* AIJ = Lm + (I * kTile) * Kp + J * kTile;
      tile_mm(AIJ, Kp, DJ, kTile, true, Tw + w * kTile * kTile, kTile, 0, Bs[w]);
      // copy back (tile_mm cannot write in place: it reads A rows lazily)
      for (int e = lane; e < kTile * kTile; e += 64)
        AIJ[(e / kTile) * Kp + e % kTile] = Tw[w * kTile * kTile + e];
      wave_lds_sync();
    }
    __syncthreads();
    // trailing update: A_IK -= L_IJ L_KJ^T for J < K <= I
    int idx = 0;
    for (int I = J + 1; I < nt; ++I)
      for (int Kq = J + 1; Kq <= I; ++Kq, ++idx) {
        if (idx % 4 != w) continue;
        tile_mm(Lm + (I * kTile) * Kp + J * kTile, Kp, Lm + (Kq * kTile) * Kp + J * kTile, Kp, true,
                Lm + (I * kTile) * Kp + Kq * kTile, Kp, 1, Bs[w]);
      }
    __syncthreads();
  }
  // inverse by diagonals: Li_II = Dinv_I; Li_IJ = -Dinv_I sum_{J<=Kq<I} L_IKq Li_KqJ
  for (int I = w; I < nt; I += 4)
    for (int e = lane; e < kTile * kTile; e += 64)
      Li[(I * kTile + e / kTile) * Kp + I * kTile + e % kTile] = Dinv[I * kTile * kTile + e];
  __syncthreads();
  for (int dl = 1; dl < nt; ++dl) {
    for (int J = w; J + dl < nt; J += 4) {
      const int I = J + dl;
      double* T = Tw + w * kTile * kTile;
      for (int e = lane; e < kTile * kTile; e += 64) T[e] = 0.0;
      wave_lds_sync();
      for (int Kq = J; Kq < I; ++Kq) {
        // T -= -(L_IKq Li_KqJ)  ==  T += L_IKq Li_KqJ  (accumulated as T -= (-1) ...)
        double* Tn = Tw + (4 + w) * kTile * kTile;
        tile_mm(Lm + (I * kTile) * Kp + Kq * kTile, Kp, Li + (Kq * kTile) * Kp + J * kTile, Kp,
                false, Tn, kTile, 0, Bs[w]);
        for (int e = lane; e < kTile * kTile; e += 64) T[e] += Tn[e];
        wave_lds_sync();
      }
      tile_mm(Dinv + I * kTile * kTile, kTile, T, kTile, false,
              Li + (I * kTile) * Kp + J * kTile, Kp, 2, Bs[w]);
    }
    __syncthreads();
  }
  for (int e = tid; e < Kp * Kp; e += 256) Linv[e] = (float)Li[e];
}

// cold start: rows of P^T drawn from N(0, 1) with Philox (key seed ^ const)
__global__ void k_sub_random(float* __restrict__ Pt, int K, int64_t d, uint32_t k0, uint32_t k1,
                             uint32_t mat) {
  const int64_t n4 = (d + 3) / 4;
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t q = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; q < (int64_t)K * n4; q += stride) {
    const int k = (int)(q / n4);
    const int64_t c = q % n4;
    float z[4];
    normals4((uint32_t)c, (uint32_t)k, mat, 0xFFFFFFFFu, k0, k1, z);
#pragma unroll
    for (int e = 0; e < 4; ++e)
      if (4 * c + e < d) Pt[(int64_t)k * d + 4 * c + e] = z[e];
  }
}

__global__ void k_sum_double(const double* __restrict__ x, int n, double* __restrict__ out) {
  __shared__ double red[4];
  double s = 0.0;
  for (int i = threadIdx.x; i < n; i += blockDim.x) s += x[i];
  s = wave_sum(s);
  if (lane_id() == 0) red[wave_id()] = s;
  __syncthreads();
  if (threadIdx.x == 0) *out = red[0] + red[1] + red[2] + red[3];
}

__global__ void k_sub_reset(SubCtl* sc) {
  if (threadIdx.x == 0) {
    sc->iters = 0;
    sc->converged = 0;
    sc->change2 = 0.0;
  }
}

__global__ void k_sub_step(SubCtl* sc, int K, float tol) {
  if (threadIdx.x != 0 || sc->converged) return;
  const double ch = sqrt(sc->change2 / (double)K);
  if (sc->iters < kHistory) sc->history[sc->iters] = __float_as_uint((float)ch);
  sc->iters += 1;
  if (ch <= (double)tol) sc->converged = 1;
}

// ---------------------------------------------------------------------------
// host side
// ---------------------------------------------------------------------------
size_t sub_part_floats(int K, int64_t d, int64_t D) {
  size_t mx = 0;
  auto upd = [&](int M, int N, int Kc) {
    const GemmPlan p = plan_splits(M, N, Kc);
    const size_t n = (size_t)p.splits * M * N;
    if (n > mx) mx = n;
  };
  upd(K, K, (int)D);
  upd(K, K, (int)d);
  upd(K, (int)d, (int)D);
  return mx;
}
static hipError_t orth_rows(const MatView& v, float* Y, float* Ytmp, int K, int64_t L, hipStream_t s) {
  const int Kp = (K + kTile - 1) / kTile * kTile;
  for (int pass = 0; pass < 2; ++pass) {
    GemmPlan pg = plan_splits(K, K, (int)L);
    gemm_launch<true, 0>(Y, L, Y, L, v.sub_part, K, K, K, (int)L, pg, (int64_t)K * K, nullptr, nullptr, s);
    hipLaunchKernelGGL(k_reduce_splits, dim3(grid_n((int64_t)K * K)), dim3(256), 0, s, v.sub_part,
                       pg.splits, (int64_t)K * K, (float*)nullptr, v.sub_S);
    hipLaunchKernelGGL(k_chol_inv, dim3(1), dim3(256), 0, s, v.sub_S, K, Kp, v.sub_L, v.sub_Dinv,
                       v.sub_Li, v.sub_T, v.sub_Linv, v.status);
    GemmPlan p1{1, K};
    gemm_launch<false, 0>(v.sub_Linv, Kp, Y, L, Ytmp, L, K, (int)L, K, p1, 0, nullptr, nullptr, s);
    hipError_t e = hipMemcpyAsync(Y, Ytmp, (size_t)K * L * 4, hipMemcpyDeviceToDevice, s);
    if (e != hipSuccess) return e;
  }
  return hipGetLastError();
}

hipError_t launch_sub_start(const MatView& v, bool warm, uint64_t seed, hipStream_t s) {
  const int K = sub_block(v.r, v.d);
  if (warm) {
    hipError_t e = hipMemcpyAsync(v.sub_P, v.Ut, (size_t)K * v.d * 4, hipMemcpyDeviceToDevice, s);
    if (e != hipSuccess) return e;
  } else {
    const uint32_t k0 = (uint32_t)(seed & 0xFFFFFFFFu) ^ 0xA5A5A5A5u;
    const uint32_t k1 = (uint32_t)(seed >> 32) ^ 0x3C3C3C3Cu;
    hipLaunchKernelGGL(k_sub_random, dim3(grid_n((int64_t)K * ((v.d + 3) / 4))), dim3(256), 0, s,
                       v.sub_P, K, v.d, k0, k1, (uint32_t)v.mat);
  }
  hipLaunchKernelGGL(k_sub_reset, dim3(1), dim3(64), 0, s, v.sub_ctl);
  return orth_rows(v, v.sub_P, v.sub_Pn, K, v.d, s);
}

// one iteration; writes the subspace change into sub_ctl
hipError_t launch_sub_iter(const MatView& v, float tol, hipStream_t s) {
  const int K = sub_block(v.r, v.d);
  const int64_t d = v.d, D = v.D;
  // Z = P^T Mo  (K x D)
  GemmPlan p1{1, (int)d};
  if (v.right)   // Mo[a][b] = Mbar[b][a]: B(k=a, j=b) at Mbar[b d + a]
    gemm_launch<true, 0>(v.sub_P, d, v.Mbar, d, v.sub_Z, D, K, (int)D, (int)d, p1, 0, nullptr, nullptr, s);
  else           // Mo = Mbar (d x D): B(k=a, j=b) at Mbar[a D + b]
    gemm_launch<false, 0>(v.sub_P, d, v.Mbar, D, v.sub_Z, D, K, (int)D, (int)d, p1, 0, nullptr, nullptr, s);
  hipError_t e = orth_rows(v, v.sub_Z, v.sub_Zt, K, D, s);
  if (e != hipSuccess) return e;
  // P_new = Z Mo^T  (K x d): B(k=b, j=a) = Mo[a][b]
  GemmPlan p2 = plan_splits(K, (int)d, (int)D);
  if (v.right)   // Mbar[b d + a]: contiguous along j
    gemm_launch<false, 0>(v.sub_Z, D, v.Mbar, d, v.sub_part, d, K, (int)d, (int)D, p2, (int64_t)K * d, nullptr, nullptr, s);
  else           // Mbar[a D + b]: contiguous along k
    gemm_launch<true, 0>(v.sub_Z, D, v.Mbar, D, v.sub_part, d, K, (int)d, (int)D, p2, (int64_t)K * d, nullptr, nullptr, s);
  hipLaunchKernelGGL(k_reduce_splits, dim3(grid_n((int64_t)K * d)), dim3(256), 0, s, v.sub_part,
                     p2.splits, (int64_t)K * d, v.sub_Pn, (double*)nullptr);
  e = orth_rows(v, v.sub_Pn, v.sub_R, K, d, s);
  if (e != hipSuccess) return e;
  // change: R = P_new - (P_new P^T) P ;  C = P_new P^T (K x K)
  GemmPlan pc = plan_splits(K, K, (int)d);
  gemm_launch<true, 0>(v.sub_Pn, d, v.sub_P, d, v.sub_part, K, K, K, (int)d, pc, (int64_t)K * K, nullptr, nullptr, s);
  hipLaunchKernelGGL(k_reduce_splits, dim3(grid_n((int64_t)K * K)), dim3(256), 0, s, v.sub_part,
                     pc.splits, (int64_t)K * K, v.sub_C, (double*)nullptr);
  GemmPlan p3{1, K};
  gemm_launch<false, 1>(v.sub_C, K, v.sub_P, d, v.sub_R, d, K, (int)d, K, p3, 0, v.sub_Pn, v.sub_sums, s);
  const int nb = (int)(((d + 127) / 128) * ((K + 127) / 128));
  hipLaunchKernelGGL(k_sum_double, dim3(1), dim3(256), 0, s, v.sub_sums, nb, &v.sub_ctl->change2);
  hipLaunchKernelGGL(k_sub_step, dim3(1), dim3(64), 0, s, v.sub_ctl, K, tol);
  // P <- P_new
  e = hipMemcpyAsync(v.sub_P, v.sub_Pn, (size_t)K * d * 4, hipMemcpyDeviceToDevice, s);
  if (e != hipSuccess) return e;
  return hipGetLastError();
}

// Rayleigh-Ritz: B = P^T Mo (K x D) into sub_Z; a MatView whose block Jacobi
// computes the SVD of B (rows): B = Y Sigma V^T, Y written to rr_Y, Sigma to
// the state's sigma, J = 0..r-1, info and status as for a full refresh.
hipError_t launch_sub_rr_begin(const MatView& v, MatView* rr, hipStream_t s) {
  const int K = sub_block(v.r, v.d);
  const int64_t d = v.d, D = v.D;
  GemmPlan p1{1, (int)d};
  if (v.right)
    gemm_launch<true, 0>(v.sub_P, d, v.Mbar, d, v.sub_Z, D, K, (int)D, (int)d, p1, 0, nullptr, nullptr, s);
  else
    gemm_launch<false, 0>(v.sub_P, d, v.Mbar, D, v.sub_Z, D, K, (int)D, (int)d, p1, 0, nullptr, nullptr, s);
  *rr = v;
  rr->d = K;
  rr->D = D;
  rr->right = false;
  rr->W = v.sub_Z;
  rr->Utw = v.rr_Utw;
  rr->Ut = v.rr_Y;
  rr->gram_part = v.rr_gram;
  rr->Vrot = v.rr_V;
  rr->skip = v.rr_skip;
  rr->ctl = v.rr_ctl;
  rr->sigma_w = v.rr_sigw;
  rr->perm = v.rr_perm;
  hipError_t e = launch_eye(v.rr_Utw, K, s);
  if (e != hipSuccess) return e;
  return launch_jac_reset(*rr, s);
}

// U^T rows 0..K-1 = Y P^T (the Ritz vectors, by descending Ritz value)
hipError_t launch_sub_rr_end(const MatView& v, hipStream_t s) {
  const int K = sub_block(v.r, v.d);
  const int64_t d = v.d;
  GemmPlan p1{1, K};
  gemm_launch<false, 0>(v.rr_Y, K, v.sub_P, d, v.Ut, d, K, (int)d, K, p1, 0, nullptr, nullptr, s);
  return hipGetLastError();
}

}  // namespace glr
