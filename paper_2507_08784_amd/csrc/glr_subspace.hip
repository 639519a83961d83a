// Refresh step when only the top-r block of U is consumed (tau = 1: every
// step is a refresh and J = {0..r-1}, so only span(U[:, :r]) matters).
//
// Block subspace iteration on K = min(d, r + max(32, r / 4)) directions, orthonormalised
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
//   EPI 2: C = X - acc
// A launch whose gate word is set returns at once (a section of the tau = 1
// refresh that the device skipped: converged, or no repair to finish).
// The grid is one-dimensional: the gy row tiles of a (column tile, slice)
// pair run one after another on one XCD (workgroups go to the XCDs in turn,
// so 8 launch slots apart), so that the slice of B they share is read from
// HBM once and then from that XCD's L2.  VEC: every operand slice loads as
// whole float4s (checked by gemm_launch).
// ---------------------------------------------------------------------------
template <int BM, int BN, int WM, int WN, bool B_KC, int EPI, bool VEC>
__global__ void __launch_bounds__(256)
k_gemm(const float* __restrict__ A, int64_t lda, const float* __restrict__ B, int64_t ldb,
       float* __restrict__ C, int64_t ldc, int M, int N, int Kc, int kslice, int64_t cstride,
       const float* __restrict__ X, double* __restrict__ sums, const int* __restrict__ gate, int gx, int gy,
       int ngroups) {
  if (gate && *gate) return;
  const int L = blockIdx.x, slot = L >> 3;
  const int grp = (slot / gy) * 8 + (L & 7), bxy = slot % gy;
  if (grp >= ngroups) return;
  const int bxx = grp % gx, bz = grp / gx;
  using T = MfmaTile<BM, BN, WM, WN>;
  __shared__ __align__(16) float smem[T::LDS_FLOATS];
  const int n0 = bxx * BN, m0 = bxy * BM;
  const int k0 = bz * kslice;
  const int klen = (Kc - k0 < kslice) ? Kc - k0 : kslice;
  T tile;
  if (klen > 0) {
    LoadK<BM, 32, false, false, float, VEC> la(A + k0, nullptr, lda, m0, M, klen, nullptr);
    if (B_KC) {
      LoadK<BN, 32, false, false, float, VEC> lb(B + k0, nullptr, ldb, n0, N, klen, nullptr);
      tile.run(la, lb, klen, smem);
    } else {
      LoadR<BN, 32, false, false, float, VEC> lb(B + (int64_t)k0 * ldb, nullptr, ldb, n0, N, klen);
      tile.run(la, lb, klen, smem);
    }
  }
  float* Cz = C + (int64_t)bz * cstride;
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
        } else if (EPI == 2) {
          Cz[(int64_t)i * ldc + j] = X[(int64_t)i * ldc + j] - tile.acc[tm][tn][v];
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
      sums[(int64_t)bxy * gx + bxx] = red[0] + red[1] + red[2] + red[3];
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

// Z = P^T Mo (K x D over d): the K x D tiles alone leave part of the chip
// idle for a whole d-long contraction (1120 tiles of 64 x 128 at K = 320,
// D = 28672), so the contraction is split into slices of at least 2048
// (fp32 partials added in fp64 by k_reduce_splits)
GemmPlan plan_z(int K, int64_t D, int64_t d) {
  GemmPlan p = plan_splits(K, (int)D, (int)d, 2048);
  if (p.kslice < 2048) {
    p.kslice = (int)std::min<int64_t>(2048, (d + 31) / 32 * 32);
    p.splits = (int)((d + p.kslice - 1) / p.kslice);
  }
  return p;
}

template <bool B_KC, int EPI>
static void gemm_launch(const float* A, int64_t lda, const float* B, int64_t ldb, float* C,
                        int64_t ldc, int M, int N, int Kc, GemmPlan p, int64_t cstride,
                        const float* X, double* sums, hipStream_t s, const int* gate = nullptr) {
  // 64-row tiles when M is not a multiple of 128 (no half-empty last row of tiles)
  const int bm = gemm_rows(M);
  const int gx = (N + 127) / 128, gy = (M + bm - 1) / bm, ngroups = gx * p.splits;
  const dim3 grid((unsigned)(((ngroups + 7) / 8) * 8 * gy));
  // the loaders' float4 conditions for every slice: leading dimensions and
  // Kc (hence every slice start and length) multiples of 4, B's row length
  // too when it is read along rows, and both operands 16-byte aligned
  const bool vec = lda % 4 == 0 && ldb % 4 == 0 && Kc % 4 == 0 && p.kslice % 4 == 0 && (B_KC || N % 4 == 0) &&
                   (reinterpret_cast<uintptr_t>(A) & 15) == 0 && (reinterpret_cast<uintptr_t>(B) & 15) == 0;
#define GLR_GEMM(BM, WM, WN, VE)                                                                         \
  hipLaunchKernelGGL((k_gemm<BM, 128, WM, WN, B_KC, EPI, VE>), grid, dim3(256), 0, s, A, lda, B, ldb, C, \
                     ldc, M, N, Kc, p.kslice, cstride, X, sums, gate, gx, gy, ngroups)
  if (bm == 64) {
    if (vec) GLR_GEMM(64, 1, 4, true);
    else GLR_GEMM(64, 1, 4, false);
  } else {
    if (vec) GLR_GEMM(128, 2, 2, true);
    else GLR_GEMM(128, 2, 2, false);
  }
#undef GLR_GEMM
}

// out[i] = sum over splits of part[s * count + i], in a fixed order, fp64
__global__ void k_reduce_splits(const float* __restrict__ part, int splits, int64_t count,
                                float* __restrict__ out32, double* __restrict__ out64,
                                const int* __restrict__ gate) {
  if (gate && *gate) return;
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
// fp64-accumulated Gram products of fp32 rows, C = A B^T (A: M x Kc, B: N x Kc,
// row-major and contiguous along k): fp32 inputs widened to fp64, fp64 MFMA
// on 64 x 64 tiles (each wave a 32 x 32 quadrant), grid.z splitting the
// contraction into slices of kslice.
//   EPI 0: slice z of C (fp64) at out64 + z M ldo (tiles below the block
//          diagonal skipped: only the upper blocks of a symmetric C are read)
//   EPI 1: out32 = (C - I) / 2 (one slice): the Newton-Schulz correction;
//          A = B and C symmetric: the upper tiles only, each entry written
//          to (i, j) and (j, i)
//   EPI 2: C packed by 16 x 16 blocks (a <= b) at out64 (one slice), ldo = nb
// ---------------------------------------------------------------------------
template <int EPI>
__global__ void __launch_bounds__(256)
k_gram64(const float* __restrict__ A, int64_t lda, const float* __restrict__ B, int64_t ldb, int M,
         int N, int Kc, int kslice, double* __restrict__ out64, float* __restrict__ out32, int64_t ldo) {
  __shared__ float As[32][65];
  __shared__ float Bs[32][65];
  const int tid = threadIdx.x, lane = lane_id(), w = wave_id();
  const int m0 = blockIdx.y * 64, n0 = blockIdx.x * 64;
  if (m0 >= n0 + 64) return;
  const int k0 = blockIdx.z * kslice;
  const int k1 = Kc < k0 + kslice ? Kc : k0 + kslice;
  const int lr = tid >> 2, kq = (tid & 3) * 8;     // loader: row, k offset
  const bool aok = m0 + lr < M, bok = n0 + lr < N;
  const float* ap = A + (int64_t)(aok ? m0 + lr : 0) * lda;
  const float* bp = B + (int64_t)(bok ? n0 + lr : 0) * ldb;
  const int wi = (w >> 1) * 32, wj = (w & 1) * 32;
  f64x4 acc[2][2];
#pragma unroll
  for (int x = 0; x < 2; ++x)
#pragma unroll
    for (int y = 0; y < 2; ++y) acc[x][y] = f64x4{0.0, 0.0, 0.0, 0.0};
  float ra[8], rb[8];
  auto fetch = [&](int kb) {
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const int k = kb + kq + e;
      ra[e] = (aok && k < k1) ? ap[k] : 0.f;
      rb[e] = (bok && k < k1) ? bp[k] : 0.f;
    }
  };
  if (k0 < k1) fetch(k0);
  for (int kb = k0; kb < k1; kb += 32) {
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      As[kq + e][lr] = ra[e];
      Bs[kq + e][lr] = rb[e];
    }
    __syncthreads();
    if (kb + 32 < k1) fetch(kb + 32);
#pragma unroll
    for (int ks = 0; ks < 32; ks += 4) {
      const int k = ks + (lane >> 4);
      const double a0 = As[k][wi + (lane & 15)], a1 = As[k][wi + 16 + (lane & 15)];
      const double b0 = Bs[k][wj + (lane & 15)], b1 = Bs[k][wj + 16 + (lane & 15)];
      acc[0][0] = mfma64(a0, b0, acc[0][0]);
      acc[0][1] = mfma64(a0, b1, acc[0][1]);
      acc[1][0] = mfma64(a1, b0, acc[1][0]);
      acc[1][1] = mfma64(a1, b1, acc[1][1]);
    }
    __syncthreads();
  }
#pragma unroll
  for (int x = 0; x < 2; ++x)
#pragma unroll
    for (int y = 0; y < 2; ++y)
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        const int i = m0 + wi + 16 * x + 4 * v + (lane >> 4);
        const int j = n0 + wj + 16 * y + (lane & 15);
        if (i >= M || j >= N) continue;
        if (EPI == 0) {
          out64[((int64_t)blockIdx.z * M + i) * ldo + j] = acc[x][y][v];
        } else if (EPI == 1) {
          if (i > j) continue;   // the mirror of (j, i), written by that entry
          const float c = (float)(0.5 * (acc[x][y][v] - (i == j ? 1.0 : 0.0)));
          out32[(int64_t)i * ldo + j] = c;
          out32[(int64_t)j * ldo + i] = c;
        } else if (i / kJB <= j / kJB) {
          out64[pk_off(i / kJB, j / kJB, (int)ldo) + (i % kJB) * kJB + (j % kJB)] = acc[x][y][v];
        }
      }
}

// out[i] = sum over splits of part[s * count + i] in a fixed order (fp64)
__global__ void k_reduce_splits64(const double* __restrict__ part, int splits, int64_t count,
                                  double* __restrict__ out) {
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < count; i += stride) {
    double s = 0.0;
    for (int z0 = 0; z0 < splits; z0 += 8) {
      double t[8];
#pragma unroll
      for (int j = 0; j < 8; ++j) t[j] = z0 + j < splits ? part[(int64_t)(z0 + j) * count + i] : 0.0;
#pragma unroll
      for (int j = 0; j < 8; ++j) s += t[j];
    }
    out[i] = s;
  }
}

// packed upper blocks of the sum over splits of n x n partials (fixed order)
__global__ void k_reduce_pack(const double* __restrict__ part, int splits, int n, int nb,
                              double* __restrict__ Apk) {
  const int64_t count = (int64_t)n * n;
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t e = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; e < count; e += stride) {
    const int i = (int)(e / n), j = (int)(e % n);
    if (i / kJB > j / kJB) continue;
    double s = 0.0;
    for (int z0 = 0; z0 < splits; z0 += 8) {
      double t[8];
#pragma unroll
      for (int q = 0; q < 8; ++q) t[q] = z0 + q < splits ? part[(int64_t)(z0 + q) * count + e] : 0.0;
#pragma unroll
      for (int q = 0; q < 8; ++q) s += t[q];
    }
    Apk[pk_off(i / kJB, j / kJB, nb) + (i % kJB) * kJB + (j % kJB)] = s;
  }
}

// the Newton-Schulz correction (C - I) / 2 (fp32, K x K, both triangles)
// from the fp64 partials of k_gram64<0> (upper tiles), summed in split order
__global__ void k_ns_reduce(const double* __restrict__ part, int splits, int K, float* __restrict__ out) {
  const int64_t count = (int64_t)K * K;
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t e = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; e < count; e += stride) {
    const int i = (int)(e / K), j = (int)(e % K);
    const int64_t src = (int64_t)(i < j ? i : j) * K + (i < j ? j : i);
    double c = 0.0;
    for (int z = 0; z < splits; ++z) c += part[(int64_t)z * count + src];
    out[e] = (float)(0.5 * (c - (i == j ? 1.0 : 0.0)));
  }
}

// contraction splits of the n x n Gram over Kc: enough workgroups for the
// chip when the tiles alone are few, slices of at least 512
int gram_splits(int64_t n, int64_t Kc) {
  const int64_t t = (n + 63) / 64;
  const int64_t tiles = t * (t + 1) / 2;
  if (tiles >= 256) return 1;
  int64_t sp = (512 + tiles - 1) / tiles;
  const int64_t mx = (Kc + 511) / 512;
  if (sp > mx) sp = mx;
  return sp < 1 ? 1 : (int)sp;
}

hipError_t launch_gram_packed(const float* W, int64_t ld, int64_t n, int64_t Kc, double* Apk, double* part64,
                              hipStream_t s) {
  const int nb = (int)((n + kJB - 1) / kJB);
  hipError_t e = launch_fill_zero(Apk, (size_t)pk_doubles(nb) * 8, s);
  if (e != hipSuccess) return e;
  const int t = (int)((n + 63) / 64);
  const int splits = part64 ? gram_splits(n, Kc) : 1;
  if (splits == 1) {
    hipLaunchKernelGGL(k_gram64<2>, dim3(t, t, 1), dim3(256), 0, s, W, ld, W, ld, (int)n, (int)n, (int)Kc,
                       (int)Kc, Apk, (float*)nullptr, (int64_t)nb);
  } else {
    const int kslice = (int)(((Kc + splits - 1) / splits + 31) / 32 * 32);
    hipLaunchKernelGGL(k_gram64<0>, dim3(t, t, splits), dim3(256), 0, s, W, ld, W, ld, (int)n, (int)n,
                       (int)Kc, kslice, part64, (float*)nullptr, n);
    hipLaunchKernelGGL(k_reduce_pack, dim3(grid_n(n * n)), dim3(256), 0, s, part64, splits, (int)n, nb, Apk);
  }
  return hipGetLastError();
}

// One Newton-Schulz step towards the nearest orthonormal rows,
//   U^T <- U^T - (U^T U - I) U^T / 2,
// with the Gram in fp64: it removes the orthogonality drift that the fp32
// rotations of a refresh accumulate.  Uses W (d x D >= d x d) and Utw as
// scratch.
hipError_t launch_reorth(const MatView& v, hipStream_t s) {
  const int d = (int)v.d;
  dim3 g64((d + 63) / 64, (d + 63) / 64, 1);
  hipLaunchKernelGGL(k_gram64<1>, g64, dim3(256), 0, s, v.Ut, (int64_t)d, v.Ut, (int64_t)d, d, d, d, d,
                     (double*)nullptr, v.Utw, (int64_t)d);
  GemmPlan p1{1, d};
  gemm_launch<false, 2>(v.Utw, d, v.Ut, d, v.W, d, d, d, d, p1, 0, v.Ut, nullptr, s);
  hipError_t e = hipMemcpyAsync(v.Ut, v.W, (size_t)d * d * 4, hipMemcpyDeviceToDevice, s);
  if (e != hipSuccess) return e;
  return hipGetLastError();
}


// ---------------------------------------------------------------------------
// Cholesky S = L L^T and X = L^-1 of the K x K Gram (fp64), blocked in 64 x 64
// tiles (Kp = K rounded up to 64; the padding is the identity).  One launch
// per block column p after a first launch that factors tile (0, 0):
//   trailing tiles (I, Kq), p < Kq <= I:  L_Ip = S_Ip D_p^T,  L_Kqp likewise,
//       S_IKq -= L_Ip L_Kqp^T; the tile (p+1, p+1) then factors itself and
//       inverts its factor into D_{p+1} (in LDS);
//   block row p of X:  X_pp = D_p,  X_pc = -D_p sum_{c <= k < p} L_pk X_kc.
// Every tile a launch reads was finished by an earlier launch.  Products are
// fp64 MFMA on LDS tiles.  The result is written as fp32 Linv (Kp x Kp, zero
// above the diagonal).  A pivot at or below kPivotFloor (a row that depends on
// the rows before it: a rank-deficient block, zero gradients included) is
// taken as 1 and its row is marked, so that the pass can replace it.
// ---------------------------------------------------------------------------
constexpr int CT = kCholTile;
constexpr int CLD = CT + 1;
typedef double CTile[CLD];

__device__ __forceinline__ int chol_row(int x, int v) {
  return (wave_id() >> 1) * 32 + 16 * x + 4 * v + (lane_id() >> 4);
}
__device__ __forceinline__ int chol_col(int y) { return (wave_id() & 1) * 32 + 16 * y + (lane_id() & 15); }

// acc (+)= sign * A B^T, A and B 64 x 64 in LDS (rows of B are output columns);
// each wave owns one 32 x 32 quadrant of the output
__device__ __forceinline__ void tile_abt(const CTile* A, const CTile* B, double sign, f64x4 (&acc)[2][2]) {
  const int lane = lane_id(), w = wave_id();
  const int ri = (w >> 1) * 32 + (lane & 15), cj = (w & 1) * 32 + (lane & 15);
  const int kk = lane >> 4;
#pragma unroll 4
  for (int k0 = 0; k0 < CT; k0 += 4) {
    const int k = k0 + kk;
    const double a0 = sign * A[ri][k], a1 = sign * A[ri + 16][k];
    const double b0 = B[cj][k], b1 = B[cj + 16][k];
    acc[0][0] = mfma64(a0, b0, acc[0][0]);
    acc[0][1] = mfma64(a0, b1, acc[0][1]);
    acc[1][0] = mfma64(a1, b0, acc[1][0]);
    acc[1][1] = mfma64(a1, b1, acc[1][1]);
  }
}

__device__ __forceinline__ void acc_zero(f64x4 (&acc)[2][2]) {
#pragma unroll
  for (int x = 0; x < 2; ++x)
#pragma unroll
    for (int y = 0; y < 2; ++y) acc[x][y] = f64x4{0.0, 0.0, 0.0, 0.0};
}

// LDS tile <- global tile (row-major, ld), optionally transposed
__device__ __forceinline__ void tile_load(const double* __restrict__ src, int64_t ld, CTile* dst, bool tr) {
  for (int e = threadIdx.x; e < CT * CT; e += 256) {
    const int i = e / CT, j = e % CT;
    const double x = src[(int64_t)i * ld + j];
    if (tr) dst[j][i] = x;
    else dst[i][j] = x;
  }
}

// global tile <- LDS tile (lower triangle only when `lower`: zeros above)
__device__ __forceinline__ void tile_store(const CTile* src, double* __restrict__ dst, int64_t ld, bool lower) {
  for (int e = threadIdx.x; e < CT * CT; e += 256) {
    const int i = e / CT, j = e % CT;
    dst[(int64_t)i * ld + j] = (lower && j > i) ? 0.0 : src[i][j];
  }
}

// 1 / sqrt(S_ii) for i < K (1 where S_ii is not positive, and in the padding)
__device__ __forceinline__ double chol_scale(const double* __restrict__ S, int K, int i) {
  if (i >= K) return 1.0;
  const double dii = S[(int64_t)i * K + i];
  return dii > 0.0 ? 1.0 / sqrt(dii) : 1.0;
}

// global fp32 tile <- LDS tile with column j scaled by 1 / sqrt(S_cc), c = c0 + j
__device__ __forceinline__ void tile_store32(const CTile* src, float* __restrict__ dst, int64_t ld,
                                             const double* __restrict__ S, int K, int c0) {
  for (int e = threadIdx.x; e < CT * CT; e += 256) {
    const int i = e / CT, j = e % CT;
    dst[(int64_t)i * ld + j] = (float)(src[i][j] * chol_scale(S, K, c0 + j));
  }
}

__device__ __forceinline__ void acc_to_lds(const f64x4 (&acc)[2][2], CTile* dst, bool tr) {
#pragma unroll
  for (int x = 0; x < 2; ++x)
#pragma unroll
    for (int y = 0; y < 2; ++y)
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        const int i = chol_row(x, v), j = chol_col(y);
        if (tr) dst[j][i] = acc[x][y][v];
        else dst[i][j] = acc[x][y][v];
      }
}

__device__ __forceinline__ double lane_bcast(double x, int l) {
  const uint64_t u = __builtin_bit_cast(uint64_t, x);
  const uint32_t lo = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)u, l);
  const uint32_t hi = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)(u >> 32), l);
  return __builtin_bit_cast(double, ((uint64_t)hi << 32) | lo);
}

// One wave factors the 16 x 16 diagonal block of T at offset o and inverts
// the factor: lane l holds row l % 16 in registers.  Right-looking: after step
// j, column j of L is final and row j of X = L^-1 is final once scaled by
// 1 / L_jj; the later rows then subtract L_ij X_j.  L replaces the block
// (zeros above the diagonal), X goes into Dl at the same place.  A pivot at
// or below kPivotFloor (the row depends on the rows before it) is taken as 1
// with a zero column below it, and the row (global index row0 + o + j) is
// marked in `bad` for replacement.
__device__ __forceinline__ void chol16(CTile* T, CTile* Dl, int o, int row0, int* __restrict__ bad,
                                       bool& marked) {
  const int li = lane_id() & 15;
  double a[16], y[16];
#pragma unroll
  for (int k = 0; k < 16; ++k) {
    a[k] = T[o + li][o + k];
    y[k] = (k == li) ? 1.0 : 0.0;
  }
#pragma unroll
  for (int j = 0; j < 16; ++j) {
    double piv = lane_bcast(a[j], j);
    const bool dep = !(piv > kPivotFloor);
    if (dep) {
      piv = 1.0;
      marked = true;
      if (lane_id() == 0 && bad) bad[row0 + o + j] = 1;
    }
    const double ljj = sqrt(piv), inv = 1.0 / ljj;
    a[j] = (li > j) ? (dep ? 0.0 : a[j] * inv) : ((li == j) ? ljj : 0.0);
#pragma unroll
    for (int k = j + 1; k < 16; ++k) a[k] = fma(-a[j], lane_bcast(a[j], k), a[k]);
    const double sc = (li == j) ? inv : 1.0;
    const double coef = (li > j) ? a[j] : 0.0;
#pragma unroll
    for (int c = 0; c <= j; ++c) {
      y[c] *= sc;
      y[c] = fma(-coef, lane_bcast(y[c], j), y[c]);
    }
  }
  if (lane_id() < 16) {
#pragma unroll
    for (int k = 0; k < 16; ++k) {
      T[o + li][o + k] = a[k];
      Dl[o + li][o + k] = y[k];
    }
  }
}

// acc (+)= sign * X Y^T for 16 x 16 blocks of LDS tiles: X at (xr, xc) of
// tile Xs, Y at (yr, yc) of tile Ys; output C[4v + lane/16][lane % 16]
__device__ __forceinline__ f64x4 blk_abt(const CTile* Xs, int xr, int xc, const CTile* Ys, int yr, int yc,
                                         double sign, f64x4 acc) {
  const int l = lane_id(), r = l & 15, kk = l >> 4;
#pragma unroll
  for (int k0 = 0; k0 < 16; k0 += 4)
    acc = mfma64(sign * Xs[xr + r][xc + k0 + kk], Ys[yr + r][yc + k0 + kk], acc);
  return acc;
}
// acc (+)= sign * X Y for 16 x 16 blocks (Y read down its columns)
__device__ __forceinline__ f64x4 blk_ab(const CTile* Xs, int xr, int xc, const CTile* Ys, int yr, int yc,
                                        double sign, f64x4 acc) {
  const int l = lane_id(), r = l & 15, kk = l >> 4;
#pragma unroll
  for (int k0 = 0; k0 < 16; k0 += 4)
    acc = mfma64(sign * Xs[xr + r][xc + k0 + kk], Ys[yr + k0 + kk][yc + r], acc);
  return acc;
}
__device__ __forceinline__ void blk_store(CTile* Cs, int cr, int cc, f64x4 acc) {
  const int l = lane_id();
#pragma unroll
  for (int v = 0; v < 4; ++v) Cs[cr + 4 * v + (l >> 4)][cc + (l & 15)] = acc[v];
}
__device__ __forceinline__ f64x4 blk_load(const CTile* Cs, int cr, int cc) {
  const int l = lane_id();
  f64x4 acc;
#pragma unroll
  for (int v = 0; v < 4; ++v) acc[v] = Cs[cr + 4 * v + (l >> 4)][cc + (l & 15)];
  return acc;
}

// In-place Cholesky of the SPD tile T (lower triangle; zeros above), then
// Dl = T^-1.  Blocked in 16-column panels: one wave factors and inverts the
// diagonal block, the blocks below it become L_iq = A_iq X_qq^T and the
// trailing lower blocks take A_ij -= L_iq L_jq^T (fp64 MFMA, one block per
// wave).  The off-diagonal blocks of X then follow block row by block row:
// X_ij = -X_ii sum_{j <= k < i} L_ik X_kj.  Dependent rows are marked (see
// chol16); row0 is the global index of the tile's first row.
__device__ void chol_tile(CTile* T, CTile* Dl, int row0, int* __restrict__ bad) {
  const int w = wave_id();
  for (int e = threadIdx.x; e < CT * CT; e += 256) Dl[e / CT][e % CT] = 0.0;
  bool marked = false;
  __syncthreads();
  for (int q = 0; q < 4; ++q) {
    const int o = 16 * q;
    if (w == 0) chol16(T, Dl, o, row0, bad, marked);
    __syncthreads();
    if (w < 3 - q) {
      const int i = 16 * (q + 1 + w);
      const f64x4 acc = blk_abt(T, i, o, Dl, o, o, 1.0, f64x4{0.0, 0.0, 0.0, 0.0});
      blk_store(T, i, o, acc);
    }
    __syncthreads();
    const int nblk = (3 - q) * (4 - q) / 2;
    for (int b = w; b < nblk; b += 4) {
      int bi = q + 1, rem = b;
      while (rem > bi - q - 1) { rem -= bi - q; ++bi; }
      const int bj = q + 1 + rem;
      f64x4 acc = blk_load(T, 16 * bi, 16 * bj);
      acc = blk_abt(T, 16 * bi, o, T, 16 * bj, o, -1.0, acc);
      blk_store(T, 16 * bi, 16 * bj, acc);
    }
    __syncthreads();
  }
  (void)marked;
  for (int bi = 1; bi < 4; ++bi) {
    if (w < bi) {
      f64x4 acc{0.0, 0.0, 0.0, 0.0};
      for (int k = w; k < bi; ++k) acc = blk_ab(T, 16 * bi, 16 * k, Dl, 16 * k, 16 * w, 1.0, acc);
      blk_store(Dl, 16 * bi, 16 * w, acc);
    }
    __syncthreads();
    if (w < bi) {
      const f64x4 acc = blk_ab(Dl, 16 * bi, 16 * bi, Dl, 16 * bi, 16 * w, -1.0, f64x4{0.0, 0.0, 0.0, 0.0});
      blk_store(Dl, 16 * bi, 16 * w, acc);
    }
    __syncthreads();
  }
}

// copy the scaled Gram D^-1/2 S D^-1/2 (K x K, D = diag S) into the padded
// work matrix; block 0 factors tile (0, 0)
__global__ void __launch_bounds__(256)
k_chol_first(const double* __restrict__ S, int K, int Kp, double* __restrict__ Sw,
             double* __restrict__ Lm, double* __restrict__ Dm, int* __restrict__ bad,
             const int* __restrict__ gate) {
  if (*gate) return;
  const int64_t n = (int64_t)Kp * Kp;
  for (int64_t e = blockIdx.x * 256 + threadIdx.x; e < n; e += (int64_t)gridDim.x * 256) {
    const int i = (int)(e / Kp), j = (int)(e % Kp);
    Sw[e] = (i < K && j < K) ? S[(int64_t)i * K + j] * chol_scale(S, K, i) * chol_scale(S, K, j)
                             : (i == j ? 1.0 : 0.0);
  }
  if (blockIdx.x != 0) return;
  __shared__ CTile T[CT], Dl[CT];
  for (int e = threadIdx.x; e < CT * CT; e += 256) {
    const int i = e / CT, j = e % CT;
    T[i][j] = (i < K && j < K) ? S[(int64_t)i * K + j] * chol_scale(S, K, i) * chol_scale(S, K, j)
                               : (i == j ? 1.0 : 0.0);
  }
  __syncthreads();
  chol_tile(T, Dl, 0, bad);
  tile_store(T, Lm, Kp, true);
  tile_store(Dl, Dm, CT, false);
}

__global__ void __launch_bounds__(256)
k_chol_step(int p, int Kp, double* __restrict__ Sw, double* __restrict__ Lm, double* __restrict__ Dm,
            double* __restrict__ Xm, float* __restrict__ Linv, const double* __restrict__ S, int K,
            int* __restrict__ bad, const int* __restrict__ gate) {
  if (*gate) return;
  __shared__ CTile A[CT], B[CT], C[CT];
  const int nt = Kp / CT;
  const int mrows = nt - p - 1;
  const int ntrail = mrows * (mrows + 1) / 2;
  const int b = blockIdx.x;
  const double* Dp = Dm + (int64_t)p * CT * CT;
  auto tile = [&](double* base, int I, int J) { return base + (int64_t)I * CT * Kp + (int64_t)J * CT; };
  f64x4 acc[2][2];
  if (b < ntrail) {
    int ip = 0;
    while ((ip + 1) * (ip + 2) / 2 <= b) ++ip;
    const int jp = b - ip * (ip + 1) / 2;
    const int I = p + 1 + ip, Kq = p + 1 + jp;
    tile_load(Dp, CT, A, false);
    tile_load(tile(Sw, I, p), Kp, B, false);
    __syncthreads();
    acc_zero(acc);
    tile_abt(B, A, 1.0, acc);          // L_Ip = S_Ip D_p^T
    __syncthreads();
    acc_to_lds(acc, B, false);
    if (Kq != I) {
      tile_load(tile(Sw, Kq, p), Kp, C, false);
      __syncthreads();
      acc_zero(acc);
      tile_abt(C, A, 1.0, acc);        // L_Kqp
      __syncthreads();
      acc_to_lds(acc, C, false);
    }
    __syncthreads();
    const CTile* Lk = (Kq != I) ? C : B;
    // acc = S_IKq - L_Ip L_Kqp^T
    double* sik = tile(Sw, I, Kq);
#pragma unroll
    for (int x = 0; x < 2; ++x)
#pragma unroll
      for (int y = 0; y < 2; ++y)
#pragma unroll
        for (int v = 0; v < 4; ++v) acc[x][y][v] = sik[(int64_t)chol_row(x, v) * Kp + chol_col(y)];
    tile_abt(B, Lk, -1.0, acc);
    if (Kq == p + 1) tile_store(B, tile(Lm, I, p), Kp, false);
    if (I == p + 1 && Kq == p + 1) {
      __syncthreads();
      acc_to_lds(acc, A, false);
      __syncthreads();
      chol_tile(A, B, I * CT, bad);
      tile_store(A, tile(Lm, I, I), Kp, true);
      tile_store(B, Dm + (int64_t)I * CT * CT, CT, false);
    } else {
#pragma unroll
      for (int x = 0; x < 2; ++x)
#pragma unroll
        for (int y = 0; y < 2; ++y)
#pragma unroll
          for (int v = 0; v < 4; ++v) sik[(int64_t)chol_row(x, v) * Kp + chol_col(y)] = acc[x][y][v];
    }
    return;
  }
  // block row p of X = L^-1, column block c
  const int c = b - ntrail;
  float* lo = Linv + (int64_t)p * CT * Kp + (int64_t)c * CT;
  if (c > p) {
    for (int e = threadIdx.x; e < CT * CT; e += 256) lo[(int64_t)(e / CT) * Kp + e % CT] = 0.f;
    return;
  }
  tile_load(Dp, CT, A, false);
  if (c == p) {
    __syncthreads();
    tile_store(A, tile(Xm, p, p), Kp, false);
    tile_store32(A, lo, Kp, S, K, c * CT);
    return;
  }
  acc_zero(acc);
  for (int k = c; k < p; ++k) {
    tile_load(tile(Lm, p, k), Kp, B, false);
    tile_load(tile(Xm, k, c), Kp, C, true);
    __syncthreads();
    tile_abt(B, C, 1.0, acc);          // T += L_pk X_kc
    __syncthreads();
  }
  acc_to_lds(acc, C, true);            // C = T^T
  __syncthreads();
  acc_zero(acc);
  tile_abt(A, C, -1.0, acc);           // X_pc = -D_p T
  __syncthreads();
  acc_to_lds(acc, B, false);
  __syncthreads();
  tile_store(B, tile(Xm, p, c), Kp, false);
  tile_store32(B, lo, Kp, S, K, c * CT);
}

static hipError_t launch_chol_inv(const MatView& v, int K, const int* gate, hipStream_t s) {
  const int Kp = chol_pad(K), nt = Kp / CT;
  hipLaunchKernelGGL(k_chol_first, dim3(16), dim3(256), 0, s, v.sub_S, K, Kp, v.sub_T, v.sub_L,
                     v.sub_Dinv, v.sub_bad, gate);
  for (int p = 0; p < nt; ++p) {
    const int m = nt - p - 1;
    hipLaunchKernelGGL(k_chol_step, dim3(m * (m + 1) / 2 + nt), dim3(256), 0, s, p, Kp, v.sub_T,
                       v.sub_L, v.sub_Dinv, v.sub_Li, v.sub_Linv, v.sub_S, K, v.sub_bad, gate);
  }
  return hipGetLastError();
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

__global__ void k_sum_double(const double* __restrict__ x, int n, double* __restrict__ out,
                             const int* __restrict__ gate) {
  if (gate && *gate) return;
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
    sc->stop = 0;
    sc->change2 = 0.0;
    sc->e_in = 0.0;
    sc->e_out = 0.0;
    sc->gate_iter = 0;
    sc->gate_pass = 0;
    sc->repaired = 0;
    sc->reuse_z = 0;
  }
}

// relative eigengap at r of the previous refresh's Ritz values (sigma, K of
// them, descending); a cold start counts as open
__device__ __forceinline__ bool sub_gap_open(const float* __restrict__ sigma, int r, bool cold) {
  if (cold) return true;
  const double s1 = sigma[0], a = sigma[r - 1], b = sigma[r];
  if (!(s1 > 0.0)) return false;
  return (a * a - b * b) / (s1 * s1) >= kSubGapOpen;
}

// after an iteration: the change of the leading r rows, and whether another
// iteration runs (see kSubMinIters)
__global__ void k_sub_step(SubCtl* sc, int r, float tol, const float* __restrict__ sigma, int cold, int cap) {
  if (threadIdx.x != 0 || sc->stop) return;
  const double ch = sqrt(sc->change2 / (double)r);
  if (sc->iters < kHistory) sc->history[sc->iters] = __float_as_uint((float)ch);
  sc->iters += 1;
  if (ch <= (double)tol) sc->converged = 1;
  if (sc->converged || sc->iters >= cap || (sc->iters >= kSubMinIters && !sub_gap_open(sigma, r, cold != 0)))
    sc->stop = 1;
  // converged from a warm start: the basis this iteration started from is
  // within the tolerance of the new one, and its Z (not orthonormalised on a
  // warm start) is the Rayleigh-Ritz product of that basis
  sc->reuse_z = (sc->converged && !cold) ? 1 : 0;
}

// part[b] = the sum of squares (fp64) of the elements b, b + nb, ... of the
// first `count` elements of x (a fixed order: deterministic)
__global__ void k_sumsq_part(const float* __restrict__ x, int64_t count, double* __restrict__ part,
                             const int* __restrict__ gate) {
  if (gate && *gate) return;
  __shared__ double red[4];
  double s = 0.0;
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < count; i += stride) {
    const double v = (double)x[i];
    s += v * v;
  }
  s = wave_sum(s);
  if (lane_id() == 0) red[wave_id()] = s;
  __syncthreads();
  if (threadIdx.x == 0) part[blockIdx.x] = red[0] + red[1] + red[2] + red[3];
}

// *out = 1 (skip the next section) when *skip is set, or when `need` is given
// and *need is not set; 0 otherwise
__global__ void k_gate(int* __restrict__ out, const int* __restrict__ skip, const int* __restrict__ need) {
  if (threadIdx.x == 0) *out = ((skip && *skip) || (need && !*need)) ? 1 : 0;
}

// start of a CholeskyQR pass: no row marked, nothing replaced yet
__global__ void k_pass_reset(int* __restrict__ bad, int K, int* __restrict__ repaired,
                             const int* __restrict__ gate) {
  if (*gate) return;
  for (int k = threadIdx.x; k < K; k += blockDim.x) bad[k] = 0;
  if (threadIdx.x == 0) *repaired = 0;
}

__global__ void k_copy_gated(const float* __restrict__ src, float* __restrict__ dst, int64_t n,
                             const int* __restrict__ gate, const int* __restrict__ gate2) {
  if (*gate || (gate2 && *gate2)) return;
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < n; i += stride) dst[i] = src[i];
}

// Each row k of Y (K x L) that the pass's factorisation marked as dependent
// is replaced by a row of N(0, 1) values (Philox, counter (c, k, mat, tag)):
// a direction that is independent of the other rows with probability one, so
// that the next pass completes the orthonormal block.  In the last pass a
// pass may run, a marked row means the block could not be completed: the
// breakdown bit of the status word.
__global__ void k_orth_repair(float* __restrict__ Y, int64_t L, const int* __restrict__ bad,
                              int* __restrict__ repaired, const int* __restrict__ gate, uint32_t k0,
                              uint32_t k1, uint32_t mat, uint32_t tag, int last_pass,
                              uint32_t* __restrict__ status) {
  if (*gate) return;
  const int k = blockIdx.x;
  if (!bad[k]) return;
  const int64_t n4 = (L + 3) / 4;
  for (int64_t c = threadIdx.x; c < n4; c += blockDim.x) {
    float z[4];
    normals4((uint32_t)c, (uint32_t)k, mat, tag, k0, k1, z);
#pragma unroll
    for (int e = 0; e < 4; ++e)
      if (4 * c + e < L) Y[(int64_t)k * L + 4 * c + e] = z[e];
  }
  if (threadIdx.x == 0) {
    atomicOr(repaired, 1);
    atomicOr(status, last_pass ? kStatusBreakdown : kStatusRepaired);
  }
}

// The refresh's iteration record (iterations; the relative gain of the
// energy ||P Mo||^2 the whole K-row block captures over the last iteration),
// and its status: not converged when the iterations reached their cap with
// the leading rows still moving by more than tol and the block still gaining
// more than tol of captured energy.  (The leading rows alone converge at the
// rate (sigma_{r+1} / sigma_r)^2; the Rayleigh-Ritz step draws the top r from
// the whole oversampled block, so movement without energy gain is not a
// failure.  With the eigengap at r closed the top-r subspace is not
// determined by the data: the block iteration stops after kSubMinIters.)
__global__ void k_sub_finish(const SubCtl* __restrict__ sc, int* __restrict__ info, uint32_t* __restrict__ status,
                             float tol, int cap) {
  if (threadIdx.x != 0) return;
  const double gain = sc->e_out > 0.0 ? (sc->e_out - sc->e_in) / sc->e_out : 0.0;
  info[kInfoSubIters] = sc->iters;
  info[kInfoSubGain] = (int)__float_as_uint((float)gain);
  if (!sc->converged && sc->iters >= cap && gain > (double)tol) atomicOr(status, kStatusSubNotConverged);
}

// energy of the leading r rows of a block (r x L, contiguous) into *out
static void block_energy(const MatView& v, const float* Z, int r, int64_t L, double* out, const int* gate,
                         hipStream_t s) {
  const int nb = kEnergyParts;
  hipLaunchKernelGGL(k_sumsq_part, dim3(nb), dim3(256), 0, s, Z, (int64_t)r * L, v.sub_sums, gate);
  hipLaunchKernelGGL(k_sum_double, dim3(1), dim3(256), 0, s, v.sub_sums, nb, out, gate);
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
  const GemmPlan pz = plan_z(K, D, d);
  mx = std::max(mx, (size_t)pz.splits * K * D);
  return mx;
}

// Philox key of the replacement rows of step t
static void repair_key(uint64_t seed, int64_t t, uint32_t* k0, uint32_t* k1) {
  *k0 = (uint32_t)(seed & 0xFFFFFFFFu) ^ 0x0F1E2D3Cu;
  *k1 = (uint32_t)(seed >> 32) ^ (uint32_t)t ^ 0x4B5A6978u;
}

// the largest oversampled block: r + r / 4 at the largest subspace rank
constexpr int kSubMaxBlock = kMaxSubK + kMaxSubK / 4;
static_assert(kMaxSubK / 4 >= 32, "sub_block takes r + max(32, r / 4)");

// *out = 1 when *gate is set or the K x K Gram S (fp64) is the identity to
// within kOrthSkip: the rows it came from are orthonormal, and the rest of
// their CholeskyQR pass is skipped
__global__ void __launch_bounds__(1024) k_orth_check(const double* __restrict__ S, int K, const int* __restrict__ gate,
                                                     int* __restrict__ out) {
  __shared__ double red[16];
  __shared__ double rs[kSubMaxBlock];   // 1 / sqrt(S_ii) (0 for a zero row)
  if (*gate) {
    if (threadIdx.x == 0) *out = 1;
    return;
  }
  double mx = 0.0;
  for (int i = threadIdx.x; i < K; i += blockDim.x) {
    const double sii = S[(int64_t)i * K + i];
    rs[i] = sii > 0.0 ? 1.0 / sqrt(sii) : 0.0;
    mx = fmax(mx, fabs(sii - 1.0));
  }
  __syncthreads();
  for (int e = threadIdx.x; e < K * K; e += blockDim.x) {
    const int i = e / K, j = e - i * K;
    if (i == j) continue;
    const double si = rs[i], sj = rs[j];
    // a zero row is not orthonormal: no skip
    mx = fmax(mx, (si > 0.0 && sj > 0.0) ? fabs(S[e]) * si * sj : 1.0);
  }
  mx = wave_max(mx);
  if (lane_id() == 0) red[wave_id()] = mx;
  __syncthreads();
  if (threadIdx.x == 0) {
    double m = 0.0;
    for (int w = 0; w < (int)(blockDim.x >> 6); ++w) m = fmax(m, red[w]);
    *out = m <= kOrthSkip ? 1 : 0;
  }
}

// One CholeskyQR pass on the rows of Y (K x L), skipped when *gate is set:
// S = Y Y^T (fp32 MFMA, partial sums added in fp64), the Cholesky factor of
// the diagonally scaled S (dependent rows marked), Y <- L^-1 Y, then every
// marked row replaced by a Gaussian row (SubCtl::repaired tells whether any
// was).
static hipError_t orth_pass(const MatView& v, float* Y, float* Ytmp, int K, int64_t L, const int* gate,
                            uint32_t tag, bool last_pass, bool check, uint64_t seed, int64_t t,
                            const ProfHook& prof, hipStream_t s) {
  const int Kp = chol_pad(K);
  SubCtl* sc = v.sub_ctl;
  hipLaunchKernelGGL(k_pass_reset, dim3(1), dim3(256), 0, s, v.sub_bad, K, &sc->repaired, gate);
  GemmPlan pg = plan_splits(K, K, (int)L);
  gemm_launch<true, 0>(Y, L, Y, L, v.sub_part, K, K, K, (int)L, pg, (int64_t)K * K, nullptr, nullptr, s, gate);
  hipLaunchKernelGGL(k_reduce_splits, dim3(grid_n((int64_t)K * K)), dim3(256), 0, s, v.sub_part,
                     pg.splits, (int64_t)K * K, (float*)nullptr, v.sub_S, gate);
  if (check) {
    // a repeat pass on rows that came out orthonormal changes nothing
    hipLaunchKernelGGL(k_orth_check, dim3(1), dim3(1024), 0, s, v.sub_S, K, gate, &sc->gate_rest);
    gate = &sc->gate_rest;
  }
  prof.begin(GLR_PROF_SUB_CHOL);
  hipError_t ce = launch_chol_inv(v, K, gate, s);
  if (ce != hipSuccess) return ce;
  prof.end(GLR_PROF_SUB_CHOL);
  GemmPlan p1{1, K};
  gemm_launch<false, 0>(v.sub_Linv, Kp, Y, L, Ytmp, L, K, (int)L, K, p1, 0, nullptr, nullptr, s, gate);
  hipLaunchKernelGGL(k_copy_gated, dim3(grid_n((int64_t)K * L)), dim3(256), 0, s, Ytmp, Y, (int64_t)K * L, gate,
                     (const int*)nullptr);
  uint32_t k0, k1;
  repair_key(seed, t, &k0, &k1);
  hipLaunchKernelGGL(k_orth_repair, dim3((unsigned)K), dim3(256), 0, s, Y, L, v.sub_bad, &sc->repaired, gate, k0,
                     k1, (uint32_t)v.mat, tag, last_pass ? 1 : 0, v.status);
  return hipGetLastError();
}

// Rows of Y (K x L) <- an orthonormal basis of their span: `passes`
// CholeskyQR passes on the diagonally scaled Gram, then one more pass only
// when the last one replaced rows (a rank-deficient block); a row still
// dependent in that pass sets the breakdown bit.  Every pass is skipped while
// *outer is set (nullptr: never).
static hipError_t orth_rows(const MatView& v, float* Y, float* Ytmp, int K, int64_t L, int passes,
                            const int* outer, uint32_t tag, uint64_t seed, int64_t t, const ProfHook& prof,
                            hipStream_t s) {
  SubCtl* sc = v.sub_ctl;
  prof.begin(GLR_PROF_SUB_ORTH);
  for (int pass = 0; pass <= passes; ++pass) {
    const bool extra = pass == passes;
    hipLaunchKernelGGL(k_gate, dim3(1), dim3(64), 0, s, &sc->gate_pass, outer, extra ? &sc->repaired : nullptr);
    hipError_t e = orth_pass(v, Y, Ytmp, K, L, &sc->gate_pass, tag + (uint32_t)pass, extra, pass > 0 && !extra,
                             seed, t, prof, s);
    if (e != hipSuccess) return e;
  }
  prof.end(GLR_PROF_SUB_ORTH);
  return hipGetLastError();
}

// sub_Z = P^T Mo (K x D), skipped when *gate is set
static void launch_z(const MatView& v, int K, const int* gate, hipStream_t s) {
  const int64_t d = v.d, D = v.D;
  const GemmPlan pz = plan_z(K, D, d);
  float* out = pz.splits > 1 ? v.sub_part : v.sub_Z;
  if (v.right)   // Mo[a][b] = Mbar[b][a]: B(k=a, j=b) at Mbar[b d + a]
    gemm_launch<true, 0>(v.sub_P, d, v.Mbar, d, out, D, K, (int)D, (int)d, pz, (int64_t)K * D, nullptr, nullptr, s,
                         gate);
  else           // Mo = Mbar (d x D): B(k=a, j=b) at Mbar[a D + b]
    gemm_launch<false, 0>(v.sub_P, d, v.Mbar, D, out, D, K, (int)D, (int)d, pz, (int64_t)K * D, nullptr, nullptr, s,
                          gate);
  if (pz.splits > 1)
    hipLaunchKernelGGL(k_reduce_splits, dim3(grid_n((int64_t)K * D)), dim3(256), 0, s, v.sub_part, pz.splits,
                       (int64_t)K * D, v.sub_Z, (double*)nullptr, gate);
}

hipError_t launch_sub_start(const MatView& v, bool warm, uint64_t seed, int64_t t, hipStream_t s) {
  const int K = sub_block(v.r, v.d);
  hipLaunchKernelGGL(k_sub_reset, dim3(1), dim3(64), 0, s, v.sub_ctl);
  if (warm) {
    // the previous Ritz vectors, orthonormal already
    hipError_t e = hipMemcpyAsync(v.sub_P, v.Ut, (size_t)K * v.d * 4, hipMemcpyDeviceToDevice, s);
    if (e != hipSuccess) return e;
    return hipGetLastError();
  }
  const uint32_t k0 = (uint32_t)(seed & 0xFFFFFFFFu) ^ 0xA5A5A5A5u;
  const uint32_t k1 = (uint32_t)(seed >> 32) ^ 0x3C3C3C3Cu;
  hipLaunchKernelGGL(k_sub_random, dim3(grid_n((int64_t)K * ((v.d + 3) / 4))), dim3(256), 0, s, v.sub_P, K, v.d,
                     k0, k1, (uint32_t)v.mat);
  return orth_rows(v, v.sub_P, v.sub_Pn, K, v.d, 2, nullptr, 0xC0000000u, seed, t, ProfHook{}, s);
}

// One iteration, skipped as a whole (every launch returns at once) once an
// earlier iteration met the tolerance; writes the subspace change into
// sub_ctl.  `it` numbers the iteration within the refresh.
hipError_t launch_sub_iter(const MatView& v, float tol, uint64_t seed, int64_t t, int it, bool cold, int cap,
                           const ProfHook& prof, hipStream_t s) {
  const int K = sub_block(v.r, v.d);
  const int64_t d = v.d, D = v.D;
  SubCtl* sc = v.sub_ctl;
  const int* g = &sc->gate_iter;
  hipLaunchKernelGGL(k_gate, dim3(1), dim3(64), 0, s, &sc->gate_iter, &sc->stop, (const int*)nullptr);
  // Z = P^T Mo  (K x D)
  prof.begin(GLR_PROF_SUB_Z);
  launch_z(v, K, g, s);
  prof.end(GLR_PROF_SUB_Z);
  block_energy(v, v.sub_Z, K, D, &sc->e_in, g, s);
  // Z only carries the span into the next product.  From a cold start one
  // scaled pass keeps it well conditioned; from the previous Ritz vectors its
  // rows are already near orthogonal (scaled by the singular values), which
  // the diagonally scaled CholeskyQR of the next half step absorbs
  const uint32_t tag = 0xC0000000u | ((uint32_t)(it + 1) << 8);
  hipError_t e = hipSuccess;
  if (cold) {
    e = orth_rows(v, v.sub_Z, v.sub_Zt, K, D, 1, g, tag, seed, t, prof, s);
    if (e != hipSuccess) return e;
  }
  // P_new = Z Mo^T  (K x d): B(k=b, j=a) = Mo[a][b]
  GemmPlan p2 = plan_splits(K, (int)d, (int)D);
  prof.begin(GLR_PROF_SUB_P);
  if (v.right)   // Mbar[b d + a]: contiguous along j
    gemm_launch<false, 0>(v.sub_Z, D, v.Mbar, d, v.sub_part, d, K, (int)d, (int)D, p2, (int64_t)K * d, nullptr,
                          nullptr, s, g);
  else           // Mbar[a D + b]: contiguous along k
    gemm_launch<true, 0>(v.sub_Z, D, v.Mbar, D, v.sub_part, d, K, (int)d, (int)D, p2, (int64_t)K * d, nullptr,
                         nullptr, s, g);
  prof.end(GLR_PROF_SUB_P);
  hipLaunchKernelGGL(k_reduce_splits, dim3(grid_n((int64_t)K * d)), dim3(256), 0, s, v.sub_part,
                     p2.splits, (int64_t)K * d, v.sub_Pn, (double*)nullptr, g);
  e = orth_rows(v, v.sub_Pn, v.sub_R, K, d, 2, g, tag | 0x10u, seed, t, prof, s);
  if (e != hipSuccess) return e;
  // change of the leading r rows (their span converges to the top-r span
  // whatever happens to the oversampled rows, which may sit in a noise bulk):
  // R = P_new[:r] - (P_new[:r] P[:r]^T) P[:r] ;  C = P_new[:r] P[:r]^T (r x r)
  const int r = v.r;
  GemmPlan pc = plan_splits(r, r, (int)d);
  gemm_launch<true, 0>(v.sub_Pn, d, v.sub_P, d, v.sub_part, r, r, r, (int)d, pc, (int64_t)r * r, nullptr, nullptr, s,
                       g);
  hipLaunchKernelGGL(k_reduce_splits, dim3(grid_n((int64_t)r * r)), dim3(256), 0, s, v.sub_part,
                     pc.splits, (int64_t)r * r, v.sub_C, (double*)nullptr, g);
  GemmPlan p3{1, r};
  gemm_launch<false, 1>(v.sub_C, r, v.sub_P, d, v.sub_R, d, r, (int)d, r, p3, 0, v.sub_Pn, v.sub_sums, s, g);
  const int nb = gemm_blocks(r, (int)d);
  hipLaunchKernelGGL(k_sum_double, dim3(1), dim3(256), 0, s, v.sub_sums, nb, &sc->change2, g);
  hipLaunchKernelGGL(k_sub_step, dim3(1), dim3(64), 0, s, sc, r, tol, (const float*)v.sigma, cold ? 1 : 0, cap);
  // P <- P_new, unless this iteration converged from a warm start (then P
  // and Z stay those of the basis it started from, for the Rayleigh-Ritz step)
  hipLaunchKernelGGL(k_copy_gated, dim3(grid_n((int64_t)K * d)), dim3(256), 0, s, v.sub_Pn, v.sub_P, (int64_t)K * d,
                     g, (const int*)&sc->reuse_z);
  return hipGetLastError();
}

// Rayleigh-Ritz: B = P^T Mo (K x D) into sub_Z and its fp64 Gram; a MatView
// whose Jacobi finds the eigenvectors Y of B B^T (the left singular vectors of
// B): Y written to rr_Y, sqrt of the eigenvalues to the state's sigma,
// J = 0..r-1, info and status as for a full refresh.
hipError_t launch_sub_rr_begin(const MatView& v, MatView* rr, hipStream_t s) {
  const int K = sub_block(v.r, v.d);
  const int64_t D = v.D;
  // B = P^T Mo, or the last iteration's Z when it is that product already
  launch_z(v, K, &v.sub_ctl->reuse_z, s);
  block_energy(v, v.sub_Z, K, D, &v.sub_ctl->e_out, nullptr, s);
  *rr = v;
  rr->d = K;
  rr->D = D;
  rr->right = false;
  rr->W = v.sub_Z;
  rr->Utw = v.rr_Utw;
  rr->Ut = v.rr_Y;
  rr->Apk = v.rr_Apk;
  rr->Vrot = v.rr_V;
  rr->V64 = v.rr_V64;
  rr->gpart = v.rr_gpart;
  rr->skip = v.rr_skip;
  rr->ctl = v.rr_ctl;
  rr->sigma_w = v.rr_sigw;
  rr->perm = v.rr_perm;
  hipError_t e = launch_eye(v.rr_Utw, K, s);
  if (e != hipSuccess) return e;
  e = launch_gram_packed(v.sub_Z, D, K, D, v.rr_Apk, v.rr_gpart, s);
  if (e != hipSuccess) return e;
  return launch_jac_reset(*rr, s);
}

// U^T rows 0..K-1 = Y P^T (the Ritz vectors, by descending Ritz value), and
// the iteration record
hipError_t launch_sub_rr_end(const MatView& v, float tol, int cap, hipStream_t s) {
  const int K = sub_block(v.r, v.d);
  const int64_t d = v.d;
  GemmPlan p1{1, K};
  gemm_launch<false, 0>(v.rr_Y, K, v.sub_P, d, v.Ut, d, K, (int)d, K, p1, 0, nullptr, nullptr, s);
  // one Newton-Schulz step on the K rows, U^T <- U^T - (U^T U - I) U^T / 2
  // with the Gram in fp64 (the fp32 rotations of the Rayleigh-Ritz Jacobi
  // leave drift of a few 1e-6 on rank-deficient blocks).  The K x K tiles
  // alone are too few for the chip (15 at K = 320): the d contraction is
  // split, its fp64 partials summed in order by k_ns_reduce.
  const int t64 = (K + 63) / 64;
  const int sp = gram_splits(K, d);
  if (sp > 1) {
    const int kslice = (int)(((d + sp - 1) / sp + 31) / 32 * 32);
    const int spe = (int)((d + kslice - 1) / kslice);
    hipLaunchKernelGGL(k_gram64<0>, dim3(t64, t64, spe), dim3(256), 0, s, v.Ut, d, v.Ut, d, K, K, (int)d, kslice,
                       v.rr_gpart, (float*)nullptr, (int64_t)K);
    hipLaunchKernelGGL(k_ns_reduce, dim3(grid_n((int64_t)K * K)), dim3(256), 0, s, v.rr_gpart, spe, K, v.sub_C);
  } else {
    hipLaunchKernelGGL(k_gram64<1>, dim3(t64, t64, 1), dim3(256), 0, s, v.Ut, d, v.Ut, d, K, K, (int)d, (int)d,
                       (double*)nullptr, v.sub_C, (int64_t)K);
  }
  gemm_launch<false, 2>(v.sub_C, K, v.Ut, d, v.sub_R, d, K, (int)d, K, p1, 0, v.Ut, nullptr, s);
  hipError_t e = hipMemcpyAsync(v.Ut, v.sub_R, (size_t)K * d * 4, hipMemcpyDeviceToDevice, s);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(k_sub_finish, dim3(1), dim3(64), 0, s, v.sub_ctl, v.info, v.status, tol, cap);
  return hipGetLastError();
}

}  // namespace glr
