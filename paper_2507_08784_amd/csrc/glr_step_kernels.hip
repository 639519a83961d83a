// Per-step kernels of the GreedyLore compression path on gfx950:
//   worker mean with error feedback, Approx-Top-r scores (MFMA GEMM with a
//   fused Philox/Box-Muller epilogue), top-r selection, projection,
//   fused residual + worker mean + reconstruction + optimizer.
#include "glr_device.hpp"
#include "glr_internal.hpp"

namespace glr {

// ---------------------------------------------------------------------------
// small utilities
// ---------------------------------------------------------------------------
__global__ void k_fill_zero(uint32_t* p, size_t nwords) {
  size_t i = blockIdx.x * (size_t)blockDim.x + threadIdx.x;
  size_t stride = (size_t)gridDim.x * blockDim.x;
  for (; i < nwords; i += stride) p[i] = 0u;
}

__global__ void k_eye(float* Ut, int64_t d) {
  int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x;
  int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (; i < d * d; i += stride) Ut[i] = (i / d == i % d) ? 1.0f : 0.0f;
}

static inline int grid_for(int64_t n, int per_thread = 1) {
  int64_t g = (n + (int64_t)kThreads * per_thread - 1) / ((int64_t)kThreads * per_thread);
  if (g < 1) g = 1;
  if (g > 2048 * 8) g = 2048 * 8;
  return (int)g;
}

hipError_t launch_fill_zero(void* p, size_t bytes, hipStream_t s) {
  size_t words = bytes / 4;
  if (!words) return hipSuccess;
  hipLaunchKernelGGL(k_fill_zero, dim3(grid_for((int64_t)words, 4)), dim3(kThreads), 0, s,
                     (uint32_t*)p, words);
  return hipGetLastError();
}

hipError_t launch_eye(float* Ut, int64_t d, hipStream_t s) {
  hipLaunchKernelGGL(k_eye, dim3(grid_for(d * d, 4)), dim3(kThreads), 0, s, Ut, d);
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// S1 + S2: Mbar = Ebar + (1/N) sum_i G^(i)   (m x n layout; Ebar is the mean
// of the workers' error buffers left by the previous step; G in the storage
// type ST)
// ---------------------------------------------------------------------------
template <class ST>
__device__ __forceinline__ void ef_mean_at(const ST* __restrict__ G, const float* __restrict__ Ebar,
                                           float* __restrict__ Mbar, int64_t mn, int N, uint32_t* status, int check,
                                           int64_t bx, int64_t gx) {
  const int64_t stride = (int64_t)gx * blockDim.x;
  bool bad = false;
  if ((mn & 3) == 0) {
    const int64_t q = mn >> 2;
    for (int64_t i = bx * (int64_t)blockDim.x + threadIdx.x; i < q; i += stride) {
      float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
      for (int w = 0; w < N; ++w) {
        float4 g = ld_nt_e4(G, (int64_t)w * mn + 4 * i);
        if (check) bad |= !(isfinite(g.x) && isfinite(g.y) && isfinite(g.z) && isfinite(g.w));
        acc.x += g.x; acc.y += g.y; acc.z += g.z; acc.w += g.w;
      }
      float4 e = reinterpret_cast<const float4*>(Ebar)[i];
      float4 o;
      o.x = e.x + acc.x / (float)N;
      o.y = e.y + acc.y / (float)N;
      o.z = e.z + acc.z / (float)N;
      o.w = e.w + acc.w / (float)N;
      reinterpret_cast<float4*>(Mbar)[i] = o;
    }
  } else {
    for (int64_t i = bx * (int64_t)blockDim.x + threadIdx.x; i < mn; i += stride) {
      float acc = 0.f;
      for (int w = 0; w < N; ++w) {
        float g = ld_e(G, (int64_t)w * mn + i);
        if (check) bad |= !isfinite(g);
        acc += g;
      }
      Mbar[i] = Ebar[i] + acc / (float)N;
    }
  }
  if (check && bad) atomicOr(status, 1u);
}
template <class ST>
__global__ void k_ef_mean(const ST* __restrict__ G, const float* __restrict__ Ebar,
                          float* __restrict__ Mbar, int64_t mn, int N, uint32_t* status,
                          int check) {
  ef_mean_at(G, Ebar, Mbar, mn, N, status, check, blockIdx.x, gridDim.x);
}

hipError_t launch_ef_mean(const MatView& v, bool check_finite, hipStream_t s) {
  const int64_t mn = v.m * v.n;
  if (v.st16)
    hipLaunchKernelGGL(k_ef_mean<bf16_t>, dim3(grid_for(mn, 4)), dim3(kThreads), 0, s, (const bf16_t*)v.G, v.Ebar,
                       v.Mbar, mn, v.N, v.status, check_finite ? 1 : 0);
  else
    hipLaunchKernelGGL(k_ef_mean<float>, dim3(grid_for(mn, 4)), dim3(kThreads), 0, s, (const float*)v.G, v.Ebar,
                       v.Mbar, mn, v.N, v.status, check_finite ? 1 : 0);
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// S3b: selection scores.  C[b][j] = sum_a Mo[a][b] Ut[j][a]  (C = Mo^T U,
// D x d), never stored: the epilogue folds each column j with v_j (approx:
// lambdabar_j = u_j^T Mbar v_j) or with itself (exact: ||u_j^T Mbar||^2) and
// writes one partial per 128-row tile: part[tile][j].
// ---------------------------------------------------------------------------
constexpr int SEL_BM = 128, SEL_BN = 128;

template <bool RIGHT, bool APPROX, bool BF16, bool VEC = false>
__device__ __forceinline__ void sel_scores_at(const float* __restrict__ Mbar, const float* __restrict__ Ut, int64_t d,
                                              int64_t D, float* __restrict__ part, uint32_t mat, uint32_t tstep,
                                              uint32_t key0, uint32_t key1, int bx, int by) {
  using T = MfmaTile<SEL_BM, SEL_BN, 2, 2>;
  __shared__ __align__(16) float smem[T::LDS_FLOATS];
  __shared__ float red[2][SEL_BN];
  const int m0 = by * SEL_BM;   // rows: b in [0, D)
  const int n0 = bx * SEL_BN;   // cols: j in [0, d)
  T tile;
  LoadK<SEL_BN, 32, false, false, float, VEC> lb(Ut, nullptr, d, n0, (int)d, (int)d, nullptr);
  if (RIGHT) {
    // Mo[a][b] = Mbar[b][a] : A[b][a] contiguous along a
    LoadK<SEL_BM, 32, false, false, float, VEC> la(Mbar, nullptr, d, m0, (int)D, (int)d, nullptr);
    tile.template run<BF16>(la, lb, (int)d, smem);
  } else {
    // Mo[a][b] = Mbar[a][b] : A[b][a] contiguous along b
    LoadR<SEL_BM, 32, false, false, float, VEC> la(Mbar, nullptr, D, m0, (int)D, (int)d);
    tile.template run<BF16>(la, lb, (int)d, smem);
  }
  const int lane = lane_id();
#pragma unroll
  for (int tn = 0; tn < T::TN; ++tn) {
    const int j = n0 + tile.col(tn);
    float acc = 0.f;
    if (j < d) {
#pragma unroll
      for (int tm = 0; tm < T::TM; ++tm) {
#pragma unroll
        for (int g = 0; g < 4; ++g) {
          const int b0 = m0 + tile.row(tm, 4 * g);   // multiple of 4
          if (b0 >= D) continue;
          if (APPROX) {
            float z[4];
            normals4((uint32_t)(b0 >> 2), (uint32_t)j, mat, tstep, key0, key1, z);
#pragma unroll
            for (int e = 0; e < 4; ++e)
              if (b0 + e < D) acc += tile.acc[tm][tn][4 * g + e] * z[e];
          } else {
#pragma unroll
            for (int e = 0; e < 4; ++e) {
              const float c = tile.acc[tm][tn][4 * g + e];
              acc += c * c;
            }
          }
        }
      }
    }
    acc += __shfl_xor(acc, 32, 64);
    if (lane < 32) red[tile.wm][tile.wn * T::WTN + tn * 32 + lane] = acc;
  }
  __syncthreads();
  if (threadIdx.x < SEL_BN) {
    const int j = n0 + threadIdx.x;
    if (j < d) part[(int64_t)by * d + j] = red[0][threadIdx.x] + red[1][threadIdx.x];
  }
}
// VEC: d and D multiples of 4 and both operands 16-byte aligned, so every
// operand slice loads as whole float4s
template <bool RIGHT, bool APPROX, bool BF16, bool VEC>
__global__ void __launch_bounds__(256)
k_sel_scores(const float* __restrict__ Mbar, const float* __restrict__ Ut, int64_t d, int64_t D,
             float* __restrict__ part, uint32_t mat, uint32_t tstep, uint32_t key0, uint32_t key1) {
  sel_scores_at<RIGHT, APPROX, BF16, VEC>(Mbar, Ut, d, D, part, mat, tstep, key0, key1, blockIdx.x, blockIdx.y);
}

// lambdabar / scores from the tile partials, summed in a fixed order
__device__ __forceinline__ void sel_finish_at(const float* __restrict__ part, int ntiles, int64_t d, int approx,
                                              float* __restrict__ score, int64_t bx) {
  int64_t j = bx * (int64_t)blockDim.x + threadIdx.x;
  if (j >= d) return;
  float s = 0.f;
  for (int t = 0; t < ntiles; ++t) s += part[(int64_t)t * d + j];
  score[j] = approx ? s * s : s;
}
__global__ void k_sel_finish(const float* __restrict__ part, int ntiles, int64_t d, int approx,
                             float* __restrict__ score) {
  sel_finish_at(part, ntiles, d, approx, score, blockIdx.x);
}

hipError_t launch_sel_scores(const MatView& v, bool approx, bool bf16, uint64_t seed, int64_t t, hipStream_t s) {
  if (bf16 && !approx) return hipErrorInvalidValue;
  dim3 grid((unsigned)((v.d + SEL_BN - 1) / SEL_BN), (unsigned)((v.D + SEL_BM - 1) / SEL_BM));
  const uint32_t k0 = (uint32_t)(seed & 0xFFFFFFFFu), k1 = (uint32_t)(seed >> 32);
  const uint32_t tt = (uint32_t)((uint64_t)t & 0xFFFFFFFFu);
  const bool vec = v.d % 4 == 0 && v.D % 4 == 0 && (reinterpret_cast<uintptr_t>(v.Ut) & 15) == 0 &&
                   (reinterpret_cast<uintptr_t>(v.Mbar) & 15) == 0;
#define GLR_SEL1(R, A, B, VE)                                                                         \
  hipLaunchKernelGGL((k_sel_scores<R, A, B, VE>), grid, dim3(kThreads), 0, s, v.Mbar, v.Ut, v.d, v.D, \
                     v.lam_part, (uint32_t)v.mat, tt, k0, k1)
#define GLR_SEL(R, A, B)                       \
  do {                                         \
    if (vec) GLR_SEL1(R, A, B, true);          \
    else GLR_SEL1(R, A, B, false);             \
  } while (0)
  if (v.right) {
    if (bf16) GLR_SEL(true, true, true);
    else if (approx) GLR_SEL(true, true, false);
    else GLR_SEL(true, false, false);
  } else {
    if (bf16) GLR_SEL(false, true, true);
    else if (approx) GLR_SEL(false, true, false);
    else GLR_SEL(false, false, false);
  }
#undef GLR_SEL1
#undef GLR_SEL
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(k_sel_finish, dim3(grid_for(v.d)), dim3(kThreads), 0, s, v.lam_part,
                     (int)grid.y, v.d, approx ? 1 : 0, v.score);
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// argtop_r: descending score, ties to the smaller index; J ascending.
// One block of 1024 threads; n_pad (power of two) 64-bit keys in LDS.
// ---------------------------------------------------------------------------
__device__ __forceinline__ void topr_at(const float* __restrict__ score, int d, int r, int n_pad,
                                        int* __restrict__ J, unsigned char* dyn) {
  uint64_t* keys = reinterpret_cast<uint64_t*>(dyn);
  for (int i = threadIdx.x; i < n_pad; i += blockDim.x) {
    if (i < d) {
      const uint32_t hi = ~float_order(score[i]);   // descending score
      keys[i] = ((uint64_t)hi << 32) | (uint32_t)i; // ties: smaller index first
    } else {
      keys[i] = ~0ull;
    }
  }
  __syncthreads();
  bitonic_sort(keys, n_pad);
  // winners' indices to registers, then reuse the buffer for flags and a scan
  constexpr int MAXW = 8;   // r <= d <= 8192 = 8 * 1024
  int win[MAXW];
#pragma unroll
  for (int q = 0; q < MAXW; ++q) {
    const int k = threadIdx.x + q * (int)blockDim.x;
    win[q] = k < r ? (int)(keys[k] & 0xFFFFFFFFu) : -1;
  }
  __syncthreads();
  int* sel = reinterpret_cast<int*>(dyn);
  int* scan = sel + n_pad;
  for (int i = threadIdx.x; i < d; i += blockDim.x) sel[i] = 0;
  __syncthreads();
#pragma unroll
  for (int q = 0; q < MAXW; ++q)
    if (win[q] >= 0) sel[win[q]] = 1;
  __syncthreads();
  const int per = (d + blockDim.x - 1) / blockDim.x;
  const int lo = threadIdx.x * per;
  int cnt = 0;
  for (int i = lo; i < lo + per && i < d; ++i) cnt += sel[i];
  scan[threadIdx.x] = cnt;
  __syncthreads();
  for (int off = 1; off < (int)blockDim.x; off <<= 1) {
    const int x = (threadIdx.x >= (unsigned)off) ? scan[threadIdx.x - off] : 0;
    __syncthreads();
    scan[threadIdx.x] += x;
    __syncthreads();
  }
  int pos = scan[threadIdx.x] - cnt;
  for (int i = lo; i < lo + per && i < d; ++i)
    if (sel[i]) J[pos++] = i;
}
__global__ void __launch_bounds__(1024)
k_topr(const float* __restrict__ score, int d, int r, int n_pad, int* __restrict__ J) {
  extern __shared__ __align__(16) unsigned char dyn[];
  topr_at(score, d, r, n_pad, J, dyn);
}

__global__ void k_iota(int* J, int r) {
  for (int i = threadIdx.x; i < r; i += blockDim.x) J[i] = i;
}

static int next_pow2(int64_t x) {
  int p = 1;
  while (p < x) p <<= 1;
  return p;
}

size_t topr_lds_bytes(int64_t d) {
  const int n_pad = next_pow2(d < 2 ? 2 : d);
  size_t lds = (size_t)n_pad * 8;
  if (lds < (size_t)(n_pad + 1024) * 4) lds = (size_t)(n_pad + 1024) * 4;
  return lds;
}

hipError_t launch_topr(const MatView& v, hipStream_t s) {
  const int n_pad = next_pow2(v.d < 2 ? 2 : v.d);
  hipLaunchKernelGGL(k_topr, dim3(1), dim3(1024), topr_lds_bytes(v.d), s, v.score, (int)v.d, v.r, n_pad, v.J);
  return hipGetLastError();
}

hipError_t launch_iota_J(const MatView& v, hipStream_t s) {
  hipLaunchKernelGGL(k_iota, dim3(1), dim3(256), 0, s, v.J, v.r);
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// S4: Q^(i) = P^T M^(i), r x D per worker (both orientations), with
// P^T[k][a] = Ut[J[k]][a] and M^(i) = G^(i) + E^(i) fused into the load (G
// and E in the storage type ST, widened to fp32 as they load).  VEC: every
// operand slice loads as whole float4s (proj_vec on the host).
// ---------------------------------------------------------------------------
template <int BM, int BN, int WM, int WN, bool RIGHT, bool FLUSH, class ST, bool VEC = false>
__device__ __forceinline__ void proj_at(const ST* __restrict__ G, const ST* __restrict__ E,
                                        const float* __restrict__ Ut, const int* __restrict__ J,
                                        float* __restrict__ Qpart, int64_t d, int64_t D, int r, int N, int kslice,
                                        int bx, int by, int bz) {
  using T = MfmaTile<BM, BN, WM, WN>;
  __shared__ __align__(16) float smem[T::LDS_FLOATS];
  const int n0 = bx * BN;   // b
  const int m0 = by * BM;   // k (rank index)
  const int w = bz % N;     // worker
  const int z = bz / N;     // slice of the d contraction
  const int64_t k0 = (int64_t)z * kslice;
  const int klen = (int)(d - k0 < kslice ? d - k0 : kslice);
  const int64_t dD = d * D;
  const ST* Gi = G + (int64_t)w * dD;
  const ST* Ei = E + (int64_t)w * dD;
  T tile;
  // fp32 accumulators are added into fp64 ones every 512 terms of the slice
  // (FLUSH), or the slice itself is at most 512 terms
  double dacc[FLUSH ? T::TM : 1][FLUSH ? T::TN : 1][16];
  if (FLUSH) {
#pragma unroll
    for (int tm = 0; tm < T::TM; ++tm)
#pragma unroll
      for (int tn = 0; tn < T::TN; ++tn)
#pragma unroll
        for (int v = 0; v < 16; ++v) dacc[FLUSH ? tm : 0][FLUSH ? tn : 0][v] = 0.0;
  }
  LoadK<BM, 32, false, true, float, VEC> la(Ut + k0, nullptr, d, m0, r, klen, J);
  if (RIGHT) {
    // M^(i) oriented: Mo[a][b] = M[b][a], M is D x d row-major
    LoadK<BN, 32, true, false, ST, VEC> lb(Gi + k0, Ei + k0, d, n0, (int)D, klen, nullptr);
    if constexpr (FLUSH) tile.run(la, lb, klen, smem, dacc);
    else tile.run(la, lb, klen, smem);
  } else {
    LoadR<BN, 32, true, false, ST, VEC> lb(Gi + k0 * D, Ei + k0 * D, D, n0, (int)D, klen);
    if constexpr (FLUSH) tile.run(la, lb, klen, smem, dacc);
    else tile.run(la, lb, klen, smem);
  }
  float* Qz = Qpart + ((int64_t)z * N + w) * r * D;
#pragma unroll
  for (int tm = 0; tm < T::TM; ++tm)
#pragma unroll
    for (int tn = 0; tn < T::TN; ++tn) {
      const int b = n0 + tile.col(tn);
      if (b >= D) continue;
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        const int k = m0 + tile.row(tm, v);
        if (k < r) Qz[(int64_t)k * D + b] = FLUSH ? (float)dacc[FLUSH ? tm : 0][FLUSH ? tn : 0][v] : tile.acc[tm][tn][v];
      }
    }
}
// gy > 1 (several rank tiles over the same columns of G and E): a 1-D grid
// in which the gy rank tiles of a (column tile, worker, slice) triple are 8
// blocks apart, so they run on the same XCD at the same time and the second
// read of those columns hits that XCD's L2 (blocks go to the XCDs in turn);
// gy = 1: the 3-D grid (x column tiles, z worker and slice)
template <int BM, int BN, int WM, int WN, bool RIGHT, bool FLUSH, class ST, bool VEC>
__global__ void __launch_bounds__(256)
k_proj(const ST* __restrict__ G, const ST* __restrict__ E, const float* __restrict__ Ut,
       const int* __restrict__ J, float* __restrict__ Qpart, int64_t d, int64_t D, int r, int N, int kslice,
       int gx, int gy, int ntiles) {
  int bx = blockIdx.x, by = blockIdx.y, bz = blockIdx.z;
  if (gy > 1) {
    const int L = blockIdx.x, xcd = L & 7, slot = L >> 3;
    by = slot % gy;
    const int tile = (slot / gy) * 8 + xcd;
    if (tile >= ntiles) return;
    bx = tile % gx;
    bz = tile / gx;
  }
  proj_at<BM, BN, WM, WN, RIGHT, FLUSH, ST, VEC>(G, E, Ut, J, Qpart, d, D, r, N, kslice, bx, by, bz);
}
// the conditions under which every loader of the projection takes its
// float4 path: rows of U^T, G and E in whole float4s (d and D multiples of
// 4, so every slice start and length is one), and the arrays aligned
static bool proj_vec(const MatView& v, size_t esz) {
  const uintptr_t al = 4 * esz - 1;
  return v.d % 4 == 0 && v.D % 4 == 0 && (reinterpret_cast<uintptr_t>(v.Ut) & 15) == 0 &&
         (reinterpret_cast<uintptr_t>(v.G) & al) == 0 && (reinterpret_cast<uintptr_t>(v.E) & al) == 0;
}

template <class ST>
static hipError_t launch_proj_st(const MatView& v, hipStream_t s) {
  const int r = v.r;
  const ST* G = static_cast<const ST*>(v.G);
  const ST* E = static_cast<const ST*>(v.E);
  const int splits = proj_splits(v.d, v.D, r, v.N);
  const int64_t kslice = proj_kslice(v.d, v.D, r, v.N);
  float* const out = splits > 1 ? v.Qpart : v.Q;
  const bool vec = proj_vec(v, sizeof(ST));
  dim3 grid;
  grid.z = (unsigned)(v.N * splits);
#define GLR_PROJ1(BM, BN, WM, WN, FL, R, VE)                                                      \
  hipLaunchKernelGGL((k_proj<BM, BN, WM, WN, R, FL, ST, VE>), gr, dim3(kThreads), 0, s, G, E, v.Ut, \
                     v.J, out, v.d, v.D, r, v.N, (int)kslice, gx, gy, ntiles)
#define GLR_PROJ(BM, BN, WM, WN, FL)                                                              \
  do {                                                                                            \
    const int gx = (int)((v.D + BN - 1) / BN), gy = (r + BM - 1) / BM;                            \
    const int ntiles = gx * (int)grid.z;                                                          \
    dim3 gr = grid;                                                                               \
    gr.x = (unsigned)gx;                                                                          \
    gr.y = (unsigned)gy;                                                                          \
    if (gy > 1) gr = dim3((unsigned)(((ntiles + 7) / 8) * 8 * gy));                               \
    if (v.right) {                                                                                \
      if (vec) GLR_PROJ1(BM, BN, WM, WN, FL, true, true);                                         \
      else GLR_PROJ1(BM, BN, WM, WN, FL, true, false);                                            \
    } else {                                                                                      \
      if (vec) GLR_PROJ1(BM, BN, WM, WN, FL, false, true);                                        \
      else GLR_PROJ1(BM, BN, WM, WN, FL, false, false);                                           \
    }                                                                                             \
  } while (0)
  // one rank tile covers all r rows, so G and E are read once.  Up to rank
  // 64 the tile adds its fp32 sums into fp64 every 512 terms; above, the
  // slices are 1024 terms and the reduction adds them in fp64, which keeps
  // fp64 accumulators out of the larger tiles (a 128-row tile holding them
  // spills).  At rank 64 the 64 x 128 tile without the fp64 sums was 10 %
  // slower than the 64 x 64 one with them (fewer, longer blocks).
  if (r <= 32) GLR_PROJ(32, 128, 1, 4, true);
  else if (r <= kProjFlushRank) GLR_PROJ(64, 64, 2, 2, true);
  else if (r <= kProjWideRank) GLR_PROJ(128, 64, 2, 2, false);
  else GLR_PROJ(256, 64, 4, 1, false);
#undef GLR_PROJ
#undef GLR_PROJ1
  return hipGetLastError();
}
hipError_t launch_proj(const MatView& v, hipStream_t s) {
  return v.st16 ? launch_proj_st<bf16_t>(v, s) : launch_proj_st<float>(v, s);
}

// S6 (with the slices of the projection): Q^(i) = sum over slices of the
// partial products, Rbar = (1/N) sum_i Q^(i); both sums in a fixed order, fp64
__device__ __forceinline__ void proj_reduce_at(const float* __restrict__ part, int splits, int N, int64_t rD,
                                               float* __restrict__ Q, float* __restrict__ Rbar, int64_t bx,
                                               int64_t gx) {
  const int64_t stride = (int64_t)gx * blockDim.x;
  for (int64_t i = bx * (int64_t)blockDim.x + threadIdx.x; i < rD; i += stride) {
    double rsum = 0.0;
    for (int w = 0; w < N; ++w) {
      double q = 0.0;
      if (splits > 1) {
        for (int z = 0; z < splits; ++z) q += (double)part[((int64_t)z * N + w) * rD + i];
        Q[(int64_t)w * rD + i] = (float)q;
      } else {
        q = (double)Q[(int64_t)w * rD + i];
      }
      rsum += q;
    }
    Rbar[i] = (float)(rsum / (double)N);
  }
}
__global__ void k_proj_reduce(const float* __restrict__ part, int splits, int N, int64_t rD, float* __restrict__ Q,
                              float* __restrict__ Rbar) {
  proj_reduce_at(part, splits, N, rD, Q, Rbar, blockIdx.x, gridDim.x);
}

hipError_t launch_rbar(const MatView& v, hipStream_t s) {
  const int64_t rD = (int64_t)v.r * v.D;
  const int splits = proj_splits(v.d, v.D, v.r, v.N);
  hipLaunchKernelGGL(k_proj_reduce, dim3(grid_for(rD)), dim3(kThreads), 0, s, v.Qpart, splits, v.N, rD, v.Q,
                     v.Rbar);
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// S5 + S7 + S8 fused, one pass over a ROWS x 64 tile of the m x n layout:
//   C^(i) = (P Q^(i)) in the caller's layout (rank-r MFMA product)
//   E^(i) <- (G^(i) - C^(i)) + E^(i)
//   Ghat  = P Rbar;  Ebar = the mean of the stored E^(i) (summed in
//   registers as they are written: Mbar - Ghat equals it in real
//   arithmetic, but when the residual is small against Mbar that difference
//   keeps only the low bits of two nearly equal fp32 values);
//   optimizer on X with Ghat.
// MFMA rows are tile rows and lanes are tile columns, so that a load or
// store of one accumulator register moves two whole 128-byte rows of 32
// columns: every written line of E, X, the optimizer state and Ebar is
// covered by one instruction (partial-line writes make the memory side
// fetch the line first).  P (gathered rows of U^T) and Q^(i) are staged
// through LDS by the tile engine, 32 rank indices at a time.
// ---------------------------------------------------------------------------
template <int OPT, bool RIGHT, int ROWS, int RO_COLS, class ST>
__device__ __forceinline__ void resid_opt_at(const ST* __restrict__ G, ST* __restrict__ E,
                                             float* __restrict__ Ebar,
            const float* __restrict__ Mbar, const float* __restrict__ Q, const float* __restrict__ Rbar,
            const float* __restrict__ Ut,
            const int* __restrict__ J,
            float* __restrict__ X, float* __restrict__ S1, float* __restrict__ S2, int64_t m,
            int64_t n, int64_t d, int64_t D, int r, int N, OptParams op, int bx, int by) {
  using T = MfmaTile<ROWS, RO_COLS, ROWS / 32, 128 / ROWS>;
  constexpr int TM = T::TM;
  static_assert(T::TN == 1, "one tile column per lane");
  __shared__ __align__(16) float smem[T::LDS_FLOATS];
  const int c0 = bx * RO_COLS;   // first column of the tile
  const int r0 = by * ROWS;      // first row of the tile
  const int64_t mn = m * n;
  // this lane's outputs: column cc, rows r0 + row(tm, v) = rb[tm] + rv(v)
  // with rv(v) = 8 (v / 4) + v % 4 the same in every lane
  T geo;
  const int64_t cc = c0 + geo.col(0);
  const bool cok = cc < n;
  // every m x n array is addressed as a buffer (m n 4 < 2^32 bytes): a
  // uniform descriptor and one 32-bit byte offset per element, shared by all
  // of them; elements outside the matrix take kBufNone
  const uint32_t bytes = (uint32_t)(mn * 4);
  uint32_t ob[TM][16];
#pragma unroll
  for (int tm = 0; tm < TM; ++tm)
#pragma unroll
    for (int v = 0; v < 16; ++v) {
      const int64_t row = r0 + geo.row(tm, v);
      ob[tm][v] = (cok && row < m) ? (uint32_t)((row * n + cc) * 4) : kBufNone;
    }
  // Ebar: the mean of the stored residuals
  float esum[TM][16];
#pragma unroll
  for (int tm = 0; tm < TM; ++tm)
#pragma unroll
    for (int v = 0; v < 16; ++v) esum[tm][v] = 0.f;
  for (int wk = 0; wk < N; ++wk) {
    const BufRsrc Gi = buf_rsrc_s(G + (int64_t)wk * mn, mn);
    const BufRsrc Ei = buf_rsrc_s(E + (int64_t)wk * mn, mn);
    const float* Qi = Q + (int64_t)wk * r * D;
    // G^(i) and E^(i) for this lane's elements, in flight during the product
    float gv[TM][16], eo[TM][16];
#pragma unroll
    for (int tm = 0; tm < TM; ++tm)
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        gv[tm][v] = buf_lde<ST>(Gi, ob[tm][v]);
        eo[tm][v] = buf_lde<ST>(Ei, ob[tm][v]);
      }
    T tile;
    if (!RIGHT) {
      // rows a < d, columns b < D: C[a][b] = sum_k Ut[J[k]][a] Q[k][b]
      LoadR<ROWS, 32, false, true> la(Ut, nullptr, d, r0, (int)d, r, J);
      LoadR<RO_COLS, 32, false> lb(Qi, nullptr, D, c0, (int)D, r);
      tile.run(la, lb, r, smem);
    } else {
      // rows b < D, columns a < d: C[b][a] = sum_k Q[k][b] Ut[J[k]][a]
      LoadR<ROWS, 32, false> la(Qi, nullptr, D, r0, (int)D, r);
      LoadR<RO_COLS, 32, false, true> lb(Ut, nullptr, d, c0, (int)d, r, J);
      tile.run(la, lb, r, smem);
    }
#pragma unroll
    for (int tm = 0; tm < TM; ++tm)
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        // (G - P Q) + E: G and P Q nearly cancel, E is the small part
        const float e = (gv[tm][v] - tile.acc[tm][0][v]) + eo[tm][v];
        buf_ste<ST>(Ei, ob[tm][v], e);
        esum[tm][v] += stored<ST>(e);
      }
  }

  // Ghat = P Rbar (the reconstruction of the averaged payload)
  T tile;
  if (!RIGHT) {
    LoadR<ROWS, 32, false, true> la(Ut, nullptr, d, r0, (int)d, r, J);
    LoadR<RO_COLS, 32, false> lb(Rbar, nullptr, D, c0, (int)D, r);
    tile.run(la, lb, r, smem);
  } else {
    LoadR<ROWS, 32, false> la(Rbar, nullptr, D, r0, (int)D, r);
    LoadR<RO_COLS, 32, false, true> lb(Ut, nullptr, d, c0, (int)d, r, J);
    tile.run(la, lb, r, smem);
  }
  const BufRsrc Xr = buf_rsrc(X, bytes), S1r = buf_rsrc(S1, bytes), Ebr = buf_rsrc(Ebar, bytes);
  const BufRsrc S2r = buf_rsrc(OPT == 1 ? S2 : S1, bytes);
#pragma unroll
  for (int tm = 0; tm < TM; ++tm)
#pragma unroll
    for (int v = 0; v < 16; ++v) {
      const uint32_t o = ob[tm][v];
      const float gh = tile.acc[tm][0][v];
      float xv = buf_ld(Xr, o);
      if (OPT == 2) {
        xv = xv - op.lr * gh;
      } else {
        float s1 = buf_ld(S1r, o);
        if (OPT == 0) {
          s1 = op.beta1 * s1 + (1.0f - op.beta1) * gh;
          xv = xv - op.lr * s1;
        } else {
          float s2 = buf_ld(S2r, o);
          s1 = op.beta1 * s1 + (1.0f - op.beta1) * gh;
          s2 = op.beta2 * s2 + (1.0f - op.beta2) * gh * gh;
          xv = xv - op.lr * s1 / (sqrtf(s2) + op.eps);
          buf_st(S2r, o, s2);
        }
        buf_st(S1r, o, s1);
      }
      const float eb = esum[tm][v] / (float)(N > 0 ? N : 1);
      buf_st(Ebr, o, op.ef ? eb : 0.0f);
      buf_st(Xr, o, xv);
    }
}
// (the stored residuals' running sum for Ebar takes 32 registers per lane
// beside the rest, so three waves per SIMD instead of four, without spills)
template <int OPT, bool RIGHT, int ROWS, int RO_COLS>
__global__ void __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(3, 3)))
k_resid_opt(const float* __restrict__ G, float* __restrict__ E, float* __restrict__ Ebar,
            const float* __restrict__ Mbar, const float* __restrict__ Q, const float* __restrict__ Rbar,
            const float* __restrict__ Ut,
            const int* __restrict__ J,
            float* __restrict__ X, float* __restrict__ S1, float* __restrict__ S2, int64_t m,
            int64_t n, int64_t d, int64_t D, int r, int N, OptParams op) {
  resid_opt_at<OPT, RIGHT, ROWS, RO_COLS, float>(G, E, Ebar, Mbar, Q, Rbar, Ut, J, X, S1, S2, m, n, d, D, r, N,
                                                 op, blockIdx.x, blockIdx.y);
}
// the same with bf16 storage
template <int OPT, bool RIGHT, int ROWS, int RO_COLS>
__global__ void __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(3, 3)))
k_resid_opt16(const bf16_t* __restrict__ G, bf16_t* __restrict__ E, float* __restrict__ Ebar,
              const float* __restrict__ Mbar, const float* __restrict__ Q, const float* __restrict__ Rbar,
              const float* __restrict__ Ut, const int* __restrict__ J, float* __restrict__ X,
              float* __restrict__ S1, float* __restrict__ S2, int64_t m, int64_t n, int64_t d, int64_t D, int r,
              int N, OptParams op) {
  resid_opt_at<OPT, RIGHT, ROWS, RO_COLS, bf16_t>(G, E, Ebar, Mbar, Q, Rbar, Ut, J, X, S1, S2, m, n, d, D, r, N,
                                                  op, blockIdx.x, blockIdx.y);
}

// S5 + S7 + S8 above rank 128, the workers side by side: one 64 x 64 output
// tile of the m x n layout per workgroup (a 32 x 32 MFMA block per wave).
// Each k-slice of P (gathered rows of U^T) is staged once and multiplied
// with the slices of Q^(w) of up to kNW workers into one accumulator per
// worker, so that the MFMAs run back to back over the whole rank-r
// contraction.  Then E^(w) <- (G^(w) - P Q^(w)) + E^(w) for each worker,
// Ghat = (1/N) sum_w P Q^(w) (= P Rbar by linearity, with no product of its
// own), Ebar = the mean of the stored residuals and the optimizer on X.  More than kNW workers take several
// groups (MULTI), the products of the earlier groups summed in registers.
constexpr int kNW = 4;
constexpr int kNWTile = 64;
// the products of one k-slice for all kNW workers of a group, with no branch
// between the MFMAs, so that the LDS reads of the unrolled loop are issued
// ahead of them (a branch per worker made every MFMA wait for its own operand
// read).  The slices of workers beyond N are zero in LDS, so their products
// are zero.
template <bool RIGHT, int BK, int SL, int PT>
__device__ __forceinline__ void nw_slice(const float* smem, int soff, int qoff, int kh, f32x16 (&acc)[kNW]) {
#pragma unroll
  for (int kk = 0; kk < BK / 2; ++kk) {
    const int row = (2 * kk + kh) * PT;
    const float sv = smem[row + soff];
#pragma unroll
    for (int w = 0; w < kNW; ++w) {
      const float qw = smem[(1 + w) * SL + row + qoff];
      acc[w] = RIGHT ? mfma32(qw, sv, acc[w]) : mfma32(sv, qw, acc[w]);
    }
  }
}
// VEC: the operand slices load through buffer descriptors as float4s (d and
// D multiples of 4, U^T and every group's Q within 2^31 bytes)
template <int OPT, bool RIGHT, bool MULTI, class ST, bool VEC>
__global__ void __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(2, 2)))
k_resid_nw(const ST* __restrict__ G, ST* __restrict__ E, float* __restrict__ Ebar,
           const float* __restrict__ Mbar, const float* __restrict__ Q, const float* __restrict__ Ut,
           const int* __restrict__ J, float* __restrict__ X, float* __restrict__ S1, float* __restrict__ S2,
           int64_t m, int64_t n, int64_t d, int64_t D, int r, int N, OptParams op, int rows_fast) {
  constexpr int BK = 32, T = kNWTile;
  constexpr int PT = T + 4, SL = BK * PT;        // LDS pitch and slice size (P, then one per worker)
  __shared__ __align__(16) float smem[(1 + kNW) * SL];
  const int lane = lane_id(), wv = wave_id();
  const int wm = wv >> 1, wn = wv & 1;
  const int kh = lane >> 5, l32 = lane & 31;
  // row tiles are the fast index: the workgroups in flight share the Q
  // slices of a few column tiles, so that each XCD's L2 holds them (and its
  // rows of P) instead of every row tile streaming all of Q again (columns
  // fast only when the column tiles exceed the grid's y extent)
  const int r0 = (rows_fast ? blockIdx.x : blockIdx.y) * T, c0 = (rows_fast ? blockIdx.y : blockIdx.x) * T;
  const int s0 = RIGHT ? c0 : r0, q0 = RIGHT ? r0 : c0;   // first P row / first Q column of the tile
  // the P operand is the MFMA's A (left: tile rows) or B (right: tile columns)
  const int soff = (RIGHT ? wn : wm) * 32 + l32, qoff = (RIGHT ? wm : wn) * 32 + l32;
  const int64_t mn = m * n;
  const uint32_t bytes = (uint32_t)(mn * 4);
  const int64_t col = c0 + wn * 32 + l32;
  float gs[MULTI ? 16 : 1];
  if (MULTI) {
#pragma unroll
    for (int v = 0; v < 16; ++v) gs[MULTI ? v : 0] = 0.f;
  }
  float esum[16];   // the stored residuals' sum over the workers (for Ebar)
#pragma unroll
  for (int v = 0; v < 16; ++v) esum[v] = 0.f;
  f32x16 acc[kNW];
  const int64_t rD = (int64_t)r * D;
  const int nk = (r + BK - 1) / BK;
  for (int w0 = 0; w0 < N; w0 += kNW) {
    const int nw = N - w0 < kNW ? N - w0 : kNW;
#pragma unroll
    for (int w = 0; w < kNW; ++w)
#pragma unroll
      for (int v = 0; v < 16; ++v) acc[w][v] = 0.f;
    // one loader per worker slot, each loading into registers of its own, so
    // that the loads of all slots are in flight together (one loader moved
    // from slot to slot made each slot's loads wait for the previous slot's
    // to land); a slot beyond N reads nothing (contraction length 0).  VEC:
    // buffer loads through one descriptor for U^T and one for this group's Q.
    static_assert(kNW == 4, "one loader per worker slot");
    using LS = std::conditional_t<VEC, LoadRB<T, BK, true>, LoadR<T, BK, false, true>>;
    using LQ = std::conditional_t<VEC, LoadRB<T, BK, false>, LoadR<T, BK, false>>;
    const BufRsrc ur = buf_rsrc(Ut, VEC ? (uint32_t)(d * d * 4) : 0u);
    const BufRsrc qr = buf_rsrc(Q + (int64_t)w0 * rD, VEC ? (uint32_t)(nw * rD * 4) : 0u);
    auto make_s = [&]() {
      if constexpr (VEC) return LS(ur, 0u, (int)d, s0, (int)d, r, J);
      else return LS(Ut, nullptr, d, s0, (int)d, r, J);
    };
    auto slot = [&](int w) {
      if constexpr (VEC) return LQ(qr, (uint32_t)((w < nw ? w : 0) * rD * 4), (int)D, q0, (int)D, w < nw ? r : 0);
      else return LQ(Q + (int64_t)(w0 + (w < nw ? w : 0)) * rD, nullptr, D, q0, (int)D, w < nw ? r : 0);
    };
    LS ls = make_s();
    LQ lq[kNW] = {slot(0), slot(1), slot(2), slot(3)};
    auto fetch = [&](int k0) {
      ls.fetch(k0);
#pragma unroll
      for (int w = 0; w < kNW; ++w) lq[w].fetch(k0);
    };
    auto put = [&]() {
      ls.template put<PT>(smem);
#pragma unroll
      for (int w = 0; w < kNW; ++w) lq[w].template put<PT>(smem + (1 + w) * SL);
    };
    fetch(0);
    put();
    __syncthreads();
    for (int kb = 0; kb < nk; ++kb) {
      const bool more = kb + 1 < nk;
      if (more) fetch((kb + 1) * BK);
      nw_slice<RIGHT, BK, SL, PT>(smem, soff, qoff, kh, acc);
      __syncthreads();
      if (more) {
        put();
        __syncthreads();
      }
    }
    // the residuals of this group's workers
#pragma unroll
    for (int w = 0; w < kNW; ++w) {
      if (w >= nw) break;
      const BufRsrc Gw = buf_rsrc_s(G + (int64_t)(w0 + w) * mn, mn);
      const BufRsrc Ew = buf_rsrc_s(E + (int64_t)(w0 + w) * mn, mn);
      uint32_t ob[16];
      float gv[16], eo[16];
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        const int64_t row = r0 + wm * 32 + mfma32_row(v, lane);
        ob[v] = (row < m && col < n) ? (uint32_t)((row * n + col) * 4) : kBufNone;
        gv[v] = buf_lde<ST>(Gw, ob[v]);
        eo[v] = buf_lde<ST>(Ew, ob[v]);
      }
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        // (G - P Q) + E: G and P Q nearly cancel, E is the small part
        const float e = (gv[v] - acc[w][v]) + eo[v];
        buf_ste<ST>(Ew, ob[v], e);
        esum[v] += stored<ST>(e);
        if (MULTI) gs[MULTI ? v : 0] += acc[w][v];
      }
      __builtin_amdgcn_sched_barrier(0);
    }
  }
  const float inv_n = 1.0f / (float)N;
  const BufRsrc Xr = buf_rsrc(X, bytes), S1r = buf_rsrc(S1, bytes), Ebr = buf_rsrc(Ebar, bytes);
  const BufRsrc S2r = buf_rsrc(OPT == 1 ? S2 : S1, bytes);
#pragma unroll
  for (int v = 0; v < 16; ++v) {
    const int64_t row = r0 + wm * 32 + mfma32_row(v, lane);
    const uint32_t o = (row < m && col < n) ? (uint32_t)((row * n + col) * 4) : kBufNone;
    // workers beyond N hold zero products
    float sum = MULTI ? gs[MULTI ? v : 0] : acc[0][v];
    if (!MULTI) {
#pragma unroll
      for (int w = 1; w < kNW; ++w) sum += acc[w][v];
    }
    const float gh = sum * inv_n;
    float xv = buf_ld(Xr, o);
    float s1 = buf_ld(S1r, o);
    if (OPT == 0) {
      s1 = op.beta1 * s1 + (1.0f - op.beta1) * gh;
      xv = xv - op.lr * s1;
    } else {
      float s2 = buf_ld(S2r, o);
      s1 = op.beta1 * s1 + (1.0f - op.beta1) * gh;
      s2 = op.beta2 * s2 + (1.0f - op.beta2) * gh * gh;
      xv = xv - op.lr * s1 / (sqrtf(s2) + op.eps);
      buf_st(S2r, o, s2);
    }
    buf_st(S1r, o, s1);
    buf_st(Ebr, o, esum[v] * inv_n);
    buf_st(Xr, o, xv);
    if ((v & 3) == 3) __builtin_amdgcn_sched_barrier(0);
  }
}

template <class ST>
static hipError_t launch_resid_opt_st(const MatView& v, const OptParams& o, hipStream_t s) {
  const ST* G = static_cast<const ST*>(v.G);
  ST* E = static_cast<ST*>(v.E);
  if (v.r > kResidWideRank && o.ef) {
    // MSGD / Adam with error feedback above rank 128 (GaLore runs without
    // error feedback): one fused pass with the workers side by side
    const bool multi = v.N > kNW;
    const unsigned rt = (unsigned)((v.m + kNWTile - 1) / kNWTile), ct = (unsigned)((v.n + kNWTile - 1) / kNWTile);
    const int rows_fast = ct <= 65535u ? 1 : 0;
    dim3 gw(rows_fast ? rt : ct, rows_fast ? ct : rt);
    // the conditions of the buffer loaders: float4 rows, and U^T and one
    // group's Q within 2^31 bytes
    const bool vec = v.d % 4 == 0 && v.D % 4 == 0 && (reinterpret_cast<uintptr_t>(v.Ut) & 3) == 0 &&
                     (reinterpret_cast<uintptr_t>(v.Q) & 3) == 0 && v.d * v.d * 4 < ((int64_t)1 << 31) &&
                     (int64_t)kNW * v.r * v.D * 4 < ((int64_t)1 << 31);
#define GLR_RW(OPT, R, MU)                                                                                   \
  do {                                                                                                       \
    if (vec)                                                                                                 \
      hipLaunchKernelGGL((k_resid_nw<OPT, R, MU, ST, true>), gw, dim3(kThreads), 0, s, G, E, v.Ebar, v.Mbar,  \
                         v.Q, v.Ut, v.J, v.X, v.S1, v.S2, v.m, v.n, v.d, v.D, v.r, v.N, o, rows_fast);       \
    else                                                                                                     \
      hipLaunchKernelGGL((k_resid_nw<OPT, R, MU, ST, false>), gw, dim3(kThreads), 0, s, G, E, v.Ebar, v.Mbar, \
                         v.Q, v.Ut, v.J, v.X, v.S1, v.S2, v.m, v.n, v.d, v.D, v.r, v.N, o, rows_fast);       \
  } while (0)
#define GLR_RW2(OPT, R) do { if (multi) GLR_RW(OPT, R, true); else GLR_RW(OPT, R, false); } while (0)
    if (o.opt == 0)      { if (v.right) GLR_RW2(0, true); else GLR_RW2(0, false); }
    else if (o.opt == 1) { if (v.right) GLR_RW2(1, true); else GLR_RW2(1, false); }
    else return hipErrorInvalidValue;
#undef GLR_RW2
#undef GLR_RW
    return hipGetLastError();
  }
  const int nfused = o.ef ? v.N : 0;   // workers whose residual k_resid_opt updates
  constexpr int rows = 64, cols = 64;
  dim3 grid((unsigned)((v.n + cols - 1) / cols), (unsigned)((v.m + rows - 1) / rows));
#define GLR_RO(OPT, R)                                                                                     \
  do {                                                                                                     \
    if constexpr (sizeof(ST) == 2)                                                                         \
      hipLaunchKernelGGL((k_resid_opt16<OPT, R, rows, cols>), grid, dim3(kThreads), 0, s, G, E, v.Ebar,    \
                         v.Mbar, v.Q, v.Rbar, v.Ut, v.J, v.X, v.S1, v.S2, v.m, v.n, v.d, v.D, v.r, nfused, o); \
    else                                                                                                   \
      hipLaunchKernelGGL((k_resid_opt<OPT, R, rows, cols>), grid, dim3(kThreads), 0, s, G, E, v.Ebar,      \
                         v.Mbar, v.Q, v.Rbar, v.Ut, v.J, v.X, v.S1, v.S2, v.m, v.n, v.d, v.D, v.r, nfused, o); \
  } while (0)
  if (o.opt == 0)      { if (v.right) GLR_RO(0, true); else GLR_RO(0, false); }
  else if (o.opt == 1) { if (v.right) GLR_RO(1, true); else GLR_RO(1, false); }
  else if (sizeof(ST) == 2) return hipErrorInvalidValue;   // GaLore runs on fp32 storage only
  else { if (v.right) GLR_RO(2, true); else GLR_RO(2, false); }
#undef GLR_RO
  return hipGetLastError();
}
hipError_t launch_resid_opt(const MatView& v, const OptParams& o, hipStream_t s) {
  return v.st16 ? launch_resid_opt_st<bf16_t>(v, o, s) : launch_resid_opt_st<float>(v, o, s);
}

// Algorithm 5 (distributed Adam-type GaLore): the Adam moments live in the
// r x D subspace (S1 = M, S2 = V, row-major r x D, oriented) and restart from
// zero at every refresh; the step direction Rhat = M / (sqrt(V) + eps)
// replaces Rbar, so that the reconstruction P Rhat and X -= lr P Rhat follow
// in k_resid_opt<2>.  Moments in the main text's form (eq-adam).
__global__ void k_galore_adam(float* __restrict__ Rbar, float* __restrict__ S1, float* __restrict__ S2, int64_t n,
                              float beta1, float beta2, float eps, int reset) {
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < n; i += stride) {
    const float g = Rbar[i];
    const float m0 = reset ? 0.0f : S1[i], v0 = reset ? 0.0f : S2[i];
    const float m1 = beta1 * m0 + (1.0f - beta1) * g;
    const float v1 = beta2 * v0 + (1.0f - beta2) * g * g;
    S1[i] = m1;
    S2[i] = v1;
    Rbar[i] = m1 / (sqrtf(v1) + eps);
  }
}

hipError_t launch_galore_adam(const MatView& v, const OptParams& o, bool reset, hipStream_t s) {
  const int64_t n = (int64_t)v.r * v.D;
  hipLaunchKernelGGL(k_galore_adam, dim3(grid_for(n)), dim3(256), 0, s, v.Rbar, v.S1, v.S2, n, o.beta1, o.beta2,
                     o.eps, reset ? 1 : 0);
  return hipGetLastError();
}

// Algorithm 3 at a refresh step: E^(i) = 0, Ebar = 0, Ghat = Mbar.
template <int OPT, class ST>
__global__ void k_full_refresh(const float* __restrict__ Mbar, ST* __restrict__ E,
                               float* __restrict__ Ebar, float* __restrict__ X,
                               float* __restrict__ S1, float* __restrict__ S2, int64_t mn, int N,
                               OptParams op) {
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < mn; i += stride) {
    const float gh = Mbar[i];
    for (int w = 0; w < N; ++w) E[(int64_t)w * mn + i] = ST(0);
    Ebar[i] = 0.f;
    float x = X[i];
    if (OPT == 0) {
      const float mm = op.beta1 * S1[i] + (1.0f - op.beta1) * gh;
      S1[i] = mm;
      x = x - op.lr * mm;
    } else {
      const float m1 = op.beta1 * S1[i] + (1.0f - op.beta1) * gh;
      const float m2 = op.beta2 * S2[i] + (1.0f - op.beta2) * gh * gh;
      S1[i] = m1;
      S2[i] = m2;
      x = x - op.lr * m1 / (sqrtf(m2) + op.eps);
    }
    X[i] = x;
  }
}

template <class ST>
static hipError_t launch_full_refresh_st(const MatView& v, const OptParams& o, hipStream_t s) {
  const int64_t mn = v.m * v.n;
  ST* E = static_cast<ST*>(v.E);
  if (o.opt == 0)
    hipLaunchKernelGGL((k_full_refresh<0, ST>), dim3(grid_for(mn, 4)), dim3(kThreads), 0, s, v.Mbar, E,
                       v.Ebar, v.X, v.S1, v.S2, mn, v.N, o);
  else
    hipLaunchKernelGGL((k_full_refresh<1, ST>), dim3(grid_for(mn, 4)), dim3(kThreads), 0, s, v.Mbar, E,
                       v.Ebar, v.X, v.S1, v.S2, mn, v.N, o);
  return hipGetLastError();
}
hipError_t launch_full_refresh(const MatView& v, const OptParams& o, hipStream_t s) {
  return v.st16 ? launch_full_refresh_st<bf16_t>(v, o, s) : launch_full_refresh_st<float>(v, o, s);
}


// ---------------------------------------------------------------------------
// Grouped selection step: every kernel of a selection step in one launch over
// all matrices.  Each matrix owns a range of blocks (tables of first blocks);
// a block finds its matrix and runs the per-matrix body with the coordinates
// it has in that matrix's own launch, so each matrix computes exactly what its
// own launches compute.  Many small matrices then fill the chip together
// instead of a few CUs each.
// ---------------------------------------------------------------------------
__device__ __forceinline__ int group_find(const int* __restrict__ first, int num, int b) {
  int lo = 0, hi = num - 1;   // the last m with first[m] <= b
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (first[mid] <= b) lo = mid;
    else hi = mid - 1;
  }
  return lo;
}

__device__ __forceinline__ int dev_next_pow2(int64_t x) {
  int p = 1;
  while (p < x) p <<= 1;
  return p;
}

// projection tiles of rank r: BM x BN, WM x WN waves, fp64 flush of the slices
#define GLR_PROJ_TIERS(X)                                   \
  if (r <= 32) X(32, 128, 1, 4, true);                      \
  else if (r <= kProjFlushRank) X(64, 64, 2, 2, true);      \
  else if (r <= kProjWideRank) X(128, 64, 2, 2, false);     \
  else X(256, 64, 4, 1, false)

template <class ST>
__global__ void k_g_ef_mean(const GroupMat* __restrict__ gm, const int* __restrict__ first, int num, int check) {
  const int m = group_find(first, num, blockIdx.x);
  const MatView& v = gm[m].v;
  ef_mean_at(static_cast<const ST*>(v.G), v.Ebar, v.Mbar, v.m * v.n, v.N, v.status, check, blockIdx.x - first[m],
             first[m + 1] - first[m]);
}

template <bool RIGHT, bool APPROX, bool BF16>
__global__ void __launch_bounds__(256)
k_g_sel_scores(const GroupMat* __restrict__ gm, const int* __restrict__ first, int num, uint32_t tstep,
               uint32_t key0, uint32_t key1) {
  const int m = group_find(first, num, blockIdx.x);
  const MatView& v = gm[m].v;
  const int local = blockIdx.x - first[m], gx = (int)((v.d + SEL_BN - 1) / SEL_BN);
  sel_scores_at<RIGHT, APPROX, BF16>(v.Mbar, v.Ut, v.d, v.D, v.lam_part, (uint32_t)v.mat, tstep, key0, key1,
                                     local % gx, local / gx);
}

__global__ void k_g_sel_finish(const GroupMat* __restrict__ gm, const int* __restrict__ first, int num, int approx) {
  const int m = group_find(first, num, blockIdx.x);
  const MatView& v = gm[m].v;
  sel_finish_at(v.lam_part, (int)((v.D + SEL_BM - 1) / SEL_BM), v.d, approx, v.score, blockIdx.x - first[m]);
}

__global__ void __launch_bounds__(1024) k_g_topr(const GroupMat* __restrict__ gm) {
  extern __shared__ __align__(16) unsigned char dyn[];
  const MatView& v = gm[blockIdx.x].v;
  topr_at(v.score, (int)v.d, v.r, dev_next_pow2(v.d < 2 ? 2 : v.d), v.J, dyn);
}

template <int BM, int BN, int WM, int WN, bool RIGHT, bool FLUSH, class ST>
__global__ void __launch_bounds__(256)
k_g_proj(const GroupMat* __restrict__ gm, const int* __restrict__ first, int num) {
  const int m = group_find(first, num, blockIdx.x);
  const GroupMat& g = gm[m];
  const MatView& v = g.v;
  const int gx = (int)((v.D + BN - 1) / BN), gy = (v.r + BM - 1) / BM;
  const int local = blockIdx.x - first[m], rest = local / gx;
  proj_at<BM, BN, WM, WN, RIGHT, FLUSH, ST>(static_cast<const ST*>(v.G), static_cast<const ST*>(v.E), v.Ut, v.J,
                                            g.splits > 1 ? v.Qpart : v.Q, v.d, v.D, v.r, v.N, g.kslice, local % gx,
                                            rest % gy, rest / gy);
}

__global__ void k_g_rbar(const GroupMat* __restrict__ gm, const int* __restrict__ first, int num) {
  const int m = group_find(first, num, blockIdx.x);
  const GroupMat& g = gm[m];
  const MatView& v = g.v;
  proj_reduce_at(v.Qpart, g.splits, v.N, (int64_t)v.r * v.D, v.Q, v.Rbar, blockIdx.x - first[m],
                 first[m + 1] - first[m]);
}

template <int OPT, bool RIGHT, class ST>
__device__ __forceinline__ void g_resid_opt_at(const GroupMat* __restrict__ gm, const int* __restrict__ first,
                                               int num, const OptParams& op) {
  const int m = group_find(first, num, blockIdx.x);
  const MatView& v = gm[m].v;
  const int local = blockIdx.x - first[m], gx = (int)((v.n + 63) / 64);
  resid_opt_at<OPT, RIGHT, 64, 64, ST>(static_cast<const ST*>(v.G), static_cast<ST*>(v.E), v.Ebar, v.Mbar, v.Q,
                                       v.Rbar, v.Ut, v.J, v.X, v.S1, v.S2, v.m, v.n, v.d, v.D, v.r, v.N, op,
                                       local % gx, local / gx);
}
template <int OPT, bool RIGHT>
__global__ void __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(3, 3)))
k_g_resid_opt(const GroupMat* __restrict__ gm, const int* __restrict__ first, int num, OptParams op) {
  g_resid_opt_at<OPT, RIGHT, float>(gm, first, num, op);
}
template <int OPT, bool RIGHT>
__global__ void __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(3, 3)))
k_g_resid_opt16(const GroupMat* __restrict__ gm, const int* __restrict__ first, int num, OptParams op) {
  g_resid_opt_at<OPT, RIGHT, bf16_t>(gm, first, num, op);
}

void group_fill(GroupMat& g, int (&blocks)[kGrpKinds]) {
  const MatView& v = g.v;
  const int r = v.r;
  g.splits = proj_splits(v.d, v.D, r, v.N);
  g.kslice = proj_kslice(v.d, v.D, r, v.N);
  blocks[kGrpEfMean] = grid_for(v.m * v.n, 4);
  blocks[kGrpSelScores] = (int)(((v.d + SEL_BN - 1) / SEL_BN) * ((v.D + SEL_BM - 1) / SEL_BM));
  blocks[kGrpSelFinish] = grid_for(v.d);
  int proj = 0;
#define GLR_PROJ_BLOCKS(BM, BN, WM, WN, FL) proj = (int)(((v.D + BN - 1) / BN) * ((r + BM - 1) / BM) * v.N * g.splits)
  GLR_PROJ_TIERS(GLR_PROJ_BLOCKS);
#undef GLR_PROJ_BLOCKS
  blocks[kGrpProj] = proj;
  blocks[kGrpRbar] = grid_for((int64_t)r * v.D);
  blocks[kGrpResid] = (int)(((v.n + 63) / 64) * ((v.m + 63) / 64));
}

template <class ST>
static hipError_t launch_group_select_st(const GroupPlan& gp, bool check_finite, bool approx, bool bf16,
                                         uint64_t seed, int64_t t, const OptParams& o, int part, hipStream_t s) {
  if (bf16 && !approx) return hipErrorInvalidValue;
  const int num = gp.num, r = gp.r;
  const bool right = gp.right;
  auto table = [&](int kind) { return gp.first + (int64_t)kind * (num + 1); };
  auto grid = [&](int kind) { return dim3((unsigned)gp.total[kind]); };
  if (part != 2)
    hipLaunchKernelGGL(k_g_ef_mean<ST>, grid(kGrpEfMean), dim3(kThreads), 0, s, gp.gm, table(kGrpEfMean), num,
                       check_finite ? 1 : 0);
  if (part == 1) return hipGetLastError();
  const uint32_t k0 = (uint32_t)(seed & 0xFFFFFFFFu), k1 = (uint32_t)(seed >> 32);
  const uint32_t tt = (uint32_t)((uint64_t)t & 0xFFFFFFFFu);
#define GLR_GSEL(R, A, B)                                                                                   \
  hipLaunchKernelGGL((k_g_sel_scores<R, A, B>), grid(kGrpSelScores), dim3(kThreads), 0, s, gp.gm,          \
                     table(kGrpSelScores), num, tt, k0, k1)
  if (right) {
    if (bf16) GLR_GSEL(true, true, true);
    else if (approx) GLR_GSEL(true, true, false);
    else GLR_GSEL(true, false, false);
  } else {
    if (bf16) GLR_GSEL(false, true, true);
    else if (approx) GLR_GSEL(false, true, false);
    else GLR_GSEL(false, false, false);
  }
#undef GLR_GSEL
  hipLaunchKernelGGL(k_g_sel_finish, grid(kGrpSelFinish), dim3(kThreads), 0, s, gp.gm, table(kGrpSelFinish), num,
                     approx ? 1 : 0);
  hipLaunchKernelGGL(k_g_topr, dim3((unsigned)num), dim3(1024), gp.topr_lds, s, gp.gm);
#define GLR_GPROJ(BM, BN, WM, WN, FL)                                                                       \
  do {                                                                                                      \
    if (right)                                                                                              \
      hipLaunchKernelGGL((k_g_proj<BM, BN, WM, WN, true, FL, ST>), grid(kGrpProj), dim3(kThreads), 0, s,    \
                         gp.gm, table(kGrpProj), num);                                                      \
    else                                                                                                    \
      hipLaunchKernelGGL((k_g_proj<BM, BN, WM, WN, false, FL, ST>), grid(kGrpProj), dim3(kThreads), 0, s,   \
                         gp.gm, table(kGrpProj), num);                                                      \
  } while (0)
  GLR_PROJ_TIERS(GLR_GPROJ);
#undef GLR_GPROJ
  hipLaunchKernelGGL(k_g_rbar, grid(kGrpRbar), dim3(kThreads), 0, s, gp.gm, table(kGrpRbar), num);
#define GLR_GRO(OPT, R)                                                                                     \
  do {                                                                                                      \
    if constexpr (sizeof(ST) == 2)                                                                          \
      hipLaunchKernelGGL((k_g_resid_opt16<OPT, R>), grid(kGrpResid), dim3(kThreads), 0, s, gp.gm,           \
                         table(kGrpResid), num, o);                                                         \
    else                                                                                                    \
      hipLaunchKernelGGL((k_g_resid_opt<OPT, R>), grid(kGrpResid), dim3(kThreads), 0, s, gp.gm,             \
                         table(kGrpResid), num, o);                                                         \
  } while (0)
  if (o.opt == 0) { if (right) GLR_GRO(0, true); else GLR_GRO(0, false); }
  else            { if (right) GLR_GRO(1, true); else GLR_GRO(1, false); }
#undef GLR_GRO
  return hipGetLastError();
}
hipError_t launch_group_select(const GroupPlan& gp, bool check_finite, bool approx, bool bf16, uint64_t seed,
                               int64_t t, const OptParams& o, int part, hipStream_t s) {
  return gp.st16 ? launch_group_select_st<bf16_t>(gp, check_finite, approx, bf16, seed, t, o, part, s)
                 : launch_group_select_st<float>(gp, check_finite, approx, bf16, seed, t, o, part, s);
}

}  // namespace glr
