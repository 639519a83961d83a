// Host runtime behind the C ABI in include/greedylore.h: configuration
// checks, the state / workspace layout, and the launch sequence of one step.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <functional>
#include <mutex>
#include <string>
#include <thread>
#include <utility>
#include <vector>

#include "../../include/greedylore.h"
#include "glr_internal.hpp"

using namespace glr;

namespace {

constexpr uint64_t kAlign = 256;
constexpr int64_t kMaxDim = (int64_t)1 << 30;
constexpr int64_t kMaxSortDim = 8192;   // LDS sort of d keys
constexpr int kMaxRank = 1024;
constexpr int kMaxWorkers = 4096;
constexpr uint64_t kHeaderBytes = 256;  // device status word + padding
constexpr int kMaxLanes = 4;            // streams the matrices of one step are spread over

inline uint64_t align_up(uint64_t x) { return (x + kAlign - 1) / kAlign * kAlign; }

thread_local std::string g_create_error;

struct WsLayout {
  uint64_t off_Mbar, off_Q, off_Qpart, off_lam, off_W, off_Utw, off_gram, off_gram2, off_V, off_V64, off_gpart, off_skip,
      off_ctl, off_sigw, off_perm;
  uint64_t off_sP, off_sPn, off_sZ, off_sZt, off_sR, off_spart, off_sS, off_sL, off_sDinv, off_sLi,
      off_sT, off_sLinv, off_sC, off_ssums, off_sctl, off_sbad;
  uint64_t off_rUtw, off_rY, off_rgram, off_rV, off_rV64, off_rgpart, off_rskip, off_rctl, off_rsigw,
      off_rperm;
  uint64_t bytes;
};

// The workspace: one scratch region per matrix, sized by that matrix (so that
// matrices on different streams, and the sweeps of a joint refresh, never
// share one), then the views of the joint refresh (two per matrix: the
// buffer parities of the reordering) and its per-launch block offsets.
struct WsPlan {
  std::vector<WsLayout> mats;
  std::vector<uint64_t> base;
  uint64_t off_views = 0, off_first = 0;
  uint64_t off_gmats = 0, off_gfirst = 0;   // the grouped selection step
  uint64_t bytes = 0;
  int lanes = 1;
};

struct Dims {
  int64_t m, n, d, D;
  int r;
  bool right;
};

Dims dims_of(const glr_config* c, int mat) {
  Dims x;
  x.m = c->shapes[mat].m;
  x.n = c->shapes[mat].n;
  x.d = x.m < x.n ? x.m : x.n;
  x.D = x.m < x.n ? x.n : x.m;
  x.r = (int)((int64_t)c->rank < x.d ? (int64_t)c->rank : x.d);
  x.right = x.m > x.n;
  return x;
}

std::string fmt(const char* f, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, f);
  vsnprintf(buf, sizeof buf, f, ap);
  va_end(ap);
  return buf;
}

glr_status check_config(const glr_config* c, std::string* why) {
  auto bad = [&](glr_status s, const std::string& m) {
    if (why) *why = m;
    return s;
  };
  if (!c) return bad(GLR_ERR_INVALID_ARG, "config is NULL");
  if (c->num_mats < 1) return bad(GLR_ERR_INVALID_ARG, "num_mats must be >= 1");
  if (!c->shapes) return bad(GLR_ERR_INVALID_ARG, "shapes is NULL");
  if (c->num_workers < 1 || c->num_workers > kMaxWorkers)
    return bad(GLR_ERR_INVALID_ARG, fmt("num_workers must be in [1, %d]", kMaxWorkers));
  if (c->rank < 1) return bad(GLR_ERR_INVALID_ARG, "rank must be >= 1");
  if (c->tau < 1) return bad(GLR_ERR_INVALID_ARG, "tau must be >= 1");
  if (c->opt != GLR_MSGD && c->opt != GLR_ADAM && c->opt != GLR_GALORE_ADAM)
    return bad(GLR_ERR_INVALID_ARG, "unknown optimizer");
  if (!(std::isfinite(c->lr) && c->lr > 0.f)) return bad(GLR_ERR_INVALID_ARG, "lr must be finite and > 0");
  if (!(c->beta1 >= 0.f && c->beta1 < 1.f)) return bad(GLR_ERR_INVALID_ARG, "beta1 must be in [0, 1)");
  if (c->opt == GLR_ADAM || c->opt == GLR_GALORE_ADAM) {
    if (!(c->beta2 >= 0.f && c->beta2 < 1.f)) return bad(GLR_ERR_INVALID_ARG, "beta2 must be in [0, 1)");
    if (!(std::isfinite(c->eps) && c->eps > 0.f)) return bad(GLR_ERR_INVALID_ARG, "eps must be finite and > 0");
  }
  if (c->refresh != GLR_REFRESH_COMPRESSED && c->refresh != GLR_REFRESH_FULL)
    return bad(GLR_ERR_INVALID_ARG, "unknown refresh mode");
  if (c->select != GLR_SELECT_APPROX && c->select != GLR_SELECT_EXACT && c->select != GLR_SELECT_APPROX_BF16 &&
      c->select != GLR_SELECT_LAZY)
    return bad(GLR_ERR_INVALID_ARG, "unknown select mode");
  if (c->opt == GLR_GALORE_ADAM && c->refresh != GLR_REFRESH_COMPRESSED)
    return bad(GLR_ERR_INVALID_ARG, "GaLore Adam (Algorithm 5) compresses at refresh steps: use GLR_REFRESH_COMPRESSED");
  if (c->max_sweeps < 1) return bad(GLR_ERR_INVALID_ARG, "max_sweeps must be >= 1");
  if (!(c->tol > 0.f && c->tol < 1.f)) return bad(GLR_ERR_INVALID_ARG, "tol must be in (0, 1)");
  if (c->flags & ~(GLR_CHECK_FINITE | GLR_COLD_START | GLR_NO_EF | GLR_STORE_BF16))
    return bad(GLR_ERR_INVALID_ARG, "unknown flag bits");
  if ((c->flags & GLR_STORE_BF16) && c->opt == GLR_GALORE_ADAM)
    return bad(GLR_ERR_INVALID_ARG, "GLR_STORE_BF16 applies to MSGD and Adam (GaLore Adam keeps no error buffers)");
  for (int i = 0; i < c->num_mats; ++i) {
    const int64_t m = c->shapes[i].m, n = c->shapes[i].n;
    if (m < 1 || n < 1) return bad(GLR_ERR_SHAPE, fmt("matrix %d: shape %lldx%lld must be positive", i, (long long)m, (long long)n));
    if (m > kMaxDim || n > kMaxDim) return bad(GLR_ERR_SHAPE, fmt("matrix %d: dimension above 2^30", i));
    if (m * n >= ((int64_t)1 << 30))   // buffer addressing of one matrix: below 4 GiB
      return bad(GLR_ERR_SHAPE, fmt("matrix %d: m*n = %lld reaches 2^30", i, (long long)(m * n)));
    const Dims x = dims_of(c, i);
    if (x.d > kMaxSortDim)
      return bad(GLR_ERR_SHAPE, fmt("matrix %d: min(m, n) = %lld exceeds %lld", i, (long long)x.d, (long long)kMaxSortDim));
    if (x.r > kMaxRank) return bad(GLR_ERR_SHAPE, fmt("matrix %d: effective rank above %d", i, kMaxRank));
    if ((int64_t)c->num_workers * m * n > ((int64_t)1 << 40))
      return bad(GLR_ERR_SHAPE, fmt("matrix %d: N*m*n too large", i));
  }
  return GLR_OK;
}

// bytes of one element of G^(i) and E^(i)
uint64_t elem_bytes(const glr_config* c) { return (c->flags & GLR_STORE_BF16) ? 2 : 4; }

void mat_layout(const glr_config* c, int mat, uint64_t base, glr_mat_layout* L, uint64_t* end) {
  const Dims x = dims_of(c, mat);
  const uint64_t N = (uint64_t)c->num_workers, mn = (uint64_t)(x.m * x.n);
  uint64_t o = base;
  auto take = [&](uint64_t bytes) {
    uint64_t at = o;
    o = align_up(o + bytes);
    return at;
  };
  L->m = x.m; L->n = x.n; L->d = x.d; L->D = x.D;
  L->right = x.right ? 1 : 0;
  L->r = x.r;
  L->off_E = take(N * mn * elem_bytes(c));
  L->off_Ebar = take(mn * 4);
  L->off_U = take((uint64_t)(x.d * x.d) * 4);
  L->off_sigma = take((uint64_t)x.d * 4);
  L->off_J = take((uint64_t)x.r * 4);
  L->off_score = take((uint64_t)x.d * 4);
  L->off_S1 = take(mn * 4);
  L->off_S2 = (c->opt == GLR_ADAM || c->opt == GLR_GALORE_ADAM) ? take(mn * 4) : 0;
  L->off_Rbar = take((uint64_t)x.r * (uint64_t)x.D * 4);
  L->off_info = take(kInfoInts * 4);
  *end = o;
}

uint64_t state_bytes_of(const glr_config* c) {
  uint64_t o = kHeaderBytes;
  for (int i = 0; i < c->num_mats; ++i) {
    glr_mat_layout L;
    mat_layout(c, i, o, &L, &o);
  }
  return o;
}

WsLayout ws_layout(const glr_config* c, int first, int last) {
  uint64_t mx_mn = 0, mx_Q = 0, mx_Qp = 0, mx_lam = 0, mx_dD = 0, mx_dd = 0, mx_gram = 0, mx_groups = 0, mx_vbuf = 0, mx_d = 0;
  uint64_t s_Kd = 0, s_KD = 0, s_part = 0, s_KK = 0, s_Kp2 = 0, s_nt = 0, s_sums = 0, s_Kp = 0;
  uint64_t r_gram = 0, r_groups = 0, r_vbuf = 0, r_gpart = 0, mx_gpart = 0;
  auto mx = [](uint64_t& a, uint64_t b) { if (b > a) a = b; };
  for (int i = first; i < last; ++i) {
    const Dims x = dims_of(c, i);
    mx(mx_mn, (uint64_t)(x.m * x.n));
    mx(mx_Q, (uint64_t)c->num_workers * (uint64_t)x.r * (uint64_t)x.D);
    const int ps = proj_splits(x.d, x.D, x.r, c->num_workers);
    if (ps > 1) mx(mx_Qp, (uint64_t)ps * c->num_workers * (uint64_t)x.r * (uint64_t)x.D);
    mx(mx_lam, (uint64_t)((x.D + 127) / 128) * (uint64_t)x.d);
    mx(mx_d, (uint64_t)x.d);
    if (use_subspace(c->tau, x.r, x.d)) {
      const int Ki = sub_block(x.r, x.d);
      const uint64_t K = (uint64_t)Ki, Kp = (uint64_t)chol_pad(Ki);
      mx(s_Kd, K * (uint64_t)x.d);
      mx(s_KD, K * (uint64_t)x.D);
      mx(s_part, (uint64_t)sub_part_floats(Ki, x.d, x.D));
      mx(r_groups, (uint64_t)jac_groups(Ki));
      mx(r_vbuf, (uint64_t)jac_vbuf(Ki));
      mx(r_gram, (uint64_t)pk_doubles(jac_blocks(Ki)));
      const int rs = gram_splits(Ki, x.D);
      if (rs > 1) mx(r_gpart, (uint64_t)rs * K * K);
      mx(s_KK, K * K);
      mx(s_Kp, Kp);
      mx(s_Kp2, Kp * Kp);
      mx(s_nt, Kp / kCholTile);
      mx(s_sums, (uint64_t)gemm_blocks(Ki, (int)x.d));
      mx(s_sums, (uint64_t)kEnergyParts);
    } else {
      mx(mx_dD, (uint64_t)(x.d * x.D));
      mx(mx_dd, (uint64_t)(x.d * x.d));
      mx(mx_gram, (uint64_t)pk_doubles(jac_blocks(x.d)));
      const int gs = gram_splits(x.d, x.D);
      if (gs > 1) mx(mx_gpart, (uint64_t)gs * (uint64_t)(x.d * x.d));
      mx(mx_groups, (uint64_t)jac_groups(x.d));
      mx(mx_vbuf, (uint64_t)jac_vbuf(x.d));
    }
  }
  WsLayout w;
  uint64_t o = 0;
  auto take = [&](uint64_t bytes) {
    uint64_t at = o;
    o = align_up(o + (bytes ? bytes : 4));
    return at;
  };
  w.off_Mbar = take(mx_mn * 4);
  w.off_Q = take(mx_Q * 4);
  w.off_Qpart = take(mx_Qp * 4);
  w.off_lam = take(mx_lam * 4);
  w.off_W = take(mx_dD * 4);
  w.off_Utw = take(mx_dd * 4);
  w.off_gram = take(mx_gram * 8);
  w.off_gram2 = take(mx_gram * 8);
  w.off_V = take(2 * mx_vbuf * 4);    // two copies: round parity
  w.off_V64 = take(2 * mx_vbuf * 8);
  w.off_gpart = take(mx_gpart * 8);
  w.off_skip = take(2 * mx_groups * 4);
  w.off_ctl = take(sizeof(JacCtl));
  w.off_sigw = take(mx_d * 4);
  w.off_perm = take(mx_d * 4);
  w.off_sP = take(s_Kd * 4);
  w.off_sPn = take(s_Kd * 4);
  w.off_sZ = take(s_KD * 4);
  w.off_sZt = take(s_KD * 4);
  w.off_sR = take(s_Kd * 4);
  w.off_spart = take(s_part * 4);
  w.off_sS = take(s_KK * 8);
  w.off_sL = take(s_Kp2 * 8);
  w.off_sDinv = take(s_nt * kCholTile * kCholTile * 8);
  w.off_sLi = take(s_Kp2 * 8);
  w.off_sT = take(s_Kp2 * 8);
  w.off_sLinv = take(s_Kp2 * 4);
  w.off_sC = take(s_KK * 4);
  w.off_ssums = take(s_sums * 8);
  w.off_sctl = take(sizeof(SubCtl));
  w.off_sbad = take(s_Kp * 4);
  w.off_rUtw = take(s_KK * 4);
  w.off_rY = take(s_KK * 4);
  w.off_rgram = take(r_gram * 8);
  w.off_rV = take(2 * r_vbuf * 4);
  w.off_rV64 = take(2 * r_vbuf * 8);
  w.off_rgpart = take(r_gpart * 8);
  w.off_rskip = take(2 * r_groups * 4);
  w.off_rctl = take(sizeof(JacCtl));
  w.off_rsigw = take(s_Kd ? 2 * kMaxSubK * 4 : 4);
  w.off_rperm = take(s_Kd ? 2 * kMaxSubK * 4 : 4);
  w.bytes = o;
  return w;
}

WsPlan ws_plan(const glr_config* c) {
  WsPlan p;
  uint64_t o = 0;
  for (int i = 0; i < c->num_mats; ++i) {
    p.mats.push_back(ws_layout(c, i, i + 1));
    p.base.push_back(o);
    o = align_up(o + p.mats.back().bytes);
  }
  p.off_views = o;
  o = align_up(o + (uint64_t)c->num_mats * sizeof(JointMat));
  p.off_first = o;   // kJointKinds tables of num_mats + 1 first blocks, then num_mats flags
  o = align_up(o + ((uint64_t)kJointKinds * ((uint64_t)c->num_mats + 1) + (uint64_t)c->num_mats) * 4);
  p.off_gmats = o;
  o = align_up(o + (uint64_t)c->num_mats * sizeof(GroupMat));
  p.off_gfirst = o;   // the tables of the parts of a grouped selection step
  o = align_up(o + (uint64_t)kGrpKinds * ((uint64_t)c->num_mats + kMaxLanes) * 4);
  p.bytes = o;
  p.lanes = c->num_mats < kMaxLanes ? c->num_mats : kMaxLanes;
  return p;
}

// Matrix -> lane by longest-processing-time-first on an estimate of each matrix's
// work over one refresh period: the per-step streaming of N m x n gradients plus
// about ten Jacobi sweeps (d^3) and the re-orthonormalisation (d^2 D) per tau steps.
std::vector<int> assign_lanes(const glr_config* c, int lanes) {
  std::vector<std::pair<double, int>> w;
  for (int i = 0; i < c->num_mats; ++i) {
    const Dims x = dims_of(c, i);
    const double d = (double)x.d, D = (double)x.D;
    const double per_step = (double)c->num_workers * (double)x.m * (double)x.n;
    w.push_back({per_step + 10.0 * (d * d * d + d * d * D) / (double)c->tau, i});
  }
  std::stable_sort(w.begin(), w.end(), [](const std::pair<double, int>& a, const std::pair<double, int>& b) {
    return a.first > b.first;
  });
  std::vector<double> load((size_t)lanes, 0.0);
  std::vector<int> lane((size_t)c->num_mats, 0);
  for (const auto& it : w) {
    int k = 0;
    for (int j = 1; j < lanes; ++j)
      if (load[(size_t)j] < load[(size_t)k]) k = j;
    lane[(size_t)it.second] = k;
    load[(size_t)k] += it.first;
  }
  return lane;
}

bool aligned(const void* p) { return ((uintptr_t)p % kAlign) == 0; }

}  // namespace

struct ProfMark {
  int group;
  hipEvent_t a, b;
};

struct glr_handle {
  glr_config cfg;
  std::vector<glr_shape> shapes;
  std::vector<glr_mat_layout> lay;
  WsPlan ws;
  char* state = nullptr;
  char* work = nullptr;
  int device = 0;
  int64_t next_t = 0;
  bool suspect = false;
  bool static_ws = false;              // the workspace is the static scratch array (glr_create_static)
  std::string err;
  int jac_inner = 1;   // inner Jacobi sweeps per pair visit
  int jac_sort = 1;    // reorder rows by descending norm before every sweep
  double jac_floor2 = 0x1p-20;  // (f / max_k |w_k|)^2 of the convergence measure
  int sub_iters_warm = kSubCapWarm, sub_iters_cold = kSubCapCold;   // tau = 1 iteration caps
  // Sweep budgets: a refresh enqueues a fixed number of Jacobi sweeps (those
  // after convergence return at once) and never waits for the device.  The
  // sweeps each matrix's last refresh needed come back through pinned host
  // memory, read only once the copy's event has completed.
  std::vector<int> known_sweeps;       // most sweeps a converged refresh took (-1: none yet)
  std::vector<int> known_conv;         // its converged flag
  std::vector<int> info_pending;       // a read-back is in flight
  int64_t repaired_total = 0;          // status reads that found replaced (dependent) rows
  int* info_host = nullptr;            // pinned, 2 ints per matrix
  std::vector<hipEvent_t> info_ev;
  bool lazy = false;                   // P kept between refreshes (Lazy-SVD, GaLore)
  bool ef = true;                      // error feedback
  bool prof = false;
  bool joint = false;                  // refresh steps sweep all matrices in shared launches
  std::vector<JointMat> jm;            // host copies of the joint tables (kept for the async upload)
  std::vector<int> jfirst;
  JointPlan jp;
  bool grouped = false;                // selection steps launch each kernel once for all matrices
  std::vector<int> gfirst;
  GroupPlan gp[kMaxLanes];             // the parts of a grouped selection step (gparts of them)
  int gparts = 0;
  hipEvent_t gev_mean[kMaxLanes] = {}; // end of each part's M-bar
  GroupMat* gring = nullptr;           // pinned host copies of the per-step table, two slots
  hipEvent_t gev[2] = {};              // the upload that last read each slot
  int gslot = 0;
  int lanes = 1;                       // streams in use (<= min(num_mats, 4))
  std::vector<int> lane_of;            // lane of each matrix
  hipStream_t lane_s[kMaxLanes] = {};  // non-blocking streams, created when ws.lanes > 1
  hipEvent_t ev_fork = nullptr;
  hipEvent_t ev_join[kMaxLanes] = {};
  std::mutex mu;                       // err and suspect, written by the lane threads
  std::vector<hipEvent_t> ev_pool;
  size_t ev_used = 0;
  std::vector<ProfMark> marks;
  double prof_ms[GLR_PROF_COUNT] = {0};
  int64_t prof_n[GLR_PROF_COUNT] = {0};
};

namespace {

glr_status fail(glr_handle* h, glr_status s, const std::string& m) {
  if (h) {
    std::lock_guard<std::mutex> lk(h->mu);
    h->err = m;
  } else {
    g_create_error = m;
  }
  return s;
}

glr_status hip_fail(glr_handle* h, hipError_t e, const char* where) {
  if (h) {
    std::lock_guard<std::mutex> lk(h->mu);
    h->suspect = true;
  }
  return fail(h, GLR_ERR_DEVICE, fmt("%s: %s", where, hipGetErrorString(e)));
}

MatView view_of(glr_handle* h, int mat, float* X, const void* G, int lane) {
  const glr_mat_layout& L = h->lay[mat];
  MatView v;
  v.m = L.m; v.n = L.n; v.d = L.d; v.D = L.D;
  v.right = L.right != 0;
  v.r = L.r;
  v.N = h->cfg.num_workers;
  v.mat = mat;
  char* s = h->state;
  v.st16 = (h->cfg.flags & GLR_STORE_BF16) != 0;
  v.E = s + L.off_E;
  v.Ebar = (float*)(s + L.off_Ebar);
  v.Ut = (float*)(s + L.off_U);
  v.sigma = (float*)(s + L.off_sigma);
  v.J = (int*)(s + L.off_J);
  v.score = (float*)(s + L.off_score);
  v.S1 = (float*)(s + L.off_S1);
  v.S2 = L.off_S2 ? (float*)(s + L.off_S2) : nullptr;
  v.Rbar = (float*)(s + L.off_Rbar);
  v.info = (int*)(s + L.off_info);
  v.status = (uint32_t*)s;
  v.X = X;
  v.G = G;
  (void)lane;
  const WsLayout& WL = h->ws.mats[(size_t)mat];
  char* w = h->work + h->ws.base[(size_t)mat];
  v.Mbar = (float*)(w + WL.off_Mbar);
  v.Q = (float*)(w + WL.off_Q);
  v.Qpart = (float*)(w + WL.off_Qpart);
  v.lam_part = (float*)(w + WL.off_lam);
  v.W = (float*)(w + WL.off_W);
  v.Utw = (float*)(w + WL.off_Utw);
  v.Apk = (double*)(w + WL.off_gram);
  v.Apk2 = (double*)(w + WL.off_gram2);
  v.Vrot = (float*)(w + WL.off_V);
  v.V64 = (double*)(w + WL.off_V64);
  v.gpart = (double*)(w + WL.off_gpart);   // sized for every matrix whose Gram is split
  v.skip = (int*)(w + WL.off_skip);
  v.ctl = (JacCtl*)(w + WL.off_ctl);
  v.sigma_w = (float*)(w + WL.off_sigw);
  v.perm = (int*)(w + WL.off_perm);
  v.sub_P = (float*)(w + WL.off_sP);
  v.sub_Pn = (float*)(w + WL.off_sPn);
  v.sub_Z = (float*)(w + WL.off_sZ);
  v.sub_Zt = (float*)(w + WL.off_sZt);
  v.sub_R = (float*)(w + WL.off_sR);
  v.sub_part = (float*)(w + WL.off_spart);
  v.sub_S = (double*)(w + WL.off_sS);
  v.sub_L = (double*)(w + WL.off_sL);
  v.sub_Dinv = (double*)(w + WL.off_sDinv);
  v.sub_Li = (double*)(w + WL.off_sLi);
  v.sub_T = (double*)(w + WL.off_sT);
  v.sub_Linv = (float*)(w + WL.off_sLinv);
  v.sub_C = (float*)(w + WL.off_sC);
  v.sub_sums = (double*)(w + WL.off_ssums);
  v.sub_ctl = (SubCtl*)(w + WL.off_sctl);
  v.sub_bad = (int*)(w + WL.off_sbad);
  v.rr_Utw = (float*)(w + WL.off_rUtw);
  v.rr_Y = (float*)(w + WL.off_rY);
  v.rr_Apk = (double*)(w + WL.off_rgram);
  v.rr_V = (float*)(w + WL.off_rV);
  v.rr_V64 = (double*)(w + WL.off_rV64);
  v.rr_gpart = (double*)(w + WL.off_rgpart);
  v.rr_skip = (int*)(w + WL.off_rskip);
  v.rr_ctl = (JacCtl*)(w + WL.off_rctl);
  v.rr_sigw = (float*)(w + WL.off_rsigw);
  v.rr_perm = (int*)(w + WL.off_rperm);
  return v;
}

hipError_t prof_event(glr_handle* h, hipEvent_t* ev) {
  if (h->ev_used == h->ev_pool.size()) {
    hipEvent_t e;
    hipError_t err = hipEventCreate(&e);
    if (err != hipSuccess) return err;
    h->ev_pool.push_back(e);
  }
  *ev = h->ev_pool[h->ev_used++];
  return hipSuccess;
}

// RAII bracket of one launch group with two events on the step's stream
struct ProfScope {
  glr_handle* h;
  hipStream_t s;
  int group;
  hipEvent_t a = nullptr;
  hipError_t err = hipSuccess;
  ProfScope(glr_handle* h_, hipStream_t s_, int g) : h(h_), s(s_), group(g) {
    if (!h->prof) return;
    err = prof_event(h, &a);
    if (err == hipSuccess) err = hipEventRecord(a, s);
  }
  ~ProfScope() {
    if (!h->prof || err != hipSuccess) return;
    hipEvent_t b;
    if (prof_event(h, &b) != hipSuccess) return;
    if (hipEventRecord(b, s) != hipSuccess) return;
    h->marks.push_back({group, a, b});
  }
};

// the same brackets for groups inside a launcher (ProfHook callback)
struct HookCtx {
  glr_handle* h;
  hipStream_t s;
  hipEvent_t open[GLR_PROF_COUNT];
};

void prof_hook_fn(void* ctx, int group, int begin) {
  HookCtx* c = static_cast<HookCtx*>(ctx);
  glr_handle* h = c->h;
  if (!h->prof || group < 0 || group >= GLR_PROF_COUNT) return;
  hipEvent_t e;
  if (prof_event(h, &e) != hipSuccess || hipEventRecord(e, c->s) != hipSuccess) return;
  if (begin) {
    c->open[group] = e;
  } else if (c->open[group]) {
    h->marks.push_back({group, c->open[group], e});
    c->open[group] = nullptr;
  }
}

// folds recorded marks into the totals (waits for them) and recycles events
hipError_t prof_collect(glr_handle* h) {
  for (const ProfMark& m : h->marks) {
    hipError_t e = hipEventSynchronize(m.b);
    if (e != hipSuccess) return e;
    float ms = 0.f;
    e = hipEventElapsedTime(&ms, m.a, m.b);
    if (e != hipSuccess) return e;
    h->prof_ms[m.group] += ms;
    h->prof_n[m.group] += 1;
  }
  h->marks.clear();
  h->ev_used = 0;
  return hipSuccess;
}

#define GLR_HIP(h, call)                                 \
  do {                                                   \
    hipError_t e_ = (call);                              \
    if (e_ != hipSuccess) return hip_fail(h, e_, #call); \
  } while (0)

// Sweeps to enqueue for a refresh of `mat`: every allowed sweep until a
// refresh of this matrix has been read back converged, then the largest count
// read back so far plus a margin of half of it (at least four): a warm
// refresh can need more sweeps than the cold one before it (7 then 10 have
// been seen on the gradients of a small network).  A refresh that runs out of
// its budget reports GLR_ERR_NOT_CONVERGED like one that runs out of
// max_sweeps, and the next refresh gets every allowed sweep again.
int sweep_budget(glr_handle* h, int mat) {
  const int mx = h->cfg.max_sweeps;
  if (!h->info_host) return mx;   // no read-back buffer (glr_create_static)
  if (h->info_pending[(size_t)mat] && hipEventQuery(h->info_ev[(size_t)mat]) == hipSuccess) {
    h->info_pending[(size_t)mat] = 0;
    const int seen = h->info_host[2 * mat], conv = h->info_host[2 * mat + 1];
    h->known_conv[(size_t)mat] = conv;
    // a miss forgets the record: the next refresh takes max_sweeps
    h->known_sweeps[(size_t)mat] = conv ? std::max(h->known_sweeps[(size_t)mat], seen) : -1;
  }
  const int k = h->known_sweeps[(size_t)mat];
  if (k < 0 || !h->known_conv[(size_t)mat]) return mx;
  const int b = k + std::max(4, k / 2);
  return b < mx ? b : mx;
}

// after a refresh's finish: its sweep count and converged flag to the host
hipError_t read_back_info(glr_handle* h, int mat, const MatView& v, hipStream_t s) {
  if (!h->info_host || h->info_pending[(size_t)mat]) return hipSuccess;   // the previous read-back is still in flight
  hipError_t e = hipMemcpyAsync(h->info_host + 2 * mat, v.info, 2 * sizeof(int), hipMemcpyDeviceToHost, s);
  if (e == hipSuccess) e = hipEventRecord(h->info_ev[(size_t)mat], s);
  if (e == hipSuccess) h->info_pending[(size_t)mat] = 1;
  return e;
}

// one sweep of the round-robin tournament: solve(0), then per round the Gram
// update and the next round's solves fused with this round's U rotation
hipError_t jacobi_sweep(glr_handle* h, const MatView& v, int rounds, int g_solve, int g_update, hipStream_t s) {
  const glr_config& c = h->cfg;
  hipError_t e;
  {
    ProfScope p(h, s, g_solve);
    if ((e = launch_jac_solve(v, 0, c.tol, h->jac_inner, h->jac_floor2, s)) != hipSuccess) return e;
  }
  for (int rd = 0; rd < rounds; ++rd) {
    {
      ProfScope p(h, s, g_update);
      if ((e = launch_jac_update(v, rd, s)) != hipSuccess) return e;
    }
    ProfScope p(h, s, g_solve);
    if (rd + 1 < rounds) e = launch_jac_solve_apply(v, rd + 1, c.tol, h->jac_inner, h->jac_floor2, s);
    else e = launch_jac_apply(v, rd, s);
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

// Semi-Lazy SVD refresh: complete U of Mbar by block Jacobi on the fp64 Gram of
// W = U_prev^T Mo
glr_status svd_begin(glr_handle* h, const MatView& v, int64_t t, hipStream_t s) {
  const bool warm = t > 0 && !(h->cfg.flags & GLR_COLD_START);
  ProfScope p(h, s, GLR_PROF_JAC_INIT);
  GLR_HIP(h, launch_jac_init(v, warm, s));
  return GLR_OK;
}

// sigma, the sorted U, and its re-orthonormalisation, from the view of the
// last sweep
glr_status svd_end(glr_handle* h, const MatView& v, hipStream_t s) {
  ProfScope p(h, s, GLR_PROF_JAC_FINISH);
  GLR_HIP(h, launch_jac_finish(v, h->cfg.max_sweeps, s));
  GLR_HIP(h, launch_reorth(v, s));
  return GLR_OK;
}

// The sweeps are enqueued up to the matrix's budget without waiting: a sweep
// after convergence returns at once, its reordering reduced to a copy into
// the other buffer of the pair (so the result is in the buffer of the last
// enqueued sweep whether that sweep ran or not).
glr_status refresh_svd(glr_handle* h, const MatView& v0, int64_t t, hipStream_t s) {
  const glr_config& c = h->cfg;
  MatView v = v0;   // the sort swaps Apk <-> Apk2 and Utw <-> W
  ProfScope all(h, s, GLR_PROF_REFRESH);
  glr_status st = svd_begin(h, v, t, s);
  if (st != GLR_OK) return st;
  const int rounds = jac_rounds(v.d);
  const int budget = sweep_budget(h, v.mat);
  for (int sw = 0; sw < budget; ++sw) {
    if (h->jac_sort == 1 || (h->jac_sort == 2 && sw == 0)) {
      GLR_HIP(h, launch_jac_sort(v, s));
      std::swap(v.Apk, v.Apk2);
      std::swap(v.Utw, v.W);
    }
    GLR_HIP(h, jacobi_sweep(h, v, rounds, GLR_PROF_JAC_SOLVE, GLR_PROF_JAC_UPDATE, s));
    GLR_HIP(h, launch_jac_check(v, c.tol, s));
  }
  st = svd_end(h, v, s);
  if (st != GLR_OK) return st;
  GLR_HIP(h, read_back_info(h, v.mat, v, s));
  return GLR_OK;
}

// tau = 1 refresh: top-r block of U by oversampled subspace iteration and a
// Rayleigh-Ritz step (block Jacobi SVD of the K x D projection)
glr_status refresh_subspace(glr_handle* h, const MatView& v, int64_t t, hipStream_t s) {
  const glr_config& c = h->cfg;
  const bool warm = t > 0 && !(c.flags & GLR_COLD_START);
  const float sub_tol = 10.0f * c.tol;
  // the cap; the device stops earlier (see kSubMinIters)
  const int iters = warm ? h->sub_iters_warm : h->sub_iters_cold;
  ProfScope all(h, s, GLR_PROF_REFRESH);
  {
    ProfScope p(h, s, GLR_PROF_JAC_INIT);
    GLR_HIP(h, launch_sub_start(v, warm, c.seed, t, s));
  }
  HookCtx hc{h, s, {}};
  const ProfHook hook{&hc, prof_hook_fn};
  for (int it = 0; it < iters; ++it) {
    ProfScope p(h, s, GLR_PROF_SUB_ITER);
    GLR_HIP(h, launch_sub_iter(v, sub_tol, c.seed, t, it, !warm, iters, hook, s));
  }
  MatView rr;
  GLR_HIP(h, launch_sub_rr_begin(v, &rr, s));
  const int rounds = jac_rounds(rr.d);
  const int budget = sweep_budget(h, v.mat);
  for (int sw = 0; sw < budget; ++sw) {
    GLR_HIP(h, jacobi_sweep(h, rr, rounds, GLR_PROF_RR_SOLVE, GLR_PROF_RR_UPDATE, s));
    GLR_HIP(h, launch_jac_check(rr, c.tol, s));
  }
  ProfScope p(h, s, GLR_PROF_JAC_FINISH);
  GLR_HIP(h, launch_jac_finish(rr, c.max_sweeps, s));
  GLR_HIP(h, launch_sub_rr_end(v, sub_tol, iters, s));
  GLR_HIP(h, read_back_info(h, v.mat, v, s));
  return GLR_OK;
}

// the error-feedback mean M-bar of one matrix
glr_status step_head(glr_handle* h, const MatView& v, hipStream_t s) {
  ProfScope p(h, s, GLR_PROF_EF_MEAN);
  GLR_HIP(h, launch_ef_mean(v, (h->cfg.flags & GLR_CHECK_FINITE) != 0, s));
  return GLR_OK;
}

// projection on the chosen columns, their mean, residual and optimizer update
glr_status step_tail(glr_handle* h, const MatView& v, bool refresh, hipStream_t s) {
  const glr_config& c = h->cfg;
  const bool galore = c.opt == GLR_GALORE_ADAM;
  OptParams op{galore ? 2 : c.opt, c.lr, c.beta1, c.beta2, c.eps, h->ef ? 1 : 0};
  {
    ProfScope p(h, s, GLR_PROF_PROJ);
    GLR_HIP(h, launch_proj(v, s));
  }
  {
    ProfScope p(h, s, GLR_PROF_RBAR);
    GLR_HIP(h, launch_rbar(v, s));
  }
  if (galore) GLR_HIP(h, launch_galore_adam(v, op, refresh, s));
  if (refresh && c.refresh == GLR_REFRESH_FULL) {
    ProfScope p(h, s, GLR_PROF_FULL_REFRESH);
    GLR_HIP(h, launch_full_refresh(v, op, s));
  } else {
    ProfScope p(h, s, GLR_PROF_RESID_OPT);
    GLR_HIP(h, launch_resid_opt(v, op, s));
  }
  return GLR_OK;
}

glr_status step_one(glr_handle* h, int mat, float* X, const void* G, int64_t t, hipStream_t s, int lane) {
  const glr_config& c = h->cfg;
  MatView v = view_of(h, mat, X, G, lane);
  const bool refresh = (t % c.tau) == 0;
  glr_status hs = step_head(h, v, s);
  if (hs != GLR_OK) return hs;
  if (refresh) {
    glr_status st = use_subspace(c.tau, v.r, v.d) ? refresh_subspace(h, v, t, s) : refresh_svd(h, v, t, s);
    if (st != GLR_OK) return st;
  } else if (v.r < v.d && !h->lazy) {
    {
      ProfScope p(h, s, GLR_PROF_SELECT);
      GLR_HIP(h, launch_sel_scores(v, c.select != GLR_SELECT_EXACT, c.select == GLR_SELECT_APPROX_BF16, c.seed, t,
                                   s));
    }
    ProfScope p(h, s, GLR_PROF_TOPR);
    GLR_HIP(h, launch_topr(v, s));
  }
  return step_tail(h, v, refresh, s);
}

// per-matrix work (matrix, lane, the lane's stream)
using MatFn = std::function<glr_status(int, int, hipStream_t)>;

// the matrices of one lane, in index order, on that lane's stream
glr_status run_lane(glr_handle* h, int lane, const MatFn& fn, hipStream_t s) {
  for (int i = 0; i < h->cfg.num_mats; ++i) {
    if (h->lane_of[(size_t)i] != lane) continue;
    glr_status st = fn(i, lane, s);
    if (st != GLR_OK) return st;
  }
  return GLR_OK;
}

// Lanes run concurrently: each on its own stream, driven by its own host thread
// (a refresh blocks its thread once per sweep on the convergence flag, so one
// thread could not keep the other streams fed).  The lanes start after the work
// already on `s` and `s` waits for all of them.
glr_status on_lanes(glr_handle* h, hipStream_t s, const MatFn& fn) {
  const int L = h->lanes;
  if (L <= 1) return run_lane(h, 0, fn, s);
  GLR_HIP(h, hipEventRecord(h->ev_fork, s));
  for (int k = 0; k < L; ++k) GLR_HIP(h, hipStreamWaitEvent(h->lane_s[k], h->ev_fork, 0));
  glr_status st[kMaxLanes];
  std::thread th[kMaxLanes];
  for (int k = 1; k < L; ++k) {
    st[k] = GLR_OK;
    try {
      th[k] = std::thread([h, k, &fn, &st] {
        const hipError_t e = hipSetDevice(h->device);
        st[k] = e == hipSuccess ? run_lane(h, k, fn, h->lane_s[k]) : hip_fail(h, e, "hipSetDevice");
      });
    } catch (...) {
      // no thread: this lane runs on the calling thread after lane 0
    }
  }
  st[0] = run_lane(h, 0, fn, h->lane_s[0]);
  for (int k = 1; k < L; ++k) {
    if (th[k].joinable()) th[k].join();
    else st[k] = run_lane(h, k, fn, h->lane_s[k]);
  }
  glr_status out = GLR_OK;
  for (int k = 0; k < L; ++k)
    if (out == GLR_OK && st[k] != GLR_OK) out = st[k];
  for (int k = 0; k < L; ++k) {
    hipError_t e = hipEventRecord(h->ev_join[k], h->lane_s[k]);
    if (e == hipSuccess) e = hipStreamWaitEvent(s, h->ev_join[k], 0);
    if (e != hipSuccess && out == GLR_OK) out = hip_fail(h, e, "joining the lane streams");
  }
  return out;
}

// A refresh step of several matrices: M-bar and the Jacobi start of every
// matrix on the lanes; then the sweeps of all matrices in shared launches on
// `s`, one convergence read per sweep for all of them (a matrix that has
// converged leaves the launches); then sigma, U and the rest of the step on the
// lanes.  Each matrix runs the same kernels on the same data as its own
// refresh, so the results are bitwise those of the per-matrix order.
glr_status step_joint(glr_handle* h, float* const* X, const void* const* G, int64_t t, hipStream_t s) {
  const glr_config& c = h->cfg;
  const int num = c.num_mats;
  glr_status st = on_lanes(h, s, [&](int i, int lane, hipStream_t ls) -> glr_status {
    const MatView v = view_of(h, i, X[i], G[i], lane);
    const glr_status r = step_head(h, v, ls);
    return r != GLR_OK ? r : svd_begin(h, v, t, ls);
  });
  if (st != GLR_OK) return st;
  const JointPlan& jp = h->jp;
  // as many sweeps as the matrix with the largest budget needs; a converged
  // matrix's later sweeps only move its data to the other buffer of the pair
  int budget = 1;
  for (int i = 0; i < num; ++i) budget = std::max(budget, sweep_budget(h, i));
  for (int sw = 0; sw < budget; ++sw) {
    const int par = sw & 1, p = par ^ 1;   // the sort reads parity par and fills the other
    GLR_HIP(h, launch_joint_sort(jp, par, s));
    GLR_HIP(h, launch_joint_solve(jp, p, 0, c.tol, h->jac_inner, h->jac_floor2, s));
    for (int k = 0; k < jp.rounds_max; ++k) {
      GLR_HIP(h, launch_joint_update(jp, p, k, s));
      GLR_HIP(h, launch_joint_solve_apply(jp, p, k + 1, c.tol, h->jac_inner, h->jac_floor2, s));
    }
    GLR_HIP(h, launch_joint_check(jp, c.tol, s));
  }
  return on_lanes(h, s, [&](int i, int lane, hipStream_t ls) -> glr_status {
    const MatView v = view_of(h, i, X[i], G[i], lane);
    const MatView& fin = h->jm[(size_t)i].v[budget & 1];
    glr_status r = svd_end(h, fin, ls);
    if (r == GLR_OK && read_back_info(h, i, v, ls) != hipSuccess) r = fail(h, GLR_ERR_DEVICE, "info read-back");
    return r != GLR_OK ? r : step_tail(h, v, true, ls);
  });
}

// the joint tables: two views per matrix (the buffer parities of the
// reordering) and the first block of each matrix in every joint launch
hipError_t joint_setup(glr_handle* h, hipStream_t s) {
  const int num = h->cfg.num_mats;
  h->jm.resize((size_t)num);
  std::vector<int> blocks((size_t)num * kJointKinds);
  JointPlan& jp = h->jp;
  jp.num = num;
  jp.ng = jac_group_blocks(h->lay[0].d);
  for (int i = 0; i < num; ++i) {
    JointMat& J = h->jm[(size_t)i];
    J.v[0] = view_of(h, i, nullptr, nullptr, 0);
    J.v[1] = J.v[0];
    std::swap(J.v[1].Apk, J.v[1].Apk2);
    std::swap(J.v[1].Utw, J.v[1].W);
    int b[kJointKinds];
    joint_fill(J, b);
    for (int k = 0; k < kJointKinds; ++k) blocks[(size_t)i * kJointKinds + k] = b[k];
    jp.rounds_max = std::max(jp.rounds_max, J.rounds);
    int n_pad = 2;
    while (n_pad < J.v[0].d) n_pad <<= 1;
    jp.npad_max = std::max(jp.npad_max, n_pad);
  }
  h->jfirst.assign((size_t)kJointKinds * (num + 1), 0);
  for (int k = 0; k < kJointKinds; ++k) {
    int64_t acc = 0;
    for (int i = 0; i < num; ++i) {
      h->jfirst[(size_t)k * (num + 1) + i] = (int)acc;
      acc += blocks[(size_t)i * kJointKinds + k];
    }
    if (acc > INT32_MAX) return hipErrorInvalidValue;
    h->jfirst[(size_t)k * (num + 1) + num] = (int)acc;
    jp.total[k] = (int)acc;
  }
  jp.jm = (const JointMat*)(h->work + h->ws.off_views);
  jp.first = (const int*)(h->work + h->ws.off_first);
  jp.flags = (int*)(h->work + h->ws.off_first) + (size_t)kJointKinds * (num + 1);
  hipError_t e = hipMemcpyAsync((void*)jp.jm, h->jm.data(), (size_t)num * sizeof(JointMat), hipMemcpyHostToDevice, s);
  if (e == hipSuccess)
    e = hipMemcpyAsync((void*)jp.first, h->jfirst.data(), h->jfirst.size() * sizeof(int), hipMemcpyHostToDevice, s);
  return e;
}

// a refresh step sweeps all matrices jointly when they take the full-basis
// refresh with one group size, the sweeps reorder every time, and no matrix is
// large enough to fill the chip with its own launches (from d = 4096 on, the
// per-matrix sweeps on concurrent streams measured a few per cent faster)
constexpr int64_t kJointMaxDim = 2048;
bool joint_allowed(const glr_handle* h) {
  const glr_config& c = h->cfg;
  if (c.num_mats < 2 || c.tau == 1 || h->jac_sort != 1) return false;
  if (const char* e = getenv("GLR_JAC_JOINT"))
    if (atoi(e) == 0) return false;
  for (int i = 0; i < c.num_mats; ++i) {
    const int64_t d = h->lay[(size_t)i].d;
    if (d > kJointMaxDim || jac_group_blocks(d) != jac_group_blocks(h->lay[0].d)) return false;
  }
  return true;
}

// A selection step of several matrices: the per-step table of views (with
// this step's X and G) goes up from a pinned slot, then each kernel of the
// step runs once over all matrices on `s`.
glr_status step_grouped(glr_handle* h, float* const* X, const void* const* G, int64_t t, hipStream_t s) {
  const glr_config& c = h->cfg;
  const int num = c.num_mats, slot = h->gslot;
  h->gslot ^= 1;
  GLR_HIP(h, hipEventSynchronize(h->gev[slot]));   // the upload that read this slot two steps ago
  GroupMat* g = h->gring + (size_t)slot * num;
  int blocks[kGrpKinds];
  for (int i = 0; i < num; ++i) {
    g[i].v = view_of(h, i, X[i], G[i], 0);
    group_fill(g[i], blocks);
  }
  GLR_HIP(h, hipMemcpyAsync((void*)h->gp[0].gm, g, (size_t)num * sizeof(GroupMat), hipMemcpyHostToDevice, s));
  GLR_HIP(h, hipEventRecord(h->gev[slot], s));
  OptParams op{c.opt, c.lr, c.beta1, c.beta2, c.eps};
  const bool fin = (c.flags & GLR_CHECK_FINITE) != 0, approx = c.select != GLR_SELECT_EXACT,
             b16 = c.select == GLR_SELECT_APPROX_BF16;
  if (h->gparts == 1) {
    GLR_HIP(h, launch_group_select(h->gp[0], fin, approx, b16, c.seed, t, op, 0, s));
    return GLR_OK;
  }
  // parts of about equal bytes, part k > 0 on lane k from the end of part
  // k - 1's M-bar on: each part's launches alternate between the HBM-bound
  // (M-bar, projection, residual) and the MFMA-bound (scores) kinds, so the
  // staggered parts overlap the two
  for (int k = 0; k < h->gparts; ++k) {
    hipStream_t ks = k == 0 ? s : h->lane_s[k];
    if (k > 0) GLR_HIP(h, hipStreamWaitEvent(ks, h->gev_mean[k - 1], 0));
    GLR_HIP(h, launch_group_select(h->gp[k], fin, approx, b16, c.seed, t, op, 1, ks));
    if (k + 1 < h->gparts) GLR_HIP(h, hipEventRecord(h->gev_mean[k], ks));
    GLR_HIP(h, launch_group_select(h->gp[k], fin, approx, b16, c.seed, t, op, 2, ks));
    if (k > 0) GLR_HIP(h, hipEventRecord(h->ev_join[k], ks));
  }
  for (int k = 1; k < h->gparts; ++k) GLR_HIP(h, hipStreamWaitEvent(s, h->ev_join[k], 0));
  return GLR_OK;
}

// selection steps are grouped when every matrix has d <= 2048, a rank below d
// and at most 128, and the same side (so the same kernel variants)
bool group_allowed(const glr_handle* h) {
  const glr_config& c = h->cfg;
  if (c.num_mats < 2 || c.tau == 1 || h->static_ws || h->lazy || !h->ef || c.opt == GLR_GALORE_ADAM) return false;
  if (const char* e = getenv("GLR_GROUPED"))
    if (atoi(e) == 0) return false;
  const glr_mat_layout& L0 = h->lay[0];
  for (int i = 0; i < c.num_mats; ++i) {
    const glr_mat_layout& L = h->lay[(size_t)i];
    if (L.d > kJointMaxDim || L.r >= L.d || L.r > kResidWideRank || L.r != L0.r || L.right != L0.right)
      return false;
  }
  return true;
}

// block tables of the grouped launches, the pinned ring and its events
hipError_t group_setup(glr_handle* h, hipStream_t s) {
  const int num = h->cfg.num_mats;
  // parts of about equal bytes, one per lane stream (two unless
  // GLR_GROUP_PARTS asks otherwise; at most one part per two matrices)
  int parts = std::min(h->lanes, 2);
  if (const char* e = getenv("GLR_GROUP_PARTS")) parts = std::min(h->lanes, std::max(1, atoi(e)));
  if (const char* e = getenv("GLR_GROUP_SPLIT"))
    if (atoi(e) == 0) parts = 1;
  parts = std::max(1, std::min(parts, num / 2));
  std::vector<int> cut(1, 0);
  {
    double tot = 0.0, acc = 0.0;
    for (int i = 0; i < num; ++i) tot += (double)h->lay[(size_t)i].m * (double)h->lay[(size_t)i].n;
    for (int i = 0; i < num && (int)cut.size() < parts; ++i) {
      const double sz = (double)h->lay[(size_t)i].m * (double)h->lay[(size_t)i].n;
      // close the part before matrix i once it holds its share
      if (i > cut.back() && acc + 0.5 * sz >= tot * (double)cut.size() / parts) cut.push_back(i);
      acc += sz;
    }
    cut.push_back(num);
  }
  std::vector<int> blocks((size_t)num * kGrpKinds);
  size_t topr_lds = 0;
  for (int i = 0; i < num; ++i) {
    GroupMat g;
    g.v = view_of(h, i, nullptr, nullptr, 0);
    int b[kGrpKinds];
    group_fill(g, b);
    for (int k = 0; k < kGrpKinds; ++k) blocks[(size_t)i * kGrpKinds + k] = b[k];
    topr_lds = std::max(topr_lds, topr_lds_bytes(g.v.d));
  }
  const GroupMat* gm = (const GroupMat*)(h->work + h->ws.off_gmats);
  const int* first = (const int*)(h->work + h->ws.off_gfirst);
  h->gfirst.clear();
  // the plan of matrices [a, b): its tables follow the previous plan's
  auto plan = [&](GroupPlan& gp, int a, int b) -> hipError_t {
    const int n = b - a;
    gp.num = n;
    gp.right = h->lay[0].right != 0;
    gp.r = h->lay[0].r;
    gp.st16 = (h->cfg.flags & GLR_STORE_BF16) != 0;
    gp.topr_lds = topr_lds;
    gp.gm = gm + a;
    gp.first = first + h->gfirst.size();
    for (int k = 0; k < kGrpKinds; ++k) {
      int64_t acc = 0;
      for (int i = a; i < b; ++i) {
        h->gfirst.push_back((int)acc);
        acc += blocks[(size_t)i * kGrpKinds + k];
      }
      if (acc > INT32_MAX) return hipErrorInvalidValue;
      h->gfirst.push_back((int)acc);
      gp.total[k] = (int)acc;
    }
    return hipSuccess;
  };
  hipError_t e = hipSuccess;
  h->gparts = (int)cut.size() - 1;
  for (int k = 0; e == hipSuccess && k < h->gparts; ++k) e = plan(h->gp[k], cut[(size_t)k], cut[(size_t)k + 1]);
  for (int k = 0; e == hipSuccess && k + 1 < h->gparts; ++k)
    e = hipEventCreateWithFlags(&h->gev_mean[k], hipEventDisableTiming);
  if (e == hipSuccess)
    e = hipMemcpyAsync((void*)first, h->gfirst.data(), h->gfirst.size() * sizeof(int), hipMemcpyHostToDevice, s);
  if (e == hipSuccess) e = hipHostMalloc((void**)&h->gring, 2 * (size_t)num * sizeof(GroupMat), hipHostMallocDefault);
  for (int k = 0; e == hipSuccess && k < 2; ++k) e = hipEventCreateWithFlags(&h->gev[k], hipEventDisableTiming);
  return e;
}

void release_group(glr_handle* h) {
  for (int k = 0; k < kMaxLanes; ++k) {
    if (h->gev_mean[k]) (void)hipEventDestroy(h->gev_mean[k]);
    h->gev_mean[k] = nullptr;
  }
  for (int k = 0; k < 2; ++k) {
    if (h->gev[k]) (void)hipEventSynchronize(h->gev[k]);
    if (h->gev[k]) (void)hipEventDestroy(h->gev[k]);
    h->gev[k] = nullptr;
  }
  if (h->gring) (void)hipHostFree(h->gring);
  h->gring = nullptr;
}

void release_info(glr_handle* h) {
  for (hipEvent_t& e : h->info_ev) {
    if (e) (void)hipEventSynchronize(e);
    if (e) (void)hipEventDestroy(e);
    e = nullptr;
  }
  if (h->info_host) (void)hipHostFree(h->info_host);
  h->info_host = nullptr;
}

void release_lanes(glr_handle* h) {
  for (int k = 0; k < kMaxLanes; ++k) {
    if (h->lane_s[k]) (void)hipStreamDestroy(h->lane_s[k]);
    if (h->ev_join[k]) (void)hipEventDestroy(h->ev_join[k]);
    h->lane_s[k] = nullptr;
    h->ev_join[k] = nullptr;
  }
  if (h->ev_fork) (void)hipEventDestroy(h->ev_fork);
  h->ev_fork = nullptr;
}

}  // namespace

extern "C" {

glr_status glr_validate_config(const glr_config* cfg) {
  std::string why;
  glr_status s = check_config(cfg, &why);
  if (s != GLR_OK) g_create_error = why;
  return s;
}

glr_status glr_workspace_bytes(const glr_config* cfg, size_t* state_bytes, size_t* ws_bytes) {
  std::string why;
  glr_status s = check_config(cfg, &why);
  if (s != GLR_OK) { g_create_error = why; return s; }
  if (!state_bytes || !ws_bytes) { g_create_error = "output pointer is NULL"; return GLR_ERR_INVALID_ARG; }
  *state_bytes = (size_t)state_bytes_of(cfg);
  *ws_bytes = (size_t)ws_plan(cfg).bytes;
  return GLR_OK;
}

glr_status glr_state_layout(const glr_config* cfg, int32_t mat, glr_mat_layout* out) {
  std::string why;
  glr_status s = check_config(cfg, &why);
  if (s != GLR_OK) { g_create_error = why; return s; }
  if (!out) { g_create_error = "output pointer is NULL"; return GLR_ERR_INVALID_ARG; }
  if (mat < 0 || mat >= cfg->num_mats) { g_create_error = "matrix index out of range"; return GLR_ERR_INVALID_ARG; }
  uint64_t o = kHeaderBytes;
  for (int i = 0; i <= mat; ++i) mat_layout(cfg, i, o, out, &o);
  return GLR_OK;
}

}  // extern "C"

namespace {

// ---------------------------------------------------------------------------
// The workspace of handles made by glr_create_static: a file-scope device
// array, which every device the library runs on holds (its own copy, at its
// own address) until the process ends.  Host code never passes the array's
// name as an address: the device address is taken once per device, with that
// device current, by hipGetSymbolAddress, and only that address is used.
// ---------------------------------------------------------------------------
constexpr size_t kStaticScratchBytes = GLR_STATIC_SCRATCH_BYTES;
static __device__ __align__(256) unsigned char scratch[kStaticScratchBytes];
constexpr int kMaxDevices = 64;
std::mutex g_static_mu;
void* g_static_ptr[kMaxDevices] = {};
bool g_static_busy[kMaxDevices] = {};

void static_release(int dev) {
  if (dev < 0 || dev >= kMaxDevices) return;
  std::lock_guard<std::mutex> lk(g_static_mu);
  g_static_busy[dev] = false;
}

glr_status create_impl(const glr_config* cfg, void* d_state, size_t state_bytes, void* d_ws, size_t ws_bytes,
                       void* stream, glr_handle** out, bool static_ws) {
  std::string why;
  glr_status s = check_config(cfg, &why);
  if (s != GLR_OK) return fail(nullptr, s, why);
  if (!out) return fail(nullptr, GLR_ERR_INVALID_ARG, "out is NULL");
  *out = nullptr;
  if (!d_state || !d_ws) return fail(nullptr, GLR_ERR_INVALID_ARG, "state or workspace pointer is NULL");
  if (!aligned(d_state) || !aligned(d_ws))
    return fail(nullptr, GLR_ERR_INVALID_ARG, "state and workspace must be 256-byte aligned");
  const uint64_t need_s = state_bytes_of(cfg);
  const WsPlan wl = ws_plan(cfg);
  if (state_bytes < need_s || ws_bytes < wl.bytes)
    return fail(nullptr, GLR_ERR_BUFFER_TOO_SMALL,
                fmt("need %llu state bytes and %llu workspace bytes", (unsigned long long)need_s,
                    (unsigned long long)wl.bytes));
  glr_handle* h = new (std::nothrow) glr_handle();
  if (!h) return fail(nullptr, GLR_ERR_INVALID_ARG, "out of host memory");
  h->cfg = *cfg;
  h->shapes.assign(cfg->shapes, cfg->shapes + cfg->num_mats);
  h->cfg.shapes = h->shapes.data();
  h->ws = wl;
  if (const char* e = getenv("GLR_JAC_FLOOR")) h->jac_floor2 = ldexp(1.0, -2 * atoi(e));
  if (const char* e = getenv("GLR_JAC_SORT")) h->jac_sort = atoi(e);
  if (const char* e = getenv("GLR_JAC_INNER")) {
    const int v = atoi(e);
    if (v >= 1 && v <= 16) h->jac_inner = v;
  }
  if (const char* e = getenv("GLR_SUB_ITERS")) {
    const int v = atoi(e);
    if (v >= kSubMinIters && v <= 64) h->sub_iters_warm = v;
  }
  h->state = (char*)d_state;
  h->work = (char*)d_ws;
  h->static_ws = static_ws;
  h->lazy = cfg->select == GLR_SELECT_LAZY || cfg->opt == GLR_GALORE_ADAM;
  h->ef = !(cfg->flags & GLR_NO_EF) && cfg->opt != GLR_GALORE_ADAM;
  uint64_t o = kHeaderBytes;
  h->lay.resize(cfg->num_mats);
  for (int i = 0; i < cfg->num_mats; ++i) mat_layout(&h->cfg, i, o, &h->lay[i], &o);
  hipError_t e = hipGetDevice(&h->device);
  hipStream_t st = (hipStream_t)stream;
  if (e == hipSuccess) e = launch_fill_zero(d_state, (size_t)need_s, st);
  for (int i = 0; e == hipSuccess && i < cfg->num_mats; ++i)
    e = launch_eye((float*)(h->state + h->lay[i].off_U), h->lay[i].d, st);
  if (e == hipSuccess) e = launch_fill_zero(d_ws, (size_t)wl.bytes, st);
  h->lanes = static_ws ? 1 : wl.lanes;   // no stream of its own without allocation
  if (const char* v = getenv("GLR_LANES")) {
    const int k = atoi(v);
    if (k >= 1 && k < h->lanes) h->lanes = k;
  }
  h->lane_of = assign_lanes(&h->cfg, h->lanes);
  for (int k = 0; e == hipSuccess && h->lanes > 1 && k < h->lanes; ++k) {
    e = hipStreamCreateWithFlags(&h->lane_s[k], hipStreamNonBlocking);
    if (e == hipSuccess) e = hipEventCreateWithFlags(&h->ev_join[k], hipEventDisableTiming);
  }
  if (e == hipSuccess && h->lanes > 1) e = hipEventCreateWithFlags(&h->ev_fork, hipEventDisableTiming);
  h->known_sweeps.assign((size_t)cfg->num_mats, -1);
  h->known_conv.assign((size_t)cfg->num_mats, 0);
  h->info_pending.assign((size_t)cfg->num_mats, 0);
  h->info_ev.assign((size_t)cfg->num_mats, nullptr);
  if (e == hipSuccess && !static_ws)
    e = hipHostMalloc((void**)&h->info_host, 2 * sizeof(int) * (size_t)cfg->num_mats, hipHostMallocDefault);
  for (int i = 0; e == hipSuccess && !static_ws && i < cfg->num_mats; ++i)
    e = hipEventCreateWithFlags(&h->info_ev[(size_t)i], hipEventDisableTiming);
  if (e == hipSuccess && joint_allowed(h)) {
    h->joint = true;
    e = joint_setup(h, st);
  }
  if (e == hipSuccess && group_allowed(h)) {
    h->grouped = true;
    e = group_setup(h, st);
  }
  if (e != hipSuccess) {
    std::string m = fmt("glr_create: %s", hipGetErrorString(e));
    release_group(h);
    release_lanes(h);
    release_info(h);
    delete h;
    return fail(nullptr, GLR_ERR_DEVICE, m);
  }
  *out = h;
  return GLR_OK;
}

}  // namespace

extern "C" {

glr_status glr_create(const glr_config* cfg, void* d_state, size_t state_bytes, void* d_ws,
                      size_t ws_bytes, void* stream, glr_handle** out) {
  return create_impl(cfg, d_state, state_bytes, d_ws, ws_bytes, stream, out, false);
}

glr_status glr_create_static(const glr_config* cfg, void* d_state, size_t state_bytes, void* stream,
                             glr_handle** out) {
  std::string why;
  glr_status s = check_config(cfg, &why);
  if (s != GLR_OK) return fail(nullptr, s, why);
  if (!out) return fail(nullptr, GLR_ERR_INVALID_ARG, "out is NULL");
  *out = nullptr;
  const uint64_t need = ws_plan(cfg).bytes;
  if (need > kStaticScratchBytes)
    return fail(nullptr, GLR_ERR_BUFFER_TOO_SMALL,
                fmt("the configuration needs %llu workspace bytes; the static scratch holds %llu "
                    "(use glr_create with a caller workspace)",
                    (unsigned long long)need, (unsigned long long)kStaticScratchBytes));
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return fail(nullptr, GLR_ERR_DEVICE, fmt("hipGetDevice: %s", hipGetErrorString(e)));
  if (dev < 0 || dev >= kMaxDevices) return fail(nullptr, GLR_ERR_DEVICE, "device index out of range");
  void* ptr = nullptr;
  {
    std::lock_guard<std::mutex> lk(g_static_mu);
    if (g_static_busy[dev])
      return fail(nullptr, GLR_ERR_STATE,
                  fmt("the static scratch of device %d belongs to another live handle (one at a time)", dev));
    if (!g_static_ptr[dev]) {
      e = hipGetSymbolAddress(&g_static_ptr[dev], HIP_SYMBOL(scratch));
      if (e != hipSuccess) {
        g_static_ptr[dev] = nullptr;
        return fail(nullptr, GLR_ERR_DEVICE, fmt("hipGetSymbolAddress(scratch): %s", hipGetErrorString(e)));
      }
    }
    ptr = g_static_ptr[dev];
    g_static_busy[dev] = true;
  }
  s = create_impl(cfg, d_state, state_bytes, ptr, kStaticScratchBytes, stream, out, true);
  if (s != GLR_OK) static_release(dev);
  return s;
}

namespace {
glr_status step_impl(glr_handle* h, float* const* X, const void* const* G, int64_t t, void* stream) {
  if (h->suspect) return fail(h, GLR_ERR_STATE, "state is suspect after an earlier error; call glr_resume");
  if (t != h->next_t)
    return fail(h, GLR_ERR_STATE, fmt("steps run in order: expected t=%lld, got %lld", (long long)h->next_t, (long long)t));
  if (!X || !G) return fail(h, GLR_ERR_INVALID_ARG, "X or G is NULL");
  for (int i = 0; i < h->cfg.num_mats; ++i) {
    if (!X[i] || !G[i]) return fail(h, GLR_ERR_INVALID_ARG, fmt("matrix %d: NULL buffer", i));
    if (!aligned(X[i]) || !aligned(G[i]))
      return fail(h, GLR_ERR_INVALID_ARG, fmt("matrix %d: buffers must be 256-byte aligned", i));
  }
  hipStream_t s = (hipStream_t)stream;
  if (h->joint && !h->prof && t % h->cfg.tau == 0) {
    glr_status st = step_joint(h, X, G, t, s);
    if (st != GLR_OK) return st;
  } else if (h->grouped && !h->prof && t % h->cfg.tau != 0) {
    glr_status st = step_grouped(h, X, G, t, s);
    if (st != GLR_OK) return st;
  } else if (h->lanes > 1 && !h->prof) {
    glr_status st = on_lanes(h, s, [&](int i, int lane, hipStream_t ls) {
      return step_one(h, i, X[i], G[i], t, ls, lane);
    });
    if (st != GLR_OK) return st;
  } else {
    // one matrix, or profiling: every matrix in order on `s` (event brackets
    // then time one launch group at a time)
    for (int i = 0; i < h->cfg.num_mats; ++i) {
      glr_status st = step_one(h, i, X[i], G[i], t, s, h->lane_of[(size_t)i]);
      if (st != GLR_OK) return st;
    }
  }
  h->next_t = t + 1;
  return GLR_OK;
}
}  // namespace

glr_status glr_step(glr_handle* h, float* const* X, const float* const* G, int64_t t, void* stream) {
  if (!h) return fail(nullptr, GLR_ERR_INVALID_ARG, "handle is NULL");
  if (h->cfg.flags & GLR_STORE_BF16)
    return fail(h, GLR_ERR_INVALID_ARG, "the handle stores G and E in bf16: call glr_step_bf16");
  return step_impl(h, X, reinterpret_cast<const void* const*>(G), t, stream);
}

glr_status glr_step_bf16(glr_handle* h, float* const* X, const uint16_t* const* G, int64_t t, void* stream) {
  if (!h) return fail(nullptr, GLR_ERR_INVALID_ARG, "handle is NULL");
  if (!(h->cfg.flags & GLR_STORE_BF16))
    return fail(h, GLR_ERR_INVALID_ARG, "the handle stores G and E in fp32: call glr_step");
  return step_impl(h, X, reinterpret_cast<const void* const*>(G), t, stream);
}

glr_status glr_sync_status(glr_handle* h, void* stream) {
  if (!h) return fail(nullptr, GLR_ERR_INVALID_ARG, "handle is NULL");
  hipStream_t s = (hipStream_t)stream;
  uint32_t word = 0;
  GLR_HIP(h, hipStreamSynchronize(s));
  GLR_HIP(h, hipMemcpy(&word, h->state, sizeof word, hipMemcpyDeviceToHost));
  if (word) {
    GLR_HIP(h, launch_fill_zero(h->state, 4, s));
    GLR_HIP(h, hipStreamSynchronize(s));
  }
  h->repaired_total += (word & kStatusRepaired) ? 1 : 0;
  if (word & kStatusNonfinite) {
    h->suspect = true;
    return fail(h, GLR_ERR_NONFINITE, "a gradient held NaN or Inf");
  }
  if (word & kStatusBreakdown) {
    h->suspect = true;
    return fail(h, GLR_ERR_BREAKDOWN, "a tau = 1 orthonormalisation found dependent rows after its repair pass");
  }
  if (word & kStatusNotConverged)
    return fail(h, GLR_ERR_NOT_CONVERGED, "a refresh ended its Jacobi sweeps (budget or max_sweeps) above tol");
  if (word & kStatusSubNotConverged)
    return fail(h, GLR_ERR_NOT_CONVERGED, "a tau = 1 block iteration ended its iterations above its tolerance");
  return GLR_OK;
}

glr_status glr_resume(glr_handle* h, int64_t next_t) {
  if (!h) return fail(nullptr, GLR_ERR_INVALID_ARG, "handle is NULL");
  if (next_t < 0) return fail(h, GLR_ERR_INVALID_ARG, "next_t must be >= 0");
  h->next_t = next_t;
  h->suspect = false;
  h->err.clear();
  return GLR_OK;
}

namespace {
// (pointer into the state, bytes) of each glr_state_view member of matrix mat,
// in member order
struct StatePart {
  uint64_t off, bytes;
};
void state_parts(const glr_handle* h, int mat, StatePart (&p)[10]) {
  const glr_mat_layout& L = h->lay[(size_t)mat];
  const uint64_t mn = (uint64_t)(L.m * L.n), N = (uint64_t)h->cfg.num_workers;
  p[0] = {L.off_E, N * mn * elem_bytes(&h->cfg)};
  p[1] = {L.off_Ebar, mn * 4};
  p[2] = {L.off_U, (uint64_t)(L.d * L.d) * 4};
  p[3] = {L.off_sigma, (uint64_t)L.d * 4};
  p[4] = {L.off_J, (uint64_t)L.r * 4};
  p[5] = {L.off_score, (uint64_t)L.d * 4};
  p[6] = {L.off_S1, mn * 4};
  p[7] = {L.off_S2, L.off_S2 ? mn * 4 : 0};
  p[8] = {L.off_Rbar, (uint64_t)L.r * (uint64_t)L.D * 4};
  p[9] = {L.off_info, (uint64_t)kInfoInts * 4};
}
void* const* view_members(const glr_state_view* v) { return reinterpret_cast<void* const*>(v); }

glr_status copy_state(glr_handle* h, int32_t mat, const glr_state_view* view, bool to_state, void* stream) {
  if (!h) return fail(nullptr, GLR_ERR_INVALID_ARG, "handle is NULL");
  if (!view) return fail(h, GLR_ERR_INVALID_ARG, "state view is NULL");
  if (mat < 0 || mat >= h->cfg.num_mats) return fail(h, GLR_ERR_INVALID_ARG, "matrix index out of range");
  static_assert(sizeof(glr_state_view) == 10 * sizeof(void*), "glr_state_view holds ten pointers");
  StatePart part[10];
  state_parts(h, mat, part);
  void* const* ptr = view_members(view);
  if (ptr[7] && part[7].bytes == 0) return fail(h, GLR_ERR_INVALID_ARG, "S2 exists only for Adam");
  hipStream_t s = (hipStream_t)stream;
  for (int k = 0; k < 10; ++k) {
    if (!ptr[k] || part[k].bytes == 0) continue;
    char* at = h->state + part[k].off;
    if (to_state) GLR_HIP(h, hipMemcpyAsync(at, ptr[k], part[k].bytes, hipMemcpyDefault, s));
    else GLR_HIP(h, hipMemcpyAsync(ptr[k], at, part[k].bytes, hipMemcpyDefault, s));
  }
  return GLR_OK;
}
}  // namespace

glr_status glr_read_state(glr_handle* h, int32_t mat, const glr_state_view* dst, void* stream) {
  return copy_state(h, mat, dst, false, stream);
}

glr_status glr_write_state(glr_handle* h, int32_t mat, const glr_state_view* src, void* stream) {
  const glr_status st = copy_state(h, mat, src, true, stream);
  if (st == GLR_OK) {
    std::lock_guard<std::mutex> lk(h->mu);
    h->suspect = false;
    h->err.clear();
  }
  return st;
}

glr_status glr_next_step(const glr_handle* h, int64_t* next_t) {
  if (!h || !next_t) return GLR_ERR_INVALID_ARG;
  *next_t = h->next_t;
  return GLR_OK;
}

glr_status glr_destroy(glr_handle* h) {
  if (!h) return GLR_OK;
  for (hipEvent_t e : h->ev_pool) (void)hipEventDestroy(e);
  release_group(h);
  release_lanes(h);
  release_info(h);
  if (h->static_ws) static_release(h->device);
  delete h;
  return GLR_OK;
}

glr_status glr_profile_enable(glr_handle* h, int32_t on) {
  if (!h) return fail(nullptr, GLR_ERR_INVALID_ARG, "handle is NULL");
  h->prof = on != 0;
  return GLR_OK;
}

glr_status glr_profile_reset(glr_handle* h) {
  if (!h) return fail(nullptr, GLR_ERR_INVALID_ARG, "handle is NULL");
  GLR_HIP(h, prof_collect(h));
  for (int i = 0; i < GLR_PROF_COUNT; ++i) { h->prof_ms[i] = 0.0; h->prof_n[i] = 0; }
  return GLR_OK;
}

glr_status glr_profile_query(glr_handle* h, int32_t group, double* total_ms, int64_t* launches) {
  if (!h) return fail(nullptr, GLR_ERR_INVALID_ARG, "handle is NULL");
  if (group < 0 || group >= GLR_PROF_COUNT || !total_ms || !launches)
    return fail(h, GLR_ERR_INVALID_ARG, "bad profile group or output pointer");
  GLR_HIP(h, prof_collect(h));
  *total_ms = h->prof_ms[group];
  *launches = h->prof_n[group];
  return GLR_OK;
}

const char* glr_status_string(glr_status s) {
  switch (s) {
    case GLR_OK: return "ok";
    case GLR_ERR_INVALID_ARG: return "invalid argument";
    case GLR_ERR_SHAPE: return "invalid shape";
    case GLR_ERR_BUFFER_TOO_SMALL: return "buffer too small";
    case GLR_ERR_STATE: return "invalid state";
    case GLR_ERR_DEVICE: return "device error";
    case GLR_ERR_NONFINITE: return "non-finite gradient";
    case GLR_ERR_NOT_CONVERGED: return "refresh not converged";
    case GLR_ERR_BREAKDOWN: return "orthonormalisation breakdown";
  }
  return "unknown status";
}

const char* glr_last_error(const glr_handle* h) {
  return h ? h->err.c_str() : g_create_error.c_str();
}

}  // extern "C"
