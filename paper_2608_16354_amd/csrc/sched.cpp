// Host-side scheduling of DriveCache (Sec. 3.1-3.2 of the paper).
//
// Built with -ffp-contract=off: every floating-point expression below is
// evaluated one IEEE-754 double operation at a time, in the written order, so
// scene costs are reproducible across compilers.  Costs are integers in units
// of 2^-40, which makes ties, budget comparisons and replanned suffix budgets
// exact.
#include <algorithm>
#include <cmath>
#include <cstdint>
#include <cstring>
#include <limits>
#include <vector>

#include "internal.h"

namespace dc {

namespace {
constexpr int64_t kUnreached = std::numeric_limits<int64_t>::max();
constexpr double kCostScale = 1099511627776.0;  // 2^40
}  // namespace

// Eq. 2 helper: signed angle difference wrapped to [-pi, pi).
static double wrap_angle(double a) {
  const double two_pi = 2.0 * M_PI;
  const double turns = std::floor((a + M_PI) / two_pi);
  return a - two_pi * turns;
}

// Eq. 2: path length and accumulated absolute heading change of a planned pose sequence.
void motion_statistics(const double* xy, const double* yaw, int n_pose, double& L, double& Th) {
  L = 0.0;
  Th = 0.0;
  for (int i = 1; i < n_pose; ++i) {
    const double dx = xy[2 * i] - xy[2 * (i - 1)];
    const double dy = xy[2 * i + 1] - xy[2 * (i - 1) + 1];
    const double sq = dx * dx + dy * dy;
    L = L + std::sqrt(sq);
    Th = Th + std::fabs(wrap_angle(yaw[i] - yaw[i - 1]));
  }
}

Status scene_tables(const dc_sched_problem& p, SceneTables& t) {
  const int K = p.K, H = p.h_max;
  double L = 0.0, Th = 0.0;
  motion_statistics(p.pose_xy, p.pose_yaw, p.n_pose, L, Th);
  // Eq. 3: position relative to the two anchors; Eq. 4: one interpolation coordinate.
  const double zL = (L - p.L0) / std::max(p.L1 - p.L0, p.eps);
  const double zTh = (Th - p.Th0) / std::max(p.Th1 - p.Th0, p.eps);
  const bool inside = zL >= 0.0 && zL <= 1.0 && zTh >= 0.0 && zTh <= 1.0;
  const double r2 = zL * zL + zTh * zTh;
  const double D = std::sqrt(r2) / std::sqrt(2.0);
  t.L = L; t.Theta = Th; t.zL = zL; t.zTh = zTh; t.D = D; t.in_support = inside;
  t.K = K; t.H = H;
  t.chat.assign(size_t(std::max(K - 1, 0)) * H, 0);
  t.dbar.assign(size_t(std::max(K - 1, 0)) * H, 0.0);
  for (int j = 0; j < K - 1; ++j) {
    double env = 0.0;
    int64_t prev = 0;
    for (int h = 0; h < H; ++h) {
      const size_t e = size_t(j) * H + h;
      // Eq. 8: only the non-negative motion-dependent difference is interpolated.
      const double qd = std::max(p.q1[e] - p.q0[e], 0.0);
      const double qs = p.q0[e] + D * qd;
      const double dd = std::max(p.d1[e] - p.d0[e], 0.0);
      t.dbar[e] = p.d0[e] + D * dd;
      // Eq. 9: running maximum over the ages seen so far, then its increment.
      env = (h == 0) ? qs : std::max(env, qs);
      const double scaled = env * kCostScale;   // exact: power-of-two scale
      if (!(std::fabs(scaled) < 4.0e18)) return Status::arg("response table value out of range");
      const int64_t Qq = std::llrint(scaled);   // round half to even (default mode)
      t.chat[e] = Qq - prev;
      prev = Qq;
    }
  }
  return Status::ok();
}

// Forward pass of Eq. 10 over steps s..K.  J has (K - s + 1) layers of
// (nmax + 1) x (H + 1) states; layer i holds step s + i.
struct DPTable {
  int s = 1, K = 0, nmax = 0, H = 0;
  std::vector<int64_t> J;
  int64_t& at(int k, int n, int h) {
    return J[(size_t(k - s) * (nmax + 1) + n) * (H + 1) + h];
  }
  int64_t get(int k, int n, int h) const {
    return J[(size_t(k - s) * (nmax + 1) + n) * (H + 1) + h];
  }
};

static bool reuse_allowed(const dc_sched_problem& p, int step, int refresh_step) {
  if (!p.legal[step - 1]) return false;
  if (p.segment && p.segment[step - 1] != p.segment[refresh_step - 1]) return false;
  return true;
}

static void dp_forward(const dc_sched_problem& p, const SceneTables& t, DPTable& T) {
  T.s = p.start_step; T.K = p.K; T.H = p.h_max;
  T.nmax = std::max(0, p.n_cap - p.spent_n);
  const int layers = p.K - p.start_step + 1;
  T.J.assign(size_t(layers) * (T.nmax + 1) * (T.H + 1), kUnreached);
  T.at(T.s, 0, 0) = 0;
  for (int k = T.s; k < p.K; ++k) {
    for (int n = 0; n <= T.nmax; ++n) {
      int64_t best = kUnreached;
      for (int h = 0; h <= T.H; ++h) best = std::min(best, T.get(k, n, h));
      T.at(k + 1, n, 0) = best;                       // full evaluation at k+1
    }
    for (int n = 0; n < T.nmax; ++n) {
      for (int h = 0; h < T.H; ++h) {
        const int64_t cur = T.get(k, n, h);
        if (cur == kUnreached) continue;
        const int j = k - h;                          // refresh step of the run
        if (!reuse_allowed(p, k + 1, j)) continue;
        const int64_t c = t.chat[size_t(j - 1) * T.H + h];   // age h+1
        const int64_t v = cur + c;
        int64_t& dst = T.at(k + 1, n + 1, h + 1);
        if (v < dst) dst = v;
      }
    }
  }
}

static void min_by_count(const DPTable& T, std::vector<int64_t>& m) {
  m.assign(size_t(T.nmax) + 1, kUnreached);
  for (int n = 0; n <= T.nmax; ++n)
    for (int h = 0; h <= T.H; ++h) m[n] = std::min(m[n], T.get(T.K, n, h));
}

Status schedule(const dc_sched_problem& p, const SceneTables& t, std::vector<uint8_t>& reuse,
                int32_t& n_reuse, int64_t& cost_q) {
  reuse.assign(size_t(p.K), 0);
  n_reuse = 0;
  cost_q = 0;
  if (!t.in_support) return Status::ok();             // outside the support: full inference
  DPTable T;
  dp_forward(p, t, T);
  std::vector<int64_t> m;
  min_by_count(T, m);
  // Eq. 11: the largest count whose cheapest schedule fits the remaining budget.
  const int64_t budget = p.tau_q - p.spent_q;
  int bstar = 0;
  for (int n = 0; n <= T.nmax; ++n)
    if (m[n] != kUnreached && m[n] <= budget) bstar = n;
  // Backtracking: smallest final age attaining the optimum, then at every full
  // state the smallest predecessor age with the same value.
  int n = bstar, h = 0;
  while (T.get(p.K, n, h) != m[n]) ++h;
  for (int k = p.K; k > T.s; --k) {
    if (h > 0) {
      reuse[size_t(k - 1)] = 1;
      --n;
      --h;
    } else {
      const int64_t target = T.get(k, n, 0);
      int hp = 0;
      while (T.get(k - 1, n, hp) != target) ++hp;
      h = hp;
    }
  }
  n_reuse = bstar;
  cost_q = m[bstar];
  return Status::ok();
}

Status validate_problem(const dc_sched_problem& p) {
  if (p.K < 1) return Status::arg("K must be >= 1");
  if (p.h_max < 1) return Status::arg("h_max must be >= 1");
  if (p.n_cap < 0 || p.n_cap > p.K - 1) return Status::arg("n_cap must be in [0, K-1]");
  if (p.tau_q < 0) return Status::arg("tau_q must be >= 0");
  if (p.start_step < 1 || p.start_step > p.K) return Status::arg("start_step must be in [1, K]");
  if (p.spent_q < 0 || p.spent_q > p.tau_q) return Status::arg("spent_q must be in [0, tau_q]");
  if (p.spent_n < 0 || p.spent_n > p.n_cap) return Status::arg("spent_n must be in [0, n_cap]");
  if (p.n_pose < 1 || !p.pose_xy || !p.pose_yaw) return Status::arg("poses missing");
  if (!p.legal) return Status::arg("legal mask missing");
  if (p.K > 1 && (!p.q0 || !p.q1 || !p.d0 || !p.d1)) return Status::arg("response/drift tables missing");
  if (!(p.eps >= 0.0)) return Status::arg("eps must be >= 0");
  return Status::ok();
}

// Sec. 3.1 anchor selection.  z-scores use the calibration set's mean and population
// standard deviation (a zero deviation is replaced by eps); the low-motion anchor has the
// smallest z^L + z^Theta; the moving-turn anchor, among clips with Theta above the
// calibration median (the mean of the two middle values for an even count) and L, Theta
// above the low-motion anchor's, has the largest z^L z^Theta; ties keep the lower index.
static void standardise(const double* x, int n, double eps, std::vector<double>& z) {
  double s = 0.0;
  for (int i = 0; i < n; ++i) s = s + x[i];
  const double mean = s / n;
  double ss = 0.0;
  for (int i = 0; i < n; ++i) {
    const double dv = x[i] - mean;
    ss = ss + dv * dv;
  }
  const double den = std::max(std::sqrt(ss / n), eps);
  z.resize(n);
  for (int i = 0; i < n; ++i) z[i] = (x[i] - mean) / den;
}

Status select_anchors(const double* L, const double* Th, int n, double eps, int& i0, int& i1) {
  if (n < 1) return Status::arg("need at least one calibration clip");
  for (int i = 0; i < n; ++i)
    if (!std::isfinite(L[i]) || !std::isfinite(Th[i])) return Status::arg("motion statistics must be finite");
  std::vector<double> zL, zT;
  standardise(L, n, eps, zL);
  standardise(Th, n, eps, zT);
  i0 = 0;
  double best = zL[0] + zT[0];
  for (int i = 1; i < n; ++i) {
    const double v = zL[i] + zT[i];
    if (v < best) { i0 = i; best = v; }
  }
  std::vector<double> srt(Th, Th + n);
  std::sort(srt.begin(), srt.end());
  const double med = (n % 2 == 1) ? srt[n / 2] : (srt[n / 2 - 1] + srt[n / 2]) / 2.0;
  i1 = -1;
  double best1 = 0.0;
  for (int i = 0; i < n; ++i) {
    if (!(Th[i] > med && L[i] > L[i0] && Th[i] > Th[i0])) continue;
    const double v = zL[i] * zT[i];
    if (i1 < 0 || v > best1) { i1 = i; best1 = v; }
  }
  return Status::ok();
}

Status select_tau(const dc_sched_problem* probs, int n, double rho, int64_t& tau) {
  if (n < 1 || !probs) return Status::arg("need at least one calibration problem");
  const int K = probs[0].K;
  std::vector<std::vector<int64_t>> curves(static_cast<size_t>(n));
  std::vector<int64_t> cands;
  for (int i = 0; i < n; ++i) {
    const dc_sched_problem& p = probs[i];
    if (p.K != K) return Status::arg("calibration problems must share K");
    Status st = validate_problem(p);
    if (!st) return st;
    SceneTables t;
    st = scene_tables(p, t);
    if (!st) return st;
    if (!t.in_support) {
      curves[i] = {0};
    } else {
      DPTable T;
      dp_forward(p, t, T);
      min_by_count(T, curves[i]);
    }
    for (int64_t v : curves[i])
      if (v != kUnreached) cands.push_back(v);
  }
  std::sort(cands.begin(), cands.end());
  cands.erase(std::unique(cands.begin(), cands.end()), cands.end());
  const int target = int(std::ceil(rho * double(K - 1)));
  std::vector<int> b(static_cast<size_t>(n));
  for (int64_t c : cands) {
    for (int i = 0; i < n; ++i) {
      int best = 0;
      for (size_t m = 0; m < curves[i].size(); ++m)
        if (curves[i][m] != kUnreached && curves[i][m] <= c) best = int(m);
      b[i] = best;
    }
    std::sort(b.begin(), b.end());
    const bool ok = (n % 2 == 1) ? b[n / 2] >= target : b[n / 2 - 1] + b[n / 2] >= 2 * target;
    if (ok) { tau = c; return Status::ok(); }
  }
  tau = cands.back();
  return Status::ok();
}

}  // namespace dc
