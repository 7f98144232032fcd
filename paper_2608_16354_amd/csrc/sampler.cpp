// The causal cache controller of Sec. 3.2 around the device steps of Eq. 1.
//
// Per scene the sampler keeps the current plan, the refresh step j of the live
// run, the cache age, the accumulated charge C (2^-40 units) and the executed
// reuse count.  Step k:
//   1. h_in = patch embedding of x_k (+ text rows), for every scene;
//   2. for scenes with a planned reuse: the observed drift of u_k against u_j
//      (one device reduction, one 4-double readback per scene, one wait);
//      accept iff drift <= dbar_{j,h} + eps and C + c_{j,h} <= tau;
//   3. scenes that refresh (planned, first step, or vetoed): snapshot u_j := u_k,
//      h := h_in, run the L blocks, store r = h - h_in; vetoed scenes replan the
//      unexecuted suffix from age zero with budget tau - C;
//   4. scenes that reuse: g = h_in[:N_v] + r (inside the fused bf16 head; otherwise
//      written to h[:N_v] by the cache-apply kernel);
//   5. head and Euler update from g (reuse) or h[:N_v] (refresh) for every scene.
#include <cmath>
#include <cstring>
#include <limits>
#include <memory>
#include <vector>

#include "internal.h"

namespace dc {

Status time_modulation(const Geo& g, const dc_model_weights* w, const double* sigmas, int K,
                       float* mod, void* ws, size_t ws_bytes, hipStream_t s);
Status patch_embed(const Geo& g, const dc_model_weights* w, const float* x, const float* txt,
                   float* h_in, const IdxList& il, void* ws, size_t ws_bytes, hipStream_t s);
Status block_forward(const Geo& g, const dc_block_weights* bw, const float* mod, float* h,
                     const IdxList& il, void* ws, size_t ws_bytes, hipStream_t s);
Status head_euler(const Geo& g, const dc_model_weights* w, const float* head_mod, const float* gin,
                  float* x, float dsigma, const IdxList& il, void* ws, size_t ws_bytes,
                  hipStream_t s, const void* resid);
Status drift_call(const Geo& g, const float* h_in, const float* mod0, void* u_ref, int snapshot,
                  double* sums, const IdxList& il, void* ws, size_t ws_bytes, hipStream_t s);
dc_status fail(const Status& s);

namespace {

// Deep copy of one scene's scheduling problem (the caller's arrays are not kept).
struct OwnedProblem {
  dc_sched_problem p{};
  std::vector<uint8_t> legal;
  std::vector<int32_t> segment;
  std::vector<double> xy, yaw, q0, q1, d0, d1;
  void assign(const dc_sched_problem& src) {
    p = src;
    const size_t K = size_t(src.K), T = size_t(std::max(src.K - 1, 0)) * src.h_max;
    legal.assign(src.legal, src.legal + K);
    if (src.segment) segment.assign(src.segment, src.segment + K);
    xy.assign(src.pose_xy, src.pose_xy + 2 * size_t(src.n_pose));
    yaw.assign(src.pose_yaw, src.pose_yaw + src.n_pose);
    q0.assign(src.q0, src.q0 + T); q1.assign(src.q1, src.q1 + T);
    d0.assign(src.d0, src.d0 + T); d1.assign(src.d1, src.d1 + T);
    p.legal = legal.data();
    p.segment = src.segment ? segment.data() : nullptr;
    p.pose_xy = xy.data(); p.pose_yaw = yaw.data();
    p.q0 = q0.data(); p.q1 = q1.data(); p.d0 = d0.data(); p.d1 = d1.data();
  }
};

struct Scene {
  OwnedProblem prob;
  SceneTables tables;
  std::vector<uint8_t> plan;   // [K], 1 = planned reuse
  int j = 1, age = 0;
  int64_t charge = 0;
  int n_done = 0, n_veto = 0;
};

}  // namespace
}  // namespace dc

struct dc_sampler {
  dc::Geo g;
  dc_model_cfg cfg;
  dc_model_weights w;
  std::vector<dc_block_weights> blocks;
  bool two = false;                  // two experts: w_low from step k_switch on
  dc_model_weights w_low{};
  std::vector<dc_block_weights> blocks_low;
  int k_switch = 0;
  float* mod_low = nullptr;
  bool cfg_on = false;               // guidance branches (entries B..2B-1 unconditional)
  float guidance = 1.0f;
  const float* txt_null = nullptr;
  int B = 0, K = 0;
  std::vector<double> sigmas;
  dc_buffers buf;
  int metric = 0;
  int next_k = 1;
  std::vector<dc::Scene> scenes;
  double* host_sums = nullptr;   // pinned [B, 4]
  ~dc_sampler() {
    if (host_sums) (void)hipHostFree(host_sums);
  }
};

namespace dc {
namespace {

Status create(const dc_model_cfg* cfg, const dc_model_weights* w, int32_t B,
              const dc_sched_problem* problems, const double* sigmas, const dc_buffers* buf,
              const dc_sampler_opts& o, hipStream_t stream, dc_sampler** out) {
  if (!out || !w || !problems || !sigmas || !buf) return Status::arg("NULL argument");
  *out = nullptr;
  const int32_t metric = o.drift_metric;
  const bool cfg_on = o.cfg != 0;
  if (B < 1 || B > (cfg_on ? DC_MAX_BATCH / 2 : DC_MAX_BATCH))
    return Status::arg("B must be in [1, DC_MAX_BATCH] (in [1, DC_MAX_BATCH / 2] with guidance)");
  if (metric != 0 && metric != 1) return Status::arg("drift_metric must be 0 or 1");
  if (o.cfg != 0 && o.cfg != 1) return Status::arg("opts->cfg must be 0 or 1");
  auto s = std::make_unique<dc_sampler>();
  DC_TRY(make_geo(cfg, s->g));
  if (!buf->x || !buf->h_in || !buf->h || !buf->resid || !buf->u_ref || !buf->mod || !buf->sums ||
      !buf->ws || (s->g.Nt > 0 && !buf->txt))
    return Status::arg("a device buffer is NULL");
  if (cfg_on && (!std::isfinite(o.guidance) || (s->g.Nt > 0 && !o.txt_null)))
    return Status::arg("guidance needs a finite scale and txt_null");
  if (buf->ws_bytes < workspace_layout(s->g, cfg_on ? 2 * B : B).total)
    return Status::make(DC_ERR_WORKSPACE, "workspace smaller than dc_workspace_bytes()");
  if (!w->blocks) return Status::arg("weights->blocks is NULL");
  s->cfg = *cfg;
  s->blocks.assign(w->blocks, w->blocks + s->g.L);
  s->w = *w;
  s->w.blocks = s->blocks.data();
  s->cfg_on = cfg_on;
  s->guidance = o.guidance;
  s->txt_null = o.txt_null;
  if (o.w_low) {
    if (!o.w_low->blocks || !o.mod_low) return Status::arg("w_low->blocks and mod_low must be set");
    if (o.k_switch < 2 || o.k_switch > problems[0].K) return Status::arg("k_switch must be in 2..K");
    s->two = true;
    s->k_switch = o.k_switch;
    s->mod_low = o.mod_low;
    s->blocks_low.assign(o.w_low->blocks, o.w_low->blocks + s->g.L);
    s->w_low = *o.w_low;
    s->w_low.blocks = s->blocks_low.data();
  }
  s->B = B;
  s->K = problems[0].K;
  s->buf = *buf;
  s->metric = metric;
  s->sigmas.assign(sigmas, sigmas + s->K + 1);
  s->scenes.resize(size_t(B));
  for (int b = 0; b < B; ++b) {
    const dc_sched_problem& p = problems[b];
    if (p.K != s->K) return Status::arg("all scenes must share K");
    if (p.start_step != 1 || p.spent_q != 0 || p.spent_n != 0)
      return Status::arg("initial problems must start at step 1 with nothing spent");
    DC_TRY(validate_problem(p));
    if (s->two && (!p.segment || p.segment[s->k_switch - 1] == p.segment[s->k_switch - 2]))
      return Status::arg("with two experts every scene's segment must change at k_switch");
    Scene& sc = s->scenes[size_t(b)];
    sc.prob.assign(p);
    DC_TRY(scene_tables(sc.prob.p, sc.tables));
    int32_t n = 0;
    int64_t c = 0;
    DC_TRY(schedule(sc.prob.p, sc.tables, sc.plan, n, c));
  }
  DC_HIP(hipHostMalloc(reinterpret_cast<void**>(&s->host_sums), sizeof(double) * 4 * B));
  DC_TRY(time_modulation(s->g, &s->w, s->sigmas.data(), s->K, buf->mod, buf->ws, buf->ws_bytes, stream));
  if (s->two)
    DC_TRY(time_modulation(s->g, &s->w_low, s->sigmas.data(), s->K, s->mod_low, buf->ws,
                           buf->ws_bytes, stream));
  *out = s.release();
  return Status::ok();
}

Status step(dc_sampler* s, int k, hipStream_t st, uint8_t* realized, double* drift_out) {
  if (!s) return Status::arg("sampler is NULL");
  if (k != s->next_k || k < 1 || k > s->K)
    return Status::make(DC_ERR_STATE, "steps must be called in order 1..K (expected " +
                                          std::to_string(s->next_k) + ")");
  const Geo& g = s->g;
  const dc_buffers& bf = s->buf;
  const int B = s->B;
  const size_t mstride = size_t(g.L + 1) * 6 * g.d;
  // the expert of this step
  const bool low = s->two && k >= s->k_switch;
  const dc_model_weights* W = low ? &s->w_low : &s->w;
  const std::vector<dc_block_weights>& blocks = low ? s->blocks_low : s->blocks;
  const float* mod_k = (low ? s->mod_low : bf.mod) + size_t(k - 1) * mstride;
  const size_t row_stride = size_t(g.N) * g.d;            // one entry of h_in / h
  // with guidance, scene b's unconditional branch is entry B + b of h_in, h, resid
  auto with_branches = [&](const std::vector<int32_t>& v) {
    std::vector<int32_t> r(v);
    if (s->cfg_on)
      for (int32_t b : v) r.push_back(B + b);
    return r;
  };

  IdxList all;
  std::vector<int32_t> ids(static_cast<size_t>(B));
  for (int b = 0; b < B; ++b) ids[size_t(b)] = b;
  DC_TRY(make_idx(ids.data(), B, all));
  DC_TRY(patch_embed(g, W, bf.x, bf.txt, bf.h_in, all, bf.ws, bf.ws_bytes, st));
  if (s->cfg_on)
    DC_TRY(patch_embed(g, W, bf.x, s->txt_null, bf.h_in + size_t(B) * row_stride, all, bf.ws,
                       bf.ws_bytes, st));

  // planned reuses: observe the drift before any backbone call
  std::vector<int32_t> planned, refresh, reuse, vetoed;
  std::vector<double> drift(size_t(B), std::numeric_limits<double>::quiet_NaN());
  for (int b = 0; b < B; ++b)
    if (k > 1 && s->scenes[size_t(b)].plan[size_t(k - 1)]) planned.push_back(b);
  if (!planned.empty()) {
    IdxList il;
    DC_TRY(make_idx(planned.data(), int(planned.size()), il));
    DC_TRY(drift_call(g, bf.h_in, mod_k, bf.u_ref, 0, bf.sums, il, bf.ws, bf.ws_bytes, st));
    for (int b : planned)
      DC_HIP(hipMemcpyAsync(s->host_sums + 4 * b, bf.sums + 4 * b, 4 * sizeof(double),
                            hipMemcpyDeviceToHost, st));
    DC_HIP(hipStreamSynchronize(st));
  }
  std::vector<uint8_t> accept(size_t(B), 0);
  for (int b : planned) {
    Scene& sc = s->scenes[size_t(b)];
    const double* S = s->host_sums + 4 * b;
    const double eps = sc.prob.p.eps;
    const double d_obs = s->metric == 0 ? S[0] / (S[1] + eps) : std::sqrt(S[2]) / (std::sqrt(S[3]) + eps);
    drift[size_t(b)] = d_obs;
    const int h = sc.age + 1;
    const bool ok = h <= sc.prob.p.h_max && d_obs <= sc.tables.threshold(sc.j, h) + eps &&
                    sc.charge + sc.tables.cost(sc.j, h) <= sc.prob.p.tau_q;
    accept[size_t(b)] = ok ? 1 : 0;
    if (!ok) vetoed.push_back(b);
  }
  for (int b = 0; b < B; ++b) (accept[size_t(b)] ? reuse : refresh).push_back(b);

  if (!refresh.empty()) {
    IdxList il, ilb;
    DC_TRY(make_idx(refresh.data(), int(refresh.size()), il));
    const std::vector<int32_t> rb = with_branches(refresh);
    DC_TRY(make_idx(rb.data(), int(rb.size()), ilb));
    DC_TRY(drift_call(g, bf.h_in, mod_k, bf.u_ref, 1, nullptr, il, bf.ws, bf.ws_bytes, st));
    for (int b : rb)
      DC_TRY(copy_rows(bf.h_in + size_t(b) * row_stride, bf.h + size_t(b) * row_stride, row_stride, st));
    for (int l = 0; l < g.L; ++l)
      DC_TRY(block_forward(g, &blocks[size_t(l)], mod_k + size_t(l) * 6 * g.d, bf.h, ilb, bf.ws,
                           bf.ws_bytes, st));
    {
      ProfScope ps(KClass::kCacheStore, st);
      DC_TRY(cache_store(bf.h, bf.h_in, bf.resid, ilb, g, st));
    }
  }
  // reuse scenes: the fused bf16 head reads h_in and r itself; other models apply the
  // cache into h first
  const bool fused_reuse = head_euler_fused_ok(g);
  if (!reuse.empty() && !fused_reuse) {
    IdxList il;
    const std::vector<int32_t> rb = with_branches(reuse);
    DC_TRY(make_idx(rb.data(), int(rb.size()), il));
    ProfScope ps(KClass::kCacheApply, st);
    DC_TRY(cache_apply(bf.h_in, bf.resid, bf.h, il, g, st));
  }
  // x += dsig v, with guidance v = v_u + w (v_c - v_u) = w v_c + (1 - w) v_u: the update is
  // linear in v, so each branch's head adds its share
  const double dsig = s->sigmas[size_t(k)] - s->sigmas[size_t(k - 1)];
  const float* head_mod = mod_k + size_t(g.L) * 6 * g.d;
  const size_t rstride = size_t(g.Nv) * g.d * g.esz;      // one entry of the residual cache
  const float dsig_c = float(s->cfg_on ? dsig * s->guidance : dsig);
  const float dsig_u = float(dsig * (1.0 - double(s->guidance)));
  const std::vector<int32_t>& from_h = fused_reuse ? refresh : ids;
  if (!from_h.empty()) {
    IdxList il;
    DC_TRY(make_idx(from_h.data(), int(from_h.size()), il));
    DC_TRY(head_euler(g, W, head_mod, bf.h, bf.x, dsig_c, il, bf.ws, bf.ws_bytes, st, nullptr));
    if (s->cfg_on)
      DC_TRY(head_euler(g, W, head_mod, bf.h + size_t(B) * row_stride, bf.x, dsig_u, il, bf.ws,
                        bf.ws_bytes, st, nullptr));
  }
  if (fused_reuse && !reuse.empty()) {
    IdxList il;
    DC_TRY(make_idx(reuse.data(), int(reuse.size()), il));
    DC_TRY(head_euler(g, W, head_mod, bf.h_in, bf.x, dsig_c, il, bf.ws, bf.ws_bytes, st, bf.resid));
    if (s->cfg_on)
      DC_TRY(head_euler(g, W, head_mod, bf.h_in + size_t(B) * row_stride, bf.x, dsig_u, il, bf.ws,
                        bf.ws_bytes, st, static_cast<const char*>(bf.resid) + size_t(B) * rstride));
  }

  // controller state
  for (int b = 0; b < B; ++b) {
    Scene& sc = s->scenes[size_t(b)];
    if (accept[size_t(b)]) {
      sc.age += 1;
      sc.charge += sc.tables.cost(sc.j, sc.age);
      sc.n_done += 1;
    } else {
      sc.j = k;
      sc.age = 0;
    }
  }
  for (int b : vetoed) {
    Scene& sc = s->scenes[size_t(b)];
    sc.n_veto += 1;
    dc_sched_problem rp = sc.prob.p;
    rp.start_step = k;
    rp.spent_q = sc.charge;
    rp.spent_n = sc.n_done;
    std::vector<uint8_t> suffix;
    int32_t n = 0;
    int64_t c = 0;
    DC_TRY(schedule(rp, sc.tables, suffix, n, c));
    for (int kk = k; kk < s->K; ++kk) sc.plan[size_t(kk)] = suffix[size_t(kk)];
  }
  if (realized)
    for (int b = 0; b < B; ++b) realized[b] = accept[size_t(b)];
  if (drift_out)
    for (int b = 0; b < B; ++b) drift_out[b] = drift[size_t(b)];
  s->next_k = k + 1;
  return Status::ok();
}

}  // namespace
}  // namespace dc

using namespace dc;

extern "C" {

dc_status dc_sampler_create(const dc_model_cfg* cfg, const dc_model_weights* w, int32_t B,
                            const dc_sched_problem* problems, const double* sigmas,
                            const dc_buffers* buf, int32_t drift_metric, hipStream_t stream,
                            dc_sampler** out) {
  try {
    dc_sampler_opts o{};
    o.drift_metric = drift_metric;
    Status st = create(cfg, w, B, problems, sigmas, buf, o, stream, out);
    return st ? DC_OK : fail(st);
  } catch (const std::exception& e) {
    return fail(Status::arg(std::string("exception: ") + e.what()));
  }
}

dc_status dc_sampler_create_ex(const dc_model_cfg* cfg, const dc_model_weights* w, int32_t B,
                               const dc_sched_problem* problems, const double* sigmas,
                               const dc_buffers* buf, const dc_sampler_opts* opts,
                               hipStream_t stream, dc_sampler** out) {
  try {
    dc_sampler_opts o{};
    if (opts) o = *opts;
    Status st = create(cfg, w, B, problems, sigmas, buf, o, stream, out);
    return st ? DC_OK : fail(st);
  } catch (const std::exception& e) {
    return fail(Status::arg(std::string("exception: ") + e.what()));
  }
}

dc_status dc_denoise_step(dc_sampler* s, int32_t k, hipStream_t stream, uint8_t* realized,
                          double* drift) {
  try {
    Status st = step(s, k, stream, realized, drift);
    return st ? DC_OK : fail(st);
  } catch (const std::exception& e) {
    return fail(Status::arg(std::string("exception: ") + e.what()));
  }
}

dc_status dc_sampler_plan(const dc_sampler* s, int32_t b, uint8_t* reuse, int32_t* n_veto,
                          int64_t* charge_q) {
  if (!s || b < 0 || b >= s->B) return fail(Status::arg("bad sampler or scene index"));
  const Scene& sc = s->scenes[size_t(b)];
  if (reuse) std::memcpy(reuse, sc.plan.data(), sc.plan.size());
  if (n_veto) *n_veto = sc.n_veto;
  if (charge_q) *charge_q = sc.charge;
  return DC_OK;
}

void dc_sampler_destroy(dc_sampler* s) { delete s; }

}  // extern "C"
