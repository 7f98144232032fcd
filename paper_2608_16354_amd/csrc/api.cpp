// C ABI of the library: argument checking, workspace layout and the device-step
// entry points.  The sampler (causal controller) is in sampler.cpp.
#include <algorithm>
#include <cstring>
#include <string>

#include "internal.h"

namespace dc {

namespace {
thread_local std::string g_last_error;

inline size_t align256(size_t v) { return (v + 255) & ~size_t(255); }
}  // namespace

Status hip_status(hipError_t e, const char* what) {
  return Status::make(DC_ERR_HIP, std::string(what) + ": " + hipGetErrorString(e));
}

dc_status fail(const Status& s) {
  g_last_error = s.msg;
  return s.code;
}

Status make_geo(const dc_model_cfg* cfg, Geo& g) {
  if (!cfg) return Status::arg("cfg is NULL");
  if (cfg->dtype != DC_F32 && cfg->dtype != DC_BF16) return Status::make(DC_ERR_DTYPE, "unknown dtype");
  g.L = cfg->n_blocks; g.d = cfg->hidden; g.H = cfg->heads; g.Dh = cfg->head_dim;
  g.F = cfg->mlp_hidden; g.C = cfg->lat_c; g.T = cfg->lat_t; g.Hl = cfg->lat_h; g.Wl = cfg->lat_w;
  g.p = cfg->patch; g.Nt = cfg->n_txt; g.eps = cfg->ln_eps;
  g.bf16 = cfg->dtype == DC_BF16;
  g.esz = g.bf16 ? 2 : 4;
  if (g.L < 1 || g.d < 1 || g.H < 1 || g.F < 1 || g.C < 1 || g.T < 1 || g.p < 1 || g.Nt < 0)
    return Status::shape("model dimensions must be positive");
  if (g.H * g.Dh != g.d) return Status::shape("heads * head_dim must equal hidden");
  if (g.d % 128 || g.d > 3072) return Status::shape("hidden must be a multiple of 128, at most 3072");
  if (g.F % 128) return Status::shape("mlp_hidden must be a multiple of 128");
  if (g.bf16 ? (g.Dh != 64 && g.Dh != 72) : (g.Dh != 64))
    return Status::shape("head_dim must be 64 (or 72 with bf16)");
  if (g.Hl % g.p || g.Wl % g.p) return Status::shape("latent height/width must be divisible by patch");
  g.P = g.C * g.p * g.p;
  if (g.P != 64) return Status::shape("lat_c * patch^2 must be 64");
  g.Hp = g.Hl / g.p; g.Wp = g.Wl / g.p;
  g.Nv = g.T * g.Hp * g.Wp;
  g.N = g.Nv + g.Nt;
  if (!(g.eps > 0.f)) return Status::shape("ln_eps must be positive");
  return Status::ok();
}

Status make_idx(const int32_t* idx, int32_t n, IdxList& out) {
  if (n < 0 || n > DC_MAX_BATCH) return Status::arg("n must be in [0, DC_MAX_BATCH]");
  if (n > 0 && !idx) return Status::arg("idx is NULL");
  out.n = n;
  for (int i = 0; i < n; ++i) {
    if (idx[i] < 0 || idx[i] >= DC_MAX_BATCH) return Status::arg("sample index out of range");
    for (int j = 0; j < i; ++j)
      if (idx[j] == idx[i]) return Status::arg("duplicate sample index");
    out.v[i] = idx[i];
  }
  for (int i = n; i < DC_MAX_BATCH; ++i) out.v[i] = 0;
  return Status::ok();
}

Workspace workspace_layout(const Geo& g, int batch) {
  Workspace w{};
  w.ldv = (g.N + 63) / 64 * 64;
  w.kTmax = 64;
  size_t off = 0;
  auto take = [&](size_t bytes) { const size_t o = off; off = align256(off + bytes); return o; };
  w.a = take(size_t(g.N) * g.d * g.esz);
  w.qk = take(size_t(w.ldv + 64) * 2 * g.d * g.esz);   // padding rows for the attention's K tiles
  w.vt = take(size_t(g.d) * w.ldv * g.esz);
  w.o = take(size_t(g.N) * g.d * g.esz);
  w.ff = take(size_t(g.N) * g.F * g.esz);
  w.patch = take(size_t(g.Nv) * 64 * 4);
  (void)batch;
  w.drift_part = take(size_t(DC_MAX_BATCH) * kDriftBlocks * 4 * sizeof(double));
  // split-tail partials of the bf16 attention: up to 64 split items per XCD, two halves of
  // 128 queries x (head_dim + 4) floats each
  w.attn_part_bytes = g.bf16 ? size_t(8) * 64 * 2 * 128 * (g.Dh + 4) * sizeof(float) : 0;
  w.attn_part = take(w.attn_part_bytes);
  w.tm_e = take(size_t(w.kTmax) * 256 * 4);
  w.tm_h = take(size_t(w.kTmax) * g.d * 4);
  w.tm_c = take(size_t(w.kTmax) * g.d * 4);
  w.tm_s = take(size_t(w.kTmax) * g.d * 4);
  w.tm_m = take(size_t(w.kTmax) * 6 * g.d * 4 + size_t(w.kTmax) * sizeof(double));
  w.total = off;
  return w;
}

static Status check_ws(const Geo& g, int batch, void* ws, size_t ws_bytes, Workspace& w) {
  w = workspace_layout(g, batch);
  if (!ws) return Status::make(DC_ERR_WORKSPACE, "workspace is NULL");
  if (reinterpret_cast<uintptr_t>(ws) % 256) return Status::make(DC_ERR_WORKSPACE, "workspace must be 256-byte aligned");
  if (ws_bytes < w.total)
    return Status::make(DC_ERR_WORKSPACE, "workspace too small: need " + std::to_string(w.total) + " bytes");
  return Status::ok();
}

static int max_index(const IdxList& il) {
  int m = -1;
  for (int i = 0; i < il.n; ++i) m = std::max(m, il.v[i]);
  return m;
}

template <class T> T* at(void* base, size_t off) {
  return reinterpret_cast<T*>(static_cast<char*>(base) + off);
}

Status time_modulation(const Geo& g, const dc_model_weights* w, const double* sigmas, int K,
                       float* mod, void* ws, size_t ws_bytes, hipStream_t s) {
  if (!w || !sigmas || !mod) return Status::arg("NULL argument");
  if (K < 1) return Status::arg("K must be >= 1");
  if (!w->blocks) return Status::arg("weights->blocks is NULL");
  Workspace L;
  DC_TRY(check_ws(g, 1, ws, ws_bytes, L));
  double* sig = at<double>(ws, L.tm_m + size_t(L.kTmax) * 6 * g.d * 4);
  for (int k0 = 0; k0 < K; k0 += L.kTmax) {
    const int kc = std::min(L.kTmax, K - k0);
    DC_HIP(hipMemcpyAsync(sig, sigmas + k0, sizeof(double) * kc, hipMemcpyHostToDevice, s));
    float* e = at<float>(ws, L.tm_e);
    float* hdn = at<float>(ws, L.tm_h);
    float* c = at<float>(ws, L.tm_c);
    float* sc = at<float>(ws, L.tm_s);
    float* m = at<float>(ws, L.tm_m);
    DC_TRY(time_features(sig, kc, e, 256, s));
    DC_TRY(gemm_f32_bias_act(e, 256, w->w_t1, 256, w->b_t1, hdn, g.d, kc, g.d, 256, Act::kSilu, s));
    DC_TRY(gemm_f32_bias_act(hdn, g.d, w->w_t2, g.d, w->b_t2, c, g.d, kc, g.d, g.d, Act::kNone, s));
    DC_TRY(silu_inplace(c, sc, size_t(kc) * g.d, s));
    DC_TRY(gemm_f32_bias_act(sc, g.d, w->w_m, g.d, w->b_m, m, 6 * g.d, kc, 6 * g.d, g.d, Act::kNone, s));
    for (int l = 0; l < g.L; ++l) {
      if (!w->blocks[l].mod_offset) return Status::arg("mod_offset is NULL");
      DC_TRY(assemble_modulation(m, c, w->blocks[l].mod_offset, kc, g.L, l, g, mod, k0, s));
    }
    DC_TRY(assemble_modulation(m, c, w->head_mod, kc, g.L, g.L, g, mod, k0, s));
  }
  return Status::ok();
}

Status patch_embed(const Geo& g, const dc_model_weights* w, const float* x, const float* txt,
                   float* h_in, const IdxList& il, void* ws, size_t ws_bytes, hipStream_t s) {
  if (!w || !x || !h_in || (g.Nt > 0 && !txt)) return Status::arg("NULL argument");
  Workspace L;
  DC_TRY(check_ws(g, max_index(il) + 1, ws, ws_bytes, L));
  float* patches = at<float>(ws, L.patch);
  const size_t lat = size_t(g.C) * g.T * g.Hl * g.Wl;
  for (int i = 0; i < il.n; ++i) {
    const int b = il.v[i];
    float* hb = h_in + size_t(b) * g.N * g.d;
    ProfScope ps(KClass::kPatchEmbed, s);
    if (g.bf16) {
      DC_TRY(patch_embed_bf16(x + size_t(b) * lat, w->w_pe, w->b_pe, static_cast<const uint16_t*>(w->pos),
                              hb, g, s));
    } else {
      DC_TRY(patchify(x + size_t(b) * lat, patches, g, s));
      DC_TRY(gemm_f32_patch_embed(patches, w->w_pe, w->b_pe, w->pos, false, hb, g.d, g.Nv, g.d, s));
    }
    if (g.Nt > 0) DC_TRY(copy_text(txt + size_t(b) * g.Nt * g.d, hb, g, s));
  }
  return Status::ok();
}

Status block_forward(const Geo& g, const dc_block_weights* bw, const float* mod, float* h,
                     const IdxList& il, void* ws, size_t ws_bytes, hipStream_t s) {
  if (!bw || !mod || !h) return Status::arg("NULL argument");
  if (!bw->w_qkv || !bw->b_qkv || !bw->w_o || !bw->b_o || !bw->w_1 || !bw->b_1 || !bw->w_2 || !bw->b_2)
    return Status::arg("block weight pointer is NULL");
  Workspace L;
  DC_TRY(check_ws(g, max_index(il) + 1, ws, ws_bytes, L));
  const int N = g.N, d = g.d, F = g.F;
  const float *shift1 = mod, *scale1 = mod + d, *gate1 = mod + 2 * d;
  const float *shift2 = mod + 3 * d, *scale2 = mod + 4 * d, *gate2 = mod + 5 * d;
  for (int i = 0; i < il.n; ++i) {
    float* hb = h + size_t(il.v[i]) * N * d;
    if (g.bf16) {
      uint16_t* a = at<uint16_t>(ws, L.a);
      uint16_t* qk = at<uint16_t>(ws, L.qk);
      uint16_t* vt = at<uint16_t>(ws, L.vt);
      uint16_t* o = at<uint16_t>(ws, L.o);
      uint16_t* ff = at<uint16_t>(ws, L.ff);
      const uint16_t* wqkv = static_cast<const uint16_t*>(bw->w_qkv);
      { ProfScope ps(KClass::kLnModulate, s); DC_TRY(ln_modulate(hb, N, d, shift1, scale1, a, d, true, g, s)); }
      { ProfScope ps(KClass::kGemmQKV, s); DC_TRY(gemm_bf16_qkv(a, wqkv, bw->b_qkv, qk, vt, L.ldv, g, N, s)); }
      {
        ProfScope ps(KClass::kAttention, s);
        DC_TRY(attention_bf16(qk, vt, L.ldv, o, g, N, at<float>(ws, L.attn_part), L.attn_part_bytes, s));
      }
      {
        ProfScope ps(KClass::kGemmOut, s);
        DC_TRY(gemm_bf16_gate_residual(o, d, static_cast<const uint16_t*>(bw->w_o), bw->b_o, gate1,
                                       hb, d, N, d, d, s));
      }
      { ProfScope ps(KClass::kLnModulate, s); DC_TRY(ln_modulate(hb, N, d, shift2, scale2, a, d, true, g, s)); }
      {
        ProfScope ps(KClass::kGemmUp, s);
        DC_TRY(gemm_bf16_gelu(a, d, static_cast<const uint16_t*>(bw->w_1), bw->b_1, ff, F, N, F, d, s));
      }
      {
        ProfScope ps(KClass::kGemmDown, s);
        DC_TRY(gemm_bf16_gate_residual(ff, F, static_cast<const uint16_t*>(bw->w_2), bw->b_2, gate2,
                                       hb, d, N, d, F, s));
      }
    } else {
      float* a = at<float>(ws, L.a);
      float* qk = at<float>(ws, L.qk);
      float* vt = at<float>(ws, L.vt);
      float* o = at<float>(ws, L.o);
      float* ff = at<float>(ws, L.ff);
      DC_TRY(ln_modulate(hb, N, d, shift1, scale1, a, d, false, g, s));
      DC_TRY(gemm_f32_qkv(a, static_cast<const float*>(bw->w_qkv), bw->b_qkv, qk, vt, L.ldv, g, N, s));
      DC_TRY(attention_f32(qk, vt, L.ldv, o, g, N, s));
      DC_TRY(gemm_f32_gate_residual(o, d, static_cast<const float*>(bw->w_o), d, bw->b_o, gate1, hb,
                                    d, N, d, d, s));
      DC_TRY(ln_modulate(hb, N, d, shift2, scale2, a, d, false, g, s));
      DC_TRY(gemm_f32_gelu(a, d, static_cast<const float*>(bw->w_1), d, bw->b_1, ff, F, N, F, d, s));
      DC_TRY(gemm_f32_gate_residual(ff, F, static_cast<const float*>(bw->w_2), F, bw->b_2, gate2, hb,
                                    d, N, d, F, s));
    }
  }
  return Status::ok();
}

// resid != NULL (bf16 models the fused head takes): the head input of sample b is
// g = gin[b] + resid[b] on the video rows, formed inside the head kernel (reuse steps).
Status head_euler(const Geo& g, const dc_model_weights* w, const float* head_mod, const float* gin,
                  float* x, float dsigma, const IdxList& il, void* ws, size_t ws_bytes,
                  hipStream_t s, const void* resid) {
  if (!w || !head_mod || !gin || !x || !w->w_head || !w->b_head) return Status::arg("NULL argument");
  if (resid && !head_euler_fused_ok(g)) return Status::shape("head with a residual input needs the fused bf16 head");
  Workspace L;
  DC_TRY(check_ws(g, max_index(il) + 1, ws, ws_bytes, L));
  const size_t lat = size_t(g.C) * g.T * g.Hl * g.Wl;
  for (int i = 0; i < il.n; ++i) {
    const int b = il.v[i];
    const float* gb = gin + size_t(b) * g.N * g.d;
    ProfScope ps(resid ? KClass::kHeadReuse : KClass::kHead, s);
    if (head_euler_fused_ok(g)) {
      const uint16_t* rb = resid ? static_cast<const uint16_t*>(resid) + size_t(b) * g.Nv * g.d : nullptr;
      DC_TRY(head_euler_bf16(gb, rb, static_cast<const uint16_t*>(w->w_head), w->b_head, head_mod,
                             head_mod + g.d, x + size_t(b) * lat, dsigma, g, s));
      continue;
    }
    DC_TRY(ln_modulate(gb, g.Nv, g.d, head_mod, head_mod + g.d, at<void>(ws, L.a), g.d, g.bf16, g, s));
    if (g.bf16)
      DC_TRY(gemm_bf16_head(at<uint16_t>(ws, L.a), g.d, static_cast<const uint16_t*>(w->w_head),
                            w->b_head, x + size_t(b) * lat, dsigma, g, g.Nv, s));
    else
      DC_TRY(gemm_f32_head(at<float>(ws, L.a), g.d, static_cast<const float*>(w->w_head), w->b_head,
                           x + size_t(b) * lat, dsigma, g, g.Nv, s));
  }
  return Status::ok();
}

Status drift_call(const Geo& g, const float* h_in, const float* mod0, void* u_ref, int snapshot,
                  double* sums, const IdxList& il, void* ws, size_t ws_bytes, hipStream_t s) {
  if (!h_in || !mod0 || !u_ref || (!snapshot && !sums)) return Status::arg("NULL argument");
  if (il.n == 0) return Status::ok();
  Workspace L;
  DC_TRY(check_ws(g, std::max(il.n, max_index(il) + 1), ws, ws_bytes, L));
  ProfScope ps(KClass::kDrift, s);
  return drift(h_in, mod0, u_ref, snapshot != 0, sums, il, g, at<double>(ws, L.drift_part), s);
}

}  // namespace dc

using namespace dc;

#define DC_ENTRY(body)                                             \
  try {                                                            \
    ::dc::Status st_ = (body);                                     \
    if (!st_) return ::dc::fail(st_);                              \
    return DC_OK;                                                  \
  } catch (const std::exception& ex_) {                            \
    return ::dc::fail(Status::arg(std::string("exception: ") + ex_.what())); \
  }

extern "C" {

const char* dc_last_error(void) { return g_last_error.c_str(); }

size_t dc_workspace_bytes(const dc_model_cfg* cfg, int32_t batch) {
  Geo g;
  if (!make_geo(cfg, g) || batch < 1 || batch > DC_MAX_BATCH) return 0;
  return workspace_layout(g, batch).total;
}

dc_status dc_time_modulation(const dc_model_cfg* cfg, const dc_model_weights* w, const double* sigmas,
                             int32_t K, float* mod, void* ws, size_t ws_bytes, hipStream_t stream) {
  DC_ENTRY(([&]() -> Status {
    Geo g;
    DC_TRY(make_geo(cfg, g));
    return time_modulation(g, w, sigmas, K, mod, ws, ws_bytes, stream);
  })());
}

dc_status dc_patch_embed(const dc_model_cfg* cfg, const dc_model_weights* w, const float* x,
                         const float* txt, float* h_in, const int32_t* idx, int32_t n, void* ws,
                         size_t ws_bytes, hipStream_t stream) {
  DC_ENTRY(([&]() -> Status {
    Geo g;
    IdxList il;
    DC_TRY(make_geo(cfg, g));
    DC_TRY(make_idx(idx, n, il));
    return patch_embed(g, w, x, txt, h_in, il, ws, ws_bytes, stream);
  })());
}

dc_status dc_block_forward(const dc_model_cfg* cfg, const dc_block_weights* blk, const float* mod,
                           float* h, const int32_t* idx, int32_t n, void* ws, size_t ws_bytes,
                           hipStream_t stream) {
  DC_ENTRY(([&]() -> Status {
    Geo g;
    IdxList il;
    DC_TRY(make_geo(cfg, g));
    DC_TRY(make_idx(idx, n, il));
    return block_forward(g, blk, mod, h, il, ws, ws_bytes, stream);
  })());
}

dc_status dc_cache_store(const dc_model_cfg* cfg, const float* h_out, const float* h_in, void* resid,
                         const int32_t* idx, int32_t n, hipStream_t stream) {
  DC_ENTRY(([&]() -> Status {
    Geo g;
    IdxList il;
    DC_TRY(make_geo(cfg, g));
    DC_TRY(make_idx(idx, n, il));
    if (!h_out || !h_in || !resid) return Status::arg("NULL argument");
    if (il.n == 0) return Status::ok();
    ProfScope ps(KClass::kCacheStore, stream);
    return cache_store(h_out, h_in, resid, il, g, stream);
  })());
}

dc_status dc_cache_apply(const dc_model_cfg* cfg, const float* h_in, const void* resid, float* gout,
                         const int32_t* idx, int32_t n, hipStream_t stream) {
  DC_ENTRY(([&]() -> Status {
    Geo g;
    IdxList il;
    DC_TRY(make_geo(cfg, g));
    DC_TRY(make_idx(idx, n, il));
    if (!h_in || !resid || !gout) return Status::arg("NULL argument");
    if (il.n == 0) return Status::ok();
    ProfScope ps(KClass::kCacheApply, stream);
    return cache_apply(h_in, resid, gout, il, g, stream);
  })());
}

dc_status dc_drift_l1(const dc_model_cfg* cfg, const float* h_in, const float* mod0, void* u_ref,
                      int32_t snapshot, double* sums, const int32_t* idx, int32_t n, void* ws,
                      size_t ws_bytes, hipStream_t stream) {
  DC_ENTRY(([&]() -> Status {
    Geo g;
    IdxList il;
    DC_TRY(make_geo(cfg, g));
    DC_TRY(make_idx(idx, n, il));
    return drift_call(g, h_in, mod0, u_ref, snapshot, sums, il, ws, ws_bytes, stream);
  })());
}

dc_status dc_drift_l1_noalloc(const dc_model_cfg* cfg, const float* h_in, const float* mod0,
                              void* u_ref, int32_t snapshot, double* sums, const int32_t* idx,
                              int32_t n, hipStream_t stream) {
  DC_ENTRY(([&]() -> Status {
    Geo g;
    IdxList il;
    DC_TRY(make_geo(cfg, g));
    DC_TRY(make_idx(idx, n, il));
    if (!h_in || !mod0 || !u_ref || (!snapshot && !sums)) return Status::arg("NULL argument");
    if (il.n == 0) return Status::ok();
    return drift_noalloc(h_in, mod0, u_ref, snapshot != 0, sums, il, g, stream);
  })());
}

dc_status dc_head_euler(const dc_model_cfg* cfg, const dc_model_weights* w, const float* head_mod,
                        const float* g_in, float* x, float dsigma, const int32_t* idx, int32_t n,
                        void* ws, size_t ws_bytes, hipStream_t stream) {
  DC_ENTRY(([&]() -> Status {
    Geo g;
    IdxList il;
    DC_TRY(make_geo(cfg, g));
    DC_TRY(make_idx(idx, n, il));
    return head_euler(g, w, head_mod, g_in, x, dsigma, il, ws, ws_bytes, stream, nullptr);
  })());
}

size_t dc_calibrate_workspace_bytes(const dc_model_cfg* cfg, int32_t K) {
  Geo g;
  if (!make_geo(cfg, g) || K < 1) return 0;
  return calibrate_workspace_bytes(g, K);
}

dc_status dc_calibrate_tables(const dc_model_cfg* cfg, const dc_model_weights* w, const float* x1,
                              const float* txt, const double* sigmas, int32_t K, int32_t h_max,
                              double eps, double* q, double* d, void* ws, size_t ws_bytes,
                              hipStream_t stream) {
  DC_ENTRY(([&]() -> Status {
    Geo g;
    DC_TRY(make_geo(cfg, g));
    return calibrate_tables(g, w, x1, txt, sigmas, K, h_max, eps, q, d, ws, ws_bytes, stream);
  })());
}

dc_status dc_schedule_dp(const dc_sched_problem* p, dc_schedule* out) {
  DC_ENTRY(([&]() -> Status {
    if (!p || !out || !out->reuse) return Status::arg("NULL argument");
    DC_TRY(validate_problem(*p));
    SceneTables t;
    DC_TRY(scene_tables(*p, t));
    std::vector<uint8_t> reuse;
    int32_t n = 0;
    int64_t c = 0;
    DC_TRY(schedule(*p, t, reuse, n, c));
    std::memcpy(out->reuse, reuse.data(), reuse.size());
    if (out->chat_q && !t.chat.empty()) std::memcpy(out->chat_q, t.chat.data(), t.chat.size() * 8);
    if (out->dbar && !t.dbar.empty()) std::memcpy(out->dbar, t.dbar.data(), t.dbar.size() * 8);
    out->n_reuse = n;
    out->cost_q = c;
    out->L = t.L; out->Theta = t.Theta; out->zL = t.zL; out->zTh = t.zTh; out->D = t.D;
    out->in_support = t.in_support ? 1 : 0;
    return Status::ok();
  })());
}

dc_status dc_motion_statistics(const double* pose_xy, const double* pose_yaw, int32_t n_pose,
                               double* L, double* Theta) {
  DC_ENTRY(([&]() -> Status {
    if (!L || !Theta || (n_pose > 0 && (!pose_xy || !pose_yaw))) return Status::arg("NULL argument");
    if (n_pose < 0) return Status::arg("n_pose must be >= 0");
    motion_statistics(pose_xy, pose_yaw, n_pose, *L, *Theta);
    return Status::ok();
  })());
}

dc_status dc_select_anchors(const double* L, const double* Theta, int32_t n, double eps, double* anchors,
                            int32_t* index) {
  DC_ENTRY(([&]() -> Status {
    if (!L || !Theta || !anchors || !index) return Status::arg("NULL argument");
    if (!(eps > 0.0)) return Status::arg("eps must be positive");
    int i0 = 0, i1 = -1;
    DC_TRY(select_anchors(L, Theta, n, eps, i0, i1));
    index[0] = i0;
    index[1] = i1;
    anchors[0] = L[i0];
    anchors[1] = Theta[i0];
    anchors[2] = i1 >= 0 ? L[i1] : L[i0];
    anchors[3] = i1 >= 0 ? Theta[i1] : Theta[i0];
    return Status::ok();
  })());
}

dc_status dc_select_tau(const dc_sched_problem* problems, int32_t n, double rho, int64_t* tau_q) {
  DC_ENTRY(([&]() -> Status {
    if (!problems || !tau_q) return Status::arg("NULL argument");
    if (!(rho >= 0.0 && rho <= 1.0)) return Status::arg("rho must be in [0, 1]");
    return select_tau(problems, n, rho, *tau_q);
  })());
}

}  // extern "C"
