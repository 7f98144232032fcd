// Anchor calibration of the run tables on the GPU (Sec. 3.1 after Eq. 4; Eq. 5-7).
//
// For one anchor clip the full (uncached) denoising trace stores, per step k, the latent
// x_k the step starts from, the backbone input u_k (block 0's modulated input of the
// video rows) and the backbone output r_k = h_out - h_in over the video rows.  For a run
// that refreshes at step j and reuses r_j for h steps:
//   Eq. 5  d_{j,h} = ||u_{j+h} - u_j||_2 / (||u_{j+h}||_2 + eps);
//   Eq. 6  e_{j,l} = H_{j+l}(x_{j+l}, r_j) - H_{j+l}(x_{j+l}, r_{j+l}), H_k(x, r) the
//          denoiser output of the head for g = h_in(x)[video] + r;
//   Eq. 7  G_{j,h} = sum_{l <= h} P_{j+l} e_{j,l},  q_{j,h} = ||G_{j,h}||_2 / (||x_out||_2 + eps),
//          with P_t e the tangent of the terminal latent when the denoiser output of step
//          t moves by e: dx = (sigma_{t+1} - sigma_t) e, then for every later step k
//          dx += (sigma_{k+1} - sigma_k) J_k dx, J_k the Jacobian of the full network at
//          x_k (a Jacobian-vector product: the network run in tangent mode).
// Runs with j + h > K price nothing and stay 0.  The trace runs the library's own
// kernels for the model's dtype (bf16 models: bf16 MFMA blocks); r, u, the perturbations
// and every tangent are fp32 (fp32 SIMT kernels, calib.hip, with bf16 weights widened
// exactly on load).
#include <algorithm>
#include <cmath>

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

namespace {

inline size_t al256(size_t v) { return (v + 255) & ~size_t(255); }

struct CalibLayout {
  size_t blk, blk_bytes, mod, xs, us, rs, h_in, h, dh, a, da, qkv, dqkv, o, dout, z, dz, patches,
      zeros, v1, v2, e, G, dx, red, red_out, total;
};

CalibLayout calib_layout(const Geo& g, int K) {
  CalibLayout c{};
  size_t off = 0;
  auto take = [&](size_t bytes) { const size_t o = off; off = al256(off + bytes); return o; };
  const size_t N = size_t(g.N), Nv = size_t(g.Nv), d = size_t(g.d), F = size_t(g.F);
  const size_t lat = size_t(g.C) * g.T * g.Hl * g.Wl;
  c.blk_bytes = workspace_layout(g, 1).total;
  c.blk = take(c.blk_bytes);
  c.mod = take(size_t(K) * (g.L + 1) * 6 * d * 4);
  c.xs = take(size_t(K + 1) * lat * 4);
  c.us = take(size_t(K) * Nv * d * 4);
  c.rs = take(size_t(K) * Nv * d * 4);
  c.h_in = take(N * d * 4);
  c.h = take(N * d * 4);
  c.dh = take(N * d * 4);
  c.a = take(N * d * 4);
  c.da = take(N * d * 4);
  c.qkv = take(N * 3 * d * 4);
  c.dqkv = take(N * 3 * d * 4);
  c.o = take(N * d * 4);
  c.dout = take(N * d * 4);
  c.z = take(N * F * 4);
  c.dz = take(N * F * 4);
  c.patches = take(Nv * 64 * 4);
  c.zeros = take(std::max(std::max(3 * d, F), size_t(64)) * 4);
  c.v1 = take(lat * 4);
  c.v2 = take(lat * 4);
  c.e = take(lat * 4);
  c.G = take(lat * 4);
  c.dx = take(lat * 4);
  c.red = take(sumsq_scratch_doubles() * 8);
  c.red_out = take(2 * 8);
  c.total = off;
  return c;
}

template <class T> T* at(void* base, size_t off) {
  return reinterpret_cast<T*>(static_cast<char*>(base) + off);
}

struct Calib {
  const Geo& g;
  const dc_model_weights* w;
  const float* txt;
  const double* sig;
  int K;
  void* ws;
  CalibLayout L;
  hipStream_t s;
  IdxList one;
  size_t lat, mstride;

  void* blk() const { return at<void>(ws, L.blk); }
  float* F(size_t off) const { return at<float>(ws, off); }
  const float* mod_k(int k) const { return F(L.mod) + size_t(k - 1) * mstride; }
  float* x_at(int k) const { return F(L.xs) + size_t(k - 1) * lat; }        // x_k, k = 1..K+1
  float* u_at(int k) const { return F(L.us) + size_t(k - 1) * g.Nv * g.d; }
  float* r_at(int k) const { return F(L.rs) + size_t(k - 1) * g.Nv * g.d; }
  float dsig(int k) const { return float(sig[k] - sig[k - 1]); }            // step k: sigma_{k+1} - sigma_k

  // (sum (a - b)^2, sum a^2) over n elements, read back (one wait)
  Status norms(const float* a, const float* b, size_t n, double out[2]) {
    DC_TRY(sumsq(a, b, n, at<double>(ws, L.red), at<double>(ws, L.red_out), s));
    DC_HIP(hipMemcpyAsync(out, at<double>(ws, L.red_out), 2 * sizeof(double), hipMemcpyDeviceToHost, s));
    DC_HIP(hipStreamSynchronize(s));
    return Status::ok();
  }

  // full trace: x_1..x_{K+1}, u_k, r_k
  Status trace(const float* x1) {
    DC_HIP(hipMemcpyAsync(x_at(1), x1, lat * 4, hipMemcpyDeviceToDevice, s));
    for (int k = 1; k <= K; ++k) {
      const float* mk = mod_k(k);
      DC_TRY(patch_embed(g, w, x_at(k), txt, F(L.h_in), one, blk(), L.blk_bytes, s));
      DC_TRY(ln_modulate(F(L.h_in), g.Nv, g.d, mk, mk + g.d, u_at(k), g.d, false, g, s));
      DC_TRY(copy_rows(F(L.h_in), F(L.h), size_t(g.N) * g.d, s));
      for (int l = 0; l < g.L; ++l)
        DC_TRY(block_forward(g, &w->blocks[l], mk + size_t(l) * 6 * g.d, F(L.h), one, blk(), L.blk_bytes, s));
      DC_TRY(lincomb(r_at(k), F(L.h), 1.0f, F(L.h_in), -1.0f, size_t(g.Nv) * g.d, s));   // r = h_out - h_in
      DC_HIP(hipMemcpyAsync(x_at(k + 1), x_at(k), lat * 4, hipMemcpyDeviceToDevice, s));
      DC_TRY(head_euler(g, w, mk + size_t(g.L) * 6 * g.d, F(L.h), x_at(k + 1), dsig(k), one, blk(),
                        L.blk_bytes, s, nullptr));
    }
    return Status::ok();
  }

  // v = H_k(x_k, r) into out: the head of g = h_in(x_k)[video] + r, as x = 0 + 1 v
  Status interface(int k, const float* r, float* out) {
    const float* mk = mod_k(k);
    DC_TRY(patch_embed(g, w, x_at(k), txt, F(L.h_in), one, blk(), L.blk_bytes, s));
    DC_TRY(lincomb(F(L.h), F(L.h_in), 1.0f, r, 1.0f, size_t(g.Nv) * g.d, s));         // g = h_in + r
    DC_HIP(hipMemsetAsync(out, 0, lat * 4, s));
    return head_euler(g, w, mk + size_t(g.L) * 6 * g.d, F(L.h), out, 1.0f, one, blk(), L.blk_bytes, s,
                      nullptr);
  }

  // the fp32 SIMT GEMMs with the model's weights (fp32, or bf16 widened on load)
  Status mm(const float* A, int lda, const void* W, int ldw, const float* bias, float* out, int ldo,
            int M, int N, int Kd) const {
    if (g.bf16)
      return gemm_f32_bias_act(A, lda, static_cast<const uint16_t*>(W), ldw, bias, out, ldo, M, N, Kd,
                               Act::kNone, s);
    return gemm_f32_bias_act(A, lda, static_cast<const float*>(W), ldw, bias, out, ldo, M, N, Kd,
                             Act::kNone, s);
  }
  Status mm_gate(const float* A, int lda, const void* W, int ldw, const float* bias, const float* gate,
                 float* h, int M, int N, int Kd) const {
    if (g.bf16)
      return gemm_f32_gate_residual(A, lda, static_cast<const uint16_t*>(W), ldw, bias, gate, h, g.d, M,
                                    N, Kd, s);
    return gemm_f32_gate_residual(A, lda, static_cast<const float*>(W), ldw, bias, gate, h, g.d, M, N,
                                  Kd, s);
  }

  // one block in tangent mode on (h, dh)
  Status block_jvp(int l, const float* m6) {
    const dc_block_weights& b = w->blocks[l];
    const int N = g.N, d = g.d, Fh = g.F;
    const float* zeros = F(L.zeros);
    const float *sh1 = m6, *sc1 = m6 + d, *g1 = m6 + 2 * d, *sh2 = m6 + 3 * d, *sc2 = m6 + 4 * d,
                *g2 = m6 + 5 * d;
    DC_TRY(ln_mod_jvp(F(L.h), F(L.dh), N, d, d, sh1, sc1, F(L.a), F(L.da), g.eps, s));
    DC_TRY(mm(F(L.a), d, b.w_qkv, d, b.b_qkv, F(L.qkv), 3 * d, N, 3 * d, d));
    DC_TRY(mm(F(L.da), d, b.w_qkv, d, zeros, F(L.dqkv), 3 * d, N, 3 * d, d));
    DC_TRY(attention_jvp_f32(F(L.qkv), F(L.dqkv), g, N, F(L.o), F(L.dout), s));
    DC_TRY(mm_gate(F(L.o), d, b.w_o, d, b.b_o, g1, F(L.h), N, d, d));
    DC_TRY(mm_gate(F(L.dout), d, b.w_o, d, zeros, g1, F(L.dh), N, d, d));
    DC_TRY(ln_mod_jvp(F(L.h), F(L.dh), N, d, d, sh2, sc2, F(L.a), F(L.da), g.eps, s));
    DC_TRY(mm(F(L.a), d, b.w_1, d, b.b_1, F(L.z), Fh, N, Fh, d));
    DC_TRY(mm(F(L.da), d, b.w_1, d, zeros, F(L.dz), Fh, N, Fh, d));
    DC_TRY(gelu_jvp(F(L.z), F(L.dz), size_t(N) * Fh, s));
    DC_TRY(mm_gate(F(L.z), Fh, b.w_2, Fh, b.b_2, g2, F(L.h), N, d, Fh));
    DC_TRY(mm_gate(F(L.dz), Fh, b.w_2, Fh, zeros, g2, F(L.dh), N, d, Fh));
    return Status::ok();
  }

  // dx += (sigma_{k+1} - sigma_k) J_k dx: the whole network at x_k in tangent mode
  Status step_jvp(int k, float* dx) {
    const float* mk = mod_k(k);
    const int d = g.d;
    DC_TRY(patch_embed(g, w, x_at(k), txt, F(L.h), one, blk(), L.blk_bytes, s));
    DC_TRY(patchify(dx, F(L.patches), g, s));              // text rows carry no tangent
    DC_TRY(gemm_f32_bias_act(F(L.patches), 64, w->w_pe, 64, F(L.zeros), F(L.dh), d, g.Nv, d, 64,
                             Act::kNone, s));
    if (g.Nt > 0)
      DC_HIP(hipMemsetAsync(F(L.dh) + size_t(g.Nv) * d, 0, size_t(g.Nt) * d * 4, s));
    for (int l = 0; l < g.L; ++l) DC_TRY(block_jvp(l, mk + size_t(l) * 6 * d));
    const float* hm = mk + size_t(g.L) * 6 * d;
    DC_TRY(ln_mod_jvp(F(L.h), F(L.dh), g.Nv, d, d, hm, hm + d, F(L.a), F(L.da), g.eps, s));
    if (g.bf16)
      return gemm_f32_head(F(L.da), d, static_cast<const uint16_t*>(w->w_head), F(L.zeros), dx, dsig(k), g,
                           g.Nv, s);
    return gemm_f32_head(F(L.da), d, static_cast<const float*>(w->w_head), F(L.zeros), dx, dsig(k), g,
                         g.Nv, s);
  }
};

}  // namespace

size_t calibrate_workspace_bytes(const Geo& g, int K) { return calib_layout(g, K).total; }

Status calibrate_tables(const Geo& g, const dc_model_weights* w, const float* x1, const float* txt,
                        const double* sigmas, int K, int h_max, double eps, double* q, double* dtab,
                        void* ws, size_t ws_bytes, hipStream_t s) {
  if (!w || !x1 || !sigmas || !q || !dtab || !ws || (g.Nt > 0 && !txt)) return Status::arg("NULL argument");
  if (g.Dh != 64) return Status::shape("calibration supports head_dim 64");
  if (K < 2 || h_max < 1) return Status::arg("calibration needs K >= 2 and h_max >= 1");
  if (!(eps >= 0.0)) return Status::arg("eps must be >= 0");
  if (!w->blocks || !w->w_head || !w->b_head || !w->w_pe) return Status::arg("weight pointer is NULL");
  for (int l = 0; l < g.L; ++l)
    if (!w->blocks[l].w_qkv || !w->blocks[l].w_o || !w->blocks[l].w_1 || !w->blocks[l].w_2 ||
        !w->blocks[l].b_qkv || !w->blocks[l].b_o || !w->blocks[l].b_1 || !w->blocks[l].b_2)
      return Status::arg("block weight pointer is NULL");
  const CalibLayout L = calib_layout(g, K);
  if (reinterpret_cast<uintptr_t>(ws) % 256) return Status::make(DC_ERR_WORKSPACE, "workspace must be 256-byte aligned");
  if (ws_bytes < L.total) return Status::make(DC_ERR_WORKSPACE, "calibration workspace too small");
  Calib c{g, w, txt, sigmas, K, ws, L, s, {}, size_t(g.C) * g.T * g.Hl * g.Wl, size_t(g.L + 1) * 6 * g.d};
  const int32_t zero = 0;
  DC_TRY(make_idx(&zero, 1, c.one));
  DC_HIP(hipMemsetAsync(c.F(L.zeros), 0, std::max(std::max(3 * size_t(g.d), size_t(g.F)), size_t(64)) * 4, s));
  DC_TRY(time_modulation(g, w, sigmas, K, c.F(L.mod), c.blk(), L.blk_bytes, s));
  DC_TRY(c.trace(x1));

  const size_t T = size_t(K - 1) * h_max;
  std::fill(q, q + T, 0.0);
  std::fill(dtab, dtab + T, 0.0);
  double nx[2];
  DC_TRY(c.norms(c.x_at(K + 1), nullptr, c.lat, nx));
  const double xn = std::sqrt(nx[1]);
  const size_t nu = size_t(g.Nv) * g.d;
  for (int j = 1; j < K; ++j) {
    DC_HIP(hipMemsetAsync(c.F(L.G), 0, c.lat * 4, s));
    for (int h = 1; h <= h_max && j + h <= K; ++h) {
      const int t = j + h;
      double du[2];
      DC_TRY(c.norms(c.u_at(t), c.u_at(j), nu, du));
      dtab[size_t(j - 1) * h_max + (h - 1)] = std::sqrt(du[0]) / (std::sqrt(du[1]) + eps);
      // Eq. 6, then the tail of Eq. 7
      DC_TRY(c.interface(t, c.r_at(j), c.F(L.v1)));
      DC_TRY(c.interface(t, c.r_at(t), c.F(L.v2)));
      DC_TRY(lincomb(c.F(L.e), c.F(L.v1), 1.0f, c.F(L.v2), -1.0f, c.lat, s));       // e = v1 - v2
      DC_TRY(lincomb(c.F(L.dx), c.F(L.e), c.dsig(t), nullptr, 0.0f, c.lat, s));     // its Euler step
      for (int k = t + 1; k <= K; ++k) DC_TRY(c.step_jvp(k, c.F(L.dx)));
      DC_TRY(lincomb(c.F(L.G), c.F(L.G), 1.0f, c.F(L.dx), 1.0f, c.lat, s));
      double gn[2];
      DC_TRY(c.norms(c.F(L.G), nullptr, c.lat, gn));
      q[size_t(j - 1) * h_max + (h - 1)] = std::sqrt(gn[1]) / (xn + eps);
    }
  }
  return Status::ok();
}

}  // namespace dc
