// Internal declarations shared by the library's host and device sources.
#pragma once

#include <cstdint>
#include <string>
#include <vector>

#include <hip/hip_runtime.h>

#include "../../include/dc.h"

namespace dc {

// ---------------------------------------------------------------------------
// status
// ---------------------------------------------------------------------------
struct Status {
  dc_status code = DC_OK;
  std::string msg;
  static Status ok() { return {}; }
  static Status make(dc_status c, std::string m) { Status s; s.code = c; s.msg = std::move(m); return s; }
  static Status arg(std::string m) { return make(DC_ERR_ARG, std::move(m)); }
  static Status shape(std::string m) { return make(DC_ERR_SHAPE, std::move(m)); }
  explicit operator bool() const { return code == DC_OK; }
};

Status hip_status(hipError_t e, const char* what);
#define DC_HIP(call)                                              \
  do {                                                            \
    hipError_t e_ = (call);                                       \
    if (e_ != hipSuccess) return ::dc::hip_status(e_, #call);     \
  } while (0)
#define DC_TRY(expr)                        \
  do {                                      \
    ::dc::Status s_ = (expr);               \
    if (!s_) return s_;                     \
  } while (0)

// ---------------------------------------------------------------------------
// host schedule (sched.cpp)
// ---------------------------------------------------------------------------
struct SceneTables {
  int K = 0, H = 0;
  double L = 0, Theta = 0, zL = 0, zTh = 0, D = 0;
  bool in_support = false;
  std::vector<int64_t> chat;   // [(K-1) * H], 2^-40 units
  std::vector<double> dbar;    // [(K-1) * H]
  int64_t cost(int j, int h) const { return chat[size_t(j - 1) * H + (h - 1)]; }
  double threshold(int j, int h) const { return dbar[size_t(j - 1) * H + (h - 1)]; }
};
Status validate_problem(const dc_sched_problem& p);
Status scene_tables(const dc_sched_problem& p, SceneTables& t);
Status schedule(const dc_sched_problem& p, const SceneTables& t, std::vector<uint8_t>& reuse,
                int32_t& n_reuse, int64_t& cost_q);
Status select_tau(const dc_sched_problem* probs, int n, double rho, int64_t& tau);
void motion_statistics(const double* xy, const double* yaw, int n_pose, double& L, double& Th);
Status select_anchors(const double* L, const double* Th, int n, double eps, int& i0, int& i1);

// ---------------------------------------------------------------------------
// model geometry
// ---------------------------------------------------------------------------
struct Geo {
  int L, d, H, Dh, F, C, T, Hl, Wl, p, Hp, Wp, Nv, Nt, N, P;
  bool bf16;
  float eps;
  size_t esz;            // bytes per element of the model dtype
};
Status make_geo(const dc_model_cfg* cfg, Geo& g);

// Kernel classes that can be timed (dc_profile_*); the numbering is part of the ABI.
enum class KClass { kAttention = 0, kGemmQKV, kGemmOut, kGemmUp, kGemmDown, kLnModulate,
                    kPatchEmbed, kDrift, kCacheStore, kCacheApply, kHead, kHeadReuse, kCount };

// RAII: brackets the launches made in its scope with events when the class is enabled.
class ProfScope {
 public:
  ProfScope(KClass c, hipStream_t s);
  ~ProfScope();
  ProfScope(const ProfScope&) = delete;
  ProfScope& operator=(const ProfScope&) = delete;

 private:
  int cls_;
  hipStream_t stream_;
  hipEvent_t start_ = nullptr;
};

// Selected samples of a batch, passed to kernels by value.
struct IdxList {
  int32_t n;
  int32_t v[DC_MAX_BATCH];
};
Status make_idx(const int32_t* idx, int32_t n, IdxList& out);

// Workspace layout (offsets in bytes, each 256-aligned).
struct Workspace {
  size_t a, qk, vt, o, ff, patch, drift_part, attn_part, attn_part_bytes, tm_e, tm_h, tm_c, tm_s, tm_m, total;
  int ldv;               // row stride of the transposed value buffer (tokens, padded)
  int kTmax;             // steps the modulation scratch can hold per pass
};
Workspace workspace_layout(const Geo& g, int batch);

constexpr int kDriftBlocks = 1024;  // fixed grid per sample: reproducible reductions

// ---------------------------------------------------------------------------
// kernel launchers (kernels_*.hip, gemm.hip, attention.hip)
// ---------------------------------------------------------------------------
enum class Act { kNone, kSilu };

// fp32 GEMM, C = A W^T (+ epilogue).  A [M, K] (lda), W [N, K] (ldw).
Status gemm_f32_bias_act(const float* A, int lda, const float* W, int ldw, const float* bias,
                         float* out, int ldo, int M, int N, int K, Act act, hipStream_t s);
Status gemm_f32_gate_residual(const float* A, int lda, const float* W, int ldw, const float* bias,
                              const float* gate, float* h, int ldh, int M, int N, int K,
                              hipStream_t s);
Status gemm_f32_gelu(const float* A, int lda, const float* W, int ldw, const float* bias,
                     float* out, int ldo, int M, int N, int K, hipStream_t s);
Status gemm_f32_patch_embed(const float* A, const float* W, const float* bias, const void* pos,
                            bool pos_bf16, float* out, int ldo, int M, int N, hipStream_t s);
Status gemm_f32_head(const float* A, int lda, const float* W, const float* bias, float* x,
                     float dsigma, const Geo& g, int M, hipStream_t s);
Status gemm_f32_qkv(const float* A, const float* W, const float* bias, float* qk, float* vt,
                    int ldv, const Geo& g, int M, hipStream_t s);
// the same fp32 SIMT GEMMs with bf16 weights (bits widened exactly on load): the tangent
// passes of the calibration on bf16 models
Status gemm_f32_bias_act(const float* A, int lda, const uint16_t* W, int ldw, const float* bias,
                         float* out, int ldo, int M, int N, int K, Act act, hipStream_t s);
Status gemm_f32_gate_residual(const float* A, int lda, const uint16_t* W, int ldw, const float* bias,
                              const float* gate, float* h, int ldh, int M, int N, int K,
                              hipStream_t s);
Status gemm_f32_head(const float* A, int lda, const uint16_t* W, const float* bias, float* x,
                     float dsigma, const Geo& g, int M, hipStream_t s);

// bf16 MFMA GEMM variants.
Status gemm_bf16_qkv(const uint16_t* A, const uint16_t* W, const float* bias, uint16_t* qk,
                     uint16_t* vt, int ldv, const Geo& g, int M, hipStream_t s);
Status gemm_bf16_gate_residual(const uint16_t* A, int lda, const uint16_t* W, const float* bias,
                               const float* gate, float* h, int ldh, int M, int N, int K,
                               hipStream_t s);
Status gemm_bf16_gelu(const uint16_t* A, int lda, const uint16_t* W, const float* bias,
                      uint16_t* out, int ldo, int M, int N, int K, hipStream_t s);
// bf16 model: fused patchify + patch embedding (+ bias + positional table) for one sample.
Status patch_embed_bf16(const float* x, const float* W, const float* bias, const uint16_t* pos,
                        float* out, const Geo& g, hipStream_t s);
Status gemm_bf16_head(const uint16_t* A, int lda, const uint16_t* W, const float* bias, float* x,
                      float dsigma, const Geo& g, int M, hipStream_t s);
// bf16 model: LN-modulation + head projection + unpatchify + Euler update of one sample's
// latent in one pass over its N_v video rows of g (head.hip); head_euler_fused_ok says
// whether the shape is supported (64 outputs, d % 32 == 0, 256 <= d <= 2048).  With
// resid != NULL the input is g = gin + resid (bf16), formed in registers (reuse steps).
bool head_euler_fused_ok(const Geo& g);
Status head_euler_bf16(const float* gin, const uint16_t* resid, const uint16_t* W, const float* bias,
                       const float* shift, const float* scale, float* x, float dsigma, const Geo& g,
                       hipStream_t s);

// Attention over one sample: qk [M, 2d] (Q | K), vt [heads][Dh][ldv], out [M, d].
// part: scratch for the split tail items (unnormalised partial outputs), part_bytes its size;
// with too little scratch the tail is not split.
Status attention_bf16(const uint16_t* qk, const uint16_t* vt, int ldv, uint16_t* out,
                      const Geo& g, int M, float* part, size_t part_bytes, hipStream_t s);
Status attention_f32(const float* qk, const float* vt, int ldv, float* out, const Geo& g, int M,
                     hipStream_t s);

// Elementwise / row kernels.
Status ln_modulate(const float* x, int rows, int ldx, const float* shift, const float* scale,
                   void* out, int ldo, bool out_bf16, const Geo& g, hipStream_t s);
Status cache_store(const float* h_out, const float* h_in, void* resid, const IdxList& idx,
                   const Geo& g, hipStream_t s);
Status cache_apply(const float* h_in, const void* resid, float* gout, const IdxList& idx,
                   const Geo& g, hipStream_t s);
Status drift(const float* h_in, const float* mod0, void* u_ref, bool snapshot, double* sums,
             const IdxList& idx, const Geo& g, double* part, hipStream_t s);
// drift() with the partial sums in the library's fixed per-GPU scratch array (no workspace)
Status drift_noalloc(const float* h_in, const float* mod0, void* u_ref, bool snapshot, double* sums,
                     const IdxList& idx, const Geo& g, hipStream_t s);
Status patchify(const float* x, float* patches, const Geo& g, hipStream_t s);

// Anchor calibration (Eq. 5-7): tangent-mode kernels of the fp32 network (calib.hip) and
// the driver (calib.cpp).  a = LN(x)(1+scale)+shift and da its tangent along dx, per row;
// o, dout = attention over qkv [M, 3d] and its tangent along dqkv; z, dz <- GELU(z) and
// its tangent; out = alpha x + beta y (y may be NULL); sumsq -> out2 = (sum (a-b)^2, sum a^2)
// (b may be NULL) in a fixed order, with sumsq_scratch_doubles() doubles of scratch.
Status ln_mod_jvp(const float* x, const float* dx, int rows, int ld, int d, const float* shift,
                  const float* scale, float* a, float* da, float eps, hipStream_t s);
Status attention_jvp_f32(const float* qkv, const float* dqkv, const Geo& g, int M, float* o,
                         float* dout, hipStream_t s);
Status gelu_jvp(float* z, float* dz, size_t n, hipStream_t s);
Status lincomb(float* out, const float* x, float alpha, const float* y, float beta, size_t n,
               hipStream_t s);
size_t sumsq_scratch_doubles();
Status sumsq(const float* a, const float* b, size_t n, double* scratch, double* out2, hipStream_t s);
size_t calibrate_workspace_bytes(const Geo& g, int K);
Status calibrate_tables(const Geo& g, const dc_model_weights* w, const float* x1, const float* txt,
                        const double* sigmas, int K, int h_max, double eps, double* q, double* dtab,
                        void* ws, size_t ws_bytes, hipStream_t s);
Status copy_text(const float* txt, float* h_in, const Geo& g, hipStream_t s);
Status copy_rows(const float* src, float* dst, size_t count, hipStream_t s);
Status time_features(const double* sig, int K, float* e, int n_freq, hipStream_t s);
Status silu_inplace(const float* in, float* out, size_t n, hipStream_t s);
Status assemble_modulation(const float* m, const float* c, const float* offset, int K, int L,
                           int l, const Geo& g, float* mod, int k0, hipStream_t s);

}  // namespace dc
