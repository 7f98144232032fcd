// Tangent-mode (forward-mode) kernels of the fp32 network, for the anchor calibration
// of the run tables (Sec. 3.1 after Eq. 4; Eq. 5-7).  The joint run response of Eq. 7
// moves an output perturbation through the frozen sampler tail with Jacobian-vector
// products of the whole network; the projections are linear, so their tangents are
// the same GEMMs without the bias, and only the nonlinear pieces need kernels here:
//   * LayerNorm with modulation: y = (x - mu) r, r = (var + eps)^-1/2,
//     dy = r (dxc - y mean(y dxc)), dxc = dx - mean(dx); a = y (1 + s) + sh, da = dy (1 + s);
//   * softmax attention per head, s = q.k c, ds = (dq.k + q.dk) c (c = 1/sqrt(d_h)):
//     o = sum_j P_j v_j, do = sum_j P_j (ds_j - sum_i P_i ds_i) v_j + P_j dv_j;
//   * GELU-tanh: g = z/2 (1 + tanh u), u = sqrt(2/pi)(z + 0.044715 z^3),
//     dg = (1/2 (1 + tanh u) + z/2 (1 - tanh^2 u) sqrt(2/pi)(1 + 3 0.044715 z^2)) dz.
// Plus a fixed-order sum-of-squares reduction (the L2 norms of Eq. 5 and Eq. 7) and a
// linear combination.  The calibration runs once per model configuration at small
// shapes, so these are plain SIMT kernels.
#include <hip/hip_runtime.h>

#include <cmath>

#include "internal.h"

namespace dc {

namespace {

constexpr int kRowThreads = 256;

__device__ inline double block_sum(double v, double* red) {
  const int t = threadIdx.x;
  red[t] = v;
  __syncthreads();
  for (int w = kRowThreads / 2; w >= 1; w >>= 1) {
    if (t < w) red[t] += red[t + w];
    __syncthreads();
  }
  const double r = red[0];
  __syncthreads();
  return r;
}

// one workgroup per row; the row statistics in double
__global__ void __launch_bounds__(kRowThreads) k_ln_mod_jvp(const float* __restrict__ x,
                                                            const float* __restrict__ dx, int ld,
                                                            int d, const float* __restrict__ shift,
                                                            const float* __restrict__ scale,
                                                            float* __restrict__ a,
                                                            float* __restrict__ da, float eps) {
  __shared__ double red[kRowThreads];
  const size_t base = size_t(blockIdx.x) * ld;
  const float* xr = x + base;
  const float* dr = dx + base;
  double s = 0.0, sd = 0.0;
  for (int c = threadIdx.x; c < d; c += kRowThreads) {
    s += xr[c];
    sd += dr[c];
  }
  const double mu = block_sum(s, red) / d;
  const double mud = block_sum(sd, red) / d;
  double q = 0.0;
  for (int c = threadIdx.x; c < d; c += kRowThreads) {
    const double xc = xr[c] - mu;
    q += xc * xc;
  }
  const double r = 1.0 / sqrt(block_sum(q, red) / d + double(eps));
  double yd = 0.0;
  for (int c = threadIdx.x; c < d; c += kRowThreads) yd += (xr[c] - mu) * r * (dr[c] - mud);
  const double m_ydxc = block_sum(yd, red) / d;
  for (int c = threadIdx.x; c < d; c += kRowThreads) {
    const double y = (xr[c] - mu) * r;
    const double dy = r * ((dr[c] - mud) - y * m_ydxc);
    const double f = 1.0 + double(scale[c]);
    a[base + c] = float(y * f + double(shift[c]));
    da[base + c] = float(dy * f);
  }
}

// one thread per (query, head, half of the head's dimensions): keys streamed through LDS
// in tiles of 32, the unnormalised sums rescaled online when the running maximum grows.
// qkv, dqkv: [M, 3d] (Q | K | V, head-major columns); o, dout: [M, d].
constexpr int kDh = 64, kHalf = 32, kKT = 32;
__global__ void __launch_bounds__(128) k_attn_jvp_f32(const float* __restrict__ qkv,
                                                      const float* __restrict__ dqkv, int M, int d,
                                                      float scale, float* __restrict__ o,
                                                      float* __restrict__ dout) {
  __shared__ float sK[kKT][kDh + 1], sdK[kKT][kDh + 1], sV[kKT][kDh + 1], sdV[kKT][kDh + 1];
  const int head = blockIdx.y;
  const int qi = threadIdx.x & 63, half = threadIdx.x >> 6;
  const int qrow = blockIdx.x * 64 + qi;
  const int ld = 3 * d;
  float qv[kDh], dq[kDh];
  for (int i = 0; i < kDh; ++i) {
    const size_t e = size_t(min(qrow, M - 1)) * ld + head * kDh + i;
    qv[i] = qkv[e];
    dq[i] = dqkv[e];
  }
  float A[kHalf], B[kHalf], Dv[kHalf];
  for (int i = 0; i < kHalf; ++i) A[i] = B[i] = Dv[i] = 0.f;
  float m = -INFINITY, l = 0.f, cs = 0.f;
  for (int k0 = 0; k0 < M; k0 += kKT) {
    for (int e = threadIdx.x; e < kKT * kDh; e += 128) {
      const int r = e / kDh, c = e % kDh;
      const int key = k0 + r;
      const bool ok = key < M;
      const size_t b = size_t(ok ? key : 0) * ld + head * kDh + c;
      sK[r][c] = ok ? qkv[b + d] : 0.f;
      sdK[r][c] = ok ? dqkv[b + d] : 0.f;
      sV[r][c] = ok ? qkv[b + 2 * d] : 0.f;
      sdV[r][c] = ok ? dqkv[b + 2 * d] : 0.f;
    }
    __syncthreads();
    const int n = min(kKT, M - k0);
    for (int j = 0; j < n; ++j) {
      float s = 0.f, ds = 0.f;
      for (int i = 0; i < kDh; ++i) {
        s += qv[i] * sK[j][i];
        ds += dq[i] * sK[j][i] + qv[i] * sdK[j][i];
      }
      s *= scale;
      ds *= scale;
      const float mn = fmaxf(m, s);
      const float al = expf(m - mn), p = expf(s - mn);
      l = l * al + p;
      cs = cs * al + p * ds;
      for (int i = 0; i < kHalf; ++i) {
        const int c = half * kHalf + i;
        B[i] = B[i] * al + p * sV[j][c];
        A[i] = A[i] * al + p * ds * sV[j][c];
        Dv[i] = Dv[i] * al + p * sdV[j][c];
      }
      m = mn;
    }
    __syncthreads();
  }
  if (qrow >= M) return;
  const float inv = 1.0f / l, c = cs * inv;
  for (int i = 0; i < kHalf; ++i) {
    const size_t e = size_t(qrow) * d + head * kDh + half * kHalf + i;
    o[e] = B[i] * inv;
    dout[e] = (A[i] - c * B[i] + Dv[i]) * inv;
  }
}

// z <- GELU_tanh(z), dz <- GELU_tanh'(z) dz
__global__ void k_gelu_jvp(float* __restrict__ z, float* __restrict__ dz, size_t n) {
  const float c = 0.7978845608028654f;
  for (size_t i = size_t(blockIdx.x) * blockDim.x + threadIdx.x; i < n; i += size_t(gridDim.x) * blockDim.x) {
    const float v = z[i];
    const float t = tanhf(c * (v + 0.044715f * v * v * v));
    const float g = 0.5f * v * (1.0f + t);
    const float dg = 0.5f * (1.0f + t) + 0.5f * v * (1.0f - t * t) * c * (1.0f + 3.0f * 0.044715f * v * v);
    z[i] = g;
    dz[i] *= dg;
  }
}

// out = alpha x + beta y (y may be NULL: out = alpha x)
__global__ void k_lincomb(float* __restrict__ out, const float* __restrict__ x, float alpha,
                          const float* __restrict__ y, float beta, size_t n) {
  for (size_t i = size_t(blockIdx.x) * blockDim.x + threadIdx.x; i < n; i += size_t(gridDim.x) * blockDim.x)
    out[i] = alpha * x[i] + (y ? beta * y[i] : 0.f);
}

// fixed-order partial sums: part[b] = (sum (a - b)^2, sum a^2) over block b's strided
// elements; k_sumsq_final adds the kSqBlocks partials in a fixed order
constexpr int kSqBlocks = 256;
__global__ void __launch_bounds__(kRowThreads) k_sumsq(const float* __restrict__ a,
                                                       const float* __restrict__ b, size_t n,
                                                       double* __restrict__ part) {
  __shared__ double red[kRowThreads];
  double s1 = 0.0, s2 = 0.0;
  for (size_t i = size_t(blockIdx.x) * kRowThreads + threadIdx.x; i < n; i += size_t(kSqBlocks) * kRowThreads) {
    const double av = a[i];
    const double dv = b ? av - double(b[i]) : av;
    s1 += dv * dv;
    s2 += av * av;
  }
  const double t1 = block_sum(s1, red);
  const double t2 = block_sum(s2, red);
  if (threadIdx.x == 0) {
    part[2 * blockIdx.x] = t1;
    part[2 * blockIdx.x + 1] = t2;
  }
}

__global__ void k_sumsq_final(const double* __restrict__ part, double* __restrict__ out) {
  if (threadIdx.x == 0) {
    double s1 = 0.0, s2 = 0.0;
    for (int i = 0; i < kSqBlocks; ++i) {
      s1 += part[2 * i];
      s2 += part[2 * i + 1];
    }
    out[0] = s1;
    out[1] = s2;
  }
}

inline unsigned grid_of(size_t n, unsigned cap) {
  const size_t g = (n + 255) / 256;
  return unsigned(g < 1 ? 1 : (g > cap ? cap : g));
}

}  // namespace

Status ln_mod_jvp(const float* x, const float* dx, int rows, int ld, int d, const float* shift,
                  const float* scale, float* a, float* da, float eps, hipStream_t s) {
  if (rows <= 0) return Status::ok();
  hipLaunchKernelGGL(k_ln_mod_jvp, dim3(rows), dim3(kRowThreads), 0, s, x, dx, ld, d, shift, scale, a,
                     da, eps);
  DC_HIP(hipGetLastError());
  return Status::ok();
}

Status attention_jvp_f32(const float* qkv, const float* dqkv, const Geo& g, int M, float* o,
                         float* dout, hipStream_t s) {
  if (g.Dh != kDh) return Status::shape("calibration attention tangent supports head_dim 64");
  const float scale = float(1.0 / std::sqrt(double(g.Dh)));
  hipLaunchKernelGGL(k_attn_jvp_f32, dim3((M + 63) / 64, g.H), dim3(128), 0, s, qkv, dqkv, M, g.d, scale,
                     o, dout);
  DC_HIP(hipGetLastError());
  return Status::ok();
}

Status gelu_jvp(float* z, float* dz, size_t n, hipStream_t s) {
  hipLaunchKernelGGL(k_gelu_jvp, dim3(grid_of(n, 4096)), dim3(256), 0, s, z, dz, n);
  DC_HIP(hipGetLastError());
  return Status::ok();
}

Status lincomb(float* out, const float* x, float alpha, const float* y, float beta, size_t n,
               hipStream_t s) {
  hipLaunchKernelGGL(k_lincomb, dim3(grid_of(n, 4096)), dim3(256), 0, s, out, x, alpha, y, beta, n);
  DC_HIP(hipGetLastError());
  return Status::ok();
}

size_t sumsq_scratch_doubles() { return 2 * kSqBlocks + 2; }

Status sumsq(const float* a, const float* b, size_t n, double* scratch, double* out2, hipStream_t s) {
  hipLaunchKernelGGL(k_sumsq, dim3(kSqBlocks), dim3(kRowThreads), 0, s, a, b, n, scratch);
  DC_HIP(hipGetLastError());
  hipLaunchKernelGGL(k_sumsq_final, dim3(1), dim3(64), 0, s, scratch, out2);
  DC_HIP(hipGetLastError());
  return Status::ok();
}

}  // namespace dc
