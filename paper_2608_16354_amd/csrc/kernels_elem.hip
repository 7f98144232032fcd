// Row-wise and elementwise kernels of the denoising step: AdaLN modulation,
// residual cache store/apply, the drift reduction, patchify, and the timestep
// conditioning.  All HBM-bound; written for 64-lane wavefronts with 16-byte
// vector accesses.
#include <hip/hip_runtime.h>

#include <mutex>
#include <type_traits>
#include <vector>

#include "internal.h"

namespace dc {

namespace {

constexpr int kWave = 64;

__device__ inline float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, kWave);
  return v;
}

__device__ inline uint16_t to_bf16(float f) {
  __bf16 b = static_cast<__bf16>(f);   // round to nearest even (v_cvt_pk_bf16_f32)
  return __builtin_bit_cast(uint16_t, b);
}
__device__ inline float from_bf16(uint16_t u) { return __uint_as_float(uint32_t(u) << 16); }

// Branch-free row load for rows of n4 float4 with NV = ceil(n4 / 64) per lane: lanes
// past the row re-read its last float4 (in bounds) and are masked in the sums, so
// all NV loads issue back to back.
template <int NV>
__device__ inline void load_row_nv(const float* __restrict__ row, int n4, int lane, float4 (&v)[NV]) {
  const float4* r4 = reinterpret_cast<const float4*>(row);
#pragma unroll
  for (int i = 0; i < NV; ++i) v[i] = r4[min(lane + i * kWave, n4 - 1)];
}

template <int NV>
__device__ inline void row_stats_nv(const float4 (&v)[NV], int n4, int lane, float eps, float& mean,
                                    float& rstd) {
  float s = 0.f;
#pragma unroll
  for (int i = 0; i < NV; ++i)
    s += (lane + i * kWave < n4) ? (v[i].x + v[i].y) + (v[i].z + v[i].w) : 0.f;
  mean = wave_sum(s) / float(4 * n4);
  float q = 0.f;
#pragma unroll
  for (int i = 0; i < NV; ++i) {
    const float a = v[i].x - mean, b = v[i].y - mean, c = v[i].z - mean, e = v[i].w - mean;
    q += (lane + i * kWave < n4) ? (a * a + b * b) + (c * c + e * e) : 0.f;
  }
  const float var = wave_sum(q) / float(4 * n4);
  rstd = 1.0f / sqrtf(var + eps);
}

__device__ inline float4 modulate4(float4 x, float mean, float rstd, float4 sh, float4 sc) {
  float4 r;
  r.x = (x.x - mean) * rstd * (1.0f + sc.x) + sh.x;
  r.y = (x.y - mean) * rstd * (1.0f + sc.y) + sh.y;
  r.z = (x.z - mean) * rstd * (1.0f + sc.z) + sh.z;
  r.w = (x.w - mean) * rstd * (1.0f + sc.w) + sh.w;
  return r;
}

__device__ inline void store4(void* out, size_t e, float4 v, bool bf) {
  if (bf) {
    ushort4 u;
    u.x = to_bf16(v.x); u.y = to_bf16(v.y); u.z = to_bf16(v.z); u.w = to_bf16(v.w);
    *reinterpret_cast<ushort4*>(static_cast<uint16_t*>(out) + e) = u;
  } else {
    *reinterpret_cast<float4*>(static_cast<float*>(out) + e) = v;
  }
}

__device__ inline float4 load4(const void* in, size_t e, bool bf) {
  if (bf) {
    const ushort4 u = *reinterpret_cast<const ushort4*>(static_cast<const uint16_t*>(in) + e);
    return make_float4(from_bf16(u.x), from_bf16(u.y), from_bf16(u.z), from_bf16(u.w));
  }
  return *reinterpret_cast<const float4*>(static_cast<const float*>(in) + e);
}

// a = LN(x)(1 + scale) + shift, one wavefront per row (NV float4 per lane).  shift and
// scale go through LDS once per block of four rows, so the L1 and L2 see each row's data
// and not four more copies of the modulation vectors (-8 % at 17,776 x 1920).
template <int NV>
__global__ void __launch_bounds__(256) k_ln_modulate(const float* __restrict__ x, int rows, int ldx,
                                                     const float* __restrict__ shift,
                                                     const float* __restrict__ scale, void* out,
                                                     int ldo, int d, float eps, bool bf) {
  __shared__ float4 s_sh[NV * kWave], s_sc[NV * kWave];
  const int n4 = d >> 2;
  for (int i = threadIdx.x; i < n4; i += 256) {
    s_sh[i] = reinterpret_cast<const float4*>(shift)[i];
    s_sc[i] = reinterpret_cast<const float4*>(scale)[i];
  }
  const int lane = threadIdx.x & 63;
  const int row = blockIdx.x * 4 + (threadIdx.x >> 6);
  float4 v[NV];
  load_row_nv<NV>(x + size_t(min(row, rows - 1)) * ldx, n4, lane, v);
  __syncthreads();
  if (row >= rows) return;
  float mean, rstd;
  row_stats_nv<NV>(v, n4, lane, eps, mean, rstd);
#pragma unroll
  for (int i = 0; i < NV; ++i) {
    const int c = min(lane + i * kWave, n4 - 1);
    const float4 u = modulate4(v[i], mean, rstd, s_sh[c], s_sc[c]);
    if (lane + i * kWave < n4) store4(out, size_t(row) * ldo + 4 * c, u, bf);
  }
}

// resid = h_out - h_in on the video rows (contiguous N_v x d per sample).
__global__ void __launch_bounds__(256) k_cache_store(const float* __restrict__ h_out,
                                                     const float* __restrict__ h_in, void* resid,
                                                     IdxList idx, size_t per_sample4,
                                                     size_t stride_h, size_t stride_r, bool bf) {
  const int b = idx.v[blockIdx.y];
  const float4* ho = reinterpret_cast<const float4*>(h_out + size_t(b) * stride_h);
  const float4* hi = reinterpret_cast<const float4*>(h_in + size_t(b) * stride_h);
  const size_t base = size_t(b) * stride_r;
  for (size_t i = size_t(blockIdx.x) * blockDim.x + threadIdx.x; i < per_sample4;
       i += size_t(gridDim.x) * blockDim.x) {
    const float4 a = ho[i], c = hi[i];
    store4(resid, base + 4 * i, make_float4(a.x - c.x, a.y - c.y, a.z - c.z, a.w - c.w), bf);
  }
}

// g = h_in + resid on the video rows.
__global__ void __launch_bounds__(256) k_cache_apply(const float* __restrict__ h_in,
                                                     const void* resid, float* __restrict__ g,
                                                     IdxList idx, size_t per_sample4,
                                                     size_t stride_h, size_t stride_r, bool bf) {
  const int b = idx.v[blockIdx.y];
  const float4* hi = reinterpret_cast<const float4*>(h_in + size_t(b) * stride_h);
  float4* go = reinterpret_cast<float4*>(g + size_t(b) * stride_h);
  const size_t base = size_t(b) * stride_r;
  for (size_t i = size_t(blockIdx.x) * blockDim.x + threadIdx.x; i < per_sample4;
       i += size_t(gridDim.x) * blockDim.x) {
    const float4 a = hi[i], r = load4(resid, base + 4 * i, bf);
    go[i] = make_float4(a.x + r.x, a.y + r.y, a.z + r.z, a.w + r.w);
  }
}

// Drift: u = LN(h_in[:N_v])(1+scale)+shift; either snapshot u into u_ref, or
// accumulate (sum|u-u_ref|, sum|u|, sum(u-u_ref)^2, sum u^2).  One wavefront per
// row; the row of u_ref is fetched together with the row of h_in (it does not
// depend on the row statistics), so each row costs one memory round trip.
// Per-lane fp32 row partials -> wave shuffle reduction -> per-block f64 partial
// in a fixed order; k_drift_reduce adds the block partials in a fixed order.
// For a given N_v the result is bitwise reproducible.
template <bool BF, int NV>
__global__ void __launch_bounds__(256) k_drift(const float* __restrict__ h_in,
                                               const float* __restrict__ mod0, void* u_ref,
                                               int snapshot, IdxList idx, int Nv, int d,
                                               size_t stride_h,
                                               size_t stride_r, float eps,
                                               double* __restrict__ part) {
  typedef typename std::conditional<BF, uint2, float4>::type RV;   // 4 elements of u_ref
  const int b = idx.v[blockIdx.y];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const float* shift = mod0;
  const float* scale = mod0 + d;
  const float* hb = h_in + size_t(b) * stride_h;
  const size_t rbase = size_t(b) * stride_r;
  const int n4 = d >> 2;
  double acc[4] = {0.0, 0.0, 0.0, 0.0};
  for (int row = blockIdx.x * 4 + wave; row < Nv; row += gridDim.x * 4) {
    float4 v[NV];
    RV r[NV];
    load_row_nv<NV>(hb + size_t(row) * d, n4, lane, v);
    const RV* rrow = reinterpret_cast<const RV*>(static_cast<const char*>(u_ref) +
                                                 (rbase + size_t(row) * d) * (BF ? 2 : 4));
    if (!snapshot) {
#pragma unroll
      for (int i = 0; i < NV; ++i) r[i] = rrow[min(lane + i * kWave, n4 - 1)];
    }
    float mean, rstd;
    row_stats_nv<NV>(v, n4, lane, eps, mean, rstd);
    float s1 = 0.f, s2 = 0.f, s3 = 0.f, s4 = 0.f;
#pragma unroll
    for (int i = 0; i < NV; ++i) {
      const bool ok = lane + i * kWave < n4;
      const int c = min(lane + i * kWave, n4 - 1);
      const float4 sh = reinterpret_cast<const float4*>(shift)[c];
      const float4 sc = reinterpret_cast<const float4*>(scale)[c];
      const float4 u = modulate4(v[i], mean, rstd, sh, sc);
      if (snapshot) {
        if (ok) store4(u_ref, rbase + size_t(row) * d + 4 * c, u, BF);
      } else {
        float4 q;
        if constexpr (BF) {
          const uint2 w = r[i];
          q = make_float4(__uint_as_float(w.x << 16), __uint_as_float(w.x & 0xFFFF0000u),
                          __uint_as_float(w.y << 16), __uint_as_float(w.y & 0xFFFF0000u));
        } else {
          q = r[i];
        }
        const float dx = u.x - q.x, dy = u.y - q.y, dz = u.z - q.z, dw = u.w - q.w;
        s1 += ok ? (fabsf(dx) + fabsf(dy)) + (fabsf(dz) + fabsf(dw)) : 0.f;
        s2 += ok ? (fabsf(u.x) + fabsf(u.y)) + (fabsf(u.z) + fabsf(u.w)) : 0.f;
        s3 += ok ? (dx * dx + dy * dy) + (dz * dz + dw * dw) : 0.f;
        s4 += ok ? (u.x * u.x + u.y * u.y) + (u.z * u.z + u.w * u.w) : 0.f;
      }
    }
    if (!snapshot) {
      s1 = wave_sum(s1); s2 = wave_sum(s2); s3 = wave_sum(s3); s4 = wave_sum(s4);
      acc[0] += double(s1); acc[1] += double(s2); acc[2] += double(s3); acc[3] += double(s4);
    }
  }
  if (snapshot) return;
  __shared__ double wsum[4][4];
  if (lane == 0)
    for (int q = 0; q < 4; ++q) wsum[wave][q] = acc[q];
  __syncthreads();
  if (threadIdx.x < 4) {
    const int q = threadIdx.x;
    part[(size_t(blockIdx.y) * gridDim.x + blockIdx.x) * 4 + q] =
        ((wsum[0][q] + wsum[1][q]) + wsum[2][q]) + wsum[3][q];
  }
}

// Second pass of the drift reduction (one workgroup per sample): the nb block
// partials in a fixed order, 64 strided f64 chains per quantity, then a fixed
// tree.  The kernel boundary orders it after every partial.
__global__ void __launch_bounds__(256) k_drift_reduce(const double* __restrict__ part, int nb,
                                                      IdxList idx, double* __restrict__ sums) {
  __shared__ double red[64][4];
  const int q = threadIdx.x & 3, j = threadIdx.x >> 2;
  const double* pb = part + size_t(blockIdx.x) * nb * 4;
  double s = 0.0;
  for (int i = j; i < nb; i += 64) s += pb[4 * i + q];
  red[j][q] = s;
  __syncthreads();
  for (int w = 32; w >= 1; w >>= 1) {
    if (j < w) red[j][q] += red[j + w][q];
    __syncthreads();
  }
  if (threadIdx.x < 4) sums[size_t(idx.v[blockIdx.x]) * 4 + threadIdx.x] = red[0][threadIdx.x];
}

// patches[n, c p^2 + a p + b] = x[c, t, p i + a, p j + b], n = (t Hp + i) Wp + j.
__global__ void __launch_bounds__(256) k_patchify(const float* __restrict__ x,
                                                  float* __restrict__ patches, int C, int T,
                                                  int Hl, int Wl, int p, int Hp, int Wp, int Nv) {
  const int P = C * p * p;
  const size_t total = size_t(Nv) * P;
  for (size_t e = size_t(blockIdx.x) * blockDim.x + threadIdx.x; e < total;
       e += size_t(gridDim.x) * blockDim.x) {
    const int n = int(e / P), q = int(e % P);
    const int c = q / (p * p), a = (q / p) % p, bb = q % p;
    const int t = n / (Hp * Wp), i = (n / Wp) % Hp, j = n % Wp;
    patches[e] = x[((size_t(c) * T + t) * Hl + (p * i + a)) * Wl + (p * j + bb)];
  }
}

__global__ void k_copy4(const float4* __restrict__ src, float4* __restrict__ dst, size_t n4) {
  for (size_t i = size_t(blockIdx.x) * blockDim.x + threadIdx.x; i < n4;
       i += size_t(gridDim.x) * blockDim.x)
    dst[i] = src[i];
}

// e[k] = [cos(t w_i), sin(t w_i)], t = 1000 sigma_k, w_i = 10000^(-i/half); in double.
__global__ void k_time_features(const double* __restrict__ sig, int K, float* __restrict__ e,
                                int n_freq) {
  const int half = n_freq / 2;
  const int k = blockIdx.x;
  for (int i = threadIdx.x; i < half; i += blockDim.x) {
    const double w = exp(-double(i) / double(half) * log(10000.0));
    const double arg = 1000.0 * sig[k] * w;
    e[size_t(k) * n_freq + i] = float(cos(arg));
    e[size_t(k) * n_freq + half + i] = float(sin(arg));
  }
}

__global__ void k_silu(const float* __restrict__ in, float* __restrict__ out, size_t n) {
  for (size_t i = size_t(blockIdx.x) * blockDim.x + threadIdx.x; i < n;
       i += size_t(gridDim.x) * blockDim.x) {
    const float v = in[i];
    out[i] = v / (1.0f + expf(-v));
  }
}

// mod[k0+k, l] = m[k] (6 rows) + offset (block l < L); for l == L rows 0, 1 = offset + c[k].
__global__ void k_assemble(const float* __restrict__ m, const float* __restrict__ c,
                           const float* __restrict__ offset, int L, int l, int d,
                           float* __restrict__ mod, int k0) {
  const int k = blockIdx.y;
  float* dst = mod + (size_t(k0 + k) * (L + 1) + l) * 6 * d;
  for (int e = blockIdx.x * blockDim.x + threadIdx.x; e < 6 * d; e += gridDim.x * blockDim.x) {
    float v;
    if (l < L) {
      v = m[size_t(k) * 6 * d + e] + offset[e];
    } else {
      const int r = e / d;
      v = (r < 2) ? offset[e] + c[size_t(k) * d + (e % d)] : 0.0f;
    }
    dst[e] = v;
  }
}

inline int grid_for(size_t n, int per_block, int cap) {
  size_t b = (n + per_block - 1) / per_block;
  if (b > size_t(cap)) b = cap;
  return int(b < 1 ? 1 : b);
}

}  // namespace

#define DC_LAUNCH_CHECK() DC_HIP(hipGetLastError())

// Calls f(std::integral_constant<int, NV>) with NV = ceil(d / 256) float4 per lane.
template <class F>
Status with_nv(int d, F&& f) {
  switch ((d + 255) / 256) {
    case 1: f(std::integral_constant<int, 1>{}); break;
    case 2: f(std::integral_constant<int, 2>{}); break;
    case 3: f(std::integral_constant<int, 3>{}); break;
    case 4: f(std::integral_constant<int, 4>{}); break;
    case 5: f(std::integral_constant<int, 5>{}); break;
    case 6: f(std::integral_constant<int, 6>{}); break;
    case 7: f(std::integral_constant<int, 7>{}); break;
    case 8: f(std::integral_constant<int, 8>{}); break;
    case 9: f(std::integral_constant<int, 9>{}); break;
    case 10: f(std::integral_constant<int, 10>{}); break;
    case 11: f(std::integral_constant<int, 11>{}); break;
    case 12: f(std::integral_constant<int, 12>{}); break;
    default: return Status::shape("row kernels support hidden sizes up to 3072");
  }
  return Status::ok();
}

Status ln_modulate(const float* x, int rows, int ldx, const float* shift, const float* scale,
                   void* out, int ldo, bool out_bf16, const Geo& g, hipStream_t s) {
  if (rows <= 0) return Status::ok();
  DC_TRY(with_nv(g.d, [&](auto nv) {
    hipLaunchKernelGGL(k_ln_modulate<decltype(nv)::value>, dim3((rows + 3) / 4), dim3(256), 0, s, x,
                       rows, ldx, shift, scale, out, ldo, g.d, g.eps, out_bf16);
  }));
  DC_LAUNCH_CHECK();
  return Status::ok();
}

Status cache_store(const float* h_out, const float* h_in, void* resid, const IdxList& idx,
                   const Geo& g, hipStream_t s) {
  const size_t n4 = size_t(g.Nv) * g.d / 4;
  hipLaunchKernelGGL(k_cache_store, dim3(grid_for(n4, 256, 4096), idx.n), dim3(256), 0, s, h_out,
                     h_in, resid, idx, n4, size_t(g.N) * g.d, size_t(g.Nv) * g.d, g.bf16);
  DC_LAUNCH_CHECK();
  return Status::ok();
}

Status cache_apply(const float* h_in, const void* resid, float* gout, const IdxList& idx,
                   const Geo& g, hipStream_t s) {
  const size_t n4 = size_t(g.Nv) * g.d / 4;
  hipLaunchKernelGGL(k_cache_apply, dim3(grid_for(n4, 256, 4096), idx.n), dim3(256), 0, s, h_in,
                     resid, gout, idx, n4, size_t(g.N) * g.d, size_t(g.Nv) * g.d, g.bf16);
  DC_LAUNCH_CHECK();
  return Status::ok();
}

Status drift(const float* h_in, const float* mod0, void* u_ref, bool snapshot, double* sums,
             const IdxList& idx, const Geo& g, double* part, hipStream_t s) {
  const int nblk = std::min(kDriftBlocks, (g.Nv + 3) / 4);
  DC_TRY(with_nv(g.d, [&](auto nv) {
    constexpr int NV = decltype(nv)::value;
    if (g.bf16)
      hipLaunchKernelGGL((k_drift<true, NV>), dim3(nblk, idx.n), dim3(256), 0, s, h_in, mod0, u_ref,
                         snapshot ? 1 : 0, idx, g.Nv, g.d, size_t(g.N) * g.d, size_t(g.Nv) * g.d,
                         g.eps, part);
    else
      hipLaunchKernelGGL((k_drift<false, NV>), dim3(nblk, idx.n), dim3(256), 0, s, h_in, mod0, u_ref,
                         snapshot ? 1 : 0, idx, g.Nv, g.d, size_t(g.N) * g.d, size_t(g.Nv) * g.d,
                         g.eps, part);
  }));
  DC_LAUNCH_CHECK();
  if (!snapshot) {
    hipLaunchKernelGGL(k_drift_reduce, dim3(idx.n), dim3(256), 0, s, part, nblk, idx, sums);
    DC_LAUNCH_CHECK();
  }
  return Status::ok();
}

Status patchify(const float* x, float* patches, const Geo& g, hipStream_t s) {
  const size_t total = size_t(g.Nv) * g.P;
  hipLaunchKernelGGL(k_patchify, dim3(grid_for(total, 256, 8192)), dim3(256), 0, s, x, patches,
                     g.C, g.T, g.Hl, g.Wl, g.p, g.Hp, g.Wp, g.Nv);
  DC_LAUNCH_CHECK();
  return Status::ok();
}

Status copy_rows(const float* src, float* dst, size_t count, hipStream_t s) {
  if (count == 0) return Status::ok();
  const size_t n4 = count / 4;
  hipLaunchKernelGGL(k_copy4, dim3(grid_for(n4, 256, 4096)), dim3(256), 0, s,
                     reinterpret_cast<const float4*>(src), reinterpret_cast<float4*>(dst), n4);
  DC_LAUNCH_CHECK();
  return Status::ok();
}

Status copy_text(const float* txt, float* h_in, const Geo& g, hipStream_t s) {
  return copy_rows(txt, h_in + size_t(g.Nv) * g.d, size_t(g.Nt) * g.d, s);
}

Status time_features(const double* sig, int K, float* e, int n_freq, hipStream_t s) {
  hipLaunchKernelGGL(k_time_features, dim3(K), dim3(128), 0, s, sig, K, e, n_freq);
  DC_LAUNCH_CHECK();
  return Status::ok();
}

Status silu_inplace(const float* in, float* out, size_t n, hipStream_t s) {
  hipLaunchKernelGGL(k_silu, dim3(grid_for(n, 256, 1024)), dim3(256), 0, s, in, out, n);
  DC_LAUNCH_CHECK();
  return Status::ok();
}

Status assemble_modulation(const float* m, const float* c, const float* offset, int K, int L,
                           int l, const Geo& g, float* mod, int k0, hipStream_t s) {
  hipLaunchKernelGGL(k_assemble, dim3(grid_for(size_t(6) * g.d, 256, 64), K), dim3(256), 0, s, m,
                     c, offset, L, l, g.d, mod, k0);
  DC_LAUNCH_CHECK();
  return Status::ok();
}

// ---------------------------------------------------------------------------
// Drift without a workspace (for callers that cannot allocate): the per-block
// partial sums live in a fixed device array, one copy per GPU, held until the
// process ends.  Capacity: DC_MAX_BATCH samples x kDriftBlocks blocks x 4 sums
// (2 MiB); every partial the second pass reads is written by the same call, so
// nothing needs clearing.  Calls that overlap on one GPU share the array and race.
// ---------------------------------------------------------------------------
constexpr size_t kDriftScratchDoubles = size_t(DC_MAX_BATCH) * kDriftBlocks * 4;
static __device__ __align__(256) double scratch[kDriftScratchDoubles];

namespace {
// Device address of this GPU's copy of `scratch` (host code must not use the
// symbol's name as a pointer), looked up once per device with that device current.
Status scratch_address(double** out) {
  static std::mutex mu;
  static std::vector<double*> per_device;
  int dev = 0;
  DC_HIP(hipGetDevice(&dev));
  std::lock_guard<std::mutex> lock(mu);
  if (size_t(dev) >= per_device.size()) per_device.resize(size_t(dev) + 1, nullptr);
  if (!per_device[size_t(dev)]) {
    void* p = nullptr;
    DC_HIP(hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)));
    if (!p) return Status::make(DC_ERR_HIP, "hipGetSymbolAddress(scratch) returned NULL");
    per_device[size_t(dev)] = static_cast<double*>(p);
  }
  *out = per_device[size_t(dev)];
  return Status::ok();
}
}  // namespace

Status drift_noalloc(const float* h_in, const float* mod0, void* u_ref, bool snapshot, double* sums,
                     const IdxList& idx, const Geo& g, hipStream_t s) {
  const size_t nblk = size_t(std::min(kDriftBlocks, (g.Nv + 3) / 4));
  if (size_t(idx.n) * nblk * 4 > kDriftScratchDoubles)
    return Status::arg("dc_drift_l1_noalloc: more samples than its fixed scratch holds (" +
                       std::to_string(DC_MAX_BATCH) + ")");
  double* part = nullptr;
  DC_TRY(scratch_address(&part));
  return drift(h_in, mod0, u_ref, snapshot, sums, idx, g, part, s);
}

}  // namespace dc
