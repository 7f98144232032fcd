// Final layer + Euler update of the bf16 model in one pass over g (Eq. 1, H_k):
//
//   x += dsigma * unpatchify( (LN(g) (1 + scale) + shift) W_head^T + b_head )
//
// The LayerNorm is folded into the projection.  For one token with mean mu and
// rstd r, and any shift K,
//   sum_k (LN(g)_k (1 + s_k) + sh_k) W_nk
//     = r (sum_k y_k W_nk - (mu - K) cs_n) + shw_n,
//   y_k = (g_k - K)(1 + s_k),  cs_n = sum_k (1 + s_k) W_nk,  shw_n = sum_k sh_k W_nk,
// so g is read once: the matrix cores take y (split v = hi + lo into two bf16
// operands, about 2^-17 relative, against the bf16 weights) while the same pass
// accumulates the row moments of g - K.
//
// Layout: one persistent workgroup per compute unit takes a contiguous range of
// tokens, 16 at a time.  Its 8 waves split d into 32-wide chunks (at d = 1920 seven
// or eight each) and keep their chunks of W_head in registers for the whole kernel;
// a wave streams its part of the 16 token rows (64 contiguous bytes per row and
// instruction) four chunks ahead through a register ring, so about 64 KB per
// compute unit is in flight.  The shift K is the row's first value (a sample of the
// row, so y stays small next to g when the row mean is large); cs and shw are computed
// once per workgroup on the matrix cores.  Per token tile the waves leave their
// 16 x 64 partial products and moments of g - K in LDS; after one barrier every thread
// combines two outputs of one token, adds shw + b and applies the Euler update to the
// two latent values they land on.  LDS is double-buffered, so one barrier per tile.
//
// On a reuse step the head input is g = h_in + r (Eq. 1 with the cached r_j): the
// kResid variant reads h_in and the bf16 residual cache and forms g in registers with
// the same fp32 addition as the cache-apply kernel, so g never goes through HBM.
#include <hip/hip_runtime.h>

#include "internal.h"

namespace dc {

namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

struct HeadGeo { int T, Hl, Wl, p, Hp, Wp; };

constexpr int kWaves = 8;           // waves per workgroup
constexpr int kChunks = 8;          // 32-wide chunks of d per wave at most (d <= 2048)
constexpr int kRing = 4;            // chunks of g in flight per wave
constexpr int kLdr = 68;            // row stride (floats) of a wave's 16 x 64 partial tile

__device__ inline float4 ld4(const float* p) { return *reinterpret_cast<const float4*>(p); }

// latent element that output n of video token m lands on (unpatchify): channel
// c = n / p^2, pixel (p i + a, p j + b) of frame t, (a, b) = ((n / p) % p, n % p)
__device__ inline size_t latent_index(const HeadGeo& hg, int m, int n) {
  const int pp = hg.p * hg.p;
  const int c = n / pp, a = (n / hg.p) % hg.p, b = n % hg.p;
  const int t = m / (hg.Hp * hg.Wp), i = (m / hg.Wp) % hg.Hp, j = m % hg.Wp;
  return ((size_t(c) * hg.T + t) * hg.Hl + (hg.p * i + a)) * hg.Wl + (hg.p * j + b);
}

// chunk j of wave w: chunks [cb, cb + kc) of the nch chunks of d
__device__ inline int chunk_begin(int w, int nch) { return (w * nch) / kWaves; }

template <bool kResid>
__global__ void __launch_bounds__(512) k_head_euler_bf16(const float* __restrict__ gin,
                                                         const uint16_t* __restrict__ resid,
                                                         const uint16_t* __restrict__ W,
                                                         const float* __restrict__ bias,
                                                         const float* __restrict__ shift,
                                                         const float* __restrict__ scale,
                                                         float* __restrict__ x, float dsigma,
                                                         int Nv, int d, float eps, HeadGeo hg) {
  __shared__ float s_sc1[kChunks * kWaves * 32];          // 1 + scale
  __shared__ float2 s_st[2][kWaves][16];                  // per wave and row: sum, sum sq of g - K
  __shared__ float s_cs[kWaves][64];                      // cs and shw over each wave's chunks
  __shared__ float s_shw[kWaves][64];
  // Staging of W_head (each wave's 64 x 128 slab, 16 KB), then shift, then the per-wave
  // partial products of the token tiles: one region, used in that order.
  __shared__ __attribute__((aligned(16))) float s_big[kWaves * 4096];
  float(*s_acc)[kWaves][16 * kLdr] = reinterpret_cast<float(*)[kWaves][16 * kLdr]>(s_big);
  __bf16* s_ab = reinterpret_cast<__bf16*>(s_big);     // [4][d]: (1 + scale), shift as hi / lo
  static_assert(2 * kWaves * 16 * kLdr <= kWaves * 4096, "partial tiles fit the staging region");

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int c16 = lane & 15, g4 = lane >> 4;
  const int nch = d >> 5;
  const int cb = chunk_begin(wave, nch);
  const int kc = chunk_begin(wave + 1, nch) - cb;
  // this workgroup's tokens [r0, r1), balanced over the grid
  const int G = gridDim.x, bid = blockIdx.x;
  const int base = Nv / G, extra = Nv % G;
  const int r0 = bid * base + min(bid, extra);
  const int r1 = r0 + base + (bid < extra ? 1 : 0);
  const int ntile = (r1 - r0 + 15) >> 4;

  // g ring: slot q holds the chunks j with j % 4 == q of a token tile.  The first tile's
  // loads go out first: their latency overlaps the staging of W below.
  // (Rows past the range, tiles past the last and chunks past kc are clamped: they
  // re-read lines already fetched, and every load stays unconditional, so the
  // compiler's wait counts do not fall back to waiting for everything at branch joins.)
  float4 ga[kRing][2];
  uint2 gr[kRing][2];                           // residual (bf16) of the same elements
  auto load_chunk = [&](int t, int j, float4 (&dst)[2], uint2 (&rdst)[2]) {
    const int m = min(r0 + 16 * min(t, ntile - 1) + c16, r1 - 1);
    const size_t e = size_t(m) * d + 32 * (cb + min(j, kc - 1)) + 4 * g4;
    dst[0] = ld4(gin + e);
    dst[1] = ld4(gin + e + 16);
    if constexpr (kResid) {
      rdst[0] = *reinterpret_cast<const uint2*>(resid + e);
      rdst[1] = *reinterpret_cast<const uint2*>(resid + e + 16);
    }
  };
  auto load_k = [&](int t) {
    const size_t e = size_t(min(r0 + 16 * min(t, ntile - 1) + c16, r1 - 1)) * d;
    if constexpr (kResid) return gin[e] + __uint_as_float(uint32_t(resid[e]) << 16);
    return gin[e];
  };
  float kcur = load_k(0), knext = 0.f;
#pragma unroll
  for (int q = 0; q < kRing; ++q) load_chunk(0, q, ga[q], gr[q]);
  // scale and shift (k = tid + 512 i), written to LDS once the slabs are done
  float scv[kChunks * kWaves * 32 / 512], shv[kChunks * kWaves * 32 / 512];
#pragma unroll
  for (int i = 0; i < kChunks * kWaves * 32 / 512; ++i) {
    const int k = min(tid + 512 * i, d - 1);
    scv[i] = scale[k];
    shv[i] = shift[k];
  }

  // W_head fragments (B operand: column n = 16 nb + c16).  Within a chunk the k order
  // is permuted the same way for both operands: slot e of lane group g4 holds
  // k = 4 g4 + e (e < 4) or 16 + 4 g4 + e - 4 (e >= 4), so a lane's 8 values of g
  // are two 16-byte runs.  The wave's columns of W go through its own LDS slab four
  // chunks at a time (64 rows x 256 bytes; each load instruction reads 4 rows x 256
  // contiguous bytes), the 16-byte pieces of a row XOR-swizzled by the row.  Slots
  // j >= kc (unused) repeat chunk kc - 1.
  bf16x8 wf[kChunks][4];
  {
    uint4* slab = reinterpret_cast<uint4*>(s_big) + wave * 1024;
    uint4 v[kChunks / 4][16];                   // both rounds' loads go out together
#pragma unroll
    for (int h = 0; h < kChunks / 4; ++h)
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        const int pz = 64 * i + lane, row = pz >> 4, pc = pz & 15;
        const int c = cb + min(4 * h + (pc >> 2), kc - 1);
        v[h][i] = *reinterpret_cast<const uint4*>(W + size_t(row) * d + 32 * c + 8 * (pc & 3));
      }
#pragma unroll
    for (int h = 0; h < kChunks / 4; ++h) {
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        const int pz = 64 * i + lane, row = pz >> 4, pc = pz & 15;
        slab[row * 16 + (pc ^ (row & 15))] = v[h][i];
      }
#pragma unroll
      for (int jj = 0; jj < 4; ++jj)
#pragma unroll
        for (int nb = 0; nb < 4; ++nb) {
          const int row = 16 * nb + c16;
          const int p0 = 4 * jj + (g4 >> 1), p1 = p0 + 2;        // pieces of k 4 g4 and 16 + 4 g4
          const uint2* r = reinterpret_cast<const uint2*>(slab + row * 16);
          const uint2 a = r[2 * (p0 ^ c16) + (g4 & 1)];
          const uint2 b = r[2 * (p1 ^ c16) + (g4 & 1)];
          wf[4 * h + jj][nb] = __builtin_bit_cast(bf16x8, make_uint4(a.x, a.y, b.x, b.y));
        }
    }
  }
  asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
  __builtin_amdgcn_s_barrier();                 // every slab is read: the region takes
  asm volatile("" ::: "memory");                // (1 + scale) and shift split to bf16 hi / lo
#pragma unroll
  for (int i = 0; i < kChunks * kWaves * 32 / 512; ++i) {
    const int k = tid + 512 * i;
    if (k < d) {
      const float f = 1.0f + scv[i];
      s_sc1[k] = f;
      const __bf16 fh = static_cast<__bf16>(f), sh = static_cast<__bf16>(shv[i]);
      s_ab[k] = fh;
      s_ab[d + k] = static_cast<__bf16>(f - static_cast<float>(fh));
      s_ab[2 * d + k] = sh;
      s_ab[3 * d + k] = static_cast<__bf16>(shv[i] - static_cast<float>(sh));
    }
  }
  asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");

  // cs_w and shw_w on the matrix cores: A rows 0 / 1 = (1 + scale) hi / lo, rows 2 / 3
  // = shift hi / lo, the other rows zero.  Rows 0..3 of the result are registers 0..3
  // of lanes 0..15.
  {
    f32x4 pc[4];
#pragma unroll
    for (int nb = 0; nb < 4; ++nb) pc[nb] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int j = 0; j < kChunks; ++j) {
      if (j < kc) {
        const __bf16* src = s_ab + min(c16, 3) * d + 32 * (cb + j) + 4 * g4;
        uint2 a = *reinterpret_cast<const uint2*>(src);
        uint2 b = *reinterpret_cast<const uint2*>(src + 16);
        if (c16 >= 4) a = b = make_uint2(0, 0);
        const bf16x8 af = __builtin_bit_cast(bf16x8, make_uint4(a.x, a.y, b.x, b.y));
#pragma unroll
        for (int nb = 0; nb < 4; ++nb)
          pc[nb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(af, wf[j][nb], pc[nb], 0, 0, 0);
      }
    }
    if (g4 == 0)
#pragma unroll
      for (int nb = 0; nb < 4; ++nb) {
        s_cs[wave][16 * nb + c16] = pc[nb][0] + pc[nb][1];
        s_shw[wave][16 * nb + c16] = pc[nb][2] + pc[nb][3];
      }
  }

  // epilogue role of this thread: token er of a tile, outputs n = 2 eq and 2 eq + 1
  const int er = tid & 15, eq = tid >> 4;
  asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
  float shw[2], cs[2];
#pragma unroll
  for (int u = 0; u < 2; ++u) {
    float v = bias[2 * eq + u], c = 0.f;
#pragma unroll
    for (int w = 0; w < kWaves; ++w) {
      v += s_shw[w][2 * eq + u];
      c += s_cs[w][2 * eq + u];
    }
    shw[u] = v;
    cs[u] = c;
  }
  const float inv_d = 1.0f / float(d);

  for (int t = 0; t < ntile; ++t) {
    const int buf = t & 1;
    // the two latent values this thread updates after the tile, loaded now
    const int em = r0 + 16 * t + er;
    const bool eok = em < r1;
    const int emc = min(em, r1 - 1);
    float xv[2];
    xv[0] = x[latent_index(hg, emc, 2 * eq)];
    xv[1] = x[latent_index(hg, emc, 2 * eq + 1)];

    f32x4 acc[4];
#pragma unroll
    for (int nb = 0; nb < 4; ++nb) acc[nb] = f32x4{0.f, 0.f, 0.f, 0.f};
    float s1 = 0.f, s2 = 0.f;
#pragma unroll
    for (int j = 0; j < kChunks; ++j) {
      if (j < kc) {
        const float4* v = ga[j % kRing];
        float e[8] = {v[0].x, v[0].y, v[0].z, v[0].w, v[1].x, v[1].y, v[1].z, v[1].w};
        if constexpr (kResid) {                 // g = h_in + r, the cache-apply addition
          const uint2* r = gr[j % kRing];
          const uint32_t rw[4] = {r[0].x, r[0].y, r[1].x, r[1].y};
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            e[2 * i] += __uint_as_float(rw[i] << 16);
            e[2 * i + 1] += __uint_as_float(rw[i] & 0xFFFF0000u);
          }
        }
        const int k0 = 32 * (cb + j) + 4 * g4;
        const float4 sa = *reinterpret_cast<const float4*>(s_sc1 + k0);
        const float4 sb = *reinterpret_cast<const float4*>(s_sc1 + k0 + 16);
        const float sc[8] = {sa.x, sa.y, sa.z, sa.w, sb.x, sb.y, sb.z, sb.w};
        bf16x8 ah, al;
#pragma unroll
        for (int i = 0; i < 8; ++i) {
          const float u = e[i] - kcur;
          s1 += u;
          s2 = fmaf(u, u, s2);
          const float y = u * sc[i];
          const __bf16 h = static_cast<__bf16>(y);
          ah[i] = h;
          al[i] = static_cast<__bf16>(y - static_cast<float>(h));
        }
#pragma unroll
        for (int nb = 0; nb < 4; ++nb) {
          acc[nb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ah, wf[j][nb], acc[nb], 0, 0, 0);
          acc[nb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(al, wf[j][nb], acc[nb], 0, 0, 0);
        }
      }
      // refill this slot with the chunk four ahead in the 8-chunk order of the tiles
      if (j + kRing < kChunks) {
        load_chunk(t, j + kRing, ga[j % kRing], gr[j % kRing]);
      } else {
        if (j == kChunks - kRing) knext = load_k(t + 1);
        load_chunk(t + 1, j + kRing - kChunks, ga[j % kRing], gr[j % kRing]);
      }
    }

    // this wave's moments of each row (the row's four lane groups) and partial products
    s1 += __shfl_xor(s1, 16, 64);
    s1 += __shfl_xor(s1, 32, 64);
    s2 += __shfl_xor(s2, 16, 64);
    s2 += __shfl_xor(s2, 32, 64);
    if (g4 == 0) s_st[buf][wave][c16] = make_float2(s1, s2);
    kcur = knext;
    float* pa = s_acc[buf][wave];
#pragma unroll
    for (int nb = 0; nb < 4; ++nb)
#pragma unroll
      for (int i = 0; i < 4; ++i) pa[(4 * g4 + i) * kLdr + 16 * nb + c16] = acc[nb][i];
    asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
    __builtin_amdgcn_s_barrier();
    asm volatile("" ::: "memory");

    // combine: mean - K and variance of the token, then
    // r (sum_w acc_w - (mu - K) cs) + shw + b
    float t1 = 0.f, t2 = 0.f, o0 = 0.f, o1 = 0.f;
#pragma unroll
    for (int w = 0; w < kWaves; ++w) {
      const float2 st = s_st[buf][w][er];
      const float2 a = *reinterpret_cast<const float2*>(&s_acc[buf][w][er * kLdr + 2 * eq]);
      t1 += st.x;
      t2 += st.y;
      o0 += a.x;
      o1 += a.y;
    }
    const float dm = t1 * inv_d;                               // mu - K
    const float var = fmaxf(t2 * inv_d - dm * dm, 0.f);
    const float rs = 1.0f / sqrtf(var + eps);
    if (eok) {
      x[latent_index(hg, em, 2 * eq)] = xv[0] + dsigma * (rs * (o0 - dm * cs[0]) + shw[0]);
      x[latent_index(hg, em, 2 * eq + 1)] = xv[1] + dsigma * (rs * (o1 - dm * cs[1]) + shw[1]);
    }
  }
}

int head_grid(int Nv) {
  static int cus[64] = {0};
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 0;
  if (cus[dev] == 0 &&
      hipDeviceGetAttribute(&cus[dev], hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess)
    return 0;
  const int tiles = (Nv + 15) / 16;
  return cus[dev] < tiles ? cus[dev] : tiles;
}

}  // namespace

bool head_euler_fused_ok(const Geo& g) {
  return g.bf16 && g.P == 64 && g.d % 32 == 0 && g.d >= 32 * kWaves && g.d <= 32 * kWaves * kChunks;
}

Status head_euler_bf16(const float* gin, const uint16_t* resid, const uint16_t* W, const float* bias,
                       const float* shift, const float* scale, float* x, float dsigma, const Geo& g,
                       hipStream_t s) {
  if (g.Nv <= 0) return Status::ok();
  if (!head_euler_fused_ok(g)) return Status::shape("fused bf16 head needs 64 outputs, d % 32 == 0 and 256 <= d <= 2048");
  const int grid = head_grid(g.Nv);
  if (grid <= 0) return Status::make(DC_ERR_HIP, "fused bf16 head: no device");
  const HeadGeo hg{g.T, g.Hl, g.Wl, g.p, g.Hp, g.Wp};
  if (resid)
    hipLaunchKernelGGL(k_head_euler_bf16<true>, dim3(grid), dim3(512), 0, s, gin, resid, W, bias, shift,
                       scale, x, dsigma, g.Nv, g.d, g.eps, hg);
  else
    hipLaunchKernelGGL(k_head_euler_bf16<false>, dim3(grid), dim3(512), 0, s, gin, resid, W, bias, shift,
                       scale, x, dsigma, g.Nv, g.d, g.eps, hg);
  DC_HIP(hipGetLastError());
  return Status::ok();
}

}  // namespace dc
