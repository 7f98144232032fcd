// Joint video + text self-attention, softmax(Q K^T / sqrt(d_h)) V per head, with
// an online softmax (flash-style: the N x N score matrix never leaves registers).
//
// bf16 path (gfx950 MFMA 32x32x16).  A workgroup is 4 waves x 32 query rows of one
// head; key/value tiles of 64 tokens are double-buffered in LDS.  Each wave
// computes the transposed scores S^T = K Q^T, so in the accumulator layout every
// lane holds scores of a single query row (lane % 32): the row max needs one
// cross-lane exchange (lanes l and l^32) and the rescale of the output is a
// per-lane multiply.  The output is accumulated transposed as well,
// O^T += V^T P^T, which needs V^T in LDS (the QKV GEMM writes V transposed).
// The K rows feeding the S^T tiles are permuted (bits 2 and 3 of the row index
// swapped) so that the eight scores a lane holds for each 16-token slice of P are
// eight consecutive tokens: P goes from the score registers straight into the
// B operand of the P V product, and V^T is read with one 16-byte LDS load.
#include <hip/hip_runtime.h>

#include <cmath>

#include "internal.h"

namespace dc {

namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));

__device__ inline uint16_t to_bf16(float f) {
  return __builtin_bit_cast(uint16_t, static_cast<__bf16>(f));
}

// LDS chunk swizzle for 128-byte tile rows.  gfx950's LDS serves 256 bytes per
// cycle (64 banks): two consecutive rows share a bank cycle, so the XOR key is
// row / 2, which gives the 16 rows that 16 consecutive lanes read (in any order,
// including the permuted K order) 16 distinct 16-byte bank groups.
__device__ inline int swz_k(int row) { return (row >> 1) & 7; }
__device__ inline int swz_v(int row) { return (row >> 1) & 7; }
__device__ inline int perm_kv(int m) { return (m & ~12) | ((m & 4) << 1) | ((m & 8) >> 1); }

constexpr float kSlack = 8.0f;   // lazy-rescale threshold of the running max (log2 units)

template <int D>
__global__ void __launch_bounds__(256) k_attn_bf16(const uint16_t* __restrict__ qk,
                                                   const uint16_t* __restrict__ vt, int ldv,
                                                   uint16_t* __restrict__ out, int M, int d,
                                                   float scale_log2) {
  constexpr int DK = (D + 15) / 16 * 16;   // contraction width of Q K^T (zero padded)
  constexpr int KC = DK / 8;               // 16-byte chunks per K row
  constexpr int DC8 = D / 8;               // chunks holding real data
  constexpr int DV = (D + 31) / 32 * 32;   // rows of the O^T accumulator
  constexpr int TV = DV / 32;
  constexpr int BKV = 64;
  constexpr int KLD = (BKV * DC8 + 255) / 256;   // K chunks per thread per tile
  constexpr int VLD = (D * 8 + 255) / 256;       // V^T chunks per thread per tile
  __shared__ uint4 sK[2][BKV * KC];
  __shared__ uint4 sV[2][DV * 8];

  const int head = blockIdx.y;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int g = lane >> 5, r32 = lane & 31;
  const int q0 = blockIdx.x * 128 + wave * 32;
  const int ldq = 2 * d;
  const uint16_t* Qb = qk + head * D;
  const uint16_t* Kb = qk + d + head * D;
  const uint16_t* Vb = vt + size_t(head) * D * ldv;
  const uint4 zero4 = make_uint4(0, 0, 0, 0);

  // zero the padding that loads never write: K chunks past D, V^T rows past D
  if constexpr (KC > DC8) {
    for (int e = tid; e < BKV * (KC - DC8); e += 256) {
      const int r = e / (KC - DC8), c = DC8 + e % (KC - DC8);
      sK[0][r * KC + c] = zero4;
      sK[1][r * KC + c] = zero4;
    }
  }
  for (int e = tid; e < (DV - D) * 8; e += 256) {
    sV[0][D * 8 + e] = zero4;
    sV[1][D * 8 + e] = zero4;
  }

  // query fragments (B operand of S^T): lane holds Q[q0 + r32][16 kk + 8 g .. + 8]
  bf16x8 qf[DK / 16];
#pragma unroll
  for (int kk = 0; kk < DK / 16; ++kk) {
    const int col = 16 * kk + 8 * g;
    const int q = q0 + r32;
    uint4 v = zero4;
    if (q < M && col < D) v = *reinterpret_cast<const uint4*>(Qb + size_t(q) * ldq + col);
    qf[kk] = __builtin_bit_cast(bf16x8, v);
  }

  uint4 rk[KLD], rv[VLD];
  auto gload = [&](int t) {
    const int kv0 = t * BKV;
#pragma unroll
    for (int i = 0; i < KLD; ++i) {
      const int e = tid + 256 * i;
      rk[i] = zero4;
      if (e < BKV * DC8) {
        const int r = e / DC8, c = e % DC8;
        if (kv0 + r < M) rk[i] = *reinterpret_cast<const uint4*>(Kb + size_t(kv0 + r) * ldq + 8 * c);
      }
    }
#pragma unroll
    for (int i = 0; i < VLD; ++i) {
      const int e = tid + 256 * i;
      rv[i] = zero4;
      if (e < D * 8) {
        const int r = e >> 3, c = e & 7;
        const int kv = kv0 + 8 * c;
        if (kv < M) {
          uint4 v = *reinterpret_cast<const uint4*>(Vb + size_t(r) * ldv + kv);
          if (kv + 8 > M) {   // ragged tail: zero the tokens past M
            uint16_t* h = reinterpret_cast<uint16_t*>(&v);
            for (int j = M - kv; j < 8; ++j) h[j] = 0;
          }
          rv[i] = v;
        }
      }
    }
  };
  auto sstore = [&](int buf) {
#pragma unroll
    for (int i = 0; i < KLD; ++i) {
      const int e = tid + 256 * i;
      if (e < BKV * DC8) {
        const int r = e / DC8, c = e % DC8;
        const int pc = (KC == 8) ? (c ^ swz_k(r)) : c;
        sK[buf][r * KC + pc] = rk[i];
      }
    }
#pragma unroll
    for (int i = 0; i < VLD; ++i) {
      const int e = tid + 256 * i;
      if (e < D * 8) {
        const int r = e >> 3, c = e & 7;
        sV[buf][r * 8 + (c ^ swz_v(r))] = rv[i];
      }
    }
  };

  f32x16 o[TV];
#pragma unroll
  for (int t = 0; t < TV; ++t)
#pragma unroll
    for (int i = 0; i < 16; ++i) o[t][i] = 0.f;
  float mrow = -INFINITY, lsum = 0.f;

  const int nkv = (M + BKV - 1) / BKV;
  gload(0);
  sstore(0);
  __syncthreads();
  for (int t = 0; t < nkv; ++t) {
    const int cur = t & 1;
    if (t + 1 < nkv) gload(t + 1);

    // S^T for two 32-token sub-tiles; sub-tile st, register i holds token
    // 32 st + 16 (i / 8) + 8 g + (i % 8) of the tile, query q0 + r32.
    f32x16 s[2];
#pragma unroll
    for (int st = 0; st < 2; ++st) {
#pragma unroll
      for (int i = 0; i < 16; ++i) s[st][i] = 0.f;
      const int row = 32 * st + perm_kv(r32);
#pragma unroll
      for (int kk = 0; kk < DK / 16; ++kk) {
        const int ch = 2 * kk + g;
        const int pc = (KC == 8) ? (ch ^ swz_k(row)) : ch;
        const bf16x8 kf = __builtin_bit_cast(bf16x8, sK[cur][row * KC + pc]);
        s[st] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf, qf[kk], s[st], 0, 0, 0);
      }
    }
    if ((t + 1) * BKV > M) {
#pragma unroll
      for (int st = 0; st < 2; ++st)
#pragma unroll
        for (int i = 0; i < 16; ++i) {
          const int kv = t * BKV + 32 * st + 16 * (i >> 3) + 8 * g + (i & 7);
          if (kv >= M) s[st][i] = -INFINITY;
        }
    }
    float mx = s[0][0];
#pragma unroll
    for (int st = 0; st < 2; ++st)
#pragma unroll
      for (int i = 0; i < 16; ++i) mx = fmaxf(mx, s[st][i]);
    mx = fmaxf(mx, __shfl_xor(mx, 32, 64)) * scale_log2;
    // Lazy rescale: keep the running max unless some row of the wave grows by
    // more than kSlack (log2 units); stale maxima only scale P and the row sum
    // by at most 2^kSlack, which fp32 accumulation absorbs.
    if (__builtin_amdgcn_ballot_w64(mx > mrow + kSlack) != 0) {
      const float mnew = fmaxf(mrow, mx);
      const float alpha = __builtin_amdgcn_exp2f(mrow - mnew);
      mrow = mnew;
      lsum *= alpha;
#pragma unroll
      for (int tv = 0; tv < TV; ++tv)
#pragma unroll
        for (int i = 0; i < 16; ++i) o[tv][i] *= alpha;
    }
    float ps = 0.f;
#pragma unroll
    for (int st = 0; st < 2; ++st)
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        const float pv = __builtin_amdgcn_exp2f(s[st][i] * scale_log2 - mrow);
        s[st][i] = pv;
        ps += pv;
      }
    lsum += ps;

    // O^T += V^T P^T over the four 16-token slices of the tile
#pragma unroll
    for (int c = 0; c < 4; ++c) {
      bf16x8 pf;
#pragma unroll
      for (int e = 0; e < 8; ++e) pf[e] = static_cast<__bf16>(s[c >> 1][8 * (c & 1) + e]);
      const int ch = 2 * c + g;
#pragma unroll
      for (int tv = 0; tv < TV; ++tv) {
        const int row = 32 * tv + r32;
        const bf16x8 vf = __builtin_bit_cast(bf16x8, sV[cur][row * 8 + (ch ^ swz_v(row))]);
        o[tv] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vf, pf, o[tv], 0, 0, 0);
      }
    }
    if (t + 1 < nkv) sstore(cur ^ 1);
    __syncthreads();
  }

  lsum += __shfl_xor(lsum, 32, 64);
  const float inv = 1.0f / lsum;
  const int q = q0 + r32;
  if (q < M) {
    uint16_t* orow = out + size_t(q) * d + head * D;
#pragma unroll
    for (int tv = 0; tv < TV; ++tv)
#pragma unroll
      for (int i4 = 0; i4 < 4; ++i4) {
        const int dh = 32 * tv + 8 * i4 + 4 * g;
        if (dh < D) {
          ushort4 u;
          u.x = to_bf16(o[tv][4 * i4 + 0] * inv);
          u.y = to_bf16(o[tv][4 * i4 + 1] * inv);
          u.z = to_bf16(o[tv][4 * i4 + 2] * inv);
          u.w = to_bf16(o[tv][4 * i4 + 3] * inv);
          *reinterpret_cast<ushort4*>(orow + dh) = u;
        }
      }
  }
}

// fp32 path: one thread per query row, key/value tiles of 64 tokens in LDS.
template <int D>
__global__ void __launch_bounds__(64) k_attn_f32(const float* __restrict__ qk,
                                                 const float* __restrict__ vt, int ldv,
                                                 float* __restrict__ out, int M, int d,
                                                 float scale) {
  __shared__ float sK[64][D + 1];
  __shared__ float sV[64][D + 1];
  const int head = blockIdx.y, tid = threadIdx.x;
  const int q = blockIdx.x * 64 + tid;
  const int ldq = 2 * d;
  float qv[D], o[D];
  for (int i = 0; i < D; ++i) {
    qv[i] = q < M ? qk[size_t(q) * ldq + head * D + i] : 0.f;
    o[i] = 0.f;
  }
  float m = -INFINITY, l = 0.f;
  for (int kv0 = 0; kv0 < M; kv0 += 64) {
    for (int e = tid; e < 64 * D; e += 64) {
      const int r = e / D, c = e % D;
      const int kv = kv0 + r;
      sK[r][c] = kv < M ? qk[size_t(kv) * ldq + d + head * D + c] : 0.f;
      const int r2 = e % 64, c2 = e / 64;
      sV[r2][c2] = (kv0 + r2) < M ? vt[size_t(head * D + c2) * ldv + kv0 + r2] : 0.f;
    }
    __syncthreads();
    const int n = min(64, M - kv0);
    for (int j = 0; j < n; ++j) {
      float sc = 0.f;
      for (int i = 0; i < D; ++i) sc += qv[i] * sK[j][i];
      sc *= scale;
      const float mn = fmaxf(m, sc);
      const float a = expf(m - mn), p = expf(sc - mn);
      l = l * a + p;
      for (int i = 0; i < D; ++i) o[i] = o[i] * a + p * sV[j][i];
      m = mn;
    }
    __syncthreads();
  }
  if (q < M)
    for (int i = 0; i < D; ++i) out[size_t(q) * d + head * D + i] = o[i] / l;
}

}  // namespace

Status attention_bf16(const uint16_t* qk, const uint16_t* vt, int ldv, uint16_t* out,
                      const Geo& g, int M, hipStream_t s) {
  const float scale_log2 = float(1.4426950408889634 / std::sqrt(double(g.Dh)));
  dim3 grid((M + 127) / 128, g.H);
  if (g.Dh == 64)
    hipLaunchKernelGGL(k_attn_bf16<64>, grid, dim3(256), 0, s, qk, vt, ldv, out, M, g.d, scale_log2);
  else if (g.Dh == 72)
    hipLaunchKernelGGL(k_attn_bf16<72>, grid, dim3(256), 0, s, qk, vt, ldv, out, M, g.d, scale_log2);
  else
    return Status::shape("bf16 attention supports head_dim 64 and 72");
  DC_HIP(hipGetLastError());
  return Status::ok();
}

Status attention_f32(const float* qk, const float* vt, int ldv, float* out, const Geo& g, int M,
                     hipStream_t s) {
  if (g.Dh != 64) return Status::shape("fp32 attention supports head_dim 64");
  const float scale = float(1.0 / std::sqrt(double(g.Dh)));
  dim3 grid((M + 63) / 64, g.H);
  hipLaunchKernelGGL(k_attn_f32<64>, grid, dim3(64), 0, s, qk, vt, ldv, out, M, g.d, scale);
  DC_HIP(hipGetLastError());
  return Status::ok();
}

}  // namespace dc
