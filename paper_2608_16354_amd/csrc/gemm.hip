// GEMMs of the denoising step: C = A W^T with fused epilogues.
//
// bf16 block GEMMs (QKV, out-projection, MLP up / down): v_mfma_f32_32x32x16_bf16,
// 8 waves, block tile 384 x 192 x 64 (QKV, out-projection, MLP down: fewer operand
// lines per FLOP, the L1 miss queue being the limit) or 320 x 256 x 64 (MLP up: still
// fewer lines per FLOP, and its 30 column tiles quantise well over the rounds), tiles
// fed global -> LDS by LDS-DMA into two
// stages (the refill of the next k-step interleaved with this k-step's MFMAs),
// XOR-swizzled 128-byte rows, one barrier per k-step, XCD-aware tile order;
// epilogues take one accumulator column at a time.
// bf16 head + Euler for models wider than the one-pass head kernel takes (d > 2048):
// the same LDS-DMA GEMM with a 64 x 64 tile (N = 64 outputs) and the unpatchify +
// Euler epilogue, after LN-modulation to bf16 rows.
// bf16 patch embedding: fp32-accurate split-bf16 MFMA with the patchify gather fused.
// f32 path: a plain SIMT tiled kernel for the fp32 model and the small fp32
// GEMMs (patch embedding of the fp32 model, timestep MLP).
#include <hip/hip_runtime.h>

#include <cmath>

#include "internal.h"

namespace dc {

namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
typedef float f32x4n __attribute__((ext_vector_type(4)));

// 16-byte streaming stores for the block GEMM epilogues: every CU finishes its tile at
// about the same time, and the output (not reused by the GEMM) then does not displace
// the operand lines the next tiles read from L2 (-1 to -4 % per GEMM on MI355X)
__device__ inline void store_nt(void* p, uint4 v) {
  __builtin_nontemporal_store(__builtin_bit_cast(u32x4, v), reinterpret_cast<u32x4*>(p));
}
__device__ inline void store_nt(float* p, float4 v) {
  __builtin_nontemporal_store(__builtin_bit_cast(f32x4n, v), reinterpret_cast<f32x4n*>(p));
}
typedef float f32x16 __attribute__((ext_vector_type(16)));

__device__ inline uint16_t to_bf16(float f) {
  return __builtin_bit_cast(uint16_t, static_cast<__bf16>(f));
}
__device__ inline float from_bf16(uint16_t u) { return __uint_as_float(uint32_t(u) << 16); }
inline bool al16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15) == 0; }

// LDS chunk swizzle for 128-byte tile rows.  gfx950's LDS serves 256 bytes per
// cycle (64 banks), so two consecutive 128-byte rows share a bank cycle: keying
// the XOR on row / 2 makes the 16 rows read by 16 consecutive lanes hit 16
// distinct 16-byte bank groups.
__device__ inline int swz(int row) { return (row >> 1) & 7; }

// GELU with the tanh approximation, written as z * sigmoid(2y), y = sqrt(2/pi)(z + 0.044715 z^3)
// (0.5 (1 + tanh y) = 1 / (1 + exp(-2y))).
__device__ inline float gelu_tanh(float z) {
  const float y = 0.7978845608028654f * (z + 0.044715f * z * z * z);
  return z / (1.0f + __expf(-2.0f * y));
}
// the same with v_rcp_f32 (1 ulp) in place of the IEEE division, for bf16 outputs
__device__ inline float gelu_tanh_fast(float z) {
  const float y = 0.7978845608028654f * (z + 0.044715f * z * z * z);
  return z * __builtin_amdgcn_rcpf(1.0f + __expf(-2.0f * y));
}
__device__ inline float silu(float z) { return z / (1.0f + expf(-z)); }

// ---------------------------------------------------------------------------
// epilogues: operator()(m, n, acc) for one output element
// ---------------------------------------------------------------------------
// The MFMA GEMM hands its epilogue either one accumulator column at a time: col(mb,
// n, M, v) gets v[i] = C[mb + 8 (i / 4) + i % 4][n] for i < 16 (mb a multiple of 4),
// or, when the epilogue declares kRowVec = V > 0, V consecutive columns of NP rows:
// rows<NP>(m0, dm, n, M, v) gets v[k][j] = C[m0 + k dm][n + j] (n a multiple of V), so
// it can issue all of its loads before any store; the GEMM transposes
// each 32 x 32 accumulator tile through LDS for that, so the stores are 16 bytes
// per lane instead of one element.  isrow(n) says whether the 32-column tile that
// starts at n goes the row way (otherwise col).
// Q (columns < d) leaves pre-multiplied by qscale = log2(e)/sqrt(d_h): the bf16
// attention kernel takes its scores in log2 units.
struct EpiQKVBf16 {
  const float* bias; uint16_t* qk; uint16_t* vt; int d; int ldv; float qscale;
  static constexpr int kRowVec = 8;
  __device__ bool isrow(int n) const { return n < 2 * d; }    // Q and K rows; V^T by column
  bool rows_aligned() const { return al16(qk) && al16(bias) && d % 4 == 0; }
  template <int NP>
  __device__ void rows(int m0, int dm, int n, int M, const float (&v)[NP][8]) const {
    const float4 b0 = *reinterpret_cast<const float4*>(bias + n);
    const float4 b1 = *reinterpret_cast<const float4*>(bias + n + 4);
    const float sc = n < d ? qscale : 1.0f;
#pragma unroll
    for (int k = 0; k < NP; ++k) {
      uint4 pk;
      pk.x = uint32_t(to_bf16((v[k][0] + b0.x) * sc)) | (uint32_t(to_bf16((v[k][1] + b0.y) * sc)) << 16);
      pk.y = uint32_t(to_bf16((v[k][2] + b0.z) * sc)) | (uint32_t(to_bf16((v[k][3] + b0.w) * sc)) << 16);
      pk.z = uint32_t(to_bf16((v[k][4] + b1.x) * sc)) | (uint32_t(to_bf16((v[k][5] + b1.y) * sc)) << 16);
      pk.w = uint32_t(to_bf16((v[k][6] + b1.z) * sc)) | (uint32_t(to_bf16((v[k][7] + b1.w) * sc)) << 16);
      if (m0 + k * dm < M) store_nt(qk + size_t(m0 + k * dm) * 2 * d + n, pk);
    }
  }
  __device__ void col(int mb, int n, int M, const f32x16& v) const {
    const float b = bias[n];
    if (n < 2 * d) {
      const float sc = n < d ? qscale : 1.0f;
      uint16_t* __restrict__ q = qk + size_t(mb) * 2 * d + n;
      if (mb + 28 <= M) {                     // all 16 rows present: no per-row guards
#pragma unroll
        for (int i = 0; i < 16; ++i) q[size_t(8 * (i >> 2) + (i & 3)) * 2 * d] = to_bf16((v[i] + b) * sc);
      } else {
#pragma unroll
        for (int i = 0; i < 16; ++i)
          if (mb + 8 * (i >> 2) + (i & 3) < M) q[size_t(8 * (i >> 2) + (i & 3)) * 2 * d] = to_bf16((v[i] + b) * sc);
      }
    } else {
      // V^T row n - 2d: four consecutive tokens per 8-byte store (ldv and mb are multiples of 4).
      // The padding tokens [M, ldv) get zeros: the attention's last value tile reads them
      // (and multiplies them by zero probabilities, which NaN garbage would turn into NaN).
      // The last row tile always reaches ldv (tile heights are multiples of 64).
      uint16_t* __restrict__ r = vt + size_t(n - 2 * d) * ldv + mb;
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        uint2 pk;
        pk.x = uint32_t(to_bf16(v[4 * g] + b)) | (uint32_t(to_bf16(v[4 * g + 1] + b)) << 16);
        pk.y = uint32_t(to_bf16(v[4 * g + 2] + b)) | (uint32_t(to_bf16(v[4 * g + 3] + b)) << 16);
        if (mb + 8 * g + 3 < M) {
          *reinterpret_cast<uint2*>(r + 8 * g) = pk;
        } else {
#pragma unroll
          for (int j = 0; j < 4; ++j) {
            const int m = mb + 8 * g + j;
            if (m < M) r[8 * g + j] = to_bf16(v[4 * g + j] + b);
            else if (m < ldv) r[8 * g + j] = 0;
          }
        }
      }
    }
  }
  __device__ void operator()(int m, int n, float v) const {
    v += bias[n];
    if (n < d) qk[size_t(m) * 2 * d + n] = to_bf16(v * qscale);
    else if (n < 2 * d) qk[size_t(m) * 2 * d + n] = to_bf16(v);
    else vt[size_t(n - 2 * d) * ldv + m] = to_bf16(v);
  }
};
struct EpiQKVF32 {
  const float* bias; float* qk; float* vt; int d; int ldv;
  __device__ void operator()(int m, int n, float v) const {
    v += bias[n];
    if (n < 2 * d) qk[size_t(m) * 2 * d + n] = v;
    else vt[size_t(n - 2 * d) * ldv + m] = v;
  }
};
struct EpiGateResidual {
  const float* bias; const float* gate; float* h; int ldh;
  static constexpr int kRowVec = 4;
  __device__ bool isrow(int) const { return true; }
  bool rows_aligned() const { return al16(h) && al16(bias) && al16(gate) && ldh % 4 == 0; }
  // rows m0 + k * dm (k < NP), columns n .. n + 3: all loads of h, then all stores
  template <int NP>
  __device__ void rows(int m0, int dm, int n, int M, const float (&v)[NP][4]) const {
    const float4 g = *reinterpret_cast<const float4*>(gate + n);
    const float4 b = *reinterpret_cast<const float4*>(bias + n);
    float4 o[NP];
#pragma unroll
    for (int k = 0; k < NP; ++k)
      o[k] = *reinterpret_cast<const float4*>(h + size_t(min(m0 + k * dm, M - 1)) * ldh + n);
#pragma unroll
    for (int k = 0; k < NP; ++k) {
      o[k].x += g.x * (v[k][0] + b.x);
      o[k].y += g.y * (v[k][1] + b.y);
      o[k].z += g.z * (v[k][2] + b.z);
      o[k].w += g.w * (v[k][3] + b.w);
      if (m0 + k * dm < M) store_nt(h + size_t(m0 + k * dm) * ldh + n, o[k]);
    }
  }
  __device__ void col(int mb, int n, int M, const f32x16& v) const {
    const float g = gate[n], b = bias[n];
    float* __restrict__ p = h + size_t(mb) * ldh + n;
    if (mb + 28 <= M) {                       // all 16 rows present: batched loads, no guards
      float old[16];
#pragma unroll
      for (int i = 0; i < 16; ++i) old[i] = p[size_t(8 * (i >> 2) + (i & 3)) * ldh];
#pragma unroll
      for (int i = 0; i < 16; ++i) p[size_t(8 * (i >> 2) + (i & 3)) * ldh] = old[i] + g * (v[i] + b);
      return;
    }
    float old[16];
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      const int r = min(mb + 8 * (i >> 2) + (i & 3), M - 1) - mb;   // clamped: in bounds
      old[i] = p[size_t(r) * ldh];
    }
#pragma unroll
    for (int i = 0; i < 16; ++i)
      if (mb + 8 * (i >> 2) + (i & 3) < M) p[size_t(8 * (i >> 2) + (i & 3)) * ldh] = old[i] + g * (v[i] + b);
  }
  __device__ void operator()(int m, int n, float v) const {
    float* p = h + size_t(m) * ldh + n;
    *p = *p + gate[n] * (v + bias[n]);
  }
};
struct EpiGeluBf16 {
  const float* bias; uint16_t* out; int ldo;
  static constexpr int kRowVec = 8;
  __device__ bool isrow(int) const { return true; }
  bool rows_aligned() const { return al16(out) && al16(bias) && ldo % 8 == 0; }
  template <int NP>
  __device__ void rows(int m0, int dm, int n, int M, const float (&v)[NP][8]) const {
    const float4 b0 = *reinterpret_cast<const float4*>(bias + n);
    const float4 b1 = *reinterpret_cast<const float4*>(bias + n + 4);
    const float bb[8] = {b0.x, b0.y, b0.z, b0.w, b1.x, b1.y, b1.z, b1.w};
#pragma unroll
    for (int k = 0; k < NP; ++k) {
      uint32_t w[4];
#pragma unroll
      for (int j = 0; j < 4; ++j)
        w[j] = uint32_t(to_bf16(gelu_tanh_fast(v[k][2 * j] + bb[2 * j]))) |
               (uint32_t(to_bf16(gelu_tanh_fast(v[k][2 * j + 1] + bb[2 * j + 1]))) << 16);
      if (m0 + k * dm < M) store_nt(out + size_t(m0 + k * dm) * ldo + n, make_uint4(w[0], w[1], w[2], w[3]));
    }
  }
  __device__ void col(int mb, int n, int M, const f32x16& v) const {
    const float b = bias[n];
    uint16_t* __restrict__ o = out + size_t(mb) * ldo + n;
    if (mb + 28 <= M) {
#pragma unroll
      for (int i = 0; i < 16; ++i) o[size_t(8 * (i >> 2) + (i & 3)) * ldo] = to_bf16(gelu_tanh(v[i] + b));
    } else {
#pragma unroll
      for (int i = 0; i < 16; ++i)
        if (mb + 8 * (i >> 2) + (i & 3) < M) o[size_t(8 * (i >> 2) + (i & 3)) * ldo] = to_bf16(gelu_tanh(v[i] + b));
    }
  }
  __device__ void operator()(int m, int n, float v) const {
    out[size_t(m) * ldo + n] = to_bf16(gelu_tanh(v + bias[n]));
  }
};
struct EpiGeluF32 {
  const float* bias; float* out; int ldo;
  __device__ void operator()(int m, int n, float v) const {
    out[size_t(m) * ldo + n] = gelu_tanh(v + bias[n]);
  }
};
struct EpiBiasAct {
  const float* bias; float* out; int ldo; int act;
  __device__ void operator()(int m, int n, float v) const {
    v += bias[n];
    out[size_t(m) * ldo + n] = act ? silu(v) : v;
  }
};
struct EpiPatch {
  const float* bias; const float* pos_f; const uint16_t* pos_b; float* out; int ldo;
  __device__ void operator()(int m, int n, float v) const {
    const size_t e = size_t(m) * ldo + n;
    const float p = pos_b ? from_bf16(pos_b[e]) : pos_f[e];
    out[e] = (v + bias[n]) + p;
  }
};
// Head + Euler: token m, patch-vector index n -> latent element; x += dsigma * (acc + b).
struct EpiHeadEuler {
  const float* bias; float* x; float dsigma; int T, Hl, Wl, p, Hp, Wp;
  static constexpr int kRowVec = 0;                 // scattered latent writes: by column
  __device__ bool isrow(int) const { return false; }
  bool rows_aligned() const { return false; }
  template <int NP>
  __device__ void rows(int, int, int, int, const float (&)[NP][4]) const {}
  __device__ float* at(int m, int n) const {
    const int pp = p * p;
    const int c = n / pp, a = (n / p) % p, b = n % p;
    const int t = m / (Hp * Wp), i = (m / Wp) % Hp, j = m % Wp;
    return x + ((size_t(c) * T + t) * Hl + (p * i + a)) * Wl + (p * j + b);
  }
  __device__ void col(int mb, int n, int M, const f32x16& v) const {
    float a[16];
#pragma unroll
    for (int i = 0; i < 16; ++i) a[i] = v[i];
    col(mb, n, M, a);
  }
  // rows mb + 8 (i / 4) + i % 4 of output column n: all loads, then all stores
  __device__ void col(int mb, int n, int M, const float (&v)[16]) const {
    const float bn = bias[n];
    float* dst[16];
    float old[16];
#pragma unroll
    for (int i = 0; i < 16; ++i) dst[i] = at(min(mb + 8 * (i >> 2) + (i & 3), M - 1), n);
#pragma unroll
    for (int i = 0; i < 16; ++i) old[i] = *dst[i];
#pragma unroll
    for (int i = 0; i < 16; ++i)
      if (mb + 8 * (i >> 2) + (i & 3) < M) *dst[i] = old[i] + dsigma * (v[i] + bn);
  }
  __device__ void operator()(int m, int n, float v) const {
    const int pp = p * p;
    const int c = n / pp, a = (n / p) % p, b = n % p;
    const int t = m / (Hp * Wp), i = (m / Wp) % Hp, j = m % Wp;
    float* dst = x + ((size_t(c) * T + t) * Hl + (p * i + a)) * Wl + (p * j + b);
    *dst = *dst + dsigma * (v + bias[n]);
  }
};

// ---------------------------------------------------------------------------
// bf16 MFMA GEMM, LDS-DMA pipeline.  512 threads = 8 waves (2 per SIMD), block
// tile BM x BN x 64.  Tiles go global -> LDS with global_load_lds_dwordx4 (lane i
// of an instruction lands at LDS base + 16 i, so the XOR swizzle is applied to the
// global address each lane fetches): no staging registers and no LDS write
// instructions.  Two stages, one barrier per k-step: the loads for step k+1 are
// issued among the MFMAs of the first DS 16-wide k-slices of step k (the block
// GEMMs use DS = 2, so the last refill has half a step to land).  Rows past M or N
// are clamped to the last row (their results are never stored).  Workgroups are
// renumbered so that each XCD (assigned round-robin by workgroup id) processes a
// contiguous range of tiles.
// ---------------------------------------------------------------------------
typedef __attribute__((address_space(3))) void lds_void;
// 16 bytes per lane global -> LDS (global_load_lds_dwordx4): lane i reads
// base + off (wave-uniform 64-bit base in SGPRs, per-lane 32-bit byte offset) and
// its bytes land at the wave-uniform LDS address dst + 16 i.  Issued as inline
// assembly so that the compiler neither makes LDS reads of the other stage wait
// for it nor reorders it; the kernel waits for its own fills (vmcnt) before each
// barrier.
__device__ inline void dma16(const void* base, uint32_t off, const void* dst) {
  const uint32_t lds = static_cast<uint32_t>(reinterpret_cast<uintptr_t>(dst));
  asm volatile("s_mov_b32 m0, %2\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %0, %1"
               :: "v"(off), "s"(base), "s"(lds) : "memory", "m0");
}

// s_waitcnt vmcnt(N) with the other counters left alone (gfx9 encoding: vmcnt bits
// [3:0] and [15:14], expcnt [6:4], lgkmcnt [11:8])
template <int N>
__device__ inline void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | 0x0F70);
}
constexpr int kEpiStride = 40;   // floats per row of the epilogue's per-wave LDS transpose buffer

// Epilogue of the bf16 block GEMMs.  Row-vector epilogues: each 32 x 32
// accumulator tile goes through a per-wave LDS buffer (rows of 40 floats: the two
// row groups a ds_write_b32 covers land 32 banks apart) and comes back as V
// consecutive columns of one row per lane.  The caller has finished every read of
// the LDS stages (the barrier here orders the reuse).
template <int BM, int BN, int WM, int WN, class Epi, int TM, int TN>
__device__ inline void gemm_epilogue(f32x16 (&acc)[TM][TN], uint4* lds, int m0, int n0, int M,
                                     int N, int wave, int lane, int rows_ok, const Epi& epi) {
  constexpr int WTM = BM / WM, WTN = BN / WN;
  constexpr int RV = Epi::kRowVec > 0 ? Epi::kRowVec : 4;
  constexpr int kS = kEpiStride;
  const int wm = wave % WM, wn = wave / WM;
  const int r32 = lane & 31, hi = lane >> 5;
  if constexpr (Epi::kRowVec > 0) {
    __builtin_amdgcn_s_barrier();              // every wave is done with the last stage
    asm volatile("" ::: "memory");
  }
  float* const st = reinterpret_cast<float*>(lds) + wave * 32 * kS;
#pragma unroll
  for (int b = 0; b < TN; ++b) {
    const int nb = n0 + wn * WTN + b * 32;     // first column of the tile
    if (nb >= N) continue;
    if (Epi::kRowVec > 0 && rows_ok && nb + 32 <= N && epi.isrow(nb)) {
#pragma unroll
      for (int a = 0; a < TM; ++a) {
        const int mb = m0 + wm * WTM + a * 32;
#pragma unroll
        for (int i = 0; i < 16; ++i) st[(8 * (i >> 2) + 4 * hi + (i & 3)) * kS + r32] = acc[a][b][i];
        constexpr int LPR = 32 / RV, RPI = 64 / LPR, NP = 32 / RPI;   // lanes per row, rows per pass
        const int r0 = lane / LPR, c = (lane % LPR) * RV;
        float v[NP][RV];
#pragma unroll
        for (int k = 0; k < NP; ++k)
#pragma unroll
          for (int q = 0; q < RV; q += 4) {
            const float4 t = *reinterpret_cast<const float4*>(st + (k * RPI + r0) * kS + c + q);
            v[k][q] = t.x; v[k][q + 1] = t.y; v[k][q + 2] = t.z; v[k][q + 3] = t.w;
          }
        epi.template rows<NP>(mb + r0, RPI, nb + c, M, v);
      }
    } else {
#pragma unroll
      for (int a = 0; a < TM; ++a)
        if (nb + r32 < N) epi.col(m0 + wm * WTM + a * 32 + 4 * hi, nb + r32, M, acc[a][b]);
    }
  }
}

template <int BM, int BN, int WM, int WN, int DS, class Epi>
__global__ void __launch_bounds__(WM * WN * 64) k_gemm_dma(const uint16_t* __restrict__ A, int lda,
                                                  const uint16_t* __restrict__ W, int ldw, int M,
                                                  int N, int K, int tiles_n, int tiles, int per_xcd,
                                                  int rows_ok, Epi epi) {
  constexpr int BK = 64;
  constexpr int NW = WM * WN;
  constexpr int WTM = BM / WM, WTN = BN / WN;
  constexpr int TM = WTM / 32, TN = WTN / 32;
  constexpr int AI = BM * 8 / 64 / NW, BI = BN * 8 / 64 / NW;   // DMA instructions per wave
  static_assert(TM >= 1 && TN >= 1 && AI * NW * 64 == BM * 8 && BI * NW * 64 == BN * 8,
                "tile shape");
  // one array, so every stage address is a constant offset from one base
  __shared__ uint4 lds[2 * (BM + BN) * 8];
  uint4* const sA0 = lds;
  uint4* const sB0 = lds + BM * 8;
  uint4* const sA1 = lds + (BM + BN) * 8;
  uint4* const sB1 = lds + (2 * BM + BN) * 8;

  const int t = (blockIdx.x & 7) * per_xcd + (blockIdx.x >> 3);
  if (t >= tiles) return;
  // groups of four row tiles: consecutive tiles (the ones an XCD runs together)
  // walk down a group before moving right, so their A and W k-slices share L2
  const int tiles_m = (M + BM - 1) / BM;
  const int grp = t / (4 * tiles_n), gbase = grp * 4;
  const int gsz = min(4, tiles_m - gbase);
  const int tin = t - grp * 4 * tiles_n;
  const int m0 = (gbase + tin % gsz) * BM, n0 = (tin / gsz) * BN;
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);   // uniform: DMA addresses in SGPRs
  const int wm = wave % WM, wn = wave / WM;

  // per-lane global byte offsets of this wave's DMA instructions (k-step 0); the
  // operands stay below 2^31 elements, so the byte offsets fit 32 bits
  uint32_t offA[AI], offB[BI];
#pragma unroll
  for (int i = 0; i < AI; ++i) {
    const int slot = (wave * AI + i) * 64 + lane;
    const int r = slot >> 3, c = (slot & 7) ^ swz(slot >> 3);
    offA[i] = 2u * uint32_t(min(m0 + r, M - 1) * lda + 8 * c);
  }
#pragma unroll
  for (int i = 0; i < BI; ++i) {
    const int slot = (wave * BI + i) * 64 + lane;
    const int r = slot >> 3, c = (slot & 7) ^ swz(slot >> 3);
    offB[i] = 2u * uint32_t(min(n0 + r, N - 1) * ldw + 8 * c);
  }
  f32x16 acc[TM][TN];
#pragma unroll
  for (int a = 0; a < TM; ++a)
#pragma unroll
    for (int b = 0; b < TN; ++b)
#pragma unroll
      for (int i = 0; i < 16; ++i) acc[a][b][i] = 0.f;

  const int KT = K / BK;                         // even: the launcher requires K % 128 == 0

  const int r32 = lane & 31, hi = lane >> 5;
  // one DMA instruction (j < AI + BI) of the refill of stage (da, db) with k-step kt;
  // compute() spreads the refill over its first DS k-slices
  auto dma_one = [&](uint4* da, uint4* db, int kt, int j) {
    const int k0 = kt * BK;
    if (j < AI) dma16(A + k0, offA[j], da + (wave * AI + j) * 64);
    else dma16(W + k0, offB[j - AI], db + (wave * BI + (j - AI)) * 64);
  };
  auto compute = [&](const uint4* sa, const uint4* sb, uint4* da, uint4* db, int kt) {
#pragma unroll
    for (int kk = 0; kk < BK / 16; ++kk) {
      if (kt >= 0) {
        // the refill goes out over the first DS k-slices, DPS instructions per slice
        constexpr int DPS = (AI + BI + DS - 1) / DS;
#pragma unroll
        for (int j = kk * DPS; j < (kk + 1) * DPS; ++j)
          if (j < AI + BI && kk < DS) dma_one(da, db, kt, j);
      }
      const int ch = kk * 2 + hi;
      bf16x8 af[TM], bf[TN];
#pragma unroll
      for (int a = 0; a < TM; ++a) {
        const int r = wm * WTM + a * 32 + r32;
        af[a] = __builtin_bit_cast(bf16x8, sa[r * 8 + (ch ^ swz(r))]);
      }
#pragma unroll
      for (int b = 0; b < TN; ++b) {
        const int r = wn * WTN + b * 32 + r32;
        bf[b] = __builtin_bit_cast(bf16x8, sb[r * 8 + (ch ^ swz(r))]);
      }
#pragma unroll
      for (int a = 0; a < TM; ++a)
#pragma unroll
        for (int b = 0; b < TN; ++b)
          acc[a][b] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[a], bf[b], acc[a][b], 0, 0, 0);
    }
  };

#pragma unroll
  for (int j = 0; j < AI + BI; ++j) dma_one(sA0, sB0, 0, j);
  // before each barrier: this wave's refill has landed
  for (int kt = 0; kt < KT; kt += 2) {
    wait_vmcnt<0>();
    __builtin_amdgcn_s_barrier();
    asm volatile("" ::: "memory");
    compute(sA0, sB0, sA1, sB1, kt + 1);
    wait_vmcnt<0>();
    __builtin_amdgcn_s_barrier();
    asm volatile("" ::: "memory");
    compute(sA1, sB1, sA0, sB0, kt + 2 < KT ? kt + 2 : -1);
  }

  static_assert(Epi::kRowVec == 0 || sizeof(lds) >= NW * 32 * kEpiStride * sizeof(float), "epilogue LDS");
  gemm_epilogue<BM, BN, WM, WN>(acc, lds, m0, n0, M, N, wave, lane, rows_ok, epi);
}

template <int BM, int BN, int WM, int WN, int DS, class Epi>
Status launch_dma(const uint16_t* A, int lda, const uint16_t* W, int ldw, int M, int N, int K,
                  const Epi& epi, hipStream_t s) {
  if (M <= 0) return Status::ok();
  if (K % 128 || lda % 8 || ldw % 8) return Status::shape("bf16 GEMM needs K % 128 == 0 and 16-byte rows");
  if (int64_t(M) * lda > INT32_MAX || int64_t(N) * ldw > INT32_MAX)
    return Status::shape("bf16 GEMM operand exceeds 2^31 elements");
  const int tn = (N + BN - 1) / BN, tm = (M + BM - 1) / BM;
  const int tiles = tn * tm;
  const int per = (tiles + 7) / 8;
  // row-vector epilogue stores need 16-byte aligned rows; otherwise every tile goes by column
  const int rows_ok = epi.rows_aligned() ? 1 : 0;
  hipLaunchKernelGGL((k_gemm_dma<BM, BN, WM, WN, DS, Epi>), dim3(8 * per), dim3(WM * WN * 64), 0, s, A, lda, W,
                     ldw, M, N, K, tn, tiles, per, rows_ok, epi);
  DC_HIP(hipGetLastError());
  return Status::ok();
}


// ---------------------------------------------------------------------------
// Patch embedding for the bf16 model: h_in[n] = patch(x)[n] W_pe^T + b + pos[n]
// with the fp32 latent and fp32 W_pe kept at fp32 accuracy on bf16 MFMA: each
// operand is split v = hi + lo (hi = bf16(v), lo = bf16(v - hi)) and the
// product is hi*Whi + lo*Whi + hi*Wlo (the dropped lo*Wlo is ~2^-18 relative).
// The patchify gather is fused: each lane reads its 8 patch-vector entries
// straight from the latent.  A workgroup = 8 waves x 32 tokens x a 128-wide
// column chunk; the chunk of W_pe is split once into LDS and shared.  Work items
// (token block, column chunk) are dealt so that an XCD runs every column chunk of
// a contiguous range of token blocks, so each XCD's L2 fetches only its own part
// of the latent.  Each wave's 32 x 32 result tiles go through LDS, so the output
// rows leave as 16-byte stores (8 rows x 128 bytes per instruction; ordinary stores:
// the drift check and the first block read h_in right after, partly from the caches)
// and the positional rows arrive as 8-byte loads.
// ---------------------------------------------------------------------------
struct PatchGeo { int T, Hl, Wl, p, lp, Hp, Wp; };   // lp = log2(p)

constexpr int kPeStride = 40;   // floats per row of a wave's 32 x 32 result tile in LDS

__global__ void __launch_bounds__(512) k_patch_embed_bf16(const float* __restrict__ x,
                                                          const float* __restrict__ W,
                                                          const float* __restrict__ bias,
                                                          const uint16_t* __restrict__ pos,
                                                          float* __restrict__ out, int Nv, int d,
                                                          int items, int per_xcd, PatchGeo pg) {
  __shared__ uint4 wh[128 * 8], wl[128 * 8];     // [n][16-byte chunk of k], swizzled
  __shared__ __attribute__((aligned(16))) float res[8][32 * kPeStride];
  const int item = (blockIdx.x & 7) * per_xcd + (blockIdx.x >> 3);
  if (item >= items) return;
  const int ncc = d >> 7;
  const int tb = item / ncc, cc = item - tb * ncc;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int r32 = lane & 31, hi = lane >> 5;
  const int n0 = cc * 128;
  // stage W[n0 .. n0 + 128)[0 .. 64) as bf16 hi / lo: thread -> (row, 4 chunks of 4 k)
  {
    const int n = tid >> 2, k4 = (tid & 3) * 16;    // 16 consecutive k per thread
    const float4* src = reinterpret_cast<const float4*>(W + size_t(n0 + n) * 64 + k4);
    float4 v[4];
#pragma unroll
    for (int q = 0; q < 4; ++q) v[q] = src[q];
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const float f[4] = {v[q].x, v[q].y, v[q].z, v[q].w};
      uint16_t h[4], l[4];
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        h[j] = to_bf16(f[j]);
        l[j] = to_bf16(f[j] - from_bf16(h[j]));
      }
      const int k = k4 + 4 * q;
      const int e = n * 64 + ((k >> 3) ^ swz(n)) * 8 + (k & 7);   // bf16 index, 8-byte aligned
      *reinterpret_cast<uint2*>(reinterpret_cast<uint16_t*>(wh) + e) =
          make_uint2(h[0] | (uint32_t(h[1]) << 16), h[2] | (uint32_t(h[3]) << 16));
      *reinterpret_cast<uint2*>(reinterpret_cast<uint16_t*>(wl) + e) =
          make_uint2(l[0] | (uint32_t(l[1]) << 16), l[2] | (uint32_t(l[3]) << 16));
    }
  }
  const int m0 = tb * 256 + wave * 32;
  // epilogue role of a lane: rows 8 q + lane / 8 (q < 4) of a 32 x 32 tile, columns
  // 4 (lane % 8) ..; the positional rows of the next tile are loaded one tile ahead
  // (rows clamped into the table)
  const int er = lane >> 3, ec = 4 * (lane & 7);
  auto load_pos = [&](int tile, uint2 (&pv)[4], float4& b4) {
    const int nc = n0 + 32 * tile + ec;
    b4 = *reinterpret_cast<const float4*>(bias + nc);
#pragma unroll
    for (int q = 0; q < 4; ++q)
      pv[q] = *reinterpret_cast<const uint2*>(pos + size_t(min(m0 + 8 * q + er, Nv - 1)) * d + nc);
  };
  uint2 pv[4];
  float4 b4;
  load_pos(0, pv, b4);
  // A fragments: token m, patch-vector entries 16 kk + 8 hi + e
  const int m = min(m0 + r32, Nv - 1);
  const int t = m / (pg.Hp * pg.Wp), i = (m / pg.Wp) % pg.Hp, j = m % pg.Wp;
  bf16x8 ah[4], al[4];
#pragma unroll
  for (int kk = 0; kk < 4; ++kk)
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const int q = 16 * kk + 8 * hi + e;
      const int c = q >> (2 * pg.lp), a = (q >> pg.lp) & (pg.p - 1), b = q & (pg.p - 1);
      const float v = x[((size_t(c) * pg.T + t) * pg.Hl + (pg.p * i + a)) * pg.Wl + (pg.p * j + b)];
      const __bf16 h = static_cast<__bf16>(v);
      ah[kk][e] = h;
      al[kk][e] = static_cast<__bf16>(v - static_cast<float>(h));
    }
  __syncthreads();
  float* const rt = res[wave];
#pragma unroll
  for (int tile = 0; tile < 4; ++tile) {
    f32x16 acc;
#pragma unroll
    for (int r = 0; r < 16; ++r) acc[r] = 0.f;
    const int nr = 32 * tile + r32;                 // row of the LDS chunk
#pragma unroll
    for (int kk = 0; kk < 4; ++kk) {
      const int ch = (2 * kk + hi) ^ swz(nr);
      const bf16x8 bh = __builtin_bit_cast(bf16x8, wh[nr * 8 + ch]);
      const bf16x8 bl = __builtin_bit_cast(bf16x8, wl[nr * 8 + ch]);
      acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ah[kk], bh, acc, 0, 0, 0);
      acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(al[kk], bh, acc, 0, 0, 0);
      acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ah[kk], bl, acc, 0, 0, 0);
    }
    const int nc = n0 + 32 * tile + ec;             // this lane's 4 output columns
    uint2 pn[4];
    float4 bn = b4;
    if (tile < 3) load_pos(tile + 1, pn, bn);
    // accumulator element r of lane (r32, hi): row 8 (r / 4) + 4 hi + r % 4, column r32
#pragma unroll
    for (int r = 0; r < 16; ++r) rt[(8 * (r >> 2) + 4 * hi + (r & 3)) * kPeStride + r32] = acc[r];
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int mm = m0 + 8 * q + er;
      const float4 a = *reinterpret_cast<const float4*>(rt + (8 * q + er) * kPeStride + ec);
      float4 o;
      o.x = (a.x + b4.x) + __uint_as_float(pv[q].x << 16);
      o.y = (a.y + b4.y) + __uint_as_float(pv[q].x & 0xFFFF0000u);
      o.z = (a.z + b4.z) + __uint_as_float(pv[q].y << 16);
      o.w = (a.w + b4.w) + __uint_as_float(pv[q].y & 0xFFFF0000u);
      if (mm < Nv) *reinterpret_cast<float4*>(out + size_t(mm) * d + nc) = o;
    }
    if (tile < 3) {
#pragma unroll
      for (int q = 0; q < 4; ++q) pv[q] = pn[q];
      b4 = bn;
    }
  }
}

// ---------------------------------------------------------------------------
// fp32 SIMT GEMM: 64x64 tile, k-step 16, each thread a 4x4 block of outputs
// ---------------------------------------------------------------------------
// four consecutive weights as fp32 (W in fp32, or bf16 bits widened exactly)
__device__ inline float4 load_w4(const float* W, size_t e) { return *reinterpret_cast<const float4*>(W + e); }
__device__ inline float4 load_w4(const uint16_t* W, size_t e) {
  const uint2 u = *reinterpret_cast<const uint2*>(W + e);
  return make_float4(__uint_as_float(u.x << 16), __uint_as_float(u.x & 0xFFFF0000u),
                     __uint_as_float(u.y << 16), __uint_as_float(u.y & 0xFFFF0000u));
}

template <class Epi, class WT>
__global__ void __launch_bounds__(256) k_gemm_f32(const float* __restrict__ A, int lda,
                                                  const WT* __restrict__ W, int ldw, int M,
                                                  int N, int K, Epi epi) {
  __shared__ float sA[16][64 + 4];
  __shared__ float sW[16][64 + 4];
  const int tid = threadIdx.x;
  const int tx = tid & 15, ty = tid >> 4;
  const int m0 = blockIdx.y * 64, n0 = blockIdx.x * 64;
  const int lr = tid >> 2, lk = (tid & 3) * 4;
  float acc[4][4] = {};
  for (int k0 = 0; k0 < K; k0 += 16) {
    const int gm = m0 + lr, gn = n0 + lr;
    float4 a = make_float4(0.f, 0.f, 0.f, 0.f), w = a;
    if (gm < M) a = *reinterpret_cast<const float4*>(A + size_t(gm) * lda + k0 + lk);
    if (gn < N) w = load_w4(W, size_t(gn) * ldw + k0 + lk);
    sA[lk + 0][lr] = a.x; sA[lk + 1][lr] = a.y; sA[lk + 2][lr] = a.z; sA[lk + 3][lr] = a.w;
    sW[lk + 0][lr] = w.x; sW[lk + 1][lr] = w.y; sW[lk + 2][lr] = w.z; sW[lk + 3][lr] = w.w;
    __syncthreads();
#pragma unroll
    for (int k = 0; k < 16; ++k) {
      float av[4], wv[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) av[i] = sA[k][ty * 4 + i];
#pragma unroll
      for (int j = 0; j < 4; ++j) wv[j] = sW[k][tx + 16 * j];
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j] += av[i] * wv[j];
    }
    __syncthreads();
  }
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int m = m0 + ty * 4 + i, n = n0 + tx + 16 * j;
      if (m < M && n < N) epi(m, n, acc[i][j]);
    }
}

template <class Epi, class WT>
Status launch_f32(const float* A, int lda, const WT* W, int ldw, int M, int N, int K,
                  const Epi& epi, hipStream_t s) {
  if (M <= 0 || N <= 0) return Status::ok();
  if (K % 16 || lda % 4 || ldw % 4) return Status::shape("f32 GEMM needs K % 16 == 0, aligned rows");
  dim3 grid((N + 63) / 64, (M + 63) / 64);
  hipLaunchKernelGGL((k_gemm_f32<Epi, WT>), grid, dim3(256), 0, s, A, lda, W, ldw, M, N, K, epi);
  DC_HIP(hipGetLastError());
  return Status::ok();
}

}  // namespace

// ---------------------------------------------------------------------------
// entry points
// ---------------------------------------------------------------------------
Status gemm_f32_bias_act(const float* A, int lda, const float* W, int ldw, const float* bias,
                         float* out, int ldo, int M, int N, int K, Act act, hipStream_t s) {
  return launch_f32(A, lda, W, ldw, M, N, K, EpiBiasAct{bias, out, ldo, act == Act::kSilu ? 1 : 0}, s);
}

Status gemm_f32_gate_residual(const float* A, int lda, const float* W, int ldw, const float* bias,
                              const float* gate, float* h, int ldh, int M, int N, int K,
                              hipStream_t s) {
  return launch_f32(A, lda, W, ldw, M, N, K, EpiGateResidual{bias, gate, h, ldh}, s);
}

Status gemm_f32_bias_act(const float* A, int lda, const uint16_t* W, int ldw, const float* bias,
                         float* out, int ldo, int M, int N, int K, Act act, hipStream_t s) {
  if (ldw % 4) return Status::shape("f32 GEMM with bf16 weights needs ldw % 4 == 0");
  return launch_f32(A, lda, W, ldw, M, N, K, EpiBiasAct{bias, out, ldo, act == Act::kSilu ? 1 : 0}, s);
}

Status gemm_f32_gate_residual(const float* A, int lda, const uint16_t* W, int ldw, const float* bias,
                              const float* gate, float* h, int ldh, int M, int N, int K,
                              hipStream_t s) {
  if (ldw % 4) return Status::shape("f32 GEMM with bf16 weights needs ldw % 4 == 0");
  return launch_f32(A, lda, W, ldw, M, N, K, EpiGateResidual{bias, gate, h, ldh}, s);
}

Status gemm_f32_head(const float* A, int lda, const uint16_t* W, const float* bias, float* x,
                     float dsigma, const Geo& g, int M, hipStream_t s) {
  EpiHeadEuler e{bias, x, dsigma, g.T, g.Hl, g.Wl, g.p, g.Hp, g.Wp};
  return launch_f32(A, lda, W, g.d, M, g.P, g.d, e, s);
}

Status gemm_f32_gelu(const float* A, int lda, const float* W, int ldw, const float* bias,
                     float* out, int ldo, int M, int N, int K, hipStream_t s) {
  return launch_f32(A, lda, W, ldw, M, N, K, EpiGeluF32{bias, out, ldo}, s);
}

Status gemm_f32_patch_embed(const float* A, const float* W, const float* bias, const void* pos,
                            bool pos_bf16, float* out, int ldo, int M, int N, hipStream_t s) {
  EpiPatch e{bias, pos_bf16 ? nullptr : static_cast<const float*>(pos),
             pos_bf16 ? static_cast<const uint16_t*>(pos) : nullptr, out, ldo};
  return launch_f32(A, 64, W, 64, M, N, 64, e, s);
}

Status gemm_f32_head(const float* A, int lda, const float* W, const float* bias, float* x,
                     float dsigma, const Geo& g, int M, hipStream_t s) {
  EpiHeadEuler e{bias, x, dsigma, g.T, g.Hl, g.Wl, g.p, g.Hp, g.Wp};
  return launch_f32(A, lda, W, g.d, M, g.P, g.d, e, s);
}

Status gemm_f32_qkv(const float* A, const float* W, const float* bias, float* qk, float* vt,
                    int ldv, const Geo& g, int M, hipStream_t s) {
  return launch_f32(A, g.d, W, g.d, M, 3 * g.d, g.d, EpiQKVF32{bias, qk, vt, g.d, ldv}, s);
}

Status gemm_bf16_qkv(const uint16_t* A, const uint16_t* W, const float* bias, uint16_t* qk,
                     uint16_t* vt, int ldv, const Geo& g, int M, hipStream_t s) {
  return launch_dma<384, 192, 4, 2, 2>(A, g.d, W, g.d, M, 3 * g.d, g.d,
                                    EpiQKVBf16{bias, qk, vt, g.d, ldv,
                                               float(1.4426950408889634 / std::sqrt(double(g.Dh)))},
                                    s);
}

Status gemm_bf16_gate_residual(const uint16_t* A, int lda, const uint16_t* W, const float* bias,
                               const float* gate, float* h, int ldh, int M, int N, int K,
                               hipStream_t s) {
  return launch_dma<384, 192, 4, 2, 2>(A, lda, W, K, M, N, K, EpiGateResidual{bias, gate, h, ldh}, s);
}

Status gemm_bf16_gelu(const uint16_t* A, int lda, const uint16_t* W, const float* bias,
                      uint16_t* out, int ldo, int M, int N, int K, hipStream_t s) {
  return launch_dma<320, 256, 2, 4, 2>(A, lda, W, K, M, N, K, EpiGeluBf16{bias, out, ldo}, s);
}

Status gemm_bf16_head(const uint16_t* A, int lda, const uint16_t* W, const float* bias, float* x,
                      float dsigma, const Geo& g, int M, hipStream_t s) {
  if (M <= 0) return Status::ok();
  if (g.P != 64 || g.d % 128 || lda % 8) return Status::shape("bf16 head needs 64 outputs and d % 128 == 0");
  EpiHeadEuler e{bias, x, dsigma, g.T, g.Hl, g.Wl, g.p, g.Hp, g.Wp};
  return launch_dma<64, 64, 2, 2, 4>(A, lda, W, g.d, M, 64, g.d, e, s);
}

Status patch_embed_bf16(const float* x, const float* W, const float* bias, const uint16_t* pos,
                        float* out, const Geo& g, hipStream_t s) {
  if (g.Nv <= 0) return Status::ok();
  if (g.P != 64 || g.d % 128) return Status::shape("bf16 patch embedding needs 64-entry patches, d % 128 == 0");
  int lp = 0;
  while ((1 << lp) < g.p) ++lp;
  if ((1 << lp) != g.p) return Status::shape("bf16 patch embedding needs a power-of-two patch");
  if (!al16(out) || !al16(bias) || !al16(pos) || !al16(W))
    return Status::arg("bf16 patch embedding needs 16-byte aligned device buffers");
  const PatchGeo pg{g.T, g.Hl, g.Wl, g.p, lp, g.Hp, g.Wp};
  const int items = (g.Nv + 255) / 256 * (g.d / 128), per_xcd = (items + 7) / 8;
  hipLaunchKernelGGL(k_patch_embed_bf16, dim3(8 * per_xcd), dim3(512), 0, s, x, W, bias, pos, out,
                     g.Nv, g.d, items, per_xcd, pg);
  DC_HIP(hipGetLastError());
  return Status::ok();
}

}  // namespace dc
