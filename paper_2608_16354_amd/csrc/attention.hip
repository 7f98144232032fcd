// Joint video + text self-attention, softmax(Q K^T / sqrt(d_h)) V per head, with
// an online softmax (flash-style: the N x N score matrix never leaves registers).
//
// Two bf16 kernels: k_attn16 (head_dim 64, sequences of 8,192 tokens and more; see its
// own comment below) and k_attn_bf16 (head_dim 64 below that, and head_dim 72).
//
// k_attn_bf16 (gfx950 MFMA 32x32x16).  A workgroup is 4 waves x 32 query rows of one
// head; key/value tiles of 64 tokens stream through a 3-stage LDS ring.  The QKV
// GEMM stores Q pre-multiplied by log2(e)/sqrt(d_h), so scores arrive in log2
// units and P = 2^(s - m).  Each wave
// computes the transposed scores S^T = K Q^T, so in the accumulator layout every
// lane holds scores of a single query row (lane % 32): the row max needs one
// cross-lane exchange (lanes l and l^32) and the rescale of the output is a
// per-lane multiply.  The output is accumulated transposed as well,
// O^T += V^T P^T, which needs V^T in LDS (the QKV GEMM writes V transposed).
// The K rows feeding the S^T tiles are permuted (bits 2 and 3 of the row index
// swapped) so that the eight scores a lane holds for each 16-token slice of P are
// eight consecutive tokens: P goes from the score registers straight into the
// B operand of the P V product, and V^T is read with one 16-byte LDS load.
// Per-score VALU work is kept to the exponential, half a bf16 conversion and one
// fp32 add for the row sum: the subtraction of the running maximum m rides on
// the MFMA as one extra rank-1 step (a column of ones times -m).  The row sum is
// a plain v_add chain rather than v_dot2 on the bf16 pairs: on gfx950 the dot
// instructions do not issue alongside running MFMAs, adds do.  m is set from
// the first tile's maximum and raised only when a tile's P would grow past 2^64
// (the tile's row sum is the test), so the common path takes no tile maximum;
// P and the fp32 sums stay far inside the fp32 range either way.
#include <hip/hip_runtime.h>

#include <cmath>
#include <type_traits>

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


typedef __attribute__((address_space(3))) void lds_void;

// 16 bytes per lane global -> LDS (global_load_lds_dwordx4): lane i reads
// base + off (a wave-uniform 64-bit base, a per-lane 32-bit byte offset) and its
// bytes land at the wave-uniform LDS address dst + 16 i.  Issued as inline
// assembly: the compiler cannot tell the stage being filled from the stage being
// read and would otherwise wait for every outstanding fill before each LDS read.
// The kernel waits for its own fills explicitly (vmcnt) before the barrier that
// publishes a stage.
__device__ inline void dma16(const void* base, uint32_t off, const void* dst) {
  const uint32_t lds = static_cast<uint32_t>(reinterpret_cast<uintptr_t>(dst));
  asm volatile("s_mov_b32 m0, %2\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %0, %1"
               :: "v"(off), "s"(base), "s"(lds) : "memory", "m0");
}

template <int D>
struct AttnShape {
  static constexpr int DK = (D + 15) / 16 * 16;   // contraction width of Q K^T (zero padded)
  static constexpr int KC = DK / 8;               // 16-byte chunks per K row in LDS
  static constexpr int DC8 = D / 8;               // chunks holding real data
  static constexpr int DV = (D + 31) / 32 * 32;   // rows of the O^T accumulator
  static constexpr int TV = DV / 32;
  static constexpr int BKV = 64;                  // tokens per K/V tile
  static constexpr int KSLOTS = BKV * KC;         // 16-byte LDS slots of a K tile
  static constexpr int VSLOTS = DV * 8;           // of a V^T tile (64 tokens = 8 chunks per row)
  static constexpr int KI = (KSLOTS + 255) / 256; // DMA instructions per wave (4 waves x 64 lanes)
  static constexpr int VI = (VSLOTS + 255) / 256;
};

// K/V^T tiles go global -> LDS into a ring of three stages (separate arrays),
// prefetched two tiles ahead; one barrier per tile.
// Lane i of a DMA instruction lands at the instruction's LDS base + 16 i, so each
// lane fetches the global chunk that belongs at its slot: the swizzle and the
// K-padding are applied on the global side.  Rows past the data (K rows past M,
// padding chunks, V^T rows past D) fetch real, finite data whose products are
// either multiplied by zero (padded Q columns, masked P) or never stored.
template <int D>
__global__ void __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(D == 64 ? 3 : 2)))
k_attn_bf16(const uint16_t* __restrict__ qk,
                                                   const uint16_t* __restrict__ vt, int ldv,
                                                   uint16_t* __restrict__ out, int M, int d,
                                                   int nqb, int items, int per_xcd, int full,
                                                   float* __restrict__ part) {
  using S = AttnShape<D>;
  constexpr int DK = S::DK, KC = S::KC, DC8 = S::DC8, TV = S::TV, BKV = S::BKV;
  constexpr int KI = S::KI, VI = S::VI;
  // one array, so every stage address is a constant offset from one base
  constexpr int STAGE = (KI + VI) * 256;
  __shared__ uint4 lds[3 * STAGE];
  uint4* const sK0 = lds;
  uint4* const sV0 = lds + KI * 256;
  uint4* const sK1 = lds + STAGE;
  uint4* const sV1 = lds + STAGE + KI * 256;
  uint4* const sK2 = lds + 2 * STAGE;
  uint4* const sV2 = lds + 2 * STAGE + KI * 256;

  // Work item w = head * nqb + query block.  Workgroups are dealt to the XCDs
  // round-robin, so workgroup b runs item (b % 8) * per_xcd + b / 8: each XCD
  // sweeps a contiguous range of items, i.e. the query blocks of one head at a
  // time, and that head's K and V stay in its L2.
  //
  // Tail split: XCD x owns items [x per_xcd, (x + 1) per_xcd).  Its first `full`
  // work units are whole items; every later item is split into two units, one per
  // half of the key tiles, so the last (partial) round of resident workgroups runs
  // half as long.  A split unit leaves its unnormalised output, running maximum and
  // row sum in `part` (record si = x (per_xcd - full) + index among the XCD's split
  // items); k_attn_combine merges the two halves.
  const int xcd = blockIdx.x & 7, u = blockIdx.x >> 3;
  const int ibeg = xcd * per_xcd, iend = min(items, ibeg + per_xcd);
  const int nfull = min(full, iend - ibeg);
  int w, half = -1;
  if (u < nfull) {
    w = ibeg + u;
  } else {
    w = ibeg + nfull + ((u - nfull) >> 1);
    half = (u - nfull) & 1;
  }
  if (w >= iend) return;
  const int ntile = (M + BKV - 1) / BKV;
  const int tb = half == 1 ? ntile / 2 : 0;              // key tiles [tb, te)
  const int te = half == 0 ? ntile / 2 : ntile;
  const int head = w / nqb;
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);   // uniform: DMA addresses in SGPRs
  const int g = lane >> 5, r32 = lane & 31;
  const int q0 = (w - head * nqb) * 128 + wave * 32;
  const int ldq = 2 * d;
  const uint16_t* Qb = qk + head * D;
  const uint16_t* Kb = qk + d + head * D;
  const uint16_t* Vb = vt + size_t(head) * D * ldv;
  const uint4 zero4 = make_uint4(0, 0, 0, 0);

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
  // the query fragments have landed before the first LDS-DMA is issued, so no
  // later wait on them can also hold up the tile pipeline
  __builtin_amdgcn_s_waitcnt(0x0F70);

  // per-lane source byte offsets of this wave's DMA instructions for tile 0; tile t
  // adds a uniform t * 64 rows (K) or t * 64 columns (V^T).  K rows run up to
  // 64 + 12 past the tile start: the qk buffer has ldv + 64 rows, and rows past M
  // only feed scores that the last tile masks (by assignment, so any bits are safe).
  uint32_t offK[KI], offV[VI];
#pragma unroll
  for (int i = 0; i < KI; ++i) {
    const int slot = (wave * KI + i) * 64 + lane;
    const int r = slot / KC, pc = slot % KC;
    const int c = (KC == 8) ? (pc ^ swz_k(r)) : pc;
    const int cc = c < DC8 ? c : 0;                    // padding chunk: any real chunk
    offK[i] = 2u * uint32_t(r * ldq + 8 * cc);
  }
#pragma unroll
  for (int i = 0; i < VI; ++i) {
    const int slot = (wave * VI + i) * 64 + lane;
    const int r = slot >> 3, c = (slot & 7) ^ swz_v(slot >> 3);
    offV[i] = 2u * uint32_t(min(r, D - 1) * ldv + 8 * c);
  }
  auto issue = [&](uint4* sk, uint4* sv, int t) {
    const uint16_t* kt = Kb + size_t(t) * BKV * ldq;
    const uint16_t* vtt = Vb + t * BKV;
#pragma unroll
    for (int i = 0; i < KI; ++i) dma16(kt, offK[i], sk + (wave * KI + i) * 64);
#pragma unroll
    for (int i = 0; i < VI; ++i) dma16(vtt, offV[i], sv + (wave * VI + i) * 64);
  };

  f32x16 o[TV];
#pragma unroll
  for (int t = 0; t < TV; ++t)
#pragma unroll
    for (int i = 0; i < 16; ++i) o[t][i] = 0.f;
  // Scores arrive in log2 units (Q pre-scaled by log2(e)/sqrt(d_h)).  One extra
  // rank-1 MFMA step (k = 8) adds -m to every score: A is a column of ones (the
  // first k slot of the lanes with g = 0), B holds -m of the lane's query in its
  // first k slot.  m is kept exactly representable in bf16.
  typedef short s16x4 __attribute__((ext_vector_type(4)));
  const s16x4 kaug = {short(g == 0 ? 0x3F80 : 0), 0, 0, 0};
  s16x4 qaug = {0, 0, 0, 0};
  float mrow = 0.f, lsum = 0.f;

  auto compute = [&](const uint4* sk, const uint4* sv, int t) {
    // S^T for two 32-token sub-tiles; sub-tile st, register i holds token
    // 32 st + 16 (i / 8) + 8 g + (i % 8) of the tile, query q0 + r32.
    f32x16 s[2];
#pragma unroll
    for (int st = 0; st < 2; ++st) {
      f32x16 z;
#pragma unroll
      for (int i = 0; i < 16; ++i) z[i] = 0.f;
      s[st] = __builtin_amdgcn_mfma_f32_32x32x8bf16_1k(kaug, qaug, z, 0, 0, 0);
      const int row = 32 * st + perm_kv(r32);
#pragma unroll
      for (int kk = 0; kk < DK / 16; ++kk) {
        const int ch = 2 * kk + g;
        const int pc = (KC == 8) ? (ch ^ swz_k(row)) : ch;
        const bf16x8 kf = __builtin_bit_cast(bf16x8, sk[row * KC + pc]);
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
    // raise m to the tile maximum (first tile; later only when P would grow past 2^64)
    auto raise = [&](bool first) {
      float mx = s[0][0];
#pragma unroll
      for (int st = 0; st < 2; ++st)
#pragma unroll
        for (int i = 0; i < 16; ++i) mx = fmaxf(mx, s[st][i]);
      mx = fmaxf(mx, __shfl_xor(mx, 32, 64));
      const float mnew = __uint_as_float(uint32_t(to_bf16(mrow + (first ? mx : fmaxf(mx, 0.f)))) << 16);
      const float up = mnew - mrow;
      const float alpha = __builtin_amdgcn_exp2f(-up);
      mrow = mnew;
      qaug[0] = short(to_bf16(-mnew));
      lsum *= alpha;
#pragma unroll
      for (int tv = 0; tv < TV; ++tv)
#pragma unroll
        for (int i = 0; i < 16; ++i) o[tv][i] *= alpha;
#pragma unroll
      for (int st = 0; st < 2; ++st)
#pragma unroll
        for (int i = 0; i < 16; ++i) s[st][i] -= up;
    };
    if (t == tb) raise(true);
    bf16x8 pf[4];
    float ts = 0.f;
    auto exps = [&]() {
      // two add chains over the fp32 exponentials (the MFMA consumes them rounded to bf16)
      float t2[2];
#pragma unroll
      for (int c = 0; c < 4; ++c)
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          const float p = __builtin_amdgcn_exp2f(s[c >> 1][8 * (c & 1) + e]);
          t2[e & 1] = (c == 0 && e < 2) ? p : t2[e & 1] + p;
          pf[c][e] = static_cast<__bf16>(p);
        }
      ts = t2[0] + t2[1];
    };
    exps();
    // P stays far inside fp32 range while m lags the running maximum by less than
    // about 58 (log2 units); only then is m raised (rare), so no tile maximum is
    // taken on the common path
    if (t > tb && __builtin_amdgcn_ballot_w64(!(ts < 0x1p64f)) != 0) {
      raise(false);
      exps();
    }
    lsum += ts;
#pragma unroll
    for (int c = 0; c < 4; ++c) {
      const int ch = 2 * c + g;
#pragma unroll
      for (int tv = 0; tv < TV; ++tv) {
        const int row = 32 * tv + r32;
        const bf16x8 vf = __builtin_bit_cast(bf16x8, sv[row * 8 + (ch ^ swz_v(row))]);
        o[tv] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vf, pf[c], o[tv], 0, 0, 0);
      }
    }
  };

  // vmcnt(n) with the other counters left alone
  constexpr int kPerTile = KI + VI;
  issue(sK0, sV0, tb);
  if (tb + 1 < te) issue(sK1, sV1, tb + 1);
  auto step = [&](uint4* sk, uint4* sv, uint4* nk, uint4* nv, int t) {
    if (t + 1 < te) __builtin_amdgcn_s_waitcnt(0x0F70 | kPerTile);    // tile t landed (t+1 may fly)
    else __builtin_amdgcn_s_waitcnt(0x0F70);
    __builtin_amdgcn_s_barrier();          // everyone's tile t landed; tile t-1's stage is free
    if (t + 2 < te) issue(nk, nv, t + 2);
    compute(sk, sv, t);
  };
  for (int t = tb; t < te; t += 3) {
    step(sK0, sV0, sK2, sV2, t);
    if (t + 1 >= te) break;
    step(sK1, sV1, sK0, sV0, t + 1);
    if (t + 2 >= te) break;
    step(sK2, sV2, sK1, sV1, t + 2);
  }

  lsum += __shfl_xor(lsum, 32, 64);
  if (half >= 0) {
    // split unit: unnormalised O, m and l of the wave's 32 queries; record layout
    // [half][128 queries][D + 4] floats (O, m, l, two unused: 16-byte aligned rows)
    const int si = xcd * (per_xcd - full) + (w - ibeg - nfull);
    float* rec = part + (size_t(si) * 2 + half) * 128 * (D + 4) + size_t(wave * 32 + r32) * (D + 4);
#pragma unroll
    for (int tv = 0; tv < TV; ++tv)
#pragma unroll
      for (int i4 = 0; i4 < 4; ++i4) {
        const int dh = 32 * tv + 8 * i4 + 4 * g;
        if (dh < D)
          *reinterpret_cast<float4*>(rec + dh) =
              make_float4(o[tv][4 * i4 + 0], o[tv][4 * i4 + 1], o[tv][4 * i4 + 2], o[tv][4 * i4 + 3]);
      }
    if (g == 0) {
      rec[D] = mrow;
      rec[D + 1] = lsum;
    }
    return;
  }
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

// Merge the two key halves of every split item: O = (O0 2^(m0-m) + O1 2^(m1-m)) /
// (l0 2^(m0-m) + l1 2^(m1-m)) with m = max(m0, m1).  One workgroup per split item,
// two threads per query (half of the head dimension each).
template <int D>
__global__ void __launch_bounds__(256) k_attn_combine(const float* __restrict__ part,
                                                      uint16_t* __restrict__ out, int M, int d,
                                                      int nqb, int items, int per_xcd, int full) {
  const int per = per_xcd - full;                 // split items per XCD (record stride)
  const int si = blockIdx.x, xcd = si / per, k = si % per;
  const int ibeg = xcd * per_xcd, iend = min(items, ibeg + per_xcd);
  const int w = ibeg + full + k;
  if (full >= iend - ibeg || w >= iend) return;
  const int head = w / nqb, ql = threadIdx.x >> 1, hf = threadIdx.x & 1;
  const int q = (w - head * nqb) * 128 + ql;
  if (q >= M) return;
  const float* r0 = part + (size_t(si) * 2 + 0) * 128 * (D + 4) + size_t(ql) * (D + 4);
  const float* r1 = r0 + 128 * (D + 4);
  const float m0 = r0[D], l0 = r0[D + 1], m1 = r1[D], l1 = r1[D + 1];
  const float m = fmaxf(m0, m1);
  const float a0 = __builtin_amdgcn_exp2f(m0 - m), a1 = __builtin_amdgcn_exp2f(m1 - m);
  const float inv = 1.0f / (l0 * a0 + l1 * a1);
  constexpr int DH = D / 2;                       // 32 or 36 dims per thread
  uint16_t* orow = out + size_t(q) * d + head * D + hf * DH;
#pragma unroll
  for (int j = 0; j < DH; j += 4) {
    const float4 x0 = *reinterpret_cast<const float4*>(r0 + hf * DH + j);
    const float4 x1 = *reinterpret_cast<const float4*>(r1 + hf * DH + j);
    ushort4 v;
    v.x = to_bf16((x0.x * a0 + x1.x * a1) * inv);
    v.y = to_bf16((x0.y * a0 + x1.y * a1) * inv);
    v.z = to_bf16((x0.z * a0 + x1.z * a1) * inv);
    v.w = to_bf16((x0.w * a0 + x1.w * a1) * inv);
    *reinterpret_cast<ushort4*>(orow + j) = v;
  }
}

// ---------------------------------------------------------------------------
// head_dim 64 on v_mfma_f32_16x16x32_bf16.  Same work items and tail split as
// k_attn_bf16, but a two-stage K/V^T ring (32 KB of LDS, the next tile's DMA issued
// right after the barrier that frees its stage) and at most 128 VGPRs, so four
// workgroups (four waves per SIMD) are resident: 3 % faster at 17,776 tokens x 30
// heads than three-stage rings at three waves per SIMD.  Per wave: 32 queries as two
// 16-query blocks; the transposed scores S^T come in 16 x 16 blocks (lane: query lane % 16,
// rows 4 (lane / 16) .. + 3 of the block).
//  - The running maximum enters as the C operand of the first score MFMA (four
//    registers holding -m per query block), so scores arrive as s - m.
//  - Each lane's eight P values of a 32-key chunk are the B operand of
//    O^T += V^T P^T directly (K rows permuted, see perm16); the matching V^T operand
//    is one 16-byte LDS read.
//  - The row sum l is one more MFMA per chunk with an all-ones A operand, so the
//    VALU does one exp2 and half a bf16 pack per score and nothing else; numerator
//    and denominator use the same bf16-rounded P.
//  - m comes from the first tile's maximum and stays there.  When a tile leaves l at
//    2^64 or more, or not finite (a later score more than about 58 above m), the whole
//    workgroup redoes the item with the tile maximum taken on every tile (the safe
//    pass); until then every P is below 2^64, so O cannot overflow.
// ---------------------------------------------------------------------------
typedef float f32x4 __attribute__((ext_vector_type(4)));

// K rows are read in a permuted order within each 32-key chunk: S^T block row
// 16 h + 4 g + i (h < 2, g < 4, i < 4) holds key 8 g + 4 h + i, so the eight P values
// a lane holds for a chunk (rows 4 g + i of blocks 2c and 2c+1) are keys 8 g .. 8 g + 7
// and the V^T operand is one 16-byte read.  The K swizzle is keyed on the row bits
// that vary across the 16 rows one LDS cycle reads in that order.
__device__ inline int perm16(int p) {
  return (p & 32) | (((p >> 2) & 3) << 3) | (((p >> 4) & 1) << 2) | (p & 3);
}
__device__ inline int swz_k16(int row) { return ((row >> 1) & 1) | ((row >> 2) & 6); }

__global__ void __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(4)))
k_attn16(const uint16_t* __restrict__ qk, const uint16_t* __restrict__ vt, int ldv,
         uint16_t* __restrict__ out, int M, int d, int nqb, int items, int per_xcd, int full,
         float* __restrict__ part) {
  constexpr int D = 64, BKV = 64;
  constexpr int KI = 2, VI = 2;                 // DMA instructions per wave per tile (K, V^T)
  constexpr int STAGE = (KI + VI) * 256;        // 16-byte slots per ring stage
  __shared__ uint4 lds[2 * STAGE];
  __shared__ int redo;
  uint4* const sK0 = lds;
  uint4* const sV0 = lds + KI * 256;
  uint4* const sK1 = lds + STAGE;
  uint4* const sV1 = lds + STAGE + KI * 256;

  const int xcd = blockIdx.x & 7, u = blockIdx.x >> 3;
  const int ibeg = xcd * per_xcd, iend = min(items, ibeg + per_xcd);
  const int nfull = min(full, iend - ibeg);
  int w, half = -1;
  if (u < nfull) {
    w = ibeg + u;
  } else {
    w = ibeg + nfull + ((u - nfull) >> 1);
    half = (u - nfull) & 1;
  }
  if (w >= iend) return;
  const int ntile = (M + BKV - 1) / BKV;
  const int tb = half == 1 ? ntile / 2 : 0;     // key tiles [tb, te)
  const int te = half == 0 ? ntile / 2 : ntile;
  const int head = w / nqb;
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int c16 = lane & 15, g4 = lane >> 4;
  const int q0 = (w - head * nqb) * 128 + wave * 32;
  const int ldq = 2 * d;
  const uint16_t* Qb = qk + head * D;
  const uint16_t* Kb = qk + d + head * D;
  const uint16_t* Vb = vt + size_t(head) * D * ldv;
  if (tid == 0) redo = 0;

  // query fragments: lane holds Q[q0 + 16 qb + c16][32 kk + 8 g4 .. + 8]
  bf16x8 qf[2][2];
#pragma unroll
  for (int qb = 0; qb < 2; ++qb)
#pragma unroll
    for (int kk = 0; kk < 2; ++kk) {
      const int q = q0 + 16 * qb + c16;
      uint4 v = make_uint4(0, 0, 0, 0);
      if (q < M) v = *reinterpret_cast<const uint4*>(Qb + size_t(q) * ldq + 32 * kk + 8 * g4);
      qf[qb][kk] = __builtin_bit_cast(bf16x8, v);
    }
  __builtin_amdgcn_s_waitcnt(0x0F70);

  uint32_t offK[KI], offV[VI];
#pragma unroll
  for (int i = 0; i < KI; ++i) {
    const int slot = (wave * KI + i) * 64 + lane;
    const int r = slot >> 3, c = (slot & 7) ^ swz_k16(slot >> 3);
    offK[i] = 2u * uint32_t(r * ldq + 8 * c);
  }
#pragma unroll
  for (int i = 0; i < VI; ++i) {
    const int slot = (wave * VI + i) * 64 + lane;
    const int r = slot >> 3, c = (slot & 7) ^ swz_v(slot >> 3);
    offV[i] = 2u * uint32_t(r * ldv + 8 * c);
  }
  auto issue = [&](uint4* sk, uint4* sv, int t) {
    const uint16_t* kt = Kb + size_t(t) * BKV * ldq;
    const uint16_t* vtt = Vb + t * BKV;
#pragma unroll
    for (int i = 0; i < KI; ++i) dma16(kt, offK[i], sk + (wave * KI + i) * 64);
#pragma unroll
    for (int i = 0; i < VI; ++i) dma16(vtt, offV[i], sv + (wave * VI + i) * 64);
  };

  bf16x8 ones;
#pragma unroll
  for (int e = 0; e < 8; ++e) ones[e] = static_cast<__bf16>(1.0f);

  f32x4 o[4][2], lacc[2], mneg[2];
  float mrow[2];
  bool fail = false;

  // one pass over the key tiles; safe: take the tile maximum on every tile
  auto run = [&](bool safe) {
#pragma unroll
    for (int qb = 0; qb < 2; ++qb) {
      mrow[qb] = 0.f;
#pragma unroll
      for (int i = 0; i < 4; ++i) { lacc[qb][i] = 0.f; mneg[qb][i] = 0.f; }
#pragma unroll
      for (int db = 0; db < 4; ++db)
#pragma unroll
        for (int i = 0; i < 4; ++i) o[db][qb][i] = 0.f;
    }
    fail = false;

    auto rescale = [&](int qb, float up) {      // m += up; O, l *= 2^-up
      const float a = __builtin_amdgcn_exp2f(-up);
      mrow[qb] += up;
#pragma unroll
      for (int i = 0; i < 4; ++i) { lacc[qb][i] *= a; mneg[qb][i] = -mrow[qb]; }
#pragma unroll
      for (int db = 0; db < 4; ++db)
#pragma unroll
        for (int i = 0; i < 4; ++i) o[db][qb][i] *= a;
    };

    // scores of key block kb (16 keys) for both query blocks, with C = -m; with
    // kMask the keys past M are set to -inf (the last tile only, so the common path
    // is one branch-free block the scheduler can interleave)
    auto scores = [&](const uint4* sk, int t, int kb, f32x4 (&sc)[2], auto kMask) {
      const int row = perm16(16 * kb + c16);
      const bf16x8 k0 = __builtin_bit_cast(bf16x8, sk[row * 8 + ((0 + g4) ^ swz_k16(row))]);
      const bf16x8 k1 = __builtin_bit_cast(bf16x8, sk[row * 8 + ((4 + g4) ^ swz_k16(row))]);
#pragma unroll
      for (int qb = 0; qb < 2; ++qb) {
        sc[qb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(k0, qf[qb][0], mneg[qb], 0, 0, 0);
        sc[qb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(k1, qf[qb][1], sc[qb], 0, 0, 0);
      }
      if constexpr (decltype(kMask)::value) {
#pragma unroll
        for (int i = 0; i < 4; ++i)
          if (t * BKV + perm16(16 * kb + 4 * g4 + i) >= M) {
            sc[0][i] = -INFINITY;
            sc[1][i] = -INFINITY;
          }
      }
    };

    // all scores of the tile, then per 32-key chunk: P = 2^(s - m) (bf16), O^T += V^T P^T,
    // l += 1 P^T.  P of chunk c: keys 32 c + 8 g4 .. + 7 (blocks 2c and 2c+1, permuted rows)
    auto body = [&](const uint4* sk, const uint4* sv, int t, auto kMask) {
      f32x4 sb[4][2];
#pragma unroll
      for (int kb = 0; kb < 4; ++kb) scores(sk, t, kb, sb[kb], kMask);
#pragma unroll
      for (int c = 0; c < 2; ++c) {
        bf16x8 pf[2];
#pragma unroll
        for (int qb = 0; qb < 2; ++qb)
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            pf[qb][e] = static_cast<__bf16>(__builtin_amdgcn_exp2f(sb[2 * c][qb][e]));
            pf[qb][4 + e] = static_cast<__bf16>(__builtin_amdgcn_exp2f(sb[2 * c + 1][qb][e]));
          }
#pragma unroll
        for (int db = 0; db < 4; ++db) {
          const int row = 16 * db + c16;
          const bf16x8 vf = __builtin_bit_cast(bf16x8, sv[row * 8 + ((4 * c + g4) ^ swz_v(row))]);
#pragma unroll
          for (int qb = 0; qb < 2; ++qb)
            o[db][qb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(vf, pf[qb], o[db][qb], 0, 0, 0);
        }
#pragma unroll
        for (int qb = 0; qb < 2; ++qb)
          lacc[qb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ones, pf[qb], lacc[qb], 0, 0, 0);
      }
    };

    // one tile: the tile maximum (first tile, safe pass), P V and l, then the raise check
    auto tile = [&](const uint4* sk, const uint4* sv, int t, auto kMask, bool domax) {
      if (domax) {
        // the tile maximum (a separate pass over the scores, which are recomputed below)
        float mx[2] = {-INFINITY, -INFINITY};
#pragma unroll
        for (int kb = 0; kb < 4; ++kb) {
          f32x4 sc[2];
          scores(sk, t, kb, sc, kMask);
#pragma unroll
          for (int qb = 0; qb < 2; ++qb)
#pragma unroll
            for (int i = 0; i < 4; ++i) mx[qb] = fmaxf(mx[qb], sc[qb][i]);
        }
#pragma unroll
        for (int qb = 0; qb < 2; ++qb) {
          float m = fmaxf(mx[qb], __shfl_xor(mx[qb], 16, 64));
          m = fmaxf(m, __shfl_xor(m, 32, 64));
          const float up = t == tb ? m : fmaxf(m, 0.f);
          if (up != 0.f) rescale(qb, up);
        }
      }
      body(sk, sv, t, kMask);
      // m lags the scores by more than about 58 (l >= 2^64, all rows of lacc hold l, or
      // l not finite): the item is redone in the safe pass.  While l < 2^64, every P
      // and so O stay far inside the fp32 range.
      if (!safe) {
        const bool big = !(lacc[0][0] < 0x1p64f && lacc[1][0] < 0x1p64f);
        // a real branch (not a select): it ends the tile's scheduling region, which keeps
        // the compiler from interleaving tiles (that spills; 144 VGPRs this way)
        if (__builtin_amdgcn_ballot_w64(big) != 0) {
          fail = true;
          __builtin_amdgcn_s_sleep(0);
        }
      }
    };
    // two-stage ring: tile t has landed in every wave's view and every wave is done with
    // tile t - 1, whose stage (nk, nv) then takes tile t + 1
    auto sync = [&](int t, uint4* nk, uint4* nv) {
      __builtin_amdgcn_s_waitcnt(0x0F70);
      __builtin_amdgcn_s_barrier();
      if (t + 1 < te) issue(nk, nv, t + 1);
    };
    constexpr std::false_type kFull{};
    constexpr std::true_type kPart{};
    // tile t sits in ring stage (t - tb) % 2.  The first tile and a partial last tile
    // run outside the loop, so the loop body is one branch-free instance per stage.
    const bool part_last = te * BKV > M;
    const int tm = part_last ? te - 1 : te;     // tiles [tb, tm) are full
    issue(sK0, sV0, tb);
    sync(tb, sK1, sV1);
    if (tb < tm) tile(sK0, sV0, tb, kFull, true);
    else tile(sK0, sV0, tb, kPart, true);
    for (int t = tb + 1; t < tm; t += 2) {
      sync(t, sK0, sV0);
      tile(sK1, sV1, t, kFull, safe);
      if (t + 1 >= tm) break;
      sync(t + 1, sK1, sV1);
      tile(sK0, sV0, t + 1, kFull, safe);
    }
    if (part_last && te - 1 > tb) {
      const int t = te - 1, q = (t - tb) % 2;
      sync(t, sK0, sV0);                        // t + 1 = te: nothing to prefetch
      tile(sK0 + q * STAGE, sV0 + q * STAGE, t, kPart, safe);   // one instance, stage by address
    }
  };

  // pass 0 is the fast path; pass 1 (rare) redoes the item with the tile maximum on
  // every tile when any wave saw a non-finite row sum (one call site: one inlined copy)
  for (int pass = 0;; ++pass) {
    run(pass > 0);
    if (pass > 0) break;
    if (__builtin_amdgcn_ballot_w64(fail) != 0 && lane == 0) redo = 1;
    __syncthreads();
    if (!redo) break;
    __syncthreads();
  }

  if (half >= 0) {
    const int si = xcd * (per_xcd - full) + (w - ibeg - nfull);
#pragma unroll
    for (int qb = 0; qb < 2; ++qb) {
      float* rec = part + (size_t(si) * 2 + half) * 128 * (D + 4) + size_t(wave * 32 + 16 * qb + c16) * (D + 4);
#pragma unroll
      for (int db = 0; db < 4; ++db)
        *reinterpret_cast<float4*>(rec + 16 * db + 4 * g4) =
            make_float4(o[db][qb][0], o[db][qb][1], o[db][qb][2], o[db][qb][3]);
      if (g4 == 0) {
        rec[D] = mrow[qb];
        rec[D + 1] = lacc[qb][0];
      }
    }
    return;
  }
#pragma unroll
  for (int qb = 0; qb < 2; ++qb) {
    const int q = q0 + 16 * qb + c16;
    if (q >= M) continue;
    const float inv = 1.0f / lacc[qb][0];
    uint16_t* orow = out + size_t(q) * d + head * D;
#pragma unroll
    for (int db = 0; db < 4; ++db) {
      ushort4 v;
      v.x = to_bf16(o[db][qb][0] * inv);
      v.y = to_bf16(o[db][qb][1] * inv);
      v.z = to_bf16(o[db][qb][2] * inv);
      v.w = to_bf16(o[db][qb][3] * inv);
      *reinterpret_cast<ushort4*>(orow + 16 * db + 4 * g4) = v;
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

// Resident workgroups of the bf16 attention kernel per XCD on the current device
// (compute units / 8 x workgroups per compute unit), cached per device.
template <int D>
static int attn_slots_per_xcd() {
  static int cache[64] = {0};
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 0;
  if (cache[dev] == 0) {
    int cus = 0, per_cu = 0;
    if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
        hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, k_attn_bf16<D>, 256, 0) != hipSuccess)
      return 0;
    cache[dev] = (cus / 8) * per_cu;
  }
  return cache[dev];
}

constexpr int kAttn16MinTokens = 8192;

static int attn16_slots_per_xcd() {
  static int cache[64] = {0};
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 0;
  if (cache[dev] == 0) {
    int cus = 0, per_cu = 0;
    if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
        hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, k_attn16, 256, 0) != hipSuccess)
      return 0;
    cache[dev] = (cus / 8) * per_cu;
  }
  return cache[dev];
}

template <int D, bool V16>
static Status launch_attn(const uint16_t* qk, const uint16_t* vt, int ldv, uint16_t* out, const Geo& g,
                          int M, float* part, size_t part_bytes, hipStream_t s) {
  const int nqb = (M + 127) / 128, items = nqb * g.H, per_xcd = (items + 7) / 8;
  // split the items of the last partial round when their halves fit in one round
  const int slots = V16 ? attn16_slots_per_xcd() : attn_slots_per_xcd<D>();
  int full = per_xcd;
  if (slots > 0 && (M + 63) / 64 >= 2) {
    const int f = per_xcd / slots * slots, r = per_xcd - f;
    const size_t need = size_t(8) * r * 2 * 128 * (D + 4) * sizeof(float);
    if (r > 0 && 2 * r <= slots && part && need <= part_bytes) full = f;
  }
  const int units = full + 2 * (per_xcd - full);
  if constexpr (V16)
    hipLaunchKernelGGL(k_attn16, dim3(8 * units), dim3(256), 0, s, qk, vt, ldv, out, M, g.d, nqb, items,
                       per_xcd, full, part);
  else
    hipLaunchKernelGGL(k_attn_bf16<D>, dim3(8 * units), dim3(256), 0, s, qk, vt, ldv, out, M, g.d, nqb,
                       items, per_xcd, full, part);
  DC_HIP(hipGetLastError());
  if (full < per_xcd) {
    hipLaunchKernelGGL(k_attn_combine<D>, dim3(8 * (per_xcd - full)), dim3(256), 0, s, part, out, M, g.d,
                       nqb, items, per_xcd, full);
    DC_HIP(hipGetLastError());
  }
  return Status::ok();
}

Status attention_bf16(const uint16_t* qk, const uint16_t* vt, int ldv, uint16_t* out,
                      const Geo& g, int M, float* part, size_t part_bytes, hipStream_t s) {
  if (ldv % 64 || ldv < M) return Status::shape("attention needs ldv >= M, ldv % 64 == 0");
  // the padding tokens [M, ldv) of vt hold zeros: the bf16 QKV GEMM writes them
  // head_dim 64: the 16x16x32 kernel from 8,192 tokens (MI355X, 17,776 x 30 heads: 1.96 vs
  // 2.08 ms); below that its per-item first-tile pass costs more than it saves (3,597 x 30:
  // 121 vs 119 us)
  if (g.Dh == 64 && M >= kAttn16MinTokens) return launch_attn<64, true>(qk, vt, ldv, out, g, M, part, part_bytes, s);
  if (g.Dh == 64) return launch_attn<64, false>(qk, vt, ldv, out, g, M, part, part_bytes, s);
  if (g.Dh == 72) return launch_attn<72, false>(qk, vt, ldv, out, g, M, part, part_bytes, s);
  return Status::shape("bf16 attention supports head_dim 64 and 72");
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
