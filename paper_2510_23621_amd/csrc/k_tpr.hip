// Edge tensor product of Eq. 26 with the last radial layer computed in place,
// fused with the receiver neighbour sum; and its vector-Jacobian product.
//
//   R[e][p][k]  = sum_j a3[e][j] W3[j][p K + k]                 (last radial layer)
//   At[i][p][m3][k] = inv_c * sum_{e: rcv_e = i} R[e][p][k]
//                     * sum_{m1,m2} C^{lo}_{lh ly}[m1][m2][m3] h[src_e][lh,m1][k] Y[e][ly,m2]
//
// R is never stored: for a K = 128 model with ten paths it would be 5 KB per
// edge each way. One wave owns a (receiver, 16-channel tile) pair and walks
// the receiver's edges (CSR order) in tiles of 16. For each tile it forms R
// with FP32 MFMA (v_mfma_f32_16x16x4_f32; lane l supplies A[l%16][l/16] and
// B[l/16][l%16], result register r holds D[4(l/16)+r][l%16]): rows are the
// tile's edges, columns the wave's channels. Lane l therefore holds R for
// channel l%16 and the four edges 4(l/16)..4(l/16)+3, and contracts exactly
// those edges; the four lane groups are summed by a fixed butterfly at the
// end of the receiver, so the result does not depend on scheduling.
//
// A block is a few waves on as many receivers, sharing one channel tile; the
// tile's slice of W3 (64 x P x 16 floats) sits in LDS for the block's life,
// and each wave stages the Y rows of its current edge tile in LDS.
#include <algorithm>

#include "mace_internal.h"
#include "static_loops.h"

namespace mace {

typedef float f4 __attribute__((ext_vector_type(4)));

constexpr int kWPitch = 68;   // LDS row pitch of the W3 slice: 64 + 4 (4 mod 32)
constexpr int kTPitch = 17;   // 16 x 16 transpose tile
constexpr int kYPitch = 20;   // Y tile row: 16 floats + 4 (float4-aligned)
// Launch shape per (l_max, direction): waves per block (all on one channel
// tile) and the waves per SIMD the register budget is cut for. Two 8-wave
// blocks per CU fit the LDS below l = 2 and give four waves per SIMD at 128
// VGPRs; the l = 1 backward needs more registers (dE/dAt of the receiver
// stays live) and runs two 4-wave blocks per CU at 256 (at 168 it spills);
// for l = 2 the W3 slice alone fills half the LDS, and the l = 2 backward
// runs one 4-wave block per CU, one wave per SIMD, so that its state fits the
// whole register file (VGPRs and AGPRs; at two waves per SIMD it spilled
// about 300 bytes per lane to scratch, 1.3x slower). The MFMA phases raise
// the wave's priority so that they issue ahead of the other waves' vector
// work on the SIMD.
// The split-BF16 backward (RM = 2) keeps both layouts of the three W3 parts
// in LDS (120 KB at P = 10): one 8-wave block per CU at l = 1.
template <int LHMAX, bool BWD, int RM = 0>
struct TprShape {
  static constexpr bool split_bwd = BWD && (RM == 2 || RM == 3);
  static constexpr int waves = ((BWD && LHMAX == 1 && !split_bwd) || (BWD && LHMAX == 2)) ? 4 : 8;
  static constexpr int per_simd = (BWD && LHMAX == 2) ? 1 : (LHMAX == 2 ? 2 : ((BWD && LHMAX == 1) ? 2 : 4));
  static constexpr int blocks_per_cu = 4 * per_simd / waves;
};

__device__ __forceinline__ f4 mfma4(float a, float b, f4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, c, 0, 0, 0);
}

// sW[(p*16 + kk)*kWPitch + j] = W3[j][p K + 16 ct + kk]
template <int P>
__device__ __forceinline__ void load_w3_slice(const float* __restrict__ W3, int K, int ct, float* sW) {
  const int PK = P * K;
  for (int idx = threadIdx.x; idx < P * 16 * 64; idx += blockDim.x) {
    const int kk = idx & 15, j = (idx >> 4) & 63, p = idx >> 10;
    sW[(p * 16 + kk) * kWPitch + j] = W3[(size_t)j * PK + p * K + 16 * ct + kk];
  }
}

// MFMA row of the tile that carries edge e0 + rho: rho itself, or with TRP the
// transposed order 4 (rho % 4) + rho / 4, which puts edge e0 + 4 q + (l/16) in
// result register q of lane l (a tile of n edges then needs ceil(n / 4) edge
// iterations per lane instead of min(n, 4)).
template <bool TRP>
__device__ __forceinline__ int tile_edge(int rho) { return TRP ? 4 * (rho & 3) + (rho >> 2) : rho; }

// R of the 16 edges e0 .. e0+15 (edges at or past e_end get R = 0) for the
// wave's channel tile: r[p][q] = R[e0 + 4(l/16) + q][p][16 ct + l%16]
// (R[e0 + 4 q + l/16] with TRP).
// The 64-long reduction runs in the order j = 16 qq + 4 s + c so that every
// lane reads its A operand as four float4.
template <int P, bool TRP = false>
__device__ __forceinline__ void tile_radial(const float* __restrict__ a3, int e0, int e_end,
                                            const float* __restrict__ sW, f4* r) {
  const int l = threadIdx.x & 63;
  const int row = e0 + tile_edge<TRP>(l & 15);
  const float keep = row < e_end ? 1.f : 0.f;
  const f4* arow = reinterpret_cast<const f4*>(a3 + (size_t)min(row, e_end - 1) * 64 + 4 * (l >> 4));
  f4 a[4];
#pragma unroll
  for (int qq = 0; qq < 4; ++qq) a[qq] = arow[4 * qq] * keep;
  const float* wb = sW + (l & 15) * kWPitch + 4 * (l >> 4);
  __builtin_amdgcn_s_setprio(1);
#pragma unroll
  for (int p = 0; p < P; ++p) {
    __builtin_amdgcn_sched_barrier(0);   // B fragments are loaded path by path
    f4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int qq = 0; qq < 4; ++qq) {
      const f4 b = *reinterpret_cast<const f4*>(wb + p * 16 * kWPitch + 16 * qq);
      acc = mfma4(a[qq][0], b[0], acc);
      acc = mfma4(a[qq][1], b[1], acc);
      acc = mfma4(a[qq][2], b[2], acc);
      acc = mfma4(a[qq][3], b[3], acc);
    }
    r[p] = acc;
  }
  __builtin_amdgcn_s_setprio(0);
}

// ---- BF16 radial mode: R = bf16(a3) bf16(W3) and dE/da3 = bf16(dR) bf16(W3)^T
// on v_mfma_f32_16x16x32_bf16 (FP32 accumulation); lane l supplies
// A[l%16][8(l/16)+i] and B[8(l/16)+i][l%16], i = 0..7.
typedef __bf16 bf8v __attribute__((ext_vector_type(8)));
typedef unsigned short us8v __attribute__((ext_vector_type(8)));
constexpr int kWbPitch = 72;   // bf16 per row of the forward slice: 64 + 8 (36 dwords, 4 mod 32)
constexpr int kWtPitch = 24;   // bf16 per row of the transposed slice: 16 + 8 (16-byte aligned)
constexpr int kT2Pitch = 20;   // floats per row of the two-path transpose tile (16-byte aligned)

__device__ __forceinline__ f4 mfma_bf16(us8v a, us8v b, f4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf8v, a), __builtin_bit_cast(bf8v, b), c, 0, 0,
                                                 0);
}
// bfloat16 bits of eight values, rounded to nearest even by the packed
// hardware conversion (for finite values the bits of bf16_bits)
__device__ __forceinline__ us8v to_bf16x8(f4 lo, f4 hi) {
  typedef unsigned u4v_ __attribute__((ext_vector_type(4)));
  const u4v_ w = {bf16_pack2(f2v{lo[0], lo[1]}), bf16_pack2(f2v{lo[2], lo[3]}), bf16_pack2(f2v{hi[0], hi[1]}),
                  bf16_pack2(f2v{hi[2], hi[3]})};
  return __builtin_bit_cast(us8v, w);
}

// Forward slice sWb[(p*16 + kk)*kWbPitch + j] = bf16(W3[j][p K + 16 ct + kk]);
// with `transposed`, also sWt[(p*64 + j)*kWtPitch + kk] (the dE/da3 operand).
template <int P>
__device__ __forceinline__ void load_w3_slice_bf16(const float* __restrict__ W3, int K, int ct,
                                                   unsigned short* sWb, unsigned short* sWt) {
  const int PK = P * K;
  for (int idx = threadIdx.x; idx < P * 16 * 64; idx += blockDim.x) {
    const int kk = idx & 15, j = (idx >> 4) & 63, p = idx >> 10;
    const unsigned short v = bf16_bits(W3[(size_t)j * PK + p * K + 16 * ct + kk]);
    sWb[(p * 16 + kk) * kWbPitch + j] = v;
    if (sWt) sWt[(p * 64 + j) * kWtPitch + kk] = v;
  }
}

// As tile_radial, on BF16 operands: two MFMAs (k = 32 each) per path. The W3
// operands are read kBf16Ahead paths ahead of their MFMAs, so that the LDS
// reads do not stall each path's pair of products.
constexpr int kBf16Ahead = 4;
template <int P, bool TRP = false>
__device__ __forceinline__ void tile_radial_bf16(const float* __restrict__ a3, int e0, int e_end,
                                                 const unsigned short* __restrict__ sWb, f4* r) {
  const int l = threadIdx.x & 63;
  const int row = e0 + tile_edge<TRP>(l & 15);
  const float keep = row < e_end ? 1.f : 0.f;
  const f4* arow = reinterpret_cast<const f4*>(a3 + (size_t)min(row, e_end - 1) * 64 + 8 * (l >> 4));
  const unsigned short* wb = sWb + (l & 15) * kWbPitch + 8 * (l >> 4);
  constexpr int D = kBf16Ahead < P ? kBf16Ahead : P;
  us8v bw[D][2];
  auto load_b = [&](int p, us8v (&b)[2]) {
    b[0] = *reinterpret_cast<const us8v*>(wb + p * 16 * kWbPitch);
    b[1] = *reinterpret_cast<const us8v*>(wb + p * 16 * kWbPitch + 32);
  };
#pragma unroll
  for (int p = 0; p < D; ++p) load_b(p, bw[p]);
  us8v a[2];
#pragma unroll
  for (int ks = 0; ks < 2; ++ks) a[ks] = to_bf16x8(arow[8 * ks] * keep, arow[8 * ks + 1] * keep);
  __builtin_amdgcn_s_setprio(1);
  static_for<0, P>([&](auto PI) {
    constexpr int p = decltype(PI)::value;
    __builtin_amdgcn_sched_barrier(0);
    const us8v b0 = bw[p % D][0], b1 = bw[p % D][1];
    if constexpr (p + D < P) load_b(p + D, bw[p % D]);
    r[p] = mfma_bf16(a[1], b1, mfma_bf16(a[0], b0, f4{0.f, 0.f, 0.f, 0.f}));
  });
  __builtin_amdgcn_s_setprio(0);
}

// ---- Split-BF16 radial layer (FP32-accurate): every FP32 operand x is carried
// as x0 + x1 + x2 with x0 = bf16(x), x1 = bf16(x - x0), x2 = bf16(x - x0 - x1)
// (each difference is exact in FP32, so the three parts hold all 24
// significand bits), and a b = a0 b0 + (a0 b1 + a1 b0) + (a0 b2 + a1 b1 + a2 b0)
// up to terms of relative size 2^-27, on v_mfma_f32_16x16x32_bf16 with FP32
// accumulation: six BF16 MFMAs (16 cycles each) in place of eight FP32 ones
// (32 cycles each) per 16 x 16 x 32 block.
__device__ __forceinline__ void split3(float x, unsigned short& b0, unsigned short& b1, unsigned short& b2) {
  const __bf16 h0 = (__bf16)x;
  const float r1 = x - (float)h0;
  const __bf16 h1 = (__bf16)r1;
  const float r2 = r1 - (float)h1;
  const __bf16 h2 = (__bf16)r2;
  b0 = __builtin_bit_cast(unsigned short, h0);
  b1 = __builtin_bit_cast(unsigned short, h1);
  b2 = __builtin_bit_cast(unsigned short, h2);
}

// split3 of eight values (lo, hi) into the three MFMA operands of their
// parts, two values per conversion: v_cvt_pk_bf16_f32 rounds a pair to nearest
// even and packs it as one operand word (first value in the low half), and the
// rounded values are unpacked by shifts and masks to form the next remainder.
typedef unsigned u4v __attribute__((ext_vector_type(4)));
__device__ __forceinline__ void split3_x8(f4 lo, f4 hi, us8v& a0, us8v& a1, us8v& a2) {
  u4v w0, w1, w2;
#pragma unroll
  for (int h = 0; h < 4; ++h) {
    const f2v x = h < 2 ? f2v{lo[2 * h], lo[2 * h + 1]} : f2v{hi[2 * h - 4], hi[2 * h - 3]};
    unsigned p0, p1, p2;
    split3_pair(x, p0, p1, p2);
    w0[h] = p0;
    w1[h] = p1;
    w2[h] = p2;
  }
  a0 = __builtin_bit_cast(us8v, w0);
  a1 = __builtin_bit_cast(us8v, w1);
  a2 = __builtin_bit_cast(us8v, w2);
}

// The parts of a3[row][32 ks + 8 (l/16) .. +7] from the pre-split rows
// ([E][3][64] bfloat16), zero where keep is false (rows past the tile's end).
__device__ __forceinline__ void load_a3_parts(const unsigned short* __restrict__ a3x, int row, bool keep, int ks,
                                              us8v& a0, us8v& a1, us8v& a2) {
  const int l = threadIdx.x & 63;
  const unsigned short* base = a3x + (size_t)row * 192 + 32 * ks + 8 * (l >> 4);
  const us8v z = {0, 0, 0, 0, 0, 0, 0, 0};
  a0 = keep ? *reinterpret_cast<const us8v*>(base) : z;
  a1 = keep ? *reinterpret_cast<const us8v*>(base + 64) : z;
  a2 = keep ? *reinterpret_cast<const us8v*>(base + 128) : z;
}

// The three parts of the forward slice, part q at sWx + q P 16 kWbPitch, in the
// layout of load_w3_slice_bf16.
template <int P>
__device__ __forceinline__ void load_w3_slice_x3(const float* __restrict__ W3, int K, int ct, unsigned short* sWx) {
  const int PK = P * K;
  constexpr int part = P * 16 * kWbPitch;
  for (int idx = threadIdx.x; idx < P * 16 * 64; idx += blockDim.x) {
    const int kk = idx & 15, j = (idx >> 4) & 63, p = idx >> 10;
    const int o = (p * 16 + kk) * kWbPitch + j;
    split3(W3[(size_t)j * PK + p * K + 16 * ct + kk], sWx[o], sWx[part + o], sWx[2 * part + o]);
  }
}

// tile_radial_x3 below l = 2 (described there)
template <int P, bool PRE = false, bool TRP = false>
__device__ __forceinline__ void tile_radial_x3_chain(const float* __restrict__ a3, int e0, int e_end,
                                                     const unsigned short* __restrict__ sWx, f4* r) {
  constexpr int part = P * 16 * kWbPitch;
  const int l = threadIdx.x & 63;
  const int row = e0 + tile_edge<TRP>(l & 15);
  const float keep = row < e_end ? 1.f : 0.f;
  const int crow = min(row, e_end - 1);
  const f4* arow = reinterpret_cast<const f4*>(a3 + (size_t)crow * 64 + 8 * (l >> 4));
  const unsigned short* wb = sWx + (l & 15) * kWbPitch + 8 * (l >> 4);
#pragma unroll
  for (int p = 0; p < P; ++p) r[p] = f4{0.f, 0.f, 0.f, 0.f};
  __builtin_amdgcn_s_setprio(1);
#pragma unroll
  for (int ks = 0; ks < 2; ++ks) {
    __builtin_amdgcn_sched_barrier(0);
    us8v a0, a1, a2;
    if constexpr (PRE) {
      load_a3_parts(reinterpret_cast<const unsigned short*>(a3), crow, row < e_end, ks, a0, a1, a2);
    } else {
      const f4 lo = arow[8 * ks] * keep, hi = arow[8 * ks + 1] * keep;
      split3_x8(lo, hi, a0, a1, a2);
    }
#pragma unroll
    for (int p = 0; p < P; ++p) {
      __builtin_amdgcn_sched_barrier(0);   // one path's B parts live at a time
      const unsigned short* q = wb + p * 16 * kWbPitch + 32 * ks;
      const us8v b0 = *reinterpret_cast<const us8v*>(q);
      const us8v b1 = *reinterpret_cast<const us8v*>(q + part);
      const us8v b2 = *reinterpret_cast<const us8v*>(q + 2 * part);
      f4 acc = r[p];
      acc = mfma_bf16(a2, b0, acc);
      acc = mfma_bf16(a1, b1, acc);
      acc = mfma_bf16(a0, b2, acc);
      acc = mfma_bf16(a1, b0, acc);
      acc = mfma_bf16(a0, b1, acc);
      r[p] = mfma_bf16(a0, b0, acc);
    }
  }
  __builtin_amdgcn_s_setprio(0);
}

// As tile_radial, FP32-accurate on split BF16 operands: within each K step the
// terms are added from the smallest to the largest.
// PRE: a3 points at the pre-split parts ([E][3][64] bfloat16) instead.
// Below l = 2 (P <= 10, four waves per SIMD at 128 registers) one path's chain
// of six products at a time, only one K step's A parts live; at l = 2 (P = 17,
// two waves per SIMD) both K steps' A parts are loaded first and the paths go
// in pairs (below).
template <int P, bool PRE = false, bool TRP = false>
__device__ __forceinline__ void tile_radial_x3(const float* __restrict__ a3, int e0, int e_end,
                                               const unsigned short* __restrict__ sWx, f4* r) {
  if constexpr (P <= 10) {
    tile_radial_x3_chain<P, PRE, TRP>(a3, e0, e_end, sWx, r);
    return;
  }
  constexpr int part = P * 16 * kWbPitch;
  const int l = threadIdx.x & 63;
  const int row = e0 + tile_edge<TRP>(l & 15);
  const float keep = row < e_end ? 1.f : 0.f;
  const int crow = min(row, e_end - 1);
  const f4* arow = reinterpret_cast<const f4*>(a3 + (size_t)crow * 64 + 8 * (l >> 4));
  const unsigned short* wb = sWx + (l & 15) * kWbPitch + 8 * (l >> 4);
#pragma unroll
  for (int p = 0; p < P; ++p) r[p] = f4{0.f, 0.f, 0.f, 0.f};
  __builtin_amdgcn_s_setprio(1);
  us8v a[2][3];
#pragma unroll
  for (int ks = 0; ks < 2; ++ks) {
    if constexpr (PRE) {
      load_a3_parts(reinterpret_cast<const unsigned short*>(a3), crow, row < e_end, ks, a[ks][0], a[ks][1], a[ks][2]);
    } else {
      const f4 lo = arow[8 * ks] * keep, hi = arow[8 * ks + 1] * keep;
      split3_x8(lo, hi, a[ks][0], a[ks][1], a[ks][2]);
    }
  }
  // Steps s = ks P + p taken in pairs: the next pair's W3 parts are requested
  // before this pair's MFMAs, and the two paths' six-product chains alternate
  // so that neither waits on its own previous product. Each path's products
  // are added in the same order as in a single chain.
  constexpr int NS = 2 * P;   // even: the pairs are (2t, 2t + 1), t < P
  us8v bb[2][2][3];
  auto load_b = [&](int s, us8v (&b)[3]) {
    const int ks = s / P, p = s % P;
    const unsigned short* q = wb + p * 16 * kWbPitch + 32 * ks;
    b[0] = *reinterpret_cast<const us8v*>(q);
    b[1] = *reinterpret_cast<const us8v*>(q + part);
    b[2] = *reinterpret_cast<const us8v*>(q + 2 * part);
  };
  load_b(0, bb[0][0]);
  load_b(1, bb[0][1]);
  static_for<0, P>([&](auto TI) {
    constexpr int t = decltype(TI)::value;
    constexpr int s0 = 2 * t, s1 = 2 * t + 1;
    __builtin_amdgcn_sched_barrier(0);
    if constexpr (s1 + 2 < NS) {
      load_b(s0 + 2, bb[(t + 1) & 1][0]);
      load_b(s1 + 2, bb[(t + 1) & 1][1]);
    }
    constexpr int ks0 = s0 / P, p0 = s0 % P, ks1 = s1 / P, p1 = s1 % P;
    const us8v(&b0)[3] = bb[t & 1][0];
    const us8v(&b1)[3] = bb[t & 1][1];
    f4 x = r[p0], y = r[p1];
    x = mfma_bf16(a[ks0][2], b0[0], x);
    y = mfma_bf16(a[ks1][2], b1[0], y);
    x = mfma_bf16(a[ks0][1], b0[1], x);
    y = mfma_bf16(a[ks1][1], b1[1], y);
    x = mfma_bf16(a[ks0][0], b0[2], x);
    y = mfma_bf16(a[ks1][0], b1[2], y);
    x = mfma_bf16(a[ks0][1], b0[0], x);
    y = mfma_bf16(a[ks1][1], b1[0], y);
    x = mfma_bf16(a[ks0][0], b0[1], x);
    y = mfma_bf16(a[ks1][0], b1[1], y);
    x = mfma_bf16(a[ks0][0], b0[0], x);
    y = mfma_bf16(a[ks1][0], b1[0], y);
    r[p0] = x;
    r[p1] = y;
  });
  __builtin_amdgcn_s_setprio(0);
}

// Split parts in the backward, without row padding: a 16-byte chunk c of row r
// sits at chunk c ^ s(r), so that the 16 lanes of an MFMA operand read hit 16
// distinct 16-byte bank groups. Forward layout: row r = p 16 + kk of 64
// elements (8 chunks of j), s(r) = (r >> 1) & 7. Transposed layout: row
// r = p 64 + j of 16 elements (2 chunks of kk), s(r) = (r >> 3) & 1.
__device__ __forceinline__ int swz_fwd(int r, int c) { return r * 64 + 8 * (c ^ ((r >> 1) & 7)); }
__device__ __forceinline__ int swz_tr(int r, int c) { return r * 16 + 8 * (c ^ ((r >> 3) & 1)); }

template <int P>
__device__ __forceinline__ void load_w3_slices_x3_swz(const float* __restrict__ W3, int K, int ct,
                                                      unsigned short* sWf, unsigned short* sWt) {
  const int PK = P * K;
  constexpr int part = P * 16 * 64;
  for (int idx = threadIdx.x; idx < P * 16 * 64; idx += blockDim.x) {
    const int kk = idx & 15, j = (idx >> 4) & 63, p = idx >> 10;
    unsigned short x0, x1, x2;
    split3(W3[(size_t)j * PK + p * K + 16 * ct + kk], x0, x1, x2);
    const int of = swz_fwd(p * 16 + kk, j >> 3) + (j & 7);
    const int ot = swz_tr(p * 64 + j, kk >> 3) + (kk & 7);
    sWf[of] = x0;
    sWf[part + of] = x1;
    sWf[2 * part + of] = x2;
    sWt[ot] = x0;
    sWt[part + ot] = x1;
    sWt[2 * part + ot] = x2;
  }
}

// tile_radial_x3 on the swizzled forward layout
template <int P>
__device__ __forceinline__ void tile_radial_x3s(const float* __restrict__ a3, int e0, int e_end,
                                                const unsigned short* __restrict__ sWf, f4* r) {
  constexpr int part = P * 16 * 64;
  const int l = threadIdx.x & 63;
  const int row = e0 + (l & 15);
  const float keep = row < e_end ? 1.f : 0.f;
  const f4* arow = reinterpret_cast<const f4*>(a3 + (size_t)min(row, e_end - 1) * 64 + 8 * (l >> 4));
#pragma unroll
  for (int p = 0; p < P; ++p) r[p] = f4{0.f, 0.f, 0.f, 0.f};
  __builtin_amdgcn_s_setprio(1);
#pragma unroll
  for (int ks = 0; ks < 2; ++ks) {
    __builtin_amdgcn_sched_barrier(0);
    const f4 lo = arow[8 * ks] * keep, hi = arow[8 * ks + 1] * keep;
    us8v a0, a1, a2;
    split3_x8(lo, hi, a0, a1, a2);
#pragma unroll
    for (int p = 0; p < P; ++p) {
      __builtin_amdgcn_sched_barrier(0);
      const unsigned short* q = sWf + swz_fwd(p * 16 + (l & 15), 4 * ks + (l >> 4));
      const us8v b0 = *reinterpret_cast<const us8v*>(q);
      const us8v b1 = *reinterpret_cast<const us8v*>(q + part);
      const us8v b2 = *reinterpret_cast<const us8v*>(q + 2 * part);
      f4 acc = r[p];
      acc = mfma_bf16(a2, b0, acc);
      acc = mfma_bf16(a1, b1, acc);
      acc = mfma_bf16(a0, b2, acc);
      acc = mfma_bf16(a1, b0, acc);
      acc = mfma_bf16(a0, b1, acc);
      r[p] = mfma_bf16(a0, b0, acc);
    }
  }
  __builtin_amdgcn_s_setprio(0);
}

// dE/da3 partial on split BF16 operands (dR split per tile, W3 parts from the
// swizzled transposed layout); otherwise as tile_da3_bf16.
template <int P>
__device__ __forceinline__ void tile_da3_x3(const f4* r, const unsigned short* __restrict__ sWt, float* tw,
                                            f4* d3) {
  constexpr int part = P * 16 * 64;
  const int l = threadIdx.x & 63, g = l >> 4, kk = l & 15;
#pragma unroll
  for (int jt = 0; jt < 4; ++jt) d3[jt] = f4{0.f, 0.f, 0.f, 0.f};
  __builtin_amdgcn_s_setprio(1);
#pragma unroll
  for (int ks = 0; ks < (P + 1) / 2; ++ks) {
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int pl = 0; pl < 2; ++pl)
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const int p = 2 * ks + pl;
        tw[(pl * 16 + 4 * g + q) * kT2Pitch + kk] = (p < P) ? r[p < P ? p : 0][q] : 0.f;
      }
    __builtin_amdgcn_wave_barrier();
    const float* src = tw + ((g >> 1) * 16 + kk) * kT2Pitch + 8 * (g & 1);
    const f4 lo = *reinterpret_cast<const f4*>(src), hi = *reinterpret_cast<const f4*>(src + 4);
    __builtin_amdgcn_wave_barrier();
    us8v a0, a1, a2;
    split3_x8(lo, hi, a0, a1, a2);
    const int p = min(2 * ks + (g >> 1), P - 1);   // a missing odd path reads a valid row; its A is zero
#pragma unroll
    for (int jt = 0; jt < 4; ++jt) {
      const unsigned short* q = sWt + swz_tr(p * 64 + 16 * jt + kk, g & 1);
      const us8v b0 = *reinterpret_cast<const us8v*>(q);
      const us8v b1 = *reinterpret_cast<const us8v*>(q + part);
      const us8v b2 = *reinterpret_cast<const us8v*>(q + 2 * part);
      f4 acc = d3[jt];
      acc = mfma_bf16(a2, b0, acc);
      acc = mfma_bf16(a1, b1, acc);
      acc = mfma_bf16(a0, b2, acc);
      acc = mfma_bf16(a1, b0, acc);
      acc = mfma_bf16(a0, b1, acc);
      d3[jt] = mfma_bf16(a0, b0, acc);
    }
  }
  __builtin_amdgcn_s_setprio(0);
}

// dE/da3 partial on BF16 operands: D[e][j] = sum over (p, kk) of
// bf16(dR[e][p][kk]) bf16(W3[j][p K + 16 ct + kk]); the reduction index
// 32 ks + 8 (l/16) + i is path 2 ks + (l/16)/2, channel 8 ((l/16)%2) + i. Each
// pair of dR tiles goes through the wave's transpose buffer tw (2 x 16 x
// kT2Pitch floats) to put the edge on l%16.
template <int P>
__device__ __forceinline__ void tile_da3_bf16(const f4* r, const unsigned short* __restrict__ sWt, float* tw,
                                              f4* d3) {
  const int l = threadIdx.x & 63, g = l >> 4, kk = l & 15;
#pragma unroll
  for (int jt = 0; jt < 4; ++jt) d3[jt] = f4{0.f, 0.f, 0.f, 0.f};
  __builtin_amdgcn_s_setprio(1);
#pragma unroll
  for (int ks = 0; ks < (P + 1) / 2; ++ks) {
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int pl = 0; pl < 2; ++pl)
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const int p = 2 * ks + pl;
        tw[(pl * 16 + 4 * g + q) * kT2Pitch + kk] = (p < P) ? r[p < P ? p : 0][q] : 0.f;
      }
    __builtin_amdgcn_wave_barrier();
    const float* src = tw + ((g >> 1) * 16 + kk) * kT2Pitch + 8 * (g & 1);
    const us8v a = to_bf16x8(*reinterpret_cast<const f4*>(src), *reinterpret_cast<const f4*>(src + 4));
    __builtin_amdgcn_wave_barrier();
    const int p = min(2 * ks + (g >> 1), P - 1);   // a missing odd path reads a valid row; its A is zero
#pragma unroll
    for (int jt = 0; jt < 4; ++jt) {
      const us8v b = *reinterpret_cast<const us8v*>(sWt + (p * 64 + 16 * jt + kk) * kWtPitch + 8 * (g & 1));
      d3[jt] = mfma_bf16(a, b, d3[jt]);
    }
  }
  __builtin_amdgcn_s_setprio(0);
}

// Y rows of the wave's 16-edge tile into LDS: sy[row][m], row pitch kYPitch.
// Lane l moves float4 number l%4 of row l/4.
// The precision study's operand rounding of the edge product (rnd: 0 none,
// 1 bfloat16, 2 binary16, round to nearest even) of the radial weights of a
// tile; the harmonics and the sender features arrive rounded (the host runtime
// rounds those buffers in place).
template <int P>
__device__ __forceinline__ void round_tile(f4* r, int rnd) {
  if (!rnd) return;
#pragma unroll
  for (int p = 0; p < P; ++p)
#pragma unroll
    for (int q = 0; q < 4; ++q) r[p][q] = lowp_round(r[p][q], rnd);
}

__device__ __forceinline__ void stage_y(const float* __restrict__ Y, int e0, int e_end, float* sy) {
  const int l = threadIdx.x & 63;
  const int row = l >> 2, ch = l & 3;
  const int e = min(e0 + row, e_end - 1);
  const f4 v = reinterpret_cast<const f4*>(Y + (size_t)e * 16)[ch];
  *reinterpret_cast<f4*>(sy + row * kYPitch + 4 * ch) = v;
}

__device__ __forceinline__ void read_y(const float* sy, int row, float* y) {
#pragma unroll
  for (int v = 0; v < 4; ++v) {
    const f4 t4 = *reinterpret_cast<const f4*>(sy + row * kYPitch + 4 * v);
    y[4 * v] = t4[0];
    y[4 * v + 1] = t4[1];
    y[4 * v + 2] = t4[2];
    y[4 * v + 3] = t4[3];
  }
}

// Source rows in h of the edges e_first .. e_first + 3 (clamped to the last
// valid edge): the sender itself, or its species-table row through src_map.
__device__ __forceinline__ void sender_rows(const int* __restrict__ snd, const int* __restrict__ src_map,
                                            int e_first, int e_end, int* srcq) {
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const int s = snd[min(e_first + q, e_end - 1)];
    srcq[q] = src_map ? src_map[s] : s;
  }
}

template <int DIN>
__device__ __forceinline__ void load_h_row(const float* __restrict__ h, int src, int K, int k, float* hv) {
#pragma unroll
  for (int c = 0; c < DIN; ++c) hv[c] = h[((size_t)src * DIN + c) * K + k];
}

// RM, the operands of the last radial layer: 0 FP32, 1 BF16, 2 split BF16 (FP32-accurate),
// 3 split BF16 with a3 arriving as its three parts (the a3 argument then points at
// [E][3][64] bfloat16 written by the edge prologue)
// KC: K as a compile-time constant (0: the argument K), so that the sender
// rows' component strides become immediate load offsets.
template <int LHMAX, int RM, int NW = TprShape<LHMAX, false>::waves, int KC = 0>
__global__ void __launch_bounds__(64 * NW)
__attribute__((amdgpu_waves_per_eu(TprShape<LHMAX, false>::per_simd, TprShape<LHMAX, false>::per_simd)))
tpr_fwd_kernel(
    int N, int K_arg, const int* __restrict__ rcv_off, const int* __restrict__ snd, const int* __restrict__ src_map,
    const float* __restrict__ a3, const float* __restrict__ W3, const float* __restrict__ Y,
    const float* __restrict__ h, float inv_c, float* __restrict__ At, int rnd) {
  const int K = KC ? KC : K_arg;
  constexpr int P = path_count(LHMAX);
  constexpr int MID = mid_count(LHMAX);
  constexpr int DIN = (LHMAX + 1) * (LHMAX + 1);
  constexpr bool SPLIT = RM == 2 || RM == 3;
  constexpr int kSlice = RM == 1 ? (P * 16 * kWbPitch + 1) / 2
                        : (SPLIT ? (3 * P * 16 * kWbPitch + 1) / 2 : P * 16 * kWPitch);   // floats
  __shared__ __align__(16) float sW[kSlice];
  __shared__ float sY[NW][16 * kYPitch];
  const int ct = blockIdx.y;
  if constexpr (RM == 1) load_w3_slice_bf16<P>(W3, K, ct, reinterpret_cast<unsigned short*>(sW), nullptr);
  else if constexpr (SPLIT) load_w3_slice_x3<P>(W3, K, ct, reinterpret_cast<unsigned short*>(sW));
  else load_w3_slice<P>(W3, K, ct, sW);
  __syncthreads();
  const int l = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int g = l >> 4;
  const int k = 16 * ct + (l & 15);
  float* sy = sY[w];
  for (int i = blockIdx.x * NW + w; i < N; i += gridDim.x * NW) {
    float acc[MID];
#pragma unroll
    for (int c = 0; c < MID; ++c) acc[c] = 0.f;
    const int e_beg = rcv_off[i], e_end = rcv_off[i + 1];
    for (int e0 = e_beg; e0 < e_end; e0 += 16) {
      // sender rows of the lane's four edges (edges past e_end carry R = 0),
      // requested before the radial MFMAs so that their latency is hidden
      // edge e0 + 4 q + g is the lane's q-th (transposed tile rows)
      int srcq[4];
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const int sq = snd[min(e0 + 4 * q + g, e_end - 1)];
        srcq[q] = src_map ? src_map[sq] : sq;
      }
      stage_y(Y, e0, e_end, sy);
      f4 r[P];
      if constexpr (RM == 1) tile_radial_bf16<P, true>(a3, e0, e_end, reinterpret_cast<const unsigned short*>(sW), r);
      else if constexpr (SPLIT)
        tile_radial_x3<P, RM == 3, true>(a3, e0, e_end, reinterpret_cast<const unsigned short*>(sW), r);
      else tile_radial<P, true>(a3, e0, e_end, sW, r);
      round_tile<P>(r, rnd);
      // a tile of n edges fills registers q < ceil(n / 4) (edges past e_end
      // carry R = 0); the scheduling barrier keeps one edge's operands live at
      // a time, and the next edge's h row is requested while this one is contracted
      const int nq = min(4, (e_end - e0 + 3) >> 2);
      // the sender rows of edges q and q + 1 (in flight); at l = 2 the two
      // buffers alternate, below it the next row is copied over (fewer registers)
      constexpr bool ALT = LHMAX == 2;
      float hb[2][DIN];
      load_h_row<DIN>(h, srcq[0], K, k, hb[0]);
      static_for<0, 4>([&](auto QI) {
        constexpr int q = decltype(QI)::value;
        constexpr int cur = ALT ? (q & 1) : 0, nxt = ALT ? ((q + 1) & 1) : 1;
        __builtin_amdgcn_sched_barrier(0);
        if (q >= nq) return;
        const int row = 4 * q + g;   // the lane's edge e0 + row
        if constexpr (q < 3) load_h_row<DIN>(h, srcq[q + 1], K, k, hb[nxt]);
        const float(&hv)[DIN] = hb[cur];
        float y[16];
        read_y(sy, row, y);
        for_paths<LHMAX>([&](auto tag) {
          using T = decltype(tag);
          constexpr int lh = T::lh, ly = T::ly, lo = T::lo;
          // R folded into the sender features (R h[m1]) and the coefficients'
          // magnitudes into the harmonics (|C| Y[m2], one product per distinct
          // pair of the path): acc[m3] += (+-R h[m1]) (|C| Y[m2]), one
          // multiply-add per coefficient with its sign on an operand
          using C = mt::CG<lh, ly, lo>;
          const float rv = r[T::index][q];
          float hr[2 * lh + 1];
#pragma unroll
          for (int m = 0; m < 2 * lh + 1; ++m) hr[m] = rv * hv[lh * lh + m];
          float yc[C::nyc];
          C::each_yc([&](int m2, float av, int u) { yc[u] = av * y[ly * ly + m2]; });
          C::each_ys([&](int m1, int m2, int m3, int sg, int u) {
            acc[T::offset + m3] = __builtin_fmaf(sg > 0 ? hr[m1] : -hr[m1], yc[u], acc[T::offset + m3]);
          });
        });
        if constexpr (!ALT && q < 3) {
#pragma unroll
          for (int c = 0; c < DIN; ++c) hb[0][c] = hb[1][c];
        }
      });
    }
    // lane groups 0+1 and 2+3, then the two pairs: every lane ends with the same sum
#pragma unroll
    for (int c = 0; c < MID; ++c) {
      acc[c] += __shfl_xor(acc[c], 16);
      acc[c] += __shfl_xor(acc[c], 32);
    }
#pragma unroll
    for (int c = 0; c < MID; ++c)
      if ((c & 3) == g) At[((size_t)i * MID + c) * K + k] = acc[c] * inv_c;
  }
}

// One halving step of group_reduce16: lanes with bit HALF set keep the upper
// half of v[0 .. 2 HALF) and receive their partner's, the others the lower.
template <int HALF>
__device__ __forceinline__ void reduce_stage(float* v, int lane) {
  const bool hi = lane & HALF;
#pragma unroll
  for (int q = 0; q < HALF; ++q) {
    const float send = hi ? v[q] : v[q + HALF];
    const float keep = hi ? v[q + HALF] : v[q];
    v[q] = keep + __shfl_xor(send, HALF);
  }
}

// Sum of 16 values over the 16 lanes of a lane group: afterwards lane l holds
// the total of index l%16.
__device__ __forceinline__ float group_reduce16(float* v, int lane) {
  reduce_stage<8>(v, lane);
  reduce_stage<4>(v, lane);
  reduce_stage<2>(v, lane);
  reduce_stage<1>(v, lane);
  return v[0];
}

// VJP of tpr_fwd. Given g = dE/dAt, per edge e (receiver i) and channel k,
// with G_p[m1][m2] = sum_m3 C g[i][p][m3] (per receiver and channel, kept in
// LDS for the receiver's edges, one value per coupled (m1, m2) pair),
// Bm_p[m2] = sum_m1 G_p[m1][m2] h[m1] and Dm_p[m1] = sum_m2 G_p[m1][m2] Y[m2]:
//   dR[e][p][k]    = inv_c sum_m2 Bm_p[m2] Y[m2]
//   dY[e][ly,m2]  += inv_c sum_k sum_p R Bm_p[m2]                    (channel-tile partial)
//   Q[e][lh,m1][k] = inv_c sum_p R Dm_p[m1]                          (per-edge sender gradient)
//   da3[e][j]     += sum_{p,k} dR[e][p][k] W3[j][p K + k]           (channel-tile partial)
// The partials of channel tile ct go to dYp[ct][e][16] and da3p[ct][e][64];
// their sum over tiles (fixed order) is taken by the hidden-layer backward.
// G_p is formed once per receiver (GF) where its table fits beside the
// weight slice at the kernel's occupancy; otherwise each edge contracts C
// with g directly (product form C (g h), C (g Y)).
template <int LHMAX, int RM>
constexpr bool tpr_bwd_gform() { return LHMAX == 0 || (LHMAX == 1 && RM == 0); }

// RM as in tpr_fwd_kernel (split BF16 for l <= 1 only: at l = 2 the two
// layouts of the parts do not fit the LDS). This body keeps the forward's lane
// layout (one channel, four edges per lane); the split-BF16 backward at
// l_h <= 1 uses tpr_bwd_edge_lanes below.
template <int LHMAX, int RM, int NW>
__device__ __forceinline__ void tpr_bwd_channel_lanes(
    int N, int K, int E, const int* __restrict__ rcv_off, const int* __restrict__ snd,
    const int* __restrict__ src_map, const float* __restrict__ a3, const float* __restrict__ W3,
    const float* __restrict__ Y, const float* __restrict__ h, float inv_c, const float* __restrict__ dAt,
    float* __restrict__ dYp, float* __restrict__ Q, float* __restrict__ da3p, int rnd) {
  constexpr int P = path_count(LHMAX);
  constexpr int MID = mid_count(LHMAX);
  constexpr int DIN = (LHMAX + 1) * (LHMAX + 1);
  static_assert(RM != 2 || LHMAX <= 1, "split-BF16 backward for l <= 1");
  static_assert(RM != 3, "pre-split a3: edge-lane backward only");
  constexpr bool RB = RM == 1;
  constexpr int kSlice = RM == 1 ? (P * 16 * kWbPitch + P * 64 * kWtPitch + 1) / 2
                        : (RM == 2 ? 3 * P * 16 * 64 : P * 16 * kWPitch);   // floats
  __shared__ __align__(16) float sW[kSlice];
  __shared__ float sY[NW][16 * kYPitch];
  __shared__ __align__(16) float sT[NW][RM != 0 ? 2 * 16 * kT2Pitch : 16 * kTPitch];
  constexpr bool GF = tpr_bwd_gform<LHMAX, RM>();
  constexpr int NPAIR = PairCount<LHMAX>::value;
  __shared__ float sG[GF ? NW : 1][GF ? NPAIR * 16 : 1];   // [pair][channel]
  unsigned short* sWb = reinterpret_cast<unsigned short*>(sW);
  unsigned short* sWt = sWb + (RM == 2 ? 3 * P * 16 * 64 : P * 16 * kWbPitch);
  const int ct = blockIdx.y;
  if constexpr (RM == 1) load_w3_slice_bf16<P>(W3, K, ct, sWb, sWt);
  else if constexpr (RM == 2) load_w3_slices_x3_swz<P>(W3, K, ct, sWb, sWt);
  else load_w3_slice<P>(W3, K, ct, sW);
  __syncthreads();
  const int l = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int g = l >> 4, kk = l & 15;
  const int k = 16 * ct + kk;
  float* sy = sY[w];
  float* tw = sT[w];
  float* sg = sG[GF ? w : 0];
  float* dYc = dYp + (size_t)ct * E * 16;
  float* da3c = da3p + (size_t)ct * E * 64;
  for (int i = blockIdx.x * NW + w; i < N; i += gridDim.x * NW) {
    float gv[MID];
#pragma unroll
    for (int c = 0; c < MID; ++c) gv[c] = dAt[((size_t)i * MID + c) * K + k] * inv_c;
    const int e_beg = rcv_off[i], e_end = rcv_off[i + 1];
    if constexpr (GF) {
      // G_p of this receiver and channel; the four lane groups hold the same
      // channels, the first one stores
      __builtin_amdgcn_wave_barrier();   // the previous receiver's reads come first
      for_paths<LHMAX>([&](auto tag) {
        using T = decltype(tag);
        using C = mt::CG<T::lh, T::ly, T::lo>;
        constexpr int goff = PathPairOffset<T::index>::value;
        float Gp[C::npair];
#pragma unroll
        for (int u = 0; u < C::npair; ++u) Gp[u] = 0.f;
        C::each_p([&](int m1, int m2, int m3, float cg, int pi) { Gp[pi] += cg * gv[T::offset + m3]; });
        if (g == 0) {
#pragma unroll
          for (int u = 0; u < C::npair; ++u) sg[(goff + u) * 16 + kk] = Gp[u];
        }
      });
      __builtin_amdgcn_wave_barrier();
    }
    for (int e0 = e_beg; e0 < e_end; e0 += 16) {
      int srcq[4];
      sender_rows(snd, src_map, e0 + 4 * g, e_end, srcq);
      stage_y(Y, e0, e_end, sy);
      f4 r[P];   // R on entry; dR (zero for edges past e_end) after the edge loop
      if constexpr (RM == 1) tile_radial_bf16<P>(a3, e0, e_end, sWb, r);
      else if constexpr (RM == 2) tile_radial_x3s<P>(a3, e0, e_end, sWb, r);
      else tile_radial<P>(a3, e0, e_end, sW, r);
      round_tile<P>(r, rnd);
      const int nq = min(4, e_end - e0);
      float hv[DIN];
      load_h_row<DIN>(h, srcq[0], K, k, hv);
      static_for<0, 4>([&](auto QI) {
        constexpr int q = decltype(QI)::value;
        __builtin_amdgcn_sched_barrier(0);
        if (q >= nq) return;
        if constexpr (GF) __asm__ volatile("" ::: "memory");   // G is read from LDS per edge, not held
        const int row = 4 * g + q;
        const int e_raw = e0 + row;
        const bool valid = e_raw < e_end;
        const int e = min(e_raw, e_end - 1);
        float hn[DIN];
        if constexpr (q < 3) load_h_row<DIN>(h, srcq[q + 1], K, k, hn);
        float y[16];
        read_y(sy, row, y);
        float dy[16], dh[DIN];
#pragma unroll
        for (int m = 0; m < 16; ++m) dy[m] = 0.f;
#pragma unroll
        for (int c = 0; c < DIN; ++c) dh[c] = 0.f;
        for_paths<LHMAX>([&](auto tag) {
          using T = decltype(tag);
          constexpr int lh = T::lh, ly = T::ly, lo = T::lo;
          __builtin_amdgcn_sched_barrier(0);
          const float rv = r[T::index][q];
          // Bm[m2] = sum C h[m1] g[m3], Dm[m1] = sum C Y[m2] g[m3] (from the
          // receiver's G table, or per coupling: C g held in registers would
          // be 86 live values across the edge loop); then dR = Bm . Y,
          // dY += R Bm, dh += R Dm.
          float Bm[2 * ly + 1], Dm[2 * lh + 1];
#pragma unroll
          for (int m = 0; m < 2 * ly + 1; ++m) Bm[m] = 0.f;
#pragma unroll
          for (int m = 0; m < 2 * lh + 1; ++m) Dm[m] = 0.f;
          if constexpr (GF) {
            const float* gp = sg + PathPairOffset<T::index>::value * 16 + kk;
            mt::CG<lh, ly, lo>::each_pair([&](int m1, int m2, int pi) {
              const float gval = gp[pi * 16];
              Bm[m2] += gval * hv[lh * lh + m1];
              Dm[m1] += gval * y[ly * ly + m2];
            });
          } else {
            mt::CG<lh, ly, lo>::each([&](int m1, int m2, int m3, float cg) {
              Bm[m2] += cg * (gv[T::offset + m3] * hv[lh * lh + m1]);
              Dm[m1] += cg * (gv[T::offset + m3] * y[ly * ly + m2]);
            });
          }
          float d = 0.f;
#pragma unroll
          for (int m = 0; m < 2 * ly + 1; ++m) {
            d += Bm[m] * y[ly * ly + m];
            dy[ly * ly + m] += rv * Bm[m];
          }
#pragma unroll
          for (int m = 0; m < 2 * lh + 1; ++m) dh[lh * lh + m] += rv * Dm[m];
          r[T::index][q] = valid ? d : 0.f;
        });
        const float tot = group_reduce16(dy, l);
        if (valid) {
          dYc[(size_t)e * 16 + kk] = tot;
          if (Q) {
#pragma unroll
            for (int c = 0; c < DIN; ++c) Q[((size_t)e * DIN + c) * K + k] = dh[c];
          }
        }
        if constexpr (q < 3) {
#pragma unroll
          for (int c = 0; c < DIN; ++c) hv[c] = hn[c];
        }
      });
      // da3 partial: D[e][j] = sum_{p, k} dR[e][p][k] W3[j][p K + 16 ct + k]. The
      // A operand wants the edge on l%16, so each dR tile is transposed through LDS.
      f4 d3[4];
      if constexpr (RM == 1) {
        tile_da3_bf16<P>(r, sWt, tw, d3);
      } else if constexpr (RM == 2) {
        tile_da3_x3<P>(r, sWt, tw, d3);
      } else {
        __builtin_amdgcn_s_setprio(1);
#pragma unroll
        for (int jt = 0; jt < 4; ++jt) d3[jt] = f4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int p = 0; p < P; ++p) {
          __builtin_amdgcn_sched_barrier(0);
#pragma unroll
          for (int q = 0; q < 4; ++q) tw[(4 * g + q) * kTPitch + kk] = r[p][q];
          __builtin_amdgcn_wave_barrier();
          float av[4];
#pragma unroll
          for (int kq = 0; kq < 4; ++kq) av[kq] = tw[kk * kTPitch + 4 * kq + g];
          __builtin_amdgcn_wave_barrier();
#pragma unroll
          for (int kq = 0; kq < 4; ++kq) {
            const float* wrow = sW + (p * 16 + 4 * kq + g) * kWPitch + kk;
#pragma unroll
            for (int jt = 0; jt < 4; ++jt) d3[jt] = mfma4(av[kq], wrow[16 * jt], d3[jt]);
          }
        }
        __builtin_amdgcn_s_setprio(0);
      }
#pragma unroll
      for (int rr = 0; rr < 4; ++rr) {
        const int e = e0 + 4 * g + rr;
        if (e < e_end) {
#pragma unroll
          for (int jt = 0; jt < 4; ++jt) da3c[(size_t)e * 64 + 16 * jt + kk] = d3[jt][rr];
        }
      }
    }
  }
}

// ---- Split-BF16 backward at l_h <= 1 in the edge-lane layout.
//
// The radial MFMAs take the weight slice as the A operand and a3 as B, so the
// result puts the edge on l%16: lane l holds R for edge e0 + l%16 and the four
// channels 16 ct + 4(l/16) .. +3. Each lane then contracts one edge over four
// channels:
//   - the Y row and the sender's h rows are the lane's own (float4 loads);
//   - the couplings come from the receiver's G table in LDS, one float4 over
//     the four channels per (m1, m2) pair: Dm[m1] += G Y[m2] and
//     dY[m2] += G (R h[m1]), two multiply-adds per pair and channel in place of
//     two products and two multiply-adds per coupling coefficient;
//   - dE/dY is summed over the lane's four channels in registers and over the
//     four lane groups by two halving exchange steps;
//   - dR is the A operand of the dE/da3 MFMA as it stands: in K step ks the
//     reduction index 8(l/16) + i stands for path 2 ks + i/4 and channel
//     4(l/16) + i%4, and W3's parts sit in LDS in that order, so no transpose
//     through LDS is needed.
// LDS: both layouts of the three W3 parts (120 KB at P = 10) and a G table of
// PairCount x 16 floats per wave (38 KB for eight waves).

// Edge-lane layout of a W3 part for the dE/da3 product:
// element (((ks 64 + j) 4 + q) 2 + pl) 4 + c of the part is W3[j][p K + 16 ct + 4 q + c]
// with p = 2 ks + pl, so that lane (l/16 = q, l%16) of K step ks reads its
// eight reduction values as one 16-byte row.
__device__ __forceinline__ int el_tr(int ks, int j, int q) { return ((ks * 64 + j) * 4 + q) * 8; }

template <int P>
__device__ __forceinline__ void load_w3_slices_x3_el(const float* __restrict__ W3, int K, int ct,
                                                     unsigned short* sWf, unsigned short* sWe) {
  static_assert(P % 2 == 0, "paths come in pairs per K step");
  const int PK = P * K;
  constexpr int part = P * 16 * 64;
  for (int idx = threadIdx.x; idx < P * 16 * 64; idx += blockDim.x) {
    const int kk = idx & 15, j = (idx >> 4) & 63, p = idx >> 10;
    unsigned short x0, x1, x2;
    split3(W3[(size_t)j * PK + p * K + 16 * ct + kk], x0, x1, x2);
    const int of = swz_fwd(p * 16 + kk, j >> 3) + (j & 7);
    const int oe = el_tr(p >> 1, j, kk >> 2) + 4 * (p & 1) + (kk & 3);
    sWf[of] = x0;
    sWf[part + of] = x1;
    sWf[2 * part + of] = x2;
    sWe[oe] = x0;
    sWe[part + oe] = x1;
    sWe[2 * part + oe] = x2;
  }
}

// R in the edge-lane layout: r[p][c] = R[e0 + l%16][p][16 ct + 4(l/16) + c]
// (zero for edges past e_end), split-BF16 products as in tile_radial_x3s with
// the operands exchanged.
template <int P, bool PRE = false>
__device__ __forceinline__ void tile_radial_x3_el(const float* __restrict__ a3, int e0, int e_end,
                                                  const unsigned short* __restrict__ sWf, f4* r) {
  constexpr int part = P * 16 * 64;
  const int l = threadIdx.x & 63;
  const int row = e0 + (l & 15);
  const float keep = row < e_end ? 1.f : 0.f;
  const int crow = min(row, e_end - 1);
  const f4* arow = reinterpret_cast<const f4*>(a3 + (size_t)crow * 64 + 8 * (l >> 4));
#pragma unroll
  for (int p = 0; p < P; ++p) r[p] = f4{0.f, 0.f, 0.f, 0.f};
  __builtin_amdgcn_s_setprio(1);
#pragma unroll
  for (int ks = 0; ks < 2; ++ks) {
    __builtin_amdgcn_sched_barrier(0);
    us8v a0, a1, a2;
    if constexpr (PRE) {
      load_a3_parts(reinterpret_cast<const unsigned short*>(a3), crow, row < e_end, ks, a0, a1, a2);
    } else {
      const f4 lo = arow[8 * ks] * keep, hi = arow[8 * ks + 1] * keep;
      split3_x8(lo, hi, a0, a1, a2);
    }
#pragma unroll
    for (int p = 0; p < P; ++p) {
      __builtin_amdgcn_sched_barrier(0);
      const unsigned short* q = sWf + swz_fwd(p * 16 + (l & 15), 4 * ks + (l >> 4));
      const us8v b0 = *reinterpret_cast<const us8v*>(q);
      const us8v b1 = *reinterpret_cast<const us8v*>(q + part);
      const us8v b2 = *reinterpret_cast<const us8v*>(q + 2 * part);
      f4 acc = r[p];
      acc = mfma_bf16(b0, a2, acc);
      acc = mfma_bf16(b1, a1, acc);
      acc = mfma_bf16(b2, a0, acc);
      acc = mfma_bf16(b0, a1, acc);
      acc = mfma_bf16(b1, a0, acc);
      r[p] = mfma_bf16(b0, a0, acc);
    }
  }
  __builtin_amdgcn_s_setprio(0);
}

// dE/da3 partial from dR in the edge-lane layout: d3[jt][rr] = D[e0 + 4(l/16) + rr][16 jt + l%16].
template <int P>
__device__ __forceinline__ void tile_da3_x3_el(const f4* r, const unsigned short* __restrict__ sWe, f4* d3) {
  constexpr int part = P * 16 * 64;
  const int l = threadIdx.x & 63, g = l >> 4, kk = l & 15;
#pragma unroll
  for (int jt = 0; jt < 4; ++jt) d3[jt] = f4{0.f, 0.f, 0.f, 0.f};
  __builtin_amdgcn_s_setprio(1);
#pragma unroll
  for (int ks = 0; ks < P / 2; ++ks) {
    __builtin_amdgcn_sched_barrier(0);
    us8v a0, a1, a2;
    split3_x8(r[2 * ks], r[2 * ks + 1], a0, a1, a2);
#pragma unroll
    for (int jt = 0; jt < 4; ++jt) {
      const unsigned short* q = sWe + el_tr(ks, 16 * jt + kk, g);
      const us8v b0 = *reinterpret_cast<const us8v*>(q);
      const us8v b1 = *reinterpret_cast<const us8v*>(q + part);
      const us8v b2 = *reinterpret_cast<const us8v*>(q + 2 * part);
      f4 acc = d3[jt];
      acc = mfma_bf16(a2, b0, acc);
      acc = mfma_bf16(a1, b1, acc);
      acc = mfma_bf16(a0, b2, acc);
      acc = mfma_bf16(a1, b0, acc);
      acc = mfma_bf16(a0, b1, acc);
      d3[jt] = mfma_bf16(a0, b0, acc);
    }
  }
  __builtin_amdgcn_s_setprio(0);
}

template <int LHMAX, int RM>
constexpr bool tpr_bwd_edge_lanes() { return (RM == 2 || RM == 3) && LHMAX == 1; }

// PRE: a3 arrives as its three parts (RM = 3).
template <int LHMAX, int NW, bool PRE>
__device__ __forceinline__ void tpr_bwd_edge_lanes_body(
    int N, int K, int E, const int* __restrict__ rcv_off, const int* __restrict__ snd,
    const int* __restrict__ src_map, const float* __restrict__ a3, const float* __restrict__ W3,
    const float* __restrict__ Y, const float* __restrict__ h, float inv_c, const float* __restrict__ dAt,
    float* __restrict__ dYp, float* __restrict__ Q, float* __restrict__ da3p, int rnd) {
  constexpr int P = path_count(LHMAX);
  constexpr int MID = mid_count(LHMAX);
  constexpr int DIN = (LHMAX + 1) * (LHMAX + 1);
  constexpr int NPAIR = PairCount<LHMAX>::value;
  constexpr int part = P * 16 * 64;
  __shared__ __align__(16) unsigned short sWx[6 * part];
  __shared__ __align__(16) float sG[NW][NPAIR * 16];   // [pair][channel]
  unsigned short* sWf = sWx;
  unsigned short* sWe = sWx + 3 * part;
  const int ct = blockIdx.y;
  load_w3_slices_x3_el<P>(W3, K, ct, sWf, sWe);
  __syncthreads();
  const int l = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int g = l >> 4, kk = l & 15;
  const int kb = 16 * ct + 4 * g;   // the lane's four channels in the edge loop
  float* sg = sG[w];
  float* dYc = dYp + (size_t)ct * E * 16;
  float* da3c = da3p + (size_t)ct * E * 64;
  for (int i = blockIdx.x * NW + w; i < N; i += gridDim.x * NW) {
    const int e_beg = rcv_off[i], e_end = rcv_off[i + 1];
    {
      // G_p of this receiver for channel 16 ct + l%16; the four lane groups
      // compute the same values and the first one stores
      float gv[MID];
#pragma unroll
      for (int c = 0; c < MID; ++c) gv[c] = dAt[((size_t)i * MID + c) * K + 16 * ct + kk] * inv_c;
      __builtin_amdgcn_wave_barrier();   // the previous receiver's reads come first
      for_paths<LHMAX>([&](auto tag) {
        using T = decltype(tag);
        using C = mt::CG<T::lh, T::ly, T::lo>;
        constexpr int goff = PathPairOffset<T::index>::value;
        float Gp[C::npair];
#pragma unroll
        for (int u = 0; u < C::npair; ++u) Gp[u] = 0.f;
        C::each_p([&](int m1, int m2, int m3, float cg, int pi) { Gp[pi] += cg * gv[T::offset + m3]; });
        if (g == 0) {
#pragma unroll
          for (int u = 0; u < C::npair; ++u) sg[(goff + u) * 16 + kk] = Gp[u];
        }
      });
      __builtin_amdgcn_wave_barrier();
    }
    for (int e0 = e_beg; e0 < e_end; e0 += 16) {
      __asm__ volatile("" ::: "memory");   // the G table is read per tile, not held in registers
      const int e_raw = e0 + kk;
      const bool valid = e_raw < e_end;
      const int e = min(e_raw, e_end - 1);
      int src = snd[e];
      if (src_map) src = src_map[src];
      f4 hv[DIN];
#pragma unroll
      for (int c = 0; c < DIN; ++c) hv[c] = *reinterpret_cast<const f4*>(h + ((size_t)src * DIN + c) * K + kb);
      float y[16];
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        const f4 t4 = reinterpret_cast<const f4*>(Y + (size_t)e * 16)[v];
        y[4 * v] = t4[0];
        y[4 * v + 1] = t4[1];
        y[4 * v + 2] = t4[2];
        y[4 * v + 3] = t4[3];
      }
      f4 r[P];   // R on entry (zero for edges past e_end); dR after the path loop
      tile_radial_x3_el<P, PRE>(a3, e0, e_end, sWf, r);
      round_tile<P>(r, rnd);
      float dy[16];
#pragma unroll
      for (int m = 0; m < 16; ++m) dy[m] = 0.f;
      f4 dh[DIN];
#pragma unroll
      for (int c = 0; c < DIN; ++c) dh[c] = f4{0.f, 0.f, 0.f, 0.f};
      for_paths<LHMAX>([&](auto tag) {
        using T = decltype(tag);
        constexpr int lh = T::lh, ly = T::ly;
        const f4 rv = r[T::index];
        f4 Dm[2 * lh + 1], Rh[2 * lh + 1];
#pragma unroll
        for (int m = 0; m < 2 * lh + 1; ++m) {
          Dm[m] = f4{0.f, 0.f, 0.f, 0.f};
          Rh[m] = rv * hv[lh * lh + m];
        }
        const float* gp = sg + PathPairOffset<T::index>::value * 16 + 4 * g;
        mt::CG<lh, ly, T::lo>::each_pair([&](int m1, int m2, int pi) {
          const f4 G = *reinterpret_cast<const f4*>(gp + pi * 16);
          const float yv = y[ly * ly + m2];
          Dm[m1] += G * yv;
          float t = dy[ly * ly + m2];
#pragma unroll
          for (int c = 0; c < 4; ++c) t += G[c] * Rh[m1][c];
          dy[ly * ly + m2] = t;
        });
        f4 d = f4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int m = 0; m < 2 * lh + 1; ++m) {
          d += hv[lh * lh + m] * Dm[m];
          dh[lh * lh + m] += rv * Dm[m];
        }
        // (rows past e_end keep their finite dR: a row of the dE/da3 product
        // depends on its own edge only, and those rows are not stored)
        r[T::index] = d;
      });
      // dE/dY over the tile's 16 channels: halve over lane bit 5 (l/16 >= 2
      // keeps m2 8..15), then over lane bit 4; lane group q ends with m2 = 4q .. 4q + 3
      {
        const bool hi5 = g >= 2;
#pragma unroll
        for (int m = 0; m < 8; ++m) {
          const float send = hi5 ? dy[m] : dy[m + 8];
          const float keep = hi5 ? dy[m + 8] : dy[m];
          dy[m] = keep + __shfl_xor(send, 32);
        }
        const bool hi4 = g & 1;
#pragma unroll
        for (int m = 0; m < 4; ++m) {
          const float send = hi4 ? dy[m] : dy[m + 4];
          const float keep = hi4 ? dy[m + 4] : dy[m];
          dy[m] = keep + __shfl_xor(send, 16);
        }
      }
      if (valid) {
        *reinterpret_cast<f4*>(dYc + (size_t)e * 16 + 4 * g) = f4{dy[0], dy[1], dy[2], dy[3]};
        if (Q) {
#pragma unroll
          for (int c = 0; c < DIN; ++c) *reinterpret_cast<f4*>(Q + ((size_t)e * DIN + c) * K + kb) = dh[c];
        }
      }
      f4 d3[4];
      tile_da3_x3_el<P>(r, sWe, d3);
#pragma unroll
      for (int rr = 0; rr < 4; ++rr) {
        const int ed = e0 + 4 * g + rr;
        if (ed < e_end) {
#pragma unroll
          for (int jt = 0; jt < 4; ++jt) da3c[(size_t)ed * 64 + 16 * jt + kk] = d3[jt][rr];
        }
      }
    }
  }
}

// ---- FP32-accurate backward at l_h = 2 in the edge-lane layout.
//
// Both products with W3 run on split-BF16 MFMA (FP32-accurate) from one copy of
// W3's three bfloat16 parts in LDS, the swizzled forward layout of the l_h <= 1
// backward (104 KB at P = 17; the transposed layout would not fit beside the G
// tables):
//   R recompute: A = W3's parts (rows p 16 + channel, 16-byte reads), B = a3's
//     parts split per tile in registers;
//   dE/da3: D[edge][j] = sum_(p, c) dR[edge][p, c] W3[j][p, c]; dR is already
//     on the lane that owns the edge (split per K step in registers), and W3's
//     parts reach the B operand through LDS transposing reads
//     (ds_read_b64_tr_b16), which hand each lane one column j of four
//     consecutive rows (channels) of the forward layout.
// The CG part is the edge-lane contraction of the l_h = 1 backward (G table of
// the receiver in LDS, two multiply-adds per coupling pair and channel). One
// wave per SIMD (W3's parts and four G tables take 149 KB), so the body keeps
// its own reads in flight: every LDS or global operand is requested a fixed
// number of uses ahead (a ring of registers indexed by compile-time
// constants, held in issue order by scheduling fences), the sender rows and
// harmonics of a tile are requested before its radial MFMAs, and the next
// tile's a3 and sender index before its dE/da3 products.
constexpr int kRingR = 3;    // split-W3 operand triples in flight (six MFMAs each)
constexpr int kRingW = 2;    // W3 operand sets of the dE/da3 product held (one in use, one in flight)
typedef short s4v __attribute__((ext_vector_type(4)));
constexpr int kRingG = 6;    // G-table entries in flight (one coupling pair each)

// The MFMAs of the l_h = 2 backward that run between the contraction's
// coupling pairs, in program order, at most MAXPER per pair (each runs in the
// shadow of a pair's multiply-adds):
//   - K step ks of the dE/da3 product (paths 2 ks and 2 ks + 1, 4 NPROD
//     MFMAs), once the contraction has produced dR of both paths, i.e. from
//     the first coupling pair of path 2 ks + 2;
//   - with PIPE, the next tile's R product of paths 2 ks and 2 ks + 1
//     (2 NPROD MFMAs each), into the registers of R values already
//     contracted, from the same pair and not before pair XA (the next tile's
//     a3 has to arrive).
// Both kinds keep their own order; between them the earlier K step goes
// first. Whatever the contraction cannot take (the last K step) follows it.
// order[first[gi] .. first[gi + 1]) are the MFMAs at pair gi; an MFMA id below
// ND is a dE/da3 one, the others the R product's. `valid` says that every
// dE/da3 K step is issued before its split operands' registers are reused
// (by the split of K step ks + 2, at the end of path 2 ks + 5).
template <int NPAIR, int P, int NPROD, int XA, bool PIPE, int MAXPER>
struct BwdPlan {
  static constexpr int KS = (P + 1) / 2;
  static constexpr int ND = KS * 4 * NPROD;
  static constexpr int NRM = PIPE ? P * 2 * NPROD : 0;
  static constexpr int NT = ND + NRM;
  static constexpr int kNever = 1 << 20;
  int first[NPAIR + 1];
  int order[NT];
  bool valid;
  template <class Off>
  constexpr BwdPlan(Off off) : first{}, order{}, valid(true) {
    auto avail_ks = [&](int ks) { return 2 * ks + 2 < P ? off(2 * ks + 2) : kNever; };
    auto pos_d = [&](int n) { return (n / (4 * NPROD)) * 8 * NPROD + n % (4 * NPROD); };
    auto pos_r = [&](int m) { return (m / (4 * NPROD)) * 8 * NPROD + 4 * NPROD + m % (4 * NPROD); };
    int k = 0, dn = 0, rn = 0;
    int last_d[KS] = {};
    for (int gi = 0; gi < NPAIR; ++gi) {
      first[gi] = k;
      for (int c = 0; c < MAXPER; ++c) {
        const bool dav = dn < ND && gi >= avail_ks(dn / (4 * NPROD));
        const int ra = rn < NRM ? avail_ks(rn / (4 * NPROD)) : kNever;
        const bool rav = rn < NRM && gi >= (ra > XA ? ra : XA);
        if (!dav && !rav) break;
        if (dav && (!rav || pos_d(dn) < pos_r(rn))) {
          last_d[dn / (4 * NPROD)] = gi;
          order[k++] = dn++;
        } else {
          order[k++] = ND + rn++;
        }
      }
    }
    first[NPAIR] = k;
    for (int ks = 0; ks + 2 < KS; ++ks) {
      if ((ks + 1) * 4 * NPROD > dn) valid = false;   // left for after the contraction
      else if (2 * ks + 6 < P && last_d[ks] >= off(2 * ks + 6)) valid = false;
    }
    // the rest in list order
    while (dn < ND || rn < NRM) {
      if (dn < ND && (rn >= NRM || pos_d(dn) < pos_r(rn))) order[k++] = dn++;
      else order[k++] = ND + rn++;
    }
  }
};
template <int I, int N>
constexpr int path_pair_offset_of(int p) {
  if constexpr (I >= N) return -1;
  else return p == I ? PathPairOffset<I>::value : path_pair_offset_of<I + 1, N>(p);
}

// sender rows (channels kb .. kb + 3) and harmonics of the lane's edge
template <int DIN>
__device__ __forceinline__ void el_load_hy(f4* hv, f4* y4, int src, int e, int kb, const float* __restrict__ h,
                                           const float* __restrict__ Y, int K) {
#pragma unroll
  for (int c = 0; c < DIN; ++c) hv[c] = *reinterpret_cast<const f4*>(h + ((size_t)src * DIN + c) * K + kb);
#pragma unroll
  for (int v = 0; v < 4; ++v) y4[v] = reinterpret_cast<const f4*>(Y + (size_t)e * 16)[v];
}

// the lane's a3 operands of the split R product: a3[e][32 ks + 8 g .. +7],
// a[2 ks] (first four) and a[2 ks + 1]
__device__ __forceinline__ void el_load_a3(f4* a, int e, int g, const float* __restrict__ a3) {
#pragma unroll
  for (int v = 0; v < 4; ++v)
    a[v] = *reinterpret_cast<const f4*>(a3 + (size_t)e * 64 + 32 * (v >> 1) + 8 * g + 4 * (v & 1));
}

// the lane's a3 operands of the split R product from the pre-split rows
// ([E][3][64] bfloat16): x[ks][q] = part q of a3[e][32 ks + 8 g .. +7]
__device__ __forceinline__ void el_load_a3_parts(us8v (&x)[2][3], int e, int g, const unsigned short* __restrict__ a3x) {
#pragma unroll
  for (int ks = 0; ks < 2; ++ks)
#pragma unroll
    for (int q = 0; q < 3; ++q) x[ks][q] = *reinterpret_cast<const us8v*>(a3x + (size_t)e * 192 + 64 * q + 32 * ks + 8 * g);
}

// NPROD: partial products per operand pair, 6 (split-BF16 operands,
// FP32-accurate) or 1 (the BF16 radial mode: the operands' bfloat16 roundings,
// which are the first split parts, with FP32 accumulation). PRE: a3 arrives as
// its three parts (the a3 argument then points at [E][3][64] bfloat16 written
// by the edge prologue), six products only.
template <int NW, bool RND, int NPROD, bool PRE>
__device__ __forceinline__ void tpr_bwd_l2_edge_lanes_body(
    int N, int K, int E, const int* __restrict__ rcv_off, const int* __restrict__ snd,
    const int* __restrict__ src_map, const float* __restrict__ a3, const float* __restrict__ W3,
    const float* __restrict__ Y, const float* __restrict__ h, float inv_c, const float* __restrict__ dAt,
    float* __restrict__ dYp, float* __restrict__ Q, float* __restrict__ da3p, int rnd,
    unsigned short* sWf, float* sGall) {
  constexpr int LHMAX = 2;
  constexpr int P = path_count(LHMAX);
  constexpr int MID = mid_count(LHMAX);
  constexpr int DIN = (LHMAX + 1) * (LHMAX + 1);
  constexpr int NPAIR = PairCount<LHMAX>::value;
  constexpr int part = P * 16 * 64;
  constexpr int NR = P * 2;    // (path, K step) steps of the split R product
  constexpr int ND = P * 4;    // (path, row tile) steps of the dE/da3 product
  const int ct = blockIdx.y;
  const int PK = P * K;
  {
    // W3's three parts in the swizzled forward layout: row p 16 + kk of 64 j
    for (int idx = threadIdx.x; idx < P * 16 * 64; idx += blockDim.x) {
      const int kk = idx & 15, j = (idx >> 4) & 63, p = idx >> 10;
      unsigned short x0, x1, x2;
      split3(W3[(size_t)j * PK + p * K + 16 * ct + kk], x0, x1, x2);
      const int of = swz_fwd(p * 16 + kk, j >> 3) + (j & 7);
      sWf[of] = x0;
      sWf[part + of] = x1;
      sWf[2 * part + of] = x2;
    }
  }
  __syncthreads();
  const int l = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int g = l >> 4, kk = l & 15;
  const int kb = 16 * ct + 4 * g;   // the lane's four channels
  float* sg = sGall + w * NPAIR * 16;   // this wave's G table [pair][channel]
  float* dYc = dYp + (size_t)ct * E * 16;
  float* da3c = da3p + (size_t)ct * E * 64;
  // split R operand of step f = 2 p + ks: row p 16 + kk, chunk 4 ks + g
  auto wr_at = [&](int f, us8v* o) {
    const unsigned short* q = sWf + swz_fwd((f >> 1) * 16 + kk, 4 * (f & 1) + g);
    o[0] = *reinterpret_cast<const us8v*>(q);
    if constexpr (NPROD == 6) {
      o[1] = *reinterpret_cast<const us8v*>(q + part);
      o[2] = *reinterpret_cast<const us8v*>(q + 2 * part);
    }
  };
  // dE/da3 operands from the forward-layout parts in LDS, by transposing reads
  // (ds_read_b64_tr_b16: in each 16-lane group, lane j receives element r of
  // the 8-byte row that lane 4 r + j / 4 addressed, at position j % 4). Lane kk
  // of lane group g addresses the columns 16 jt + 4 (kk % 4) .. + 3 of row
  // 4 g + kk / 4 of a path, so that it receives column 16 jt + kk of the
  // path's rows (channels) 4 g .. 4 g + 3: the B operand's K slots 4 pl .. 4 pl + 3
  // for path 2 ks + pl (zero past the last path).
  constexpr int KS = (P + 1) / 2;
  constexpr int NDX = KS * 4;   // (K step, row tile) steps
  const int t_row = 4 * g + (kk >> 2), t_col = 4 * (kk & 3);
  auto tr_at = [&](int q, int p, int jt) {
    const int col = 16 * jt + t_col;
    unsigned short* a = sWf + q * part + swz_fwd(p * 16 + t_row, col >> 3) + (col & 7);
    return __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) s4v*)a);
  };
  auto wd_at = [&](int f, us8v* o) {
    const int ks = f >> 2, jt = f & 3;
#pragma unroll
    for (int q = 0; q < (NPROD == 6 ? 3 : 1); ++q) {
      const s4v lo = tr_at(q, 2 * ks, jt);
      const s4v hi = 2 * ks + 1 < P ? tr_at(q, 2 * ks + 1, jt) : s4v{0, 0, 0, 0};
      o[q] = us8v{(unsigned short)lo[0], (unsigned short)lo[1], (unsigned short)lo[2], (unsigned short)lo[3],
                  (unsigned short)hi[0], (unsigned short)hi[1], (unsigned short)hi[2], (unsigned short)hi[3]};
    }
  };
  // PIPE (the one-product radial mode): a software pipeline over the wave's
  // tiles. The R product of the next tile (this receiver's next, else the
  // first of the wave's next receiver) runs inside the current tile's
  // contraction, into the registers of R values already contracted; its a3,
  // sender rows and harmonics are requested during the current tile, and
  // `prep` says r, hv and y4 hold the upcoming tile's. With six products per
  // operand pair the MFMAs of both products would outrun the contraction's
  // vector work (measured slower), so there each tile forms its R product
  // before its contraction, and the next tile's a3 is requested during the
  // dE/da3 product.
  constexpr bool PIPE = NPROD == 1;
  using Plan = BwdPlan<NPAIR, P, NPROD, 40, PIPE, PIPE ? 3 : 2>;
  constexpr Plan plan([](int q) { return path_pair_offset_of<0, P>(q); });
  static_assert(plan.valid, "a dE/da3 K step would outlive its split operands");
  const int stride = gridDim.x * NW;
  bool prep = false;
  int e = 0, src = 0;   // src: without PIPE, the sender of the tile's edge
  f4 r[P], hv[DIN], y4[4];
  static_assert(!(PRE && PIPE), "pre-split a3 goes with six products");
  f4 a[4];           // without PIPE, the a3 of the tile's edge
  us8v apre[2][3];   // with PRE instead, its parts
  const unsigned short* a3x = reinterpret_cast<const unsigned short*>(a3);
  // R of the tile whose a3 is a0 .. a3 (with PRE: apre), edge on the lane,
  // split-BF16 products
  auto r_standalone = [&](f4 av0, f4 av1, f4 av2, f4 av3) {
#pragma unroll
    for (int p = 0; p < P; ++p) r[p] = f4{0.f, 0.f, 0.f, 0.f};
    us8v x[2][3];
    if constexpr (PRE) {
#pragma unroll
      for (int ks = 0; ks < 2; ++ks)
#pragma unroll
        for (int q = 0; q < 3; ++q) x[ks][q] = apre[ks][q];
    } else {
      split3_x8(av0, av1, x[0][0], x[0][1], x[0][2]);
      split3_x8(av2, av3, x[1][0], x[1][1], x[1][2]);
    }
    us8v ring[kRingR][3];
#pragma unroll
    for (int f = 0; f < kRingR; ++f) wr_at(f, ring[f]);
    __builtin_amdgcn_s_setprio(1);
    static_for<0, NR>([&](auto F) {
      constexpr int f = decltype(F)::value;
      constexpr int p = f >> 1, ks = f & 1;
      __builtin_amdgcn_sched_barrier(0);   // keeps each read kRingR steps ahead of its use
      const us8v b0 = ring[f % kRingR][0], b1 = ring[f % kRingR][1], b2 = ring[f % kRingR][2];
      if constexpr (f + kRingR < NR) wr_at(f + kRingR, ring[f % kRingR]);
      f4 acc = r[p];
      if constexpr (NPROD == 6) {
        acc = mfma_bf16(b0, x[ks][2], acc);
        acc = mfma_bf16(b1, x[ks][1], acc);
        acc = mfma_bf16(b2, x[ks][0], acc);
        acc = mfma_bf16(b0, x[ks][1], acc);
        acc = mfma_bf16(b1, x[ks][0], acc);
      }
      r[p] = mfma_bf16(b0, x[ks][0], acc);
    });
    __builtin_amdgcn_s_setprio(0);
  };
  for (int i = blockIdx.x * NW + w; i < N; i += stride) {
    const int e_beg = rcv_off[i], e_end = rcv_off[i + 1];
    if (e_beg == e_end) {
      prep = false;
      continue;
    }
    int nb = 0, ne = 0;   // the wave's next receiver's edges
    if (i + stride < N) {
      nb = rcv_off[i + stride];
      ne = rcv_off[i + stride + 1];
    }
    {
      // G_p of this receiver for channel 16 ct + l%16, path by path (only the
      // path's own dE/dAt values live); the four lane groups compute the same
      // values and the first one stores
      const float* gsrc = dAt + (size_t)i * MID * K + 16 * ct + kk;
      __builtin_amdgcn_wave_barrier();   // the previous receiver's reads come first
      for_paths<LHMAX>([&](auto tag) {
        using T = decltype(tag);
        using C = mt::CG<T::lh, T::ly, T::lo>;
        constexpr int goff = PathPairOffset<T::index>::value;
        float gv[2 * T::lo + 1];
#pragma unroll
        for (int m = 0; m < 2 * T::lo + 1; ++m) gv[m] = gsrc[(size_t)(T::offset + m) * K] * inv_c;
        float Gp[C::npair];
#pragma unroll
        for (int u = 0; u < C::npair; ++u) Gp[u] = 0.f;
        C::each_p([&](int m1, int m2, int m3, float cg, int pi) { Gp[pi] += cg * gv[m3]; });
        if (g == 0) {
#pragma unroll
          for (int u = 0; u < C::npair; ++u) sg[(goff + u) * 16 + kk] = Gp[u];
        }
      });
      __builtin_amdgcn_wave_barrier();
    }
    if (!prep) {
      // the receiver's first tile (with PIPE: when no earlier tile prepared it)
      e = min(e_beg + kk, e_end - 1);
      int s0 = snd[e];
      if (src_map) s0 = src_map[s0];
      if constexpr (PIPE) {
        f4 a0[4];
        el_load_a3(a0, e, g, a3);
        el_load_hy<DIN>(hv, y4, s0, e, kb, h, Y, K);
        // (written out here: as a call of r_standalone it costs registers)
#pragma unroll
        for (int p = 0; p < P; ++p) r[p] = f4{0.f, 0.f, 0.f, 0.f};
        us8v x[2][3];
        split3_x8(a0[0], a0[1], x[0][0], x[0][1], x[0][2]);
        split3_x8(a0[2], a0[3], x[1][0], x[1][1], x[1][2]);
        us8v ring[kRingR][3];
#pragma unroll
        for (int f = 0; f < kRingR; ++f) wr_at(f, ring[f]);
        __builtin_amdgcn_s_setprio(1);
        static_for<0, NR>([&](auto F) {
          constexpr int f = decltype(F)::value;
          constexpr int p = f >> 1, ks = f & 1;
          __builtin_amdgcn_sched_barrier(0);   // keeps each read kRingR steps ahead of its use
          const us8v b0 = ring[f % kRingR][0], b1 = ring[f % kRingR][1], b2 = ring[f % kRingR][2];
          if constexpr (f + kRingR < NR) wr_at(f + kRingR, ring[f % kRingR]);
          f4 acc = r[p];
          if constexpr (NPROD == 6) {
            acc = mfma_bf16(b0, x[ks][2], acc);
            acc = mfma_bf16(b1, x[ks][1], acc);
            acc = mfma_bf16(b2, x[ks][0], acc);
            acc = mfma_bf16(b0, x[ks][1], acc);
            acc = mfma_bf16(b1, x[ks][0], acc);
          }
          r[p] = mfma_bf16(b0, x[ks][0], acc);
        });
        __builtin_amdgcn_s_setprio(0);
      } else {
        src = s0;
        if constexpr (PRE) el_load_a3_parts(apre, e, g, a3x);
        else el_load_a3(a, e, g, a3);
      }
    }
    for (int e0 = e_beg; e0 < e_end; e0 += 16) {
      __asm__ volatile("" ::: "memory");   // the G table is read per tile, not held in registers
      // Lanes past the receiver's last edge work on that edge (ec is clamped):
      // their inputs, hence every value they compute, equal the last valid
      // lane's, so they store the same values to the same rows, and the stores
      // need no branch.
      const int ec = e;
      const bool more = e0 + 16 < e_end;
      if constexpr (!PIPE) {
        el_load_hy<DIN>(hv, y4, src, e, kb, h, Y, K);
        r_standalone(a[0], a[1], a[2], a[3]);
      }
      // with PIPE, the next tile's edge; after the wave's last tile, this
      // tile's again (its products are then discarded)
      const int e_n = more ? min(e0 + 16 + kk, e_end - 1) : (nb < ne ? min(nb + kk, ne - 1) : ec);
      int src_n = 0;
      f4 an[4];
      if constexpr (PIPE) {
        src_n = snd[e_n];
        el_load_a3(an, e_n, g, a3);
      }
      if constexpr (RND) round_tile<P>(r, rnd);
      float y[16];
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        y[4 * v] = y4[v][0];
        y[4 * v + 1] = y4[v][1];
        y[4 * v + 2] = y4[v][2];
        y[4 * v + 3] = y4[v][3];
      }
      if constexpr (PIPE) {
#pragma unroll
        for (int v = 0; v < 4; ++v) y4[v] = reinterpret_cast<const f4*>(Y + (size_t)e_n * 16)[v];
      }
      float dy[16];
#pragma unroll
      for (int m = 0; m < 16; ++m) dy[m] = 0.f;
      f4 dh[DIN];
#pragma unroll
      for (int c = 0; c < DIN; ++c) dh[c] = f4{0.f, 0.f, 0.f, 0.f};
      // dE/da3 partial on split-BF16 products (dR split per K step):
      // d3[jt][rr] = D[edge e0 + 4 g + rr][j = 16 jt + kk]; in K step ks the
      // lane's eight reduction values are (path 2 ks + pl, channel 4 g + c).
      // The split dR of two K steps (x) and kRingW W3 operand sets (wring) are
      // live at a time.
      f4 d3[4];
#pragma unroll
      for (int jt = 0; jt < 4; ++jt) d3[jt] = f4{0.f, 0.f, 0.f, 0.f};
      us8v x[2][NPROD == 6 ? 3 : 1];
      us8v wring[kRingW][NPROD == 6 ? 3 : 1];
#pragma unroll
      for (int t = 0; t + 1 < kRingW; ++t) wd_at(t, wring[t]);
      // MFMA n of the dE/da3 product: operand set t = n / NPROD (K step t / 4,
      // row tile t % 4), partial product n % NPROD; the first one of a set
      // requests the set kRingW - 1 ahead
      auto da3_mfma = [&](int n) {
        const int t = n / NPROD, pr = n % NPROD;
        const int ks = t >> 2, jt = t & 3;
        if (pr == 0 && t + kRingW - 1 < NDX) wd_at(t + kRingW - 1, wring[(t + kRingW - 1) % kRingW]);
        const us8v* b = wring[t % kRingW];
        const us8v* xa = x[ks & 1];
        if constexpr (NPROD == 6) {
          // smallest terms first, as in the other split products
          constexpr int ia[6] = {2, 1, 0, 1, 0, 0}, ib[6] = {0, 1, 2, 0, 1, 0};
          d3[jt] = mfma_bf16(xa[ia[pr]], b[ib[pr]], d3[jt]);
        } else {
          d3[jt] = mfma_bf16(xa[0], b[0], d3[jt]);
        }
      };
      // MFMA m of the next tile's R product: operand set f = m / NPROD (path
      // f / 2, K step f % 2 of a3), partial product m % NPROD, in the order of
      // the standalone product (a path's first one starts from zero); the next
      // tile's a3 is split at the first one
      us8v xn[2][NPROD == 6 ? 3 : 1];
      us8v rring[2][NPROD == 6 ? 3 : 1];
      if constexpr (PIPE) wr_at(0, rring[0]);
      auto r_mfma = [&](int m) {
        const int f = m / NPROD, pr = m % NPROD;
        const int p = f >> 1, kq = f & 1;
        if (m == 0) {
          if constexpr (NPROD == 6) {
            split3_x8(an[0], an[1], xn[0][0], xn[0][1], xn[0][2]);
            split3_x8(an[2], an[3], xn[1][0], xn[1][1], xn[1][2]);
          } else {
            us8v t1, t2;
            split3_x8(an[0], an[1], xn[0][0], t1, t2);
            split3_x8(an[2], an[3], xn[1][0], t1, t2);
          }
        }
        if (pr == 0 && f + 1 < NR) wr_at(f + 1, rring[(f + 1) & 1]);
        const us8v* b = rring[f & 1];
        const f4 acc = (kq == 0 && pr == 0) ? f4{0.f, 0.f, 0.f, 0.f} : r[p];
        if constexpr (NPROD == 6) {
          constexpr int ib[6] = {0, 1, 2, 0, 1, 0}, ia[6] = {2, 1, 0, 1, 0, 0};
          r[p] = mfma_bf16(b[ib[pr]], xn[kq][ia[pr]], acc);
        } else {
          r[p] = mfma_bf16(b[0], xn[kq][0], acc);
        }
      };
      auto mfma_item = [&](int id) {
        if (id < Plan::ND) da3_mfma(id);
        else r_mfma(id - Plan::ND);
      };
      {
        const float* gq = sg + 4 * g;
        f4 gring[kRingG];
#pragma unroll
        for (int u = 0; u < kRingG; ++u) gring[u] = *reinterpret_cast<const f4*>(gq + u * 16);
        for_paths<LHMAX>([&](auto tag) {
          using T = decltype(tag);
          constexpr int lh = T::lh, ly = T::ly;
          constexpr int goff = PathPairOffset<T::index>::value;
          const f4 rv = r[T::index];
          f4 Dm[2 * lh + 1], Rh[2 * lh + 1];
#pragma unroll
          for (int m = 0; m < 2 * lh + 1; ++m) {
            Dm[m] = f4{0.f, 0.f, 0.f, 0.f};
            Rh[m] = rv * hv[lh * lh + m];
          }
          mt::CG<lh, ly, T::lo>::each_pair([&](int m1, int m2, int pi) {
            const int gi = goff + pi;   // a constant after inlining
            __builtin_amdgcn_sched_barrier(0);   // keeps each read kRingG pairs ahead of its use
            const f4 G = gring[gi % kRingG];
            if (gi + kRingG < NPAIR) gring[gi % kRingG] = *reinterpret_cast<const f4*>(gq + (gi + kRingG) * 16);
            const float yv = y[ly * ly + m2];
            Dm[m1] += G * yv;
            float t = dy[ly * ly + m2];
#pragma unroll
            for (int c = 0; c < 4; ++c) t += G[c] * Rh[m1][c];
            dy[ly * ly + m2] = t;
            // the MFMAs planned for this pair
#pragma unroll
            for (int j = plan.first[gi]; j < plan.first[gi + 1]; ++j) mfma_item(plan.order[j]);
          });
          f4 d = f4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
          for (int m = 0; m < 2 * lh + 1; ++m) {
            d += hv[lh * lh + m] * Dm[m];
            dh[lh * lh + m] += rv * Dm[m];
          }
          r[T::index] = d;   // dR
          // a completed K step of the dE/da3 product: its dR in split form
          if constexpr (T::index % 2 == 1 || T::index + 1 == P) {
            constexpr int ks = T::index / 2;
            const f4 hi = 2 * ks + 1 < P ? r[2 * ks + 1 < P ? 2 * ks + 1 : 0] : f4{0.f, 0.f, 0.f, 0.f};
            if constexpr (NPROD == 6) split3_x8(r[2 * ks], hi, x[ks & 1][0], x[ks & 1][1], x[ks & 1][2]);
            else {
              us8v x1, x2;
              split3_x8(r[2 * ks], hi, x[ks & 1][0], x1, x2);
            }
          }
          // the paths come ordered by l_h: after the last one of an l_h block
          // that block of the sender gradient is complete and leaves registers,
          // and the block's sender rows are free for the next tile's
          if constexpr (T::index + 1 == P || PathAt<T::index + 1>::lh != lh) {
#pragma unroll
            for (int m = 0; m < 2 * lh + 1; ++m)
              *reinterpret_cast<f4*>(Q + ((size_t)ec * DIN + lh * lh + m) * K + kb) = dh[lh * lh + m];
            if constexpr (!PIPE) {
            } else if constexpr (lh == 0) {
              if (src_map) src_n = src_map[src_n];
            } else if constexpr (lh == 1) {
#pragma unroll
              for (int c = 0; c < 4; ++c) hv[c] = *reinterpret_cast<const f4*>(h + ((size_t)src_n * DIN + c) * K + kb);
            }
          }
        });
      }
      // dE/dY over the tile's 16 channels: halve over lane bit 5, then bit 4;
      // lane group q ends with m2 = 4q .. 4q + 3
      {
        const bool hi5 = g >= 2;
#pragma unroll
        for (int m = 0; m < 8; ++m) {
          const float send = hi5 ? dy[m] : dy[m + 8];
          const float keep = hi5 ? dy[m + 8] : dy[m];
          dy[m] = keep + __shfl_xor(send, 32);
        }
        const bool hi4 = g & 1;
#pragma unroll
        for (int m = 0; m < 4; ++m) {
          const float send = hi4 ? dy[m] : dy[m + 4];
          const float keep = hi4 ? dy[m + 4] : dy[m];
          dy[m] = keep + __shfl_xor(send, 16);
        }
      }
      *reinterpret_cast<f4*>(dYc + (size_t)ec * 16 + 4 * g) = f4{dy[0], dy[1], dy[2], dy[3]};
      if constexpr (PIPE) {
#pragma unroll
        for (int c = 4; c < DIN; ++c) hv[c] = *reinterpret_cast<const f4*>(h + ((size_t)src_n * DIN + c) * K + kb);
      } else {
        if (more) {
          // the next tile's sender index and a3, in flight during the rest of
          // the dE/da3 product
          e = min(e0 + 16 + kk, e_end - 1);
          src = snd[e];
          if (src_map) src = src_map[src];
          if constexpr (PRE) el_load_a3_parts(apre, e, g, a3x);
          else el_load_a3(a, e, g, a3);
        }
      }
      // the MFMAs the contraction could not take
      __builtin_amdgcn_s_setprio(1);
      static_for<plan.first[NPAIR], Plan::NT>([&](auto J) {
        __builtin_amdgcn_sched_barrier(0);   // keeps each operand read one set ahead of its use
        mfma_item(plan.order[decltype(J)::value]);
      });
      __builtin_amdgcn_s_setprio(0);
      // rows past the receiver's last edge hold that edge's values (their A rows
      // came from lanes working on it): stored to its row, no branch
#pragma unroll
      for (int rr = 0; rr < 4; ++rr) {
        const size_t row = (size_t)min(e0 + 4 * g + rr, e_end - 1) * 64;
#pragma unroll
        for (int jt = 0; jt < 4; ++jt) da3c[row + 16 * jt + kk] = d3[jt][rr];
      }
      if constexpr (PIPE) e = e_n;
    }
    prep = PIPE && nb < ne;
  }
}

template <int LHMAX, int RM, int NW = TprShape<LHMAX, true, RM>::waves>
__global__ void __launch_bounds__(64 * NW)
__attribute__((amdgpu_waves_per_eu(TprShape<LHMAX, true, RM>::per_simd, TprShape<LHMAX, true, RM>::per_simd)))
tpr_bwd_kernel(
    int N, int K, int E, const int* __restrict__ rcv_off, const int* __restrict__ snd,
    const int* __restrict__ src_map, const float* __restrict__ a3, const float* __restrict__ W3,
    const float* __restrict__ Y, const float* __restrict__ h, float inv_c, const float* __restrict__ dAt,
    float* __restrict__ dYp, float* __restrict__ Q, float* __restrict__ da3p, int rnd) {
  if constexpr (tpr_bwd_edge_lanes<LHMAX, RM>())
    tpr_bwd_edge_lanes_body<LHMAX, NW, RM == 3>(N, K, E, rcv_off, snd, src_map, a3, W3, Y, h, inv_c, dAt, dYp, Q, da3p,
                                        rnd);
  else if constexpr (LHMAX == 2 && RM >= 1) {
    // W3's slice (one layout for both products) and a G table per wave; the
    // precision study's operand rounding runs as its own instance (a uniform
    // branch, taken once)
    __shared__ __align__(16) unsigned short sW[3 * path_count(2) * 16 * 64];
    __shared__ __align__(16) float sG[NW * PairCount<2>::value * 16];
    constexpr int NPROD = RM == 1 ? 1 : 6;
    if (rnd)
      tpr_bwd_l2_edge_lanes_body<NW, true, NPROD, RM == 3>(N, K, E, rcv_off, snd, src_map, a3, W3, Y, h, inv_c, dAt,
                                                           dYp, Q, da3p, rnd, sW, sG);
    else
      tpr_bwd_l2_edge_lanes_body<NW, false, NPROD, RM == 3>(N, K, E, rcv_off, snd, src_map, a3, W3, Y, h, inv_c, dAt,
                                                            dYp, Q, da3p, 0, sW, sG);
  }
  else
    tpr_bwd_channel_lanes<LHMAX, RM, NW>(N, K, E, rcv_off, snd, src_map, a3, W3, Y, h, inv_c, dAt, dYp, Q, da3p,
                                         rnd);
}

namespace {
// blocks per channel tile: the resident blocks of the whole chip shared
// among the channel tiles, a multiple of 8 where possible so that the channel
// tiles of one receiver group land on the same XCD (same L2)
int tpr_grid_x(int N, int n_ct, int waves, int blocks_per_cu) {
  const int want = std::max(8, (256 * blocks_per_cu / n_ct) & ~7);
  return std::max(1, std::min(want, (N + waves - 1) / waves));
}

template <int LH, int RM>
void tpr_fwd_launch(hipStream_t s, int N, int K, const int* rcv_off, const int* snd, const int* src_map,
                    const float* a3, const float* W3, const float* Y, const float* h, float inv_c, float* At,
                    int rnd) {
  using S = TprShape<LH, false>;
  const int n_ct = K / 16;
  dim3 grid(tpr_grid_x(N, n_ct, S::waves, S::blocks_per_cu), n_ct);
  if constexpr (LH == 2 && (RM == 3 || RM == 1)) {
    if (K == 128) {
      tpr_fwd_kernel<LH, RM, S::waves, 128><<<grid, 64 * S::waves, 0, s>>>(N, K, rcv_off, snd, src_map, a3, W3, Y, h,
                                                                            inv_c, At, rnd);
      return;
    }
  }
  tpr_fwd_kernel<LH, RM><<<grid, 64 * S::waves, 0, s>>>(N, K, rcv_off, snd, src_map, a3, W3, Y, h, inv_c, At, rnd);
}

template <int LH, int RM>
void tpr_bwd_launch(hipStream_t s, int N, int K, int E, const int* rcv_off, const int* snd, const int* src_map,
                    const float* a3, const float* W3, const float* Y, const float* h, float inv_c,
                    const float* dAt, float* dYp, float* Q, float* da3p, int rnd) {
  using S = TprShape<LH, true, RM>;
  const int n_ct = K / 16;
  dim3 grid(tpr_grid_x(N, n_ct, S::waves, S::blocks_per_cu), n_ct);
  tpr_bwd_kernel<LH, RM><<<grid, 64 * S::waves, 0, s>>>(N, K, E, rcv_off, snd, src_map, a3, W3, Y, h, inv_c, dAt, dYp,
                                                    Q, da3p, rnd);
}
}  // namespace

// Instances built: every l_h <= 2 with radial mode 0 (FP32), 1 (BF16) or 2
// (split BF16), and mode 3 (split BF16 with pre-split a3) at l_h = 1 and 2.
// The l_h = 2 backward in modes 1 to 3 (the edge-lane form) needs Q.
bool tpr_supported(int lh_max, int radial_mode) {
  if (lh_max < 0 || lh_max > 2 || radial_mode < 0 || radial_mode > 3) return false;
  return radial_mode != 3 || lh_max >= 1;
}

bool launch_tpr_fwd(hipStream_t s, int lh_max, int N, int K, const int* rcv_off, const int* snd,
                    const int* src_map, const float* a3, const float* W3, const float* Y, const float* h,
                    float inv_c, float* At, int radial_mode, int tp_round) {
  if (!tpr_supported(lh_max, radial_mode)) return false;
  if (N <= 0) return true;
#define MACE_TPRF(LH, RM) tpr_fwd_launch<LH, RM>(s, N, K, rcv_off, snd, src_map, a3, W3, Y, h, inv_c, At, tp_round)
  switch (lh_max) {
    case 0:
      if (radial_mode == 1) MACE_TPRF(0, 1);
      else if (radial_mode == 2) MACE_TPRF(0, 2);
      else MACE_TPRF(0, 0);
      break;
    case 1:
      if (radial_mode == 1) MACE_TPRF(1, 1);
      else if (radial_mode == 2) MACE_TPRF(1, 2);
      else if (radial_mode == 3) MACE_TPRF(1, 3);
      else MACE_TPRF(1, 0);
      break;
    default:
      if (radial_mode == 1) MACE_TPRF(2, 1);
      else if (radial_mode == 2) MACE_TPRF(2, 2);
      else if (radial_mode == 3) MACE_TPRF(2, 3);
      else MACE_TPRF(2, 0);
      break;
  }
#undef MACE_TPRF
  return true;
}

bool launch_tpr_bwd(hipStream_t s, int lh_max, int N, int K, int E, const int* rcv_off, const int* snd,
                    const int* src_map, const float* a3, const float* W3, const float* Y, const float* h,
                    float inv_c, const float* dAt, float* dYp, float* Q, float* da3p, int radial_mode,
                    int tp_round) {
  if (!tpr_supported(lh_max, radial_mode)) return false;
  if (lh_max == 2 && radial_mode >= 1 && !Q) return false;
  if (N <= 0 || E <= 0) return true;
#define MACE_TPRB(LH, RM) \
  tpr_bwd_launch<LH, RM>(s, N, K, E, rcv_off, snd, src_map, a3, W3, Y, h, inv_c, dAt, dYp, Q, da3p, tp_round)
  switch (lh_max) {
    case 0:
      if (radial_mode == 1) MACE_TPRB(0, 1);
      else if (radial_mode == 2) MACE_TPRB(0, 2);
      else MACE_TPRB(0, 0);
      break;
    case 1:
      if (radial_mode == 1) MACE_TPRB(1, 1);
      else if (radial_mode == 2) MACE_TPRB(1, 2);
      else if (radial_mode == 3) MACE_TPRB(1, 3);
      else MACE_TPRB(1, 0);
      break;
    default:
      if (radial_mode == 1) MACE_TPRB(2, 1);
      else if (radial_mode == 2) MACE_TPRB(2, 2);
      else if (radial_mode == 3) MACE_TPRB(2, 3);
      else MACE_TPRB(2, 0);
      break;
  }
#undef MACE_TPRB
  return true;
}

}  // namespace mace
