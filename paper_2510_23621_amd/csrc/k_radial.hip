// Radial MLP of the edge weights (conv_tp_weights): e [E][nb] -> 64 -> 64 ->
// 64 -> R [E][P*K], bias-free, SiLU between layers; and its VJP back to e.
// Weights are consecutive in the blob: W0 [nb][64], W1 [64][64], W2 [64][64],
// W3 [64][P*K], each row-major [in][out]; the backward pass also reads W3^T
// [P*K][64] from the transposed blob.
//
// The three hidden layers run here (a3 [E][64] is written out, 256 bytes per
// edge); the wide last layer is computed inside the tensor-product kernels,
// which also hand back dE/da3 as per-channel-tile partials. A block owns a
// 64-edge tile (4 row tiles of 16) and has 4 waves, wave w the 16 columns
// 16w .. 16w + 15 of a layer. The 64-wide layers (and their transposed
// products in the backward pass) run as FP32-accurate products on the
// bfloat16 MFMA pipe (v_mfma_f32_16x16x32_bf16; each FP32 operand carried as
// three bfloat16 parts, six partial products, as in the edge product): lane l
// supplies A[l%16][8(l/16) + i] and B[8(l/16) + i][l%16], i = 0..7, and result
// register r holds D[4(l/16) + r][l%16]. The weights are the A operand and
// the activations of 16 edges the B operand, so that a lane's results are four
// consecutive columns of one edge, which it splits into parts once for the
// next layer. The narrow input layer (nb <= 16 inputs) runs on FP32 MFMA
// (v_mfma_f32_16x16x4_f32, A[l%16][l/16], B[l/16][l%16]), with the same
// operand roles; the precision study's rounded instances run every layer on
// FP32 MFMA with the activations as A (results: rows 4(l/16) + r of column
// l%16).
#include <type_traits>

#include "mace_internal.h"

namespace mace {

typedef float f4 __attribute__((ext_vector_type(4)));

constexpr int kTE = 64;     // edges per block
constexpr int kH = 64;      // hidden width
constexpr int kPad = kH + 4;   // row pitch = 4 (mod 32): A-fragment reads hit 2 lanes per bank
constexpr int kXPad = 20;  // padded row of the radial-basis tile (nb <= 16)

__device__ __forceinline__ f4 mfma4(float a, float b, f4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, c, 0, 0, 0);
}

// z[e][j] = sum_i in[e][i] W[i][j] for the tile's 64 edges; wave w owns the
// columns j = 16w .. 16w+15. in: LDS rows of stride ldin, zero beyond nin
// valid inputs up to nin_pad (a multiple of 4). Writes silu(z) to out (LDS,
// stride kPad) and returns z in the result layout.
template <int NIN_PAD>
__device__ __forceinline__ void hidden_layer(const float* __restrict__ in, int ldin, int nin,
                                             const float* __restrict__ W, float* __restrict__ out, f4* z) {
  const int l = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int col = 16 * w + (l & 15);
  f4 acc[4];
#pragma unroll
  for (int rt = 0; rt < 4; ++rt) acc[rt] = f4{0.f, 0.f, 0.f, 0.f};
  float b[NIN_PAD / 4];
#pragma unroll
  for (int ks = 0; ks < NIN_PAD / 4; ++ks) {
    const int k = 4 * ks + (l >> 4);
    b[ks] = (k < nin) ? W[k * kH + col] : 0.f;
  }
#pragma unroll
  for (int ks = 0; ks < NIN_PAD / 4; ++ks) {
    const int k = 4 * ks + (l >> 4);
#pragma unroll
    for (int rt = 0; rt < 4; ++rt) acc[rt] = mfma4(in[(16 * rt + (l & 15)) * ldin + k], b[ks], acc[rt]);
  }
#pragma unroll
  for (int rt = 0; rt < 4; ++rt) {
    z[rt] = acc[rt];
#pragma unroll
    for (int r = 0; r < 4; ++r) out[(16 * rt + 4 * (l >> 4) + r) * kPad + col] = silu(acc[rt][r]);
  }
}

// The two halves of hidden_layer, so that the next layer's B fragments can
// be in flight while the current layer's MFMAs run.
template <int NIN_PAD, bool RND = false>
__device__ __forceinline__ void load_b_frag(const float* __restrict__ W, int nin, float* b, int rnd = 0) {
  const int l = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int col = 16 * w + (l & 15);
#pragma unroll
  for (int ks = 0; ks < NIN_PAD / 4; ++ks) {
    const int k = 4 * ks + (l >> 4);
    b[ks] = (k < nin) ? W[k * kH + col] : 0.f;
    if constexpr (RND) b[ks] = lowp_round(b[ks], rnd);
  }
}

template <int NIN_PAD, bool STORE = true, bool RND = false>
__device__ __forceinline__ void hidden_mma(const float* __restrict__ in, int ldin, const float* b,
                                           float* __restrict__ out, f4* z, int rnd = 0) {
  const int l = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int col = 16 * w + (l & 15);
  f4 acc[4];
#pragma unroll
  for (int rt = 0; rt < 4; ++rt) acc[rt] = f4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int ks = 0; ks < NIN_PAD / 4; ++ks) {
    const int k = 4 * ks + (l >> 4);
#pragma unroll
    for (int rt = 0; rt < 4; ++rt) acc[rt] = mfma4(in[(16 * rt + (l & 15)) * ldin + k], b[ks], acc[rt]);
  }
#pragma unroll
  for (int rt = 0; rt < 4; ++rt) {
    z[rt] = acc[rt];
    if constexpr (STORE) {
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const float a = silu(acc[rt][r]);
        out[(16 * rt + 4 * (l >> 4) + r) * kPad + col] = RND ? lowp_round(a, rnd) : a;
      }
    }
  }
}

// ---- 64-wide layers on split-BF16 MFMA
typedef unsigned short us8v __attribute__((ext_vector_type(8)));
typedef __bf16 bf8v __attribute__((ext_vector_type(8)));
typedef unsigned u4v __attribute__((ext_vector_type(4)));

__device__ __forceinline__ f4 mfma_b16(us8v a, us8v b, f4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf8v, a), __builtin_bit_cast(bf8v, b), c, 0, 0, 0);
}

// the three bfloat16 parts of eight FP32 values, element i of each operand
// word holding value i (two values per conversion)
__device__ __forceinline__ void split8(f4 lo, f4 hi, us8v& p0, us8v& p1, us8v& p2) {
  u4v w0, w1, w2;
#pragma unroll
  for (int h = 0; h < 4; ++h) {
    const f2v x = h < 2 ? f2v{lo[2 * h], lo[2 * h + 1]} : f2v{hi[2 * h - 4], hi[2 * h - 3]};
    unsigned a, b, c;
    split3_pair(x, a, b, c);
    w0[h] = a;
    w1[h] = b;
    w2[h] = c;
  }
  p0 = __builtin_bit_cast(us8v, w0);
  p1 = __builtin_bit_cast(us8v, w1);
  p2 = __builtin_bit_cast(us8v, w2);
}

// B operand parts of a 64 x 64 layer for this wave's 16 columns: W[k][col]
// (TR: W[col][k], the transposed product) for k = 32 ks + 8 (l/16) + i
template <bool TR>
__device__ __forceinline__ void load_b_parts64(const float* __restrict__ W, us8v (&b)[2][3]) {
  const int l = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int col = 16 * w + (l & 15);
#pragma unroll
  for (int ks = 0; ks < 2; ++ks) {
    float v[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const int k = 32 * ks + 8 * (l >> 4) + i;
      v[i] = TR ? W[col * kH + k] : W[k * kH + col];
    }
    split8(f4{v[0], v[1], v[2], v[3]}, f4{v[4], v[5], v[6], v[7]}, b[ks][0], b[ks][1], b[ks][2]);
  }
}

// ---- prologue layers with the operands' roles swapped: A = the weights'
// column fragment of the wave's 16 columns, B = the activations of 16 edges,
// so that result register r of lane l holds column 16w + 4(l/16) + r of edge
// 16 rt + l%16 (four consecutive columns of one edge per lane). Each layer's
// output is split into its three bfloat16 parts once, by the wave that
// produced it, into part planes in LDS (row = edge, pitch kPP), which every
// wave of the next layer reads as its B operand.
constexpr int kPP = kH + 8;          // 72 bfloat16 per plane row (36 dwords, 4 mod 32)
constexpr int kPlane = kTE * kPP;    // elements per part plane

// silu(z) (SILU) or z of the wave's columns, as three part planes
template <bool SILU = true>
__device__ __forceinline__ void store_parts_t(const f4* z, unsigned short* __restrict__ P) {
  const int l = threadIdx.x & 63, w = threadIdx.x >> 6;
  auto act = [](float x) { return SILU ? silu(x) : x; };
#pragma unroll
  for (int rt = 0; rt < 4; ++rt) {
    unsigned p0[2], p1[2], p2[2];
    split3_pair(f2v{act(z[rt][0]), act(z[rt][1])}, p0[0], p1[0], p2[0]);
    split3_pair(f2v{act(z[rt][2]), act(z[rt][3])}, p0[1], p1[1], p2[1]);
    unsigned short* d = P + (16 * rt + (l & 15)) * kPP + 16 * w + 4 * (l >> 4);
    *reinterpret_cast<uint2*>(d) = make_uint2(p0[0], p0[1]);
    *reinterpret_cast<uint2*>(d + kPlane) = make_uint2(p1[0], p1[1]);
    *reinterpret_cast<uint2*>(d + 2 * kPlane) = make_uint2(p2[0], p2[1]);
  }
}

// the narrow input layer on FP32 MFMA, operands swapped: z = (x W0) of the
// wave's columns for the tile's 64 edges (x: LDS rows of stride kXPad)
template <int NIN_PAD>
__device__ __forceinline__ void input_mma_t(const float* __restrict__ xs, const float* b, f4* z) {
  const int l = threadIdx.x & 63;
#pragma unroll
  for (int rt = 0; rt < 4; ++rt) z[rt] = f4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int ks = 0; ks < NIN_PAD / 4; ++ks)
#pragma unroll
    for (int rt = 0; rt < 4; ++rt) z[rt] = mfma4(b[ks], xs[(16 * rt + (l & 15)) * kXPad + 4 * ks + (l >> 4)], z[rt]);
}

// a 64-input layer on split-BF16 products from part planes, operands swapped;
// within each K step the six partial products go from the smallest to the
// largest
__device__ __forceinline__ void mma64_x3t(const unsigned short* __restrict__ P, const us8v (&b)[2][3], f4* z) {
  const int l = threadIdx.x & 63;
#pragma unroll
  for (int rt = 0; rt < 4; ++rt) z[rt] = f4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int ks = 0; ks < 2; ++ks)
#pragma unroll
    for (int rt = 0; rt < 4; ++rt) {
      const unsigned short* ar = P + (16 * rt + (l & 15)) * kPP + 32 * ks + 8 * (l >> 4);
      const us8v a0 = *reinterpret_cast<const us8v*>(ar);
      const us8v a1 = *reinterpret_cast<const us8v*>(ar + kPlane);
      const us8v a2 = *reinterpret_cast<const us8v*>(ar + 2 * kPlane);
      f4 c = z[rt];
      c = mfma_b16(b[ks][0], a2, c);
      c = mfma_b16(b[ks][1], a1, c);
      c = mfma_b16(b[ks][2], a0, c);
      c = mfma_b16(b[ks][0], a1, c);
      c = mfma_b16(b[ks][1], a0, c);
      z[rt] = mfma_b16(b[ks][0], a0, c);
    }
}

template <bool RND = false>
__device__ __forceinline__ void load_basis_tile(int E, int e0, const float* __restrict__ rbf, int nb, int nb_pad,
                                                float* xs, int rnd = 0) {
  for (int idx = threadIdx.x; idx < kTE * kXPad; idx += blockDim.x) {
    int e = idx / kXPad, i = idx % kXPad;
    const float v = (e0 + e < E && i < nb) ? rbf[(size_t)(e0 + e) * nb + i] : 0.f;
    xs[idx] = RND ? lowp_round(v, rnd) : v;
  }
}

// Edge prologue for a 64-edge tile: geometry of every edge (Y and the radial
// basis e, written out; the first wave computes one edge per lane in FP64),
// then the hidden layers a3 = SiLU(SiLU(SiLU(e W0) W1) W2) of the radial MLP
// of every interaction layer in rs, all from the same e. RND: the precision
// study's rounding of every layer's input and weights (rs.rnd: 1 bfloat16,
// 2 binary16); the basis is written out unrounded.
template <int NBP, bool RND>
__global__ void __launch_bounds__(256) edge_prologue_kernel(int E, const float* __restrict__ pos,
                                                            const int* __restrict__ snd, const int* __restrict__ rcv,
                                                            const double4* __restrict__ shift, double rc, int p,
                                                            int nb, float* __restrict__ Y, float* __restrict__ rbf,
                                                            RadialSet rs, int* __restrict__ status) {
  __shared__ float xs[kTE * kXPad];
  // RND: the FP32 activations ha, hb; otherwise the three part planes
  __shared__ __align__(16) float hbuf[2 * kTE * kPad];
  static_assert(3 * kPlane * sizeof(unsigned short) <= sizeof(hbuf), "part planes fit the activation buffers");
  float* ha = hbuf;
  float* hb = hbuf + kTE * kPad;
  unsigned short* P = reinterpret_cast<unsigned short*>(hbuf);
  const int e0 = blockIdx.x * kTE;
  // B fragments: bc for the layer being computed, bn for the next one (in
  // flight meanwhile); the first is requested before the geometry
  float bc[kH / 4], bn[kH / 4];
  load_b_frag<NBP, RND>(rs.W[0], nb, bc, rs.rnd);
  if (threadIdx.x < kTE) {
    const int e = e0 + threadIdx.x;
    float row[kXPad];
#pragma unroll
    for (int i = 0; i < kXPad; ++i) row[i] = 0.f;
    if (e < E) {
      float y[16];
      const int bad = edge_geometry(e, pos, snd, rcv, shift, rc, p, nb, y, row);
      if (bad) atomicOr(status, bad);
      float4* Yv = reinterpret_cast<float4*>(Y + (size_t)e * 16);
#pragma unroll
      for (int v = 0; v < 4; ++v) Yv[v] = make_float4(y[4 * v], y[4 * v + 1], y[4 * v + 2], y[4 * v + 3]);
      for (int n = 0; n < nb; ++n) rbf[(size_t)e * nb + n] = row[n];
    }
#pragma unroll
    for (int i = 0; i < kXPad; ++i) xs[threadIdx.x * kXPad + i] = RND ? lowp_round(row[i], rs.rnd) : row[i];
  }
  __syncthreads();
  for (int t = 0; t < rs.n; ++t) {
    const float* W0 = rs.W[t];
    const float* W1 = W0 + nb * kH;
    const float* W2 = W1 + kH * kH;
    f4 z[4];
    if constexpr (RND) {
      load_b_frag<kH, RND>(W1, kH, bn, rs.rnd);
      hidden_mma<NBP, true, RND>(xs, kXPad, bc, ha, z, rs.rnd);
      __syncthreads();
      load_b_frag<kH, RND>(W2, kH, bc, rs.rnd);
      hidden_mma<kH, true, RND>(ha, kPad, bn, hb, z, rs.rnd);
      __syncthreads();
      if (t + 1 < rs.n) load_b_frag<NBP, RND>(rs.W[t + 1], nb, bn, rs.rnd);
      hidden_mma<kH, true, RND>(hb, kPad, bc, ha, z, rs.rnd);
      __syncthreads();
#pragma unroll
      for (int ks = 0; ks < NBP / 4; ++ks) bc[ks] = bn[ks];
      float* a3 = rs.a3[t];
      unsigned short* a3x = rs.a3x[t];
      for (int idx = threadIdx.x; idx < kTE * kH / 4; idx += blockDim.x) {
        const int e = idx >> 4, c4 = idx & 15;
        if (e0 + e >= E) continue;
        const f4 v = *reinterpret_cast<const f4*>(ha + e * kPad + 4 * c4);
        if (a3x) {   // the three bfloat16 parts, [E][3][64]
          unsigned p0[2], p1[2], p2[2];
          split3_pair(f2v{v[0], v[1]}, p0[0], p1[0], p2[0]);
          split3_pair(f2v{v[2], v[3]}, p0[1], p1[1], p2[1]);
          unsigned short* row = a3x + (size_t)(e0 + e) * 3 * kH + 4 * c4;
          *reinterpret_cast<uint2*>(row) = make_uint2(p0[0], p0[1]);
          *reinterpret_cast<uint2*>(row + kH) = make_uint2(p1[0], p1[1]);
          *reinterpret_cast<uint2*>(row + 2 * kH) = make_uint2(p2[0], p2[1]);
        } else {
          *reinterpret_cast<f4*>(a3 + (size_t)(e0 + e) * kH + 4 * c4) = v;
        }
      }
      __syncthreads();   // ha is rewritten by the next layer's MLP
    } else {
      // the 64-wide layers on split-BF16 products from part planes split once
      // by their producer, the next layer's weight parts in flight meanwhile
      us8v b1[2][3], b2[2][3];
      load_b_parts64<false>(W1, b1);
      input_mma_t<NBP>(xs, bc, z);
      __syncthreads();   // the previous interaction layer's reads of the planes are done
      store_parts_t(z, P);
      __syncthreads();
      load_b_parts64<false>(W2, b2);
      mma64_x3t(P, b1, z);
      __syncthreads();   // every wave has read the planes
      store_parts_t(z, P);
      __syncthreads();
      if (t + 1 < rs.n) load_b_frag<NBP, false>(rs.W[t + 1], nb, bn);
      mma64_x3t(P, b2, z);
#pragma unroll
      for (int ks = 0; ks < NBP / 4; ++ks) bc[ks] = bn[ks];
      // a3 = silu(z): four consecutive columns of one edge per lane, straight
      // to memory (FP32, or the three bfloat16 parts [E][3][64])
      const int l = threadIdx.x & 63, w = threadIdx.x >> 6;
      const int c0 = 16 * w + 4 * (l >> 4);
      float* a3 = rs.a3[t];
      unsigned short* a3x = rs.a3x[t];
#pragma unroll
      for (int rt = 0; rt < 4; ++rt) {
        const int e = e0 + 16 * rt + (l & 15);
        if (e >= E) continue;
        const f4 v = {silu(z[rt][0]), silu(z[rt][1]), silu(z[rt][2]), silu(z[rt][3])};
        if (a3x) {
          unsigned p0[2], p1[2], p2[2];
          split3_pair(f2v{v[0], v[1]}, p0[0], p1[0], p2[0]);
          split3_pair(f2v{v[2], v[3]}, p0[1], p1[1], p2[1]);
          unsigned short* row = a3x + (size_t)e * 3 * kH + c0;
          *reinterpret_cast<uint2*>(row) = make_uint2(p0[0], p0[1]);
          *reinterpret_cast<uint2*>(row + kH) = make_uint2(p1[0], p1[1]);
          *reinterpret_cast<uint2*>(row + 2 * kH) = make_uint2(p2[0], p2[1]);
        } else {
          *reinterpret_cast<f4*>(a3 + (size_t)e * kH + c0) = v;
        }
      }
    }
  }
}

// de = VJP of the hidden layers given dE/da3, which arrives as n_part partials
// da3p[part][E][64] summed here in part order. The pre-activations z0, z1, z2
// are recomputed from the radial basis (three MFMA layers per 64-edge tile;
// cheaper than storing silu'(z) for every edge and reading it back), so
// the pass is dz2 = da3 silu'(z2), dz1 = (dz2 W2^T) silu'(z1),
// dz0 = (dz1 W1^T) silu'(z0), de = dz0 W0^T. The same pass folds the partials
// dYp[part][E][16] of dE/dY into dY. With accumulate set, de and dY are added
// to instead of overwritten.
template <int NBP, int NPART, bool RND>
__global__ void __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(RND ? 2 : 3))) radial_bwd_kernel(int E, const float* __restrict__ rbf, int nb,
                                                         const float* __restrict__ W,
                                                         const float* __restrict__ da3p,
                                                         const float* __restrict__ dYp,
                                                         float* __restrict__ dY, float* __restrict__ de,
                                                         int accumulate, int rnd) {
  __shared__ float xs[kTE * kXPad];
  // RND: the FP32 tiles ta, tb; otherwise three part planes and one FP32 tile
  constexpr int kPlanesF = 3 * kPlane / 2;   // floats taken by the part planes
  __shared__ __align__(16) float tbuf[kPlanesF + kTE * kPad];
  static_assert(2 * kTE * kPad <= kPlanesF + kTE * kPad, "the FP32 tiles fit");
  float* ta = tbuf;
  float* tb = tbuf + kTE * kPad;
  const int e0 = blockIdx.x * kTE;
  const float* W0 = W;
  const float* W1 = W0 + nb * kH;
  const float* W2 = W1 + kH * kH;
  const int tid = threadIdx.x;
  const int l = tid & 63, w = tid >> 6;
  const int col = 16 * w + (l & 15);
  // The partial sums of dE/da3 (thread t holds rows (t + 256 s) / 16, s = 0..3,
  // float4 column (t % 16), summed in part order) and of dE/dY (written out
  // here). Even blocks take them before the forward recompute and odd blocks
  // after it, so that the blocks that start together on a CU are not all in
  // their memory phase, or all in their MFMA phase, at the same time.
  f4 pacc[4];
  auto sum_partials = [&]() {
#pragma unroll
    for (int sr = 0; sr < 4; ++sr) {
      const int idx = tid + 256 * sr;
      const int row = idx >> 4, c4 = idx & 15;
      const int e = min(e0 + row, E - 1);
      f4 v = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int q = 0; q < NPART; ++q) v += *reinterpret_cast<const f4*>(da3p + ((size_t)q * E + e) * kH + 4 * c4);
      pacc[sr] = e0 + row < E ? v : f4{0.f, 0.f, 0.f, 0.f};
    }
    {
      const int e = e0 + (tid >> 2), c4 = tid & 3;
      if (e < E) {
        f4 v = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int q = 0; q < NPART; ++q) v += *reinterpret_cast<const f4*>(dYp + ((size_t)q * E + e) * 16 + 4 * c4);
        f4* o = reinterpret_cast<f4*>(dY + (size_t)e * 16 + 4 * c4);
        *o = accumulate ? *o + v : v;
      }
    }
  };
  const bool parts_first = (blockIdx.x & 1) == 0;
  if constexpr (!RND) {
    // The layers with the operands' roles swapped (as in the edge prologue):
    // every 64-wide product reads its activations as part planes split once
    // by the wave that produced them; lane l holds columns c0 .. c0 + 3 of
    // edge 16 rt + l%16 of every result.
    unsigned short* P = reinterpret_cast<unsigned short*>(tbuf);
    float* F = tbuf + kPlanesF;   // [edge][kPad] FP32: dE/da3, then dz0
    const int c0 = 16 * w + 4 * (l >> 4);
    if (parts_first) sum_partials();
    float bc[NBP / 4];
    us8v bp[2][3];
    load_b_frag<NBP, false>(W0, nb, bc);
    load_b_parts64<false>(W1, bp);
    load_basis_tile<false>(E, e0, rbf, nb, (nb + 3) & ~3, xs);
    __syncthreads();
    f4 z0[4], z1[4], z2[4], acc[4];
    input_mma_t<NBP>(xs, bc, z0);
    store_parts_t(z0, P);
    __syncthreads();
    mma64_x3t(P, bp, z1);
    load_b_parts64<false>(W2, bp);
    __syncthreads();   // every wave has read the planes
    store_parts_t(z1, P);
    __syncthreads();
    mma64_x3t(P, bp, z2);   // z2 only (a3 itself is not needed)
    if (!parts_first) sum_partials();
#pragma unroll
    for (int sr = 0; sr < 4; ++sr) {
      const int idx = tid + 256 * sr;
      *reinterpret_cast<f4*>(F + (idx >> 4) * kPad + 4 * (idx & 15)) = pacc[sr];
    }
    load_b_parts64<true>(W2, bp);   // A of dz2 W2^T: W2[i][j], i the wave's output column
    __syncthreads();   // dE/da3 in F; every wave has read the planes
    // dz2 = da3 silu'(z2)
#pragma unroll
    for (int rt = 0; rt < 4; ++rt) {
      const f4 g = *reinterpret_cast<const f4*>(F + (16 * rt + (l & 15)) * kPad + c0);
#pragma unroll
      for (int r = 0; r < 4; ++r) acc[rt][r] = g[r] * silu_grad(z2[rt][r]);
    }
    store_parts_t<false>(acc, P);
    __syncthreads();
    // dz1 = (dz2 W2^T) silu'(z1)
    mma64_x3t(P, bp, acc);
    load_b_parts64<true>(W1, bp);
#pragma unroll
    for (int rt = 0; rt < 4; ++rt)
#pragma unroll
      for (int r = 0; r < 4; ++r) acc[rt][r] *= silu_grad(z1[rt][r]);
    __syncthreads();   // every wave has read the planes
    store_parts_t<false>(acc, P);
    __syncthreads();
    // dz0 = (dz1 W1^T) silu'(z0), FP32 into F for the input layer's product
    mma64_x3t(P, bp, acc);
#pragma unroll
    for (int rt = 0; rt < 4; ++rt) {
      f4 v;
#pragma unroll
      for (int r = 0; r < 4; ++r) v[r] = acc[rt][r] * silu_grad(z0[rt][r]);
      *reinterpret_cast<f4*>(F + (16 * rt + (l & 15)) * kPad + c0) = v;
    }
    __syncthreads();
    ta = F;   // dz0 for the de product below
  } else {
    // the precision study's rounded instance: FP32 MFMA on rounded operands,
    // FP32 tiles in the result layout (lane l: rows 4(l/16) + r, column col)
    if (parts_first) sum_partials();
    float bc[kH / 4], bn[kH / 4];
    load_b_frag<NBP, RND>(W0, nb, bc, rnd);
    load_basis_tile<RND>(E, e0, rbf, nb, (nb + 3) & ~3, xs, rnd);
    __syncthreads();
    f4 z0[4], z1[4], z2[4];
    load_b_frag<kH, RND>(W1, kH, bn, rnd);
    hidden_mma<NBP, true, RND>(xs, kXPad, bc, ta, z0, rnd);
    __syncthreads();
    load_b_frag<kH, RND>(W2, kH, bc, rnd);
    hidden_mma<kH, true, RND>(ta, kPad, bn, tb, z1, rnd);
    __syncthreads();   // every wave is done with ta
    auto store_partials = [&]() {
#pragma unroll
      for (int sr = 0; sr < 4; ++sr) {
        const int idx = tid + 256 * sr;
        *reinterpret_cast<f4*>(ta + (idx >> 4) * kPad + 4 * (idx & 15)) = pacc[sr];
      }
    };
    if (parts_first) store_partials();
    // z2 only (a3 itself is not needed)
    hidden_mma<kH, false, RND>(tb, kPad, bc, nullptr, z2, rnd);
    if (!parts_first) {
      sum_partials();
      store_partials();
    }
    // operand of the first backward MFMA stage: B[k = j][col = i] = W2[i][j]
    float b2[kH / 4];
#pragma unroll
    for (int ks = 0; ks < kH / 4; ++ks) b2[ks] = lowp_round(W2[col * kH + 4 * ks + (l >> 4)], rnd);
    __syncthreads();
    // dz2 = da3 silu'(z2), in place
#pragma unroll
    for (int rt = 0; rt < 4; ++rt)
#pragma unroll
      for (int r = 0; r < 4; ++r) ta[(16 * rt + 4 * (l >> 4) + r) * kPad + col] *= silu_grad(z2[rt][r]);
    __syncthreads();
    f4 acc[4];
    // dz1 = (dz2 W2^T) silu'(z1) into tb
    float b1[kH / 4];
#pragma unroll
    for (int ks = 0; ks < kH / 4; ++ks) b1[ks] = lowp_round(W1[col * kH + 4 * ks + (l >> 4)], rnd);
#pragma unroll
    for (int rt = 0; rt < 4; ++rt) acc[rt] = f4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int ks = 0; ks < kH / 4; ++ks)
#pragma unroll
      for (int rt = 0; rt < 4; ++rt)
        acc[rt] = mfma4(ta[(16 * rt + (l & 15)) * kPad + 4 * ks + (l >> 4)], b2[ks], acc[rt]);
#pragma unroll
    for (int rt = 0; rt < 4; ++rt)
#pragma unroll
      for (int r = 0; r < 4; ++r) tb[(16 * rt + 4 * (l >> 4) + r) * kPad + col] = acc[rt][r] * silu_grad(z1[rt][r]);
    __syncthreads();
    // dz0 = (dz1 W1^T) silu'(z0) into ta (every wave has read ta before the barrier above)
#pragma unroll
    for (int rt = 0; rt < 4; ++rt) acc[rt] = f4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int ks = 0; ks < kH / 4; ++ks)
#pragma unroll
      for (int rt = 0; rt < 4; ++rt)
        acc[rt] = mfma4(tb[(16 * rt + (l & 15)) * kPad + 4 * ks + (l >> 4)], b1[ks], acc[rt]);
#pragma unroll
    for (int rt = 0; rt < 4; ++rt)
#pragma unroll
      for (int r = 0; r < 4; ++r) ta[(16 * rt + 4 * (l >> 4) + r) * kPad + col] = acc[rt][r] * silu_grad(z0[rt][r]);
    __syncthreads();
  }
  // de[e][i] = sum_j dz0[e][j] W0[i][j] on MFMA: wave w takes the edge rows
  // 16w .. 16w + 15, the 16 result columns are i (zero past nb <= 16)
  {
    const int i = l & 15;
    f4 d = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int ks = 0; ks < kH / 4; ++ks) {
      float bw = i < nb ? W0[i * kH + 4 * ks + (l >> 4)] : 0.f;
      if constexpr (RND) bw = lowp_round(bw, rnd);
      d = mfma4(ta[(16 * w + (l & 15)) * kPad + 4 * ks + (l >> 4)], bw, d);
    }
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int e = e0 + 16 * w + 4 * (l >> 4) + r;
      if (e < E && i < nb) {
        const size_t o = (size_t)e * nb + i;
        de[o] = accumulate ? de[o] + d[r] : d[r];
      }
    }
  }
}

void launch_edge_prologue(hipStream_t s, int E, const float* pos, const int* snd, const int* rcv,
                          const double4* shift, double rc, int p, int nb, float* Y, float* rbf,
                          const RadialSet& rs, int* status) {
  if (E <= 0) return;
  const int g = (E + kTE - 1) / kTE;
  auto go = [&](auto R) {
    constexpr bool RND = decltype(R)::value;
    if (nb <= 8) edge_prologue_kernel<8, RND><<<g, 256, 0, s>>>(E, pos, snd, rcv, shift, rc, p, nb, Y, rbf, rs, status);
    else edge_prologue_kernel<16, RND><<<g, 256, 0, s>>>(E, pos, snd, rcv, shift, rc, p, nb, Y, rbf, rs, status);
  };
  if (rs.rnd) go(std::true_type{});
  else go(std::false_type{});
}

void launch_radial_bwd(hipStream_t s, int E, const float* rbf, int nb, const float* W, const float* da3p,
                       const float* dYp, int n_part, float* dY, float* de, int accumulate, int rnd) {
  if (E <= 0) return;
  const int g = (E + kTE - 1) / kTE;
  auto go = [&](auto NP) {
    constexpr int NPART = decltype(NP)::value;
    if (rnd) {
      if (nb <= 8) radial_bwd_kernel<8, NPART, true><<<g, 256, 0, s>>>(E, rbf, nb, W, da3p, dYp, dY, de, accumulate, rnd);
      else radial_bwd_kernel<16, NPART, true><<<g, 256, 0, s>>>(E, rbf, nb, W, da3p, dYp, dY, de, accumulate, rnd);
    } else {
      if (nb <= 8) radial_bwd_kernel<8, NPART, false><<<g, 256, 0, s>>>(E, rbf, nb, W, da3p, dYp, dY, de, accumulate, 0);
      else radial_bwd_kernel<16, NPART, false><<<g, 256, 0, s>>>(E, rbf, nb, W, da3p, dYp, dY, de, accumulate, 0);
    }
  };
  switch (n_part) {   // K / 16 for K in {32, 64, 96, 128}, or 1 (whole values)
    case 1: go(std::integral_constant<int, 1>{}); break;
    case 2: go(std::integral_constant<int, 2>{}); break;
    case 4: go(std::integral_constant<int, 4>{}); break;
    case 6: go(std::integral_constant<int, 6>{}); break;
    case 8: go(std::integral_constant<int, 8>{}); break;
  }
}

}  // namespace mace
