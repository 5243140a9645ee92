// Radial MLP of the edge weights (conv_tp_weights): e [E][nb] -> 64 -> 64 ->
// 64 -> R [E][P*K], bias-free, SiLU between layers; and its VJP back to e.
// Weights are consecutive in the blob: W0 [nb][64], W1 [64][64], W2 [64][64],
// W3 [64][P*K], each row-major [in][out]; the backward pass also reads W3^T
// [P*K][64] from the transposed blob.
//
// Dense contractions on FP32 MFMA (v_mfma_f32_16x16x4_f32). A block owns a
// 64-edge tile (4 row tiles of 16) and has 4 waves. Operand layouts of the
// 16x16x4 instruction, lane l: A[l%16][l/16], B[l/16][l%16], and result
// register r holds D[4*(l/16)+r][l%16].
#include "mace_internal.h"

namespace mace {

typedef float f4 __attribute__((ext_vector_type(4)));

constexpr int kTE = 64;     // edges per block
constexpr int kH = 64;      // hidden width
constexpr int kPad = kH + 1;
constexpr int kXPad = 17;   // padded row of the radial-basis tile (nb <= 16)

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

__device__ __forceinline__ void load_basis_tile(int E, int e0, const float* __restrict__ rbf, int nb, int nb_pad,
                                                float* xs) {
  for (int idx = threadIdx.x; idx < kTE * kXPad; idx += blockDim.x) {
    int e = idx / kXPad, i = idx % kXPad;
    xs[idx] = (e0 + e < E && i < nb) ? rbf[(size_t)(e0 + e) * nb + i] : 0.f;
  }
}

template <int NBP>
__global__ void __launch_bounds__(256) radial_fwd_kernel(int E, const float* __restrict__ rbf, int nb,
                                                         const float* __restrict__ W, int PK,
                                                         float* __restrict__ R) {
  __shared__ float xs[kTE * kXPad];
  __shared__ float ha[kTE * kPad];
  __shared__ float hb[kTE * kPad];
  const int e0 = blockIdx.x * kTE;
  const float* W0 = W;
  const float* W1 = W0 + nb * kH;
  const float* W2 = W1 + kH * kH;
  const float* W3 = W2 + kH * kH;
  const int nb_pad = (nb + 3) & ~3;
  load_basis_tile(E, e0, rbf, nb, nb_pad, xs);
  __syncthreads();
  f4 z[4];
  hidden_layer<NBP>(xs, kXPad, nb, W0, ha, z);
  __syncthreads();
  hidden_layer<kH>(ha, kPad, kH, W1, hb, z);
  __syncthreads();
  hidden_layer<kH>(hb, kPad, kH, W2, ha, z);
  __syncthreads();
  const int l = threadIdx.x & 63, w = threadIdx.x >> 6;
  // the A operand (a3) is read from LDS at each MFMA: keeping its 64
  // fragments in registers would halve the occupancy
  const int nct = PK / 16;
  // B fragments of column tile ct: W3[4 ks + l/16][16 ct + l%16], ks = 0..15
  auto load_b = [&](float* bq, int ct) {
    const float* Wc = W3 + (size_t)(l >> 4) * PK + 16 * ct + (l & 15);
#pragma unroll
    for (int ks = 0; ks < kH / 4; ++ks) bq[ks] = Wc[(size_t)(4 * ks) * PK];
  };
  auto tile = [&](const float* bq, int ct) {
    f4 acc[4];
#pragma unroll
    for (int rt = 0; rt < 4; ++rt) acc[rt] = f4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int ks = 0; ks < kH / 4; ++ks)
#pragma unroll
      for (int rt = 0; rt < 4; ++rt) acc[rt] = mfma4(ha[(16 * rt + (l & 15)) * kPad + 4 * ks + (l >> 4)], bq[ks], acc[rt]);
#pragma unroll
    for (int rt = 0; rt < 4; ++rt)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int e = e0 + 16 * rt + 4 * (l >> 4) + r;
        if (e < E) R[(size_t)e * PK + 16 * ct + (l & 15)] = acc[rt][r];
      }
  };
  // two fragment buffers: the loads of the next column tile overlap the
  // MFMAs of the current one
  float bA[kH / 4], bB[kH / 4];
  if (w < nct) load_b(bA, w);
  for (int ct = w; ct < nct; ct += 8) {
    if (ct + 4 < nct) load_b(bB, ct + 4);
    tile(bA, ct);
    if (ct + 4 < nct) {
      if (ct + 8 < nct) load_b(bA, ct + 8);
      tile(bB, ct + 4);
    }
  }
}

// VJP: da3 = dR W3^T, then back through the SiLU layers to de.
template <int NBP>
__global__ void __launch_bounds__(256) radial_bwd_kernel(int E, const float* __restrict__ rbf, int nb,
                                                         const float* __restrict__ W,
                                                         const float* __restrict__ W3T, int PK,
                                                         const float* __restrict__ dR, float* __restrict__ de,
                                                         int accumulate) {
  __shared__ float xs[kTE * kXPad];
  __shared__ float ta[kTE * kPad];
  __shared__ float tb[kTE * kPad];
  __shared__ float tc[kTE * kPad];
  const int e0 = blockIdx.x * kTE;
  const float* W0 = W;
  const float* W1 = W0 + nb * kH;
  const float* W2 = W1 + kH * kH;
  const int nb_pad = (nb + 3) & ~3;
  const int tid = threadIdx.x;
  const int l = tid & 63, w = tid >> 6;
  const int col = 16 * w + (l & 15);
  // da3[e][j] = sum_n dR[e][n] W3[j][n]: dR staged through LDS 64 columns at
  // a time, double-buffered (the global loads of chunk i+1 are in flight
  // while chunk i feeds the MFMAs); W3^T fragments prefetched likewise.
  f4 acc[4];
#pragma unroll
  for (int rt = 0; rt < 4; ++rt) acc[rt] = f4{0.f, 0.f, 0.f, 0.f};
  const int nchunk = (PK + kH - 1) / kH;
  float pre[kTE * kH / 256];
  auto fetch = [&](int ch) {
    const int n0 = ch * kH;
#pragma unroll
    for (int q = 0; q < kTE * kH / 256; ++q) {
      const int idx = tid + 256 * q, r = idx / kH, c = idx % kH;
      pre[q] = (e0 + r < E && n0 + c < PK) ? dR[(size_t)(e0 + r) * PK + n0 + c] : 0.f;
    }
  };
  auto stash = [&](float* buf) {
#pragma unroll
    for (int q = 0; q < kTE * kH / 256; ++q) {
      const int idx = tid + 256 * q;
      buf[(idx / kH) * kPad + idx % kH] = pre[q];
    }
  };
  float bw[2][kH / 4];
  auto load_w = [&](float* bq, int ch) {
    const int n0 = ch * kH;
#pragma unroll
    for (int ks = 0; ks < kH / 4; ++ks) {
      const int n = n0 + 4 * ks + (l >> 4);
      bq[ks] = (n < PK) ? W3T[(size_t)n * kH + col] : 0.f;
    }
  };
  auto chunk = [&](const float* buf, const float* bq) {
#pragma unroll
    for (int ks = 0; ks < kH / 4; ++ks)
#pragma unroll
      for (int rt = 0; rt < 4; ++rt) acc[rt] = mfma4(buf[(16 * rt + (l & 15)) * kPad + 4 * ks + (l >> 4)], bq[ks], acc[rt]);
  };
  fetch(0);
  load_w(bw[0], 0);
  stash(tb);
  __syncthreads();
  for (int ch = 0; ch < nchunk; ch += 2) {
    // even chunk in tb, odd chunk goes to tc
    if (ch + 1 < nchunk) {
      fetch(ch + 1);
      load_w(bw[1], ch + 1);
    }
    chunk(tb, bw[0]);
    if (ch + 1 < nchunk) {
      stash(tc);
      __syncthreads();
      if (ch + 2 < nchunk) {
        fetch(ch + 2);
        load_w(bw[0], ch + 2);
      }
      chunk(tc, bw[1]);
      __syncthreads();           // all waves are done with tb and tc
      if (ch + 2 < nchunk) stash(tb);
      __syncthreads();
    }
  }
  __syncthreads();
  // the hidden layers are recomputed only now, so their pre-activations are
  // not live across the long dR loop above
  load_basis_tile(E, e0, rbf, nb, nb_pad, xs);
  __syncthreads();
  f4 z0[4], z1[4], z2[4];
  hidden_layer<NBP>(xs, kXPad, nb, W0, ta, z0);
  __syncthreads();
  hidden_layer<kH>(ta, kPad, kH, W1, tb, z1);
  __syncthreads();
  hidden_layer<kH>(tb, kPad, kH, W2, ta, z2);   // a2 itself is not needed below
  __syncthreads();
  // dz2 -> ta
#pragma unroll
  for (int rt = 0; rt < 4; ++rt)
#pragma unroll
    for (int r = 0; r < 4; ++r) ta[(16 * rt + 4 * (l >> 4) + r) * kPad + col] = acc[rt][r] * silu_grad(z2[rt][r]);
  __syncthreads();
  // da1[e][i] = sum_j dz2[e][j] W2[i][j]  (B[k=j][col=i] = W2[i][j])
#pragma unroll
  for (int rt = 0; rt < 4; ++rt) acc[rt] = f4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int ks = 0; ks < kH / 4; ++ks) {
    const float b = W2[col * kH + 4 * ks + (l >> 4)];
#pragma unroll
    for (int rt = 0; rt < 4; ++rt) acc[rt] = mfma4(ta[(16 * rt + (l & 15)) * kPad + 4 * ks + (l >> 4)], b, acc[rt]);
  }
#pragma unroll
  for (int rt = 0; rt < 4; ++rt)
#pragma unroll
    for (int r = 0; r < 4; ++r) tb[(16 * rt + 4 * (l >> 4) + r) * kPad + col] = acc[rt][r] * silu_grad(z1[rt][r]);
  __syncthreads();
  // da0 = dz1 W1^T
#pragma unroll
  for (int rt = 0; rt < 4; ++rt) acc[rt] = f4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int ks = 0; ks < kH / 4; ++ks) {
    const float b = W1[col * kH + 4 * ks + (l >> 4)];
#pragma unroll
    for (int rt = 0; rt < 4; ++rt) acc[rt] = mfma4(tb[(16 * rt + (l & 15)) * kPad + 4 * ks + (l >> 4)], b, acc[rt]);
  }
  __syncthreads();   // every wave has finished reading ta (dz2)
#pragma unroll
  for (int rt = 0; rt < 4; ++rt)
#pragma unroll
    for (int r = 0; r < 4; ++r) ta[(16 * rt + 4 * (l >> 4) + r) * kPad + col] = acc[rt][r] * silu_grad(z0[rt][r]);
  __syncthreads();
  // de[e][i] = sum_j dz0[e][j] W0[i][j]
  for (int idx = tid; idx < kTE * nb; idx += blockDim.x) {
    int e = idx / nb, i = idx % nb;
    if (e0 + e >= E) continue;
    float s = 0.f;
    for (int jj = 0; jj < kH; ++jj) s += ta[e * kPad + jj] * W0[i * kH + jj];
    size_t o = (size_t)(e0 + e) * nb + i;
    de[o] = accumulate ? de[o] + s : s;
  }
}

void launch_radial_fwd(hipStream_t s, int E, const float* rbf, int nb, const float* W, int PK, float* R) {
  if (E <= 0) return;
  const int g = (E + kTE - 1) / kTE;
  switch ((nb + 3) / 4) {
    case 1: radial_fwd_kernel<4><<<g, 256, 0, s>>>(E, rbf, nb, W, PK, R); break;
    case 2: radial_fwd_kernel<8><<<g, 256, 0, s>>>(E, rbf, nb, W, PK, R); break;
    case 3: radial_fwd_kernel<12><<<g, 256, 0, s>>>(E, rbf, nb, W, PK, R); break;
    default: radial_fwd_kernel<16><<<g, 256, 0, s>>>(E, rbf, nb, W, PK, R); break;
  }
}

void launch_radial_bwd(hipStream_t s, int E, const float* rbf, int nb, const float* W, const float* W3T, int PK,
                       const float* dR, float* de, int accumulate) {
  if (E <= 0) return;
  const int g = (E + kTE - 1) / kTE;
  switch ((nb + 3) / 4) {
    case 1: radial_bwd_kernel<4><<<g, 256, 0, s>>>(E, rbf, nb, W, W3T, PK, dR, de, accumulate); break;
    case 2: radial_bwd_kernel<8><<<g, 256, 0, s>>>(E, rbf, nb, W, W3T, PK, dR, de, accumulate); break;
    case 3: radial_bwd_kernel<12><<<g, 256, 0, s>>>(E, rbf, nb, W, W3T, PK, dR, de, accumulate); break;
    default: radial_bwd_kernel<16><<<g, 256, 0, s>>>(E, rbf, nb, W, W3T, PK, dR, de, accumulate); break;
  }
}

}  // namespace mace
