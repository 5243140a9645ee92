// First interaction layer in factorised form.
//
// At layer 0 the sender features are the species table (h[j][k] =
// table[z_j][k]) and every path is (0, l, l), whose coupling is the identity,
// so the neighbour sum of Eq. 26 with the last radial layer written out is
//   At[i][c][k] = inv_c sum_{e: rcv_e = i} (sum_j a3[e][j] W3[j][p(l) K + k]) table[z_e][k] Y[e][c]
//               = sum_{s, j} U[i][c][s][j] Wf[l][s, j][k],
//   U[i][c][s][j] = sum_{e: rcv_e = i, z_e = s} a3[e][j] Y[e][c],
//   Wf[l][s, j][k] = inv_c W3[j][p(l) K + k] table[s][k],
// with c = l^2 + m the component of Y and of At, p(l) the path (0, l, l) and
// z_e the species of the edge's sender. The per-edge product is then 64 x 16
// multiply-adds into U instead of the P K-wide radial layer, and the rest is
// a node-level contraction over S * 64 channels that runs on the channel-mixing
// linear kernel (where it can be composed with the path-merging and species
// linears that follow it). The backward pass receives gU = dE/dU from the
// transposed contraction and returns per edge
//   dE/da3[e][j] = sum_c gU[i][c][z_e][j] Y[e][c],
//   dE/dY[e][c]  = sum_j gU[i][c][z_e][j] a3[e][j].
// In the BF16-radial mode a3 enters as its bfloat16 rounding (the weights
// carry the rounded W3), which is the same product as the per-edge form.
//
// U and gU are [N][16][S * 64]. One block of four waves per receiver; lane
// j = 0..63 is the radial hidden unit. Every sum has a fixed order (the
// gather's: each wave over its edges in CSR order, then the four waves in
// order), so results do not depend on scheduling.
#include "mace_internal.h"

namespace mace {

typedef float f4 __attribute__((ext_vector_type(4)));

constexpr int kL0BwdEdges = 4;   // edges per wave and iteration, their loads issued together

// Wave w takes the receiver's edges e_beg + w, e_beg + w + 4, ... (four per
// iteration, their loads issued together) for all 16 components; the waves'
// sums are added in wave order through LDS (waves 1-3 store, wave 0 adds).
template <int S, bool RB>
__global__ void __launch_bounds__(256) l0_gather_kernel(int N, const int* __restrict__ rcv_off,
                                                        const int* __restrict__ snd_z, const float* __restrict__ a3,
                                                        const float* __restrict__ Y, float* __restrict__ U) {
  constexpr int KI = 64 * S;
  __shared__ float part[3][16][KI];
  const int i = blockIdx.x;
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  float acc[S][16];
#pragma unroll
  for (int s = 0; s < S; ++s)
#pragma unroll
    for (int c = 0; c < 16; ++c) acc[s][c] = 0.f;
  const int e_beg = rcv_off[i], e_end = rcv_off[i + 1];
  for (int e = e_beg + w; e < e_end; e += 4 * kL0BwdEdges) {
    float a[kL0BwdEdges];
    f4 y[kL0BwdEdges][4];
    int z[kL0BwdEdges];
#pragma unroll
    for (int q = 0; q < kL0BwdEdges; ++q) {
      const int eq = min(e + 4 * q, e_end - 1);
      z[q] = snd_z[eq];
      a[q] = a3[(size_t)eq * 64 + lane];
#pragma unroll
      for (int v = 0; v < 4; ++v) y[q][v] = reinterpret_cast<const f4*>(Y + (size_t)eq * 16)[v];
    }
#pragma unroll
    for (int q = 0; q < kL0BwdEdges; ++q) {
      const bool valid = e + 4 * q < e_end;
      const float av = valid ? (RB ? bf16_round(a[q]) : a[q]) : 0.f;   // past e_end: adds zero
      const int zq = valid ? z[q] : -1;
#pragma unroll
      for (int s = 0; s < S; ++s)
        if (zq == s) {
#pragma unroll
          for (int c = 0; c < 16; ++c) acc[s][c] += av * y[q][c >> 2][c & 3];
        }
    }
  }
  if (w > 0) {
#pragma unroll
    for (int c = 0; c < 16; ++c)
#pragma unroll
      for (int s = 0; s < S; ++s) part[w - 1][c][64 * s + lane] = acc[s][c];
  }
  __syncthreads();
  if (w == 0) {
#pragma unroll
    for (int c = 0; c < 16; ++c)
#pragma unroll
      for (int s = 0; s < S; ++s) {
        const int o = 64 * s + lane;
        U[((size_t)i * 16 + c) * KI + o] = ((acc[s][c] + part[0][c][o]) + part[1][c][o]) + part[2][c][o];
      }
  }
}

// Wave w takes the receiver's edges e_beg + w, e_beg + w + 4, ...; it holds
// gU[i][c][s][lane] for every (s, c) in registers. dE/da3 goes to da3[e][64],
// dE/dY to dY[e][16] (both overwritten).
template <int S, bool RB>
__global__ void __launch_bounds__(256) l0_edge_bwd_kernel(int N, const int* __restrict__ rcv_off,
                                                          const int* __restrict__ snd_z,
                                                          const float* __restrict__ a3, const float* __restrict__ Y,
                                                          const float* __restrict__ gU, float* __restrict__ da3,
                                                          float* __restrict__ dY) {
  constexpr int KI = 64 * S;
  const int i = blockIdx.x;
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int e_beg = rcv_off[i], e_end = rcv_off[i + 1];
  if (e_beg + w >= e_end) return;
  float g[S][16];
#pragma unroll
  for (int s = 0; s < S; ++s)
#pragma unroll
    for (int c = 0; c < 16; ++c) g[s][c] = gU[((size_t)i * 16 + c) * KI + 64 * s + lane];
  // kL0BwdEdges edges per iteration (e, e + 4, ...), their loads issued together
  for (int e = e_beg + w; e < e_end; e += 4 * kL0BwdEdges) {
    int ee[kL0BwdEdges], z[kL0BwdEdges];
    float a[kL0BwdEdges], y[kL0BwdEdges][16];
#pragma unroll
    for (int q = 0; q < kL0BwdEdges; ++q) {
      ee[q] = min(e + 4 * q, e_end - 1);   // a missing edge repeats the last one and stores nothing
      z[q] = snd_z[ee[q]];
      a[q] = a3[(size_t)ee[q] * 64 + lane];
#pragma unroll
      for (int v4 = 0; v4 < 4; ++v4) {
        const f4 t = *reinterpret_cast<const f4*>(Y + (size_t)ee[q] * 16 + 4 * v4);
        y[q][4 * v4] = t[0];
        y[q][4 * v4 + 1] = t[1];
        y[q][4 * v4 + 2] = t[2];
        y[q][4 * v4 + 3] = t[3];
      }
    }
#pragma unroll
    for (int q = 0; q < kL0BwdEdges; ++q) {
      if (e + 4 * q >= e_end) break;
      const float av = RB ? bf16_round(a[q]) : a[q];
      float gs[16];
#pragma unroll
      for (int c = 0; c < 16; ++c) gs[c] = g[0][c];
#pragma unroll
      for (int s = 1; s < S; ++s)
        if (z[q] == s) {
#pragma unroll
          for (int c = 0; c < 16; ++c) gs[c] = g[s][c];
        }
      float d = 0.f;
#pragma unroll
      for (int c = 0; c < 16; ++c) d += gs[c] * y[q][c];
      da3[(size_t)ee[q] * 64 + lane] = d;
      float v[16];
#pragma unroll
      for (int c = 0; c < 16; ++c) v[c] = gs[c] * av;
      const float t = wave_reduce_scatter16(v, lane);
      if ((lane & 3) == 0) dY[(size_t)ee[q] * 16 + (lane >> 2)] = t;
    }
  }
}

void launch_l0_gather(hipStream_t s, int N, int S, const int* rcv_off, const int* snd_z, const float* a3,
                      const float* Y, int rb, float* U) {
  if (N <= 0) return;
  auto go = [&](auto SS) {
    constexpr int SV = decltype(SS)::value;
    if (rb) l0_gather_kernel<SV, true><<<N, 256, 0, s>>>(N, rcv_off, snd_z, a3, Y, U);
    else l0_gather_kernel<SV, false><<<N, 256, 0, s>>>(N, rcv_off, snd_z, a3, Y, U);
  };
  switch (S) {
    case 1: go(std::integral_constant<int, 1>{}); break;
    case 2: go(std::integral_constant<int, 2>{}); break;
    case 3: go(std::integral_constant<int, 3>{}); break;
    case 4: go(std::integral_constant<int, 4>{}); break;
  }
}

void launch_l0_edge_bwd(hipStream_t s, int N, int S, const int* rcv_off, const int* snd_z, const float* a3,
                        const float* Y, const float* gU, int rb, float* da3, float* dY) {
  if (N <= 0) return;
  auto go = [&](auto SS) {
    constexpr int SV = decltype(SS)::value;
    if (rb) l0_edge_bwd_kernel<SV, true><<<N, 256, 0, s>>>(N, rcv_off, snd_z, a3, Y, gU, da3, dY);
    else l0_edge_bwd_kernel<SV, false><<<N, 256, 0, s>>>(N, rcv_off, snd_z, a3, Y, gU, da3, dY);
  };
  switch (S) {
    case 1: go(std::integral_constant<int, 1>{}); break;
    case 2: go(std::integral_constant<int, 2>{}); break;
    case 3: go(std::integral_constant<int, 3>{}); break;
    case 4: go(std::integral_constant<int, 4>{}); break;
  }
}

}  // namespace mace
