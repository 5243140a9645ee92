// Edge tensor product of Eq. 26 fused with the receiver neighbour sum, and
// its vector-Jacobian product.
//
//   At[i][p][m3][k] = inv_c * sum_{e: rcv_e = i} R[e][p][k]
//                     * sum_{m1,m2} C^{lo}_{lh ly}[m1][m2][m3] h[src_e][lh,m1][k] Y[e][ly,m2]
//
// Edges arrive sorted by receiver (CSR offsets rcv_off), so one block owns a
// receiver and sums its edges in CSR order: deterministic, no atomics.
// Threads = channels (k); every coupling constant is an immediate from the
// generated CG visitors; Y of the current edge is wave-uniform.
#include "mace_internal.h"
#include "static_loops.h"

namespace mace {

template <int LHMAX>
__global__ void __launch_bounds__(128) tp_fwd_kernel(int N, int K, const int* __restrict__ rcv_off,
                                                     const int* __restrict__ snd, const int* __restrict__ src_map,
                                                     const float* __restrict__ R, const float* __restrict__ Y,
                                                     const float* __restrict__ h, float inv_c,
                                                     float* __restrict__ At) {
  constexpr int P = path_count(LHMAX);
  constexpr int MID = mid_count(LHMAX);
  constexpr int DIN = (LHMAX + 1) * (LHMAX + 1);
  const int i = blockIdx.x;
  const int k = threadIdx.x;
  if (k >= K) return;
  float acc[MID];
#pragma unroll
  for (int c = 0; c < MID; ++c) acc[c] = 0.f;
  const int e_beg = rcv_off[i], e_end = rcv_off[i + 1];
  // operands of one edge; two sets so that the loads of edge e+1 are in
  // flight while edge e is being contracted
  auto load = [&](int e, float* hv, float* y, float* r) {
    const int s = snd[e];
    const int src = src_map ? src_map[s] : s;
#pragma unroll
    for (int c = 0; c < DIN; ++c) hv[c] = h[((size_t)src * DIN + c) * K + k];
#pragma unroll
    for (int m = 0; m < 16; ++m) y[m] = Y[(size_t)e * 16 + m];
#pragma unroll
    for (int p = 0; p < P; ++p) r[p] = R[((size_t)e * P + p) * K + k];
  };
  auto contract = [&](const float* hv, const float* y, const float* r) {
    for_paths<LHMAX>([&](auto tag) {
      using T = decltype(tag);
      constexpr int lh = T::lh, ly = T::ly, lo = T::lo;
      float t[2 * lo + 1];
#pragma unroll
      for (int m = 0; m < 2 * lo + 1; ++m) t[m] = 0.f;
      mt::CG<lh, ly, lo>::each([&](int m1, int m2, int m3, float cg) {
        t[m3] += cg * (hv[lh * lh + m1] * y[ly * ly + m2]);
      });
#pragma unroll
      for (int m = 0; m < 2 * lo + 1; ++m) acc[T::offset + m] += r[T::index] * t[m];
    });
  };
  float hA[DIN], yA[16], rA[P], hB[DIN], yB[16], rB[P];
  if (e_beg < e_end) load(e_beg, hA, yA, rA);
  for (int e = e_beg; e < e_end; e += 2) {
    if (e + 1 < e_end) load(e + 1, hB, yB, rB);
    contract(hA, yA, rA);
    if (e + 1 < e_end) {
      if (e + 2 < e_end) load(e + 2, hA, yA, rA);
      contract(hB, yB, rB);
    }
  }
#pragma unroll
  for (int c = 0; c < MID; ++c) At[((size_t)i * MID + c) * K + k] = acc[c] * inv_c;
}

// Sum of 16 values over the 64 lanes of a wave: afterwards lane l holds the
// total of index (bit5,bit4,bit3,bit2 of l) read as a 4-bit number.
__device__ __forceinline__ float wave_reduce16(float* v, int lane) {
  {
    const bool hi = lane & 32;
#pragma unroll
    for (int q = 0; q < 8; ++q) {
      float send = hi ? v[q] : v[q + 8];
      float keep = hi ? v[q + 8] : v[q];
      v[q] = keep + __shfl_xor(send, 32);
    }
  }
  {
    const bool hi = lane & 16;
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      float send = hi ? v[q] : v[q + 4];
      float keep = hi ? v[q + 4] : v[q];
      v[q] = keep + __shfl_xor(send, 16);
    }
  }
  {
    const bool hi = lane & 8;
#pragma unroll
    for (int q = 0; q < 2; ++q) {
      float send = hi ? v[q] : v[q + 2];
      float keep = hi ? v[q + 2] : v[q];
      v[q] = keep + __shfl_xor(send, 8);
    }
  }
  {
    const bool hi = lane & 4;
    float send = hi ? v[0] : v[1];
    float keep = hi ? v[1] : v[0];
    v[0] = keep + __shfl_xor(send, 4);
  }
  float x = v[0];
  x += __shfl_xor(x, 2);
  x += __shfl_xor(x, 1);
  return x;
}
__device__ __forceinline__ int wave_reduce16_index(int lane) {
  return ((lane >> 5) & 1) * 8 + ((lane >> 4) & 1) * 4 + ((lane >> 3) & 1) * 2 + ((lane >> 2) & 1);
}

constexpr int kTpChunk = 32;   // edges per dY staging round

// VJP of tp_fwd. Given g = dE/dAt:
//   dR[e][p][k]  = inv_c sum_m3 g[i][p][m3][k] t_p[m3]           (written over R)
//   dY[e][ly,m2] = inv_c sum_k sum_p R sum C h[m1] g[m3]          (reduced over channels)
//   Q[e][lh,m1][k] = inv_c sum_p R sum C Y[m2] g[m3]              (per-edge sender gradient)
// blockDim = 64 * ceil(K / 64); lanes with k >= K contribute zeros.
template <int LHMAX>
__global__ void __launch_bounds__(128) tp_bwd_kernel(int N, int K, const int* __restrict__ rcv_off,
                                                     const int* __restrict__ snd, const int* __restrict__ src_map,
                                                     float* __restrict__ R_dR, const float* __restrict__ Y,
                                                     const float* __restrict__ h, float inv_c,
                                                     const float* __restrict__ dAt, float* __restrict__ dY,
                                                     int accumulate_dY, float* __restrict__ Q) {
  constexpr int P = path_count(LHMAX);
  constexpr int MID = mid_count(LHMAX);
  constexpr int DIN = (LHMAX + 1) * (LHMAX + 1);
  __shared__ float red[2][kTpChunk][16];
  const int i = blockIdx.x;
  const int k = threadIdx.x;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int nwaves = blockDim.x >> 6;
  const bool active = k < K;
  const int kc = min(k, K - 1);             // lanes past K read a valid channel ...
  const float gs = active ? inv_c : 0.f;   // ... and contribute nothing
  float g[MID];
#pragma unroll
  for (int c = 0; c < MID; ++c) g[c] = dAt[((size_t)i * MID + c) * K + kc] * gs;
  const int e_beg = rcv_off[i], e_end = rcv_off[i + 1];
  for (int c0 = e_beg; c0 < e_end; c0 += kTpChunk) {
    const int c1 = min(e_end, c0 + kTpChunk);
    for (int e = c0; e < c1; ++e) {
      const int s = snd[e];
      const int src = src_map ? src_map[s] : s;
      float hv[DIN];
#pragma unroll
      for (int c = 0; c < DIN; ++c) hv[c] = h[((size_t)src * DIN + c) * K + kc];
      float y[16];
#pragma unroll
      for (int m = 0; m < 16; ++m) y[m] = Y[(size_t)e * 16 + m];
      float r[P];
#pragma unroll
      for (int p = 0; p < P; ++p) r[p] = R_dR[((size_t)e * P + p) * K + kc];
      float dr[P], dy[16], dh[DIN];
#pragma unroll
      for (int m = 0; m < 16; ++m) dy[m] = 0.f;
#pragma unroll
      for (int c = 0; c < DIN; ++c) dh[c] = 0.f;
      for_paths<LHMAX>([&](auto tag) {
        using T = decltype(tag);
        constexpr int lh = T::lh, ly = T::ly, lo = T::lo;
        float t[2 * lo + 1], u[2 * lo + 1];
#pragma unroll
        for (int m = 0; m < 2 * lo + 1; ++m) {
          t[m] = 0.f;
          u[m] = r[T::index] * g[T::offset + m];
        }
        mt::CG<lh, ly, lo>::each([&](int m1, int m2, int m3, float cg) {
          t[m3] += cg * (hv[lh * lh + m1] * y[ly * ly + m2]);
          dy[ly * ly + m2] += cg * (hv[lh * lh + m1] * u[m3]);
          dh[lh * lh + m1] += cg * (y[ly * ly + m2] * u[m3]);
        });
        float d = 0.f;
#pragma unroll
        for (int m = 0; m < 2 * lo + 1; ++m) d += g[T::offset + m] * t[m];
        dr[T::index] = d;
      });
      if (active) {
#pragma unroll
        for (int p = 0; p < P; ++p) R_dR[((size_t)e * P + p) * K + k] = dr[p];
        if (Q) {
#pragma unroll
          for (int c = 0; c < DIN; ++c) Q[((size_t)e * DIN + c) * K + k] = dh[c];
        }
      }
      float tot = wave_reduce16(dy, lane);
      if ((lane & 3) == 0) red[wave][e - c0][wave_reduce16_index(lane)] = tot;
    }
    __syncthreads();
    for (int q = threadIdx.x; q < (c1 - c0) * 16; q += blockDim.x) {
      int el = q >> 4, m = q & 15;
      float v = red[0][el][m];
      for (int w = 1; w < nwaves; ++w) v += red[w][el][m];
      size_t o = (size_t)(c0 + el) * 16 + m;
      dY[o] = accumulate_dY ? dY[o] + v : v;
    }
    __syncthreads();
  }
}

// out[j][c][k] = sum over edges with sender j (in increasing edge order) of Q[e][c][k]
__global__ void __launch_bounds__(256) sender_sum_kernel(int N, int CK, const int* __restrict__ snd_off,
                                                         const int* __restrict__ snd_perm,
                                                         const float* __restrict__ Q, float* __restrict__ out) {
  const int j = blockIdx.x;
  const int q0 = snd_off[j], q1 = snd_off[j + 1];
  for (int ck = threadIdx.x; ck < CK; ck += blockDim.x) {
    float acc = 0.f;
    int q = q0;
    for (; q + 4 <= q1; q += 4) {
      const float v0 = Q[(size_t)snd_perm[q] * CK + ck], v1 = Q[(size_t)snd_perm[q + 1] * CK + ck];
      const float v2 = Q[(size_t)snd_perm[q + 2] * CK + ck], v3 = Q[(size_t)snd_perm[q + 3] * CK + ck];
      acc += v0;
      acc += v1;
      acc += v2;
      acc += v3;
    }
    for (; q < q1; ++q) acc += Q[(size_t)snd_perm[q] * CK + ck];
    out[(size_t)j * CK + ck] = acc;
  }
}

void launch_tp_fwd(hipStream_t s, int lh_max, int N, int K, const int* rcv_off, const int* snd,
                   const int* src_map, const float* R, const float* Y, const float* h, int /*h_stride_nodes*/,
                   float inv_c, float* At) {
  if (N <= 0) return;
  dim3 grid(N), block(K);
  switch (lh_max) {
    case 0: tp_fwd_kernel<0><<<grid, block, 0, s>>>(N, K, rcv_off, snd, src_map, R, Y, h, inv_c, At); break;
    case 1: tp_fwd_kernel<1><<<grid, block, 0, s>>>(N, K, rcv_off, snd, src_map, R, Y, h, inv_c, At); break;
    case 2: tp_fwd_kernel<2><<<grid, block, 0, s>>>(N, K, rcv_off, snd, src_map, R, Y, h, inv_c, At); break;
  }
}

void launch_tp_bwd(hipStream_t s, int lh_max, int N, int K, const int* rcv_off, const int* snd,
                   const int* src_map, float* R_dR, const float* Y, const float* h, float inv_c,
                   const float* dAt, float* dY, int accumulate_dY, float* Q) {
  if (N <= 0) return;
  dim3 grid(N), block(((K + 63) / 64) * 64);
  switch (lh_max) {
    case 0: tp_bwd_kernel<0><<<grid, block, 0, s>>>(N, K, rcv_off, snd, src_map, R_dR, Y, h, inv_c, dAt, dY, accumulate_dY, Q); break;
    case 1: tp_bwd_kernel<1><<<grid, block, 0, s>>>(N, K, rcv_off, snd, src_map, R_dR, Y, h, inv_c, dAt, dY, accumulate_dY, Q); break;
    case 2: tp_bwd_kernel<2><<<grid, block, 0, s>>>(N, K, rcv_off, snd, src_map, R_dR, Y, h, inv_c, dAt, dY, accumulate_dY, Q); break;
  }
}

void launch_sender_sum(hipStream_t s, int N, int C, int K, const int* snd_off, const int* snd_perm,
                       const float* Q, float* out) {
  if (N <= 0) return;
  sender_sum_kernel<<<N, 256, 0, s>>>(N, C * K, snd_off, snd_perm, Q, out);
}

}  // namespace mace
