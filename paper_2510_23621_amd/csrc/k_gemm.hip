// FP32 GEMM on MFMA for the two dense products of the radial MLP:
//   R   [E][P*K] = a3 [E][64]   @ W3   [64][P*K]      (forward)
//   da3 [E][64]  = dR [E][P*K]  @ W3^T [P*K][64]      (backward)
// C = A @ B with A [M][KD], B [KD][N], C [M][N], all row-major; M is the edge
// count (ragged), N a multiple of BN, KD a multiple of KC.
//
// Block = 4 waves, block tile BM x BN, wave tile (BM/WR) x (BN/WC) made of
// 16 x 16 MFMA tiles (v_mfma_f32_16x16x4_f32: lane l supplies A[l%16][l/16],
// B[l/16][l%16]; result register r holds D[4(l/16)+r][l%16]). The reduction
// runs in chunks of KC columns staged through LDS with coalesced loads,
// double-buffered: the global loads of chunk c+1 are in flight while chunk c
// feeds the MFMAs. Row pitches are 4 (mod 32) floats so that fragment reads
// put exactly two lanes on each LDS bank.
#include "mace_internal.h"

namespace mace {

typedef float f4 __attribute__((ext_vector_type(4)));

template <int BM, int BN, int KC, int WR, int WC>
struct GemmSmem {
  static constexpr int LA = KC + 4, LB = BN + 4, LC = BN + 4;   // LDS pitches (4 mod 32)
  static constexpr int kStage = 2 * BM * LA + 2 * KC * LB;
  static constexpr int kEpi = BM * LC;
  static constexpr int kFloats = kStage > kEpi ? kStage : kEpi;
};

template <int BM, int BN, int KC, int WR, int WC>
__global__ void __launch_bounds__(256) gemm_kernel(int M, int N, int KD, const float* __restrict__ A,
                                                   const float* __restrict__ B, float* __restrict__ C) {
  static_assert(WR * WC == 4, "4 waves");
  using SM = GemmSmem<BM, BN, KC, WR, WC>;
  constexpr int TM = BM / WR / 16, TN = BN / WC / 16;     // MFMA tiles per wave
  constexpr int LA = SM::LA, LB = SM::LB, LC = SM::LC;
  constexpr int NA = BM * KC / 256, NB = KC * BN / 256;    // floats each thread stages
  static_assert(NA * 256 == BM * KC && NB * 256 == KC * BN, "tile sizes");
  static_assert((BM * BN) % 1024 == 0, "epilogue: whole float4 rounds");
  __shared__ float smem[SM::kFloats];
  auto sA = [&](int buf) { return smem + buf * (BM * LA); };
  auto sB = [&](int buf) { return smem + 2 * BM * LA + buf * (KC * LB); };
  const int tid = threadIdx.x, l = tid & 63, w = tid >> 6;
  const int wr = w / WC, wc = w % WC;
  const int m0 = blockIdx.x * BM, n0 = blockIdx.y * BN;
  float pa[NA], pb[NB];
  auto fetch = [&](int kc) {
#pragma unroll
    for (int q = 0; q < NA; ++q) {
      const int idx = tid + 256 * q, r = idx / KC, c = idx % KC;
      const int row = min(m0 + r, M - 1);                  // ragged rows read a valid row
      pa[q] = A[(size_t)row * KD + kc + c];
    }
#pragma unroll
    for (int q = 0; q < NB; ++q) {
      const int idx = tid + 256 * q, r = idx / BN, c = idx % BN;
      pb[q] = B[(size_t)(kc + r) * N + n0 + c];
    }
  };
  auto stash = [&](int buf) {
#pragma unroll
    for (int q = 0; q < NA; ++q) {
      const int idx = tid + 256 * q;
      sA(buf)[(idx / KC) * LA + idx % KC] = pa[q];
    }
#pragma unroll
    for (int q = 0; q < NB; ++q) {
      const int idx = tid + 256 * q;
      sB(buf)[(idx / BN) * LB + idx % BN] = pb[q];
    }
  };
  f4 acc[TM][TN];
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j) acc[i][j] = f4{0.f, 0.f, 0.f, 0.f};
  const int nk = KD / KC;
  fetch(0);
  stash(0);
  __syncthreads();
  for (int c = 0; c < nk; ++c) {
    const int cur = c & 1;
    if (c + 1 < nk) fetch((c + 1) * KC);
    const float* a = sA(cur) + (wr * TM * 16 + (l & 15)) * LA + (l >> 4);
    const float* b = sB(cur) + (l >> 4) * LB + wc * TN * 16 + (l & 15);
#pragma unroll
    for (int ks = 0; ks < KC / 4; ++ks) {
      float av[TM], bv[TN];
#pragma unroll
      for (int i = 0; i < TM; ++i) av[i] = a[i * 16 * LA + 4 * ks];
#pragma unroll
      for (int j = 0; j < TN; ++j) bv[j] = b[4 * ks * LB + j * 16];
#pragma unroll
      for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j) acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x4f32(av[i], bv[j], acc[i][j], 0, 0, 0);
    }
    if (c + 1 < nk) stash(cur ^ 1);
    __syncthreads();
  }
  // epilogue through LDS: whole rows leave as float4 stores
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j)
#pragma unroll
      for (int r = 0; r < 4; ++r)
        smem[(wr * TM * 16 + i * 16 + 4 * (l >> 4) + r) * LC + wc * TN * 16 + j * 16 + (l & 15)] = acc[i][j][r];
  __syncthreads();
  constexpr int V = BN / 4;   // float4 per row
#pragma unroll
  for (int q = 0; q < BM * V / 256; ++q) {
    const int idx = tid + 256 * q, r = idx / V, c4 = idx % V;
    if (m0 + r < M) {
      const float* src = smem + r * LC + 4 * c4;
      *reinterpret_cast<f4*>(C + (size_t)(m0 + r) * N + n0 + 4 * c4) = f4{src[0], src[1], src[2], src[3]};
    }
  }
}

// R = a3 @ W3 (N = P*K, KD = 64)
void launch_gemm_radial_out(hipStream_t s, int E, int PK, const float* a3, const float* W3, float* R) {
  if (E <= 0) return;
  if (PK % 128 == 0) {
    dim3 grid((E + 127) / 128, PK / 128);
    gemm_kernel<128, 128, 32, 2, 2><<<grid, 256, 0, s>>>(E, PK, 64, a3, W3, R);
  } else if (PK % 64 == 0) {
    dim3 grid((E + 127) / 128, PK / 64);
    gemm_kernel<128, 64, 32, 4, 1><<<grid, 256, 0, s>>>(E, PK, 64, a3, W3, R);
  } else {   // P*K is a multiple of 32 for every supported K
    dim3 grid((E + 127) / 128, PK / 32);
    gemm_kernel<128, 32, 32, 4, 1><<<grid, 256, 0, s>>>(E, PK, 64, a3, W3, R);
  }
}

// da3 = dR @ W3^T (N = 64, KD = P*K)
void launch_gemm_radial_in(hipStream_t s, int E, int PK, const float* dR, const float* W3T, float* da3) {
  if (E <= 0) return;
  dim3 grid((E + 127) / 128, 1);
  gemm_kernel<128, 64, 32, 4, 1><<<grid, 256, 0, s>>>(E, 64, PK, dR, W3T, da3);
}

}  // namespace mace
