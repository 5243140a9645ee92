// FP64 debug precision: the whole model, energy forward and force backward,
// in double precision on the vector units, written plainly (one thread per
// output element, no MFMA, no tiling). Same definitions as the FP32 kernels:
// real harmonics l <= 3 and the Bessel x envelope radial basis of each edge
// (the graph problem statement and the ingredients of Eq. 26), the radial MLP,
// the channelwise CG edge product summed over each receiver's edges (Eq. 26),
// the channel-mixing linears, the symmetric contraction over coupling trees
// (Eq. 27 and the message), the readouts and the energies, then the reverse
// of every step for F = -dE/dr (force equation). The couplings come from the
// generated FP64 tables (17 significant digits). Its purpose is to reproduce
// an FP64 reference to FP64 rounding on the GPU, not speed.
#include <algorithm>

#include "mace_internal.h"
#include "static_loops.h"
#include "generated/mace_tables64.h"

namespace mace {

namespace {

__device__ __forceinline__ double silu64(double x) { return x / (1.0 + exp(-x)); }
__device__ __forceinline__ double silu64_grad(double x) {
  const double s = 1.0 / (1.0 + exp(-x));
  return s * (1.0 + x * (1.0 - s));
}

// ------------------------------------------------------------------ edges

__global__ void f64_geom_kernel(int E, const double* __restrict__ pos, const int* __restrict__ snd,
                                const int* __restrict__ rcv, const double4* __restrict__ shift, double rc, int p,
                                int nb, double* __restrict__ Y, double* __restrict__ rb, int* __restrict__ status) {
  const int e = blockIdx.x * blockDim.x + threadIdx.x;
  if (e >= E) return;
  const int s = snd[e], r = rcv[e];
  const double4 sh = shift[e];
  const double dx = (pos[3 * s + 0] - pos[3 * r + 0]) + sh.x;
  const double dy = (pos[3 * s + 1] - pos[3 * r + 1]) + sh.y;
  const double dz = (pos[3 * s + 2] - pos[3 * r + 2]) + sh.z;
  const double rr = sqrt(dx * dx + dy * dy + dz * dz);
  int st = 0;
  if (!isfinite(dx) || !isfinite(dy) || !isfinite(dz)) st |= kStatusNonFinite;
  else if (rr == 0.0) st |= kStatusZeroLength;
  if (st) {
    atomicOr(status, st);
    for (int m = 0; m < 16; ++m) Y[(size_t)e * 16 + m] = 0.0;
    for (int n = 0; n < nb; ++n) rb[(size_t)e * nb + n] = 0.0;
    return;
  }
  const double inv = 1.0 / rr;
  sh16<double>(dx * inv, dy * inv, dz * inv, Y + (size_t)e * 16);
  double eb[16];
  bessel_env<double>(rr, rc, p, nb, eb);
  for (int n = 0; n < nb; ++n) rb[(size_t)e * nb + n] = eb[n];
}

// hidden layers of the radial MLP, one block of 64 threads per edge:
// z1 = rb W0, z2 = silu(z1) W1, z3 = silu(z2) W2 (a3 = silu(z3))
__global__ void __launch_bounds__(64) f64_radial_fwd_kernel(int nb, const double* __restrict__ rb,
                                                            const double* __restrict__ W0,
                                                            const double* __restrict__ W1,
                                                            const double* __restrict__ W2, double* __restrict__ z1,
                                                            double* __restrict__ z2, double* __restrict__ z3) {
  __shared__ double v[64];
  const int e = blockIdx.x, j = threadIdx.x;
  double acc = 0.0;
  for (int n = 0; n < nb; ++n) acc += rb[(size_t)e * nb + n] * W0[n * 64 + j];
  z1[(size_t)e * 64 + j] = acc;
  v[j] = silu64(acc);
  __syncthreads();
  acc = 0.0;
  for (int i = 0; i < 64; ++i) acc += v[i] * W1[i * 64 + j];
  z2[(size_t)e * 64 + j] = acc;
  __syncthreads();
  v[j] = silu64(acc);
  __syncthreads();
  acc = 0.0;
  for (int i = 0; i < 64; ++i) acc += v[i] * W2[i * 64 + j];
  z3[(size_t)e * 64 + j] = acc;
}

// backward of the hidden layers from dE/da3 (a3 = silu(z3)): de = dE/d(rb),
// added to de when acc (the layers below the last add theirs)
__global__ void __launch_bounds__(64) f64_radial_bwd_kernel(int nb, const double* __restrict__ W0,
                                                            const double* __restrict__ W1,
                                                            const double* __restrict__ W2,
                                                            const double* __restrict__ z1,
                                                            const double* __restrict__ z2,
                                                            const double* __restrict__ z3,
                                                            const double* __restrict__ da3, double* __restrict__ de,
                                                            int acc) {
  __shared__ double v[64];
  const int e = blockIdx.x, j = threadIdx.x;
  v[j] = da3[(size_t)e * 64 + j] * silu64_grad(z3[(size_t)e * 64 + j]);   // dE/dz3
  __syncthreads();
  double t = 0.0;
  for (int i = 0; i < 64; ++i) t += W2[j * 64 + i] * v[i];                  // dE/d silu(z2)
  t *= silu64_grad(z2[(size_t)e * 64 + j]);
  __syncthreads();
  v[j] = t;
  __syncthreads();
  t = 0.0;
  for (int i = 0; i < 64; ++i) t += W1[j * 64 + i] * v[i];
  t *= silu64_grad(z1[(size_t)e * 64 + j]);
  __syncthreads();
  v[j] = t;                                                                 // dE/dz1
  __syncthreads();
  if (j < nb) {
    double g = 0.0;
    for (int i = 0; i < 64; ++i) g += W0[j * 64 + i] * v[i];
    de[(size_t)e * nb + j] = acc ? de[(size_t)e * nb + j] + g : g;
  }
}

// R[p] of edge e and channel k: sum_j silu(z3[e][j]) W3[j][p K + k]
template <int P>
__device__ __forceinline__ void f64_radial_row(const double* __restrict__ z3, const double* __restrict__ W3, int e,
                                               int K, int k, double* R) {
#pragma unroll
  for (int p = 0; p < P; ++p) R[p] = 0.0;
  for (int j = 0; j < 64; ++j) {
    const double a = silu64(z3[(size_t)e * 64 + j]);
#pragma unroll
    for (int p = 0; p < P; ++p) R[p] += a * W3[(size_t)j * P * K + p * K + k];
  }
}

// At[i][off_p + m3][k] = inv_c sum over edges into i of
//   R[e][p][k] sum_{m1 m2} C^{lo}_{lh ly}[m1][m2][m3] h[snd][lh, m1][k] Y[e][ly, m2]
// one thread per (receiver, channel), edges in CSR order
template <int LH>
__global__ void f64_tp_fwd_kernel(int N, int K, const int* __restrict__ rcv_off, const int* __restrict__ snd,
                                  const double* __restrict__ z3, const double* __restrict__ W3,
                                  const double* __restrict__ Y, const double* __restrict__ h, double inv_c,
                                  double* __restrict__ At) {
  constexpr int P = path_count(LH), MID = mid_count(LH), DIN = (LH + 1) * (LH + 1);
  const int idx = blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= N * K) return;
  const int i = idx / K, k = idx % K;
  double acc[MID];
#pragma unroll
  for (int c = 0; c < MID; ++c) acc[c] = 0.0;
  for (int e = rcv_off[i]; e < rcv_off[i + 1]; ++e) {
    double R[P];
    f64_radial_row<P>(z3, W3, e, K, k, R);
    const int s = snd[e];
    double hv[DIN], y[16];
#pragma unroll
    for (int c = 0; c < DIN; ++c) hv[c] = h[((size_t)s * DIN + c) * K + k];
#pragma unroll
    for (int m = 0; m < 16; ++m) y[m] = Y[(size_t)e * 16 + m];
    for_paths<LH>([&](auto tag) {
      using T = decltype(tag);
      constexpr int lh = T::lh, ly = T::ly, lo = T::lo;
      mt64::CG<lh, ly, lo>::each([&](int m1, int m2, int m3, double c) {
        acc[T::offset + m3] += R[T::index] * (c * hv[lh * lh + m1] * y[ly * ly + m2]);
      });
    });
  }
#pragma unroll
  for (int c = 0; c < MID; ++c) At[((size_t)i * MID + c) * K + k] = acc[c] * inv_c;
}

// VJP of f64_tp_fwd for edge e (one thread per edge, channels in turn), with
// g = dE/dAt: dE/dY[e] (written, or added when accY), dE/da3[e] and the
// per-edge sender gradient Q[e][c][k] (when Q is given)
template <int LH>
__global__ void f64_tp_bwd_kernel(int E, int K, const int* __restrict__ snd, const int* __restrict__ rcv,
                                  const double* __restrict__ z3, const double* __restrict__ W3,
                                  const double* __restrict__ Y, const double* __restrict__ h,
                                  const double* __restrict__ dAt, double inv_c, double* __restrict__ dY, int accY,
                                  double* __restrict__ da3, double* __restrict__ Q) {
  constexpr int P = path_count(LH), MID = mid_count(LH), DIN = (LH + 1) * (LH + 1);
  const int e = blockIdx.x * blockDim.x + threadIdx.x;
  if (e >= E) return;
  const int s = snd[e], i = rcv[e];
  double y[16], dy[16];
#pragma unroll
  for (int m = 0; m < 16; ++m) {
    y[m] = Y[(size_t)e * 16 + m];
    dy[m] = 0.0;
  }
  double a3[64], d3[64];
  for (int j = 0; j < 64; ++j) {
    a3[j] = silu64(z3[(size_t)e * 64 + j]);
    d3[j] = 0.0;
  }
  for (int k = 0; k < K; ++k) {
    double R[P], dR[P];
#pragma unroll
    for (int p = 0; p < P; ++p) {
      R[p] = 0.0;
      dR[p] = 0.0;
    }
    for (int j = 0; j < 64; ++j)
#pragma unroll
      for (int p = 0; p < P; ++p) R[p] += a3[j] * W3[(size_t)j * P * K + p * K + k];
    double hv[DIN], dh[DIN], g[MID];
#pragma unroll
    for (int c = 0; c < DIN; ++c) {
      hv[c] = h[((size_t)s * DIN + c) * K + k];
      dh[c] = 0.0;
    }
#pragma unroll
    for (int c = 0; c < MID; ++c) g[c] = dAt[((size_t)i * MID + c) * K + k] * inv_c;
    for_paths<LH>([&](auto tag) {
      using T = decltype(tag);
      constexpr int lh = T::lh, ly = T::ly, lo = T::lo;
      mt64::CG<lh, ly, lo>::each([&](int m1, int m2, int m3, double c) {
        const double t = c * g[T::offset + m3];
        dR[T::index] += t * hv[lh * lh + m1] * y[ly * ly + m2];
        dy[ly * ly + m2] += R[T::index] * t * hv[lh * lh + m1];
        dh[lh * lh + m1] += R[T::index] * t * y[ly * ly + m2];
      });
    });
    for (int j = 0; j < 64; ++j)
#pragma unroll
      for (int p = 0; p < P; ++p) d3[j] += dR[p] * W3[(size_t)j * P * K + p * K + k];
    if (Q) {
#pragma unroll
      for (int c = 0; c < DIN; ++c) Q[((size_t)e * DIN + c) * K + k] = dh[c];
    }
  }
#pragma unroll
  for (int m = 0; m < 16; ++m) dY[(size_t)e * 16 + m] = accY ? dY[(size_t)e * 16 + m] + dy[m] : dy[m];
  for (int j = 0; j < 64; ++j) da3[(size_t)e * 64 + j] = d3[j];
}

// out[n][c][k] = sum over the edges sent by n (sender CSR, increasing edge
// order) of Q[e][c][k]
__global__ void f64_sender_sum_kernel(int N, int C, int K, const int* __restrict__ snd_off,
                                      const int* __restrict__ snd_perm, const double* __restrict__ Q,
                                      double* __restrict__ out) {
  const size_t idx = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= (size_t)N * C * K) return;
  const int n = (int)(idx / ((size_t)C * K));
  const int ck = (int)(idx % ((size_t)C * K));
  double acc = 0.0;
  for (int q = snd_off[n]; q < snd_off[n + 1]; ++q) acc += Q[(size_t)snd_perm[q] * C * K + ck];
  out[idx] = acc;
}

// ------------------------------------------------------------------ nodes

// y[n][c][k] = (res[n][c][k] or 0) + sum over the terms t with
// cy[t] <= c < cy[t] + nc[t] of sum_k' W_t[k'][k] x[n][cx[t] + c - cy[t]][k']
// (W_t[k][k'] with transpose), W_t at W + woff[t] (+ z_n K K for
// species-dependent terms)
__global__ void f64_linear_kernel(int N, int K, Lin64 L, const int* __restrict__ species,
                                  const double* __restrict__ W, const double* __restrict__ x,
                                  double* __restrict__ y, const double* __restrict__ res) {
  const size_t idx = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= (size_t)N * L.cout * K) return;
  const int n = (int)(idx / ((size_t)L.cout * K));
  const int c = (int)((idx / K) % L.cout), k = (int)(idx % K);
  double acc = res ? res[idx] : 0.0;
  for (int t = 0; t < L.n_terms; ++t) {
    const int m = c - L.cy[t];
    if (m < 0 || m >= L.nc[t]) continue;
    const double* Wt = W + L.woff[t] + (L.spec[t] ? (size_t)species[n] * K * K : 0);
    const double* xr = x + ((size_t)n * L.cin + L.cx[t] + m) * K;
    if (L.transpose)
      for (int q = 0; q < K; ++q) acc += Wt[(size_t)k * K + q] * xr[q];
    else
      for (int q = 0; q < K; ++q) acc += Wt[(size_t)q * K + k] * xr[q];
  }
  y[idx] = acc;
}

template <class TT, int L>
__device__ __forceinline__ void f64_tree_eval(const double* a, double* t) {
  constexpr int nu = TT::nu, l1 = TT::l1, l2 = TT::l2, l3 = TT::l3, l12 = TT::l12;
#pragma unroll
  for (int m = 0; m < 2 * L + 1; ++m) t[m] = 0.0;
  if constexpr (nu == 1) {
#pragma unroll
    for (int m = 0; m < 2 * L + 1; ++m) t[m] = a[l1 * l1 + m];
  } else if constexpr (nu == 2) {
    mt64::CG<l1, l2, L>::each([&](int m1, int m2, int M, double c) { t[M] += c * (a[l1 * l1 + m1] * a[l2 * l2 + m2]); });
  } else {
    double x[2 * l12 + 1];
#pragma unroll
    for (int m = 0; m < 2 * l12 + 1; ++m) x[m] = 0.0;
    mt64::CG<l1, l2, l12>::each([&](int m1, int m2, int m3, double c) { x[m3] += c * (a[l1 * l1 + m1] * a[l2 * l2 + m2]); });
    mt64::CG<l12, l3, L>::each([&](int m1, int m2, int M, double c) { t[M] += c * (x[m1] * a[l3 * l3 + m2]); });
  }
}

// da += coef * d/dA <gB, Tree(A)>
template <class TT, int L>
__device__ __forceinline__ void f64_tree_vjp(const double* a, const double* gB, double coef, double* da) {
  constexpr int nu = TT::nu, l1 = TT::l1, l2 = TT::l2, l3 = TT::l3, l12 = TT::l12;
  if constexpr (nu == 1) {
#pragma unroll
    for (int m = 0; m < 2 * L + 1; ++m) da[l1 * l1 + m] += coef * gB[m];
  } else if constexpr (nu == 2) {
    mt64::CG<l1, l2, L>::each([&](int m1, int m2, int M, double c) {
      const double w = coef * c * gB[M];
      da[l1 * l1 + m1] += w * a[l2 * l2 + m2];
      da[l2 * l2 + m2] += w * a[l1 * l1 + m1];
    });
  } else {
    double x[2 * l12 + 1], dx[2 * l12 + 1];
#pragma unroll
    for (int m = 0; m < 2 * l12 + 1; ++m) {
      x[m] = 0.0;
      dx[m] = 0.0;
    }
    mt64::CG<l1, l2, l12>::each([&](int m1, int m2, int m3, double c) { x[m3] += c * (a[l1 * l1 + m1] * a[l2 * l2 + m2]); });
    mt64::CG<l12, l3, L>::each([&](int m1, int m2, int M, double c) {
      const double w = coef * c * gB[M];
      dx[m1] += w * a[l3 * l3 + m2];
      da[l3 * l3 + m2] += w * x[m1];
    });
    mt64::CG<l1, l2, l12>::each([&](int m1, int m2, int m3, double c) {
      da[l1 * l1 + m1] += c * (dx[m3] * a[l2 * l2 + m2]);
      da[l2 * l2 + m2] += c * (dx[m3] * a[l1 * l1 + m1]);
    });
  }
}

// B[n][L,M][k] = sum_nu sum_eta W^{nu}_{z_n, L}[eta][k] s_eta Tree_eta(A[n][.][k])[M]
template <int LOUT>
__global__ void f64_symcon_fwd_kernel(int N, int K, const int* __restrict__ species, const double* __restrict__ A,
                                      SymW64 w, double* __restrict__ B) {
  constexpr int DOUT = (LOUT + 1) * (LOUT + 1);
  const int idx = blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= N * K) return;
  const int n = idx / K, k = idx % K, z = species[n];
  double a[16], b[DOUT];
#pragma unroll
  for (int c = 0; c < 16; ++c) a[c] = A[((size_t)n * 16 + c) * K + k];
#pragma unroll
  for (int c = 0; c < DOUT; ++c) b[c] = 0.0;
  static_for<0, LOUT + 1>([&](auto LL) {
    constexpr int L = decltype(LL)::value;
    static_for<1, 4>([&](auto NUc) {
      constexpr int nu = decltype(NUc)::value;
      constexpr int ne = mt64::Trees<nu, L>::n;
      if constexpr (ne > 0) {
        const double* W = w.w[L][nu] + (size_t)z * ne * K + k;
        mt64::Trees<nu, L>::each([&](auto tree, int eta, double scale) {
          const double coef = W[(size_t)eta * K] * scale;
          double t[2 * L + 1];
          f64_tree_eval<decltype(tree), L>(a, t);
#pragma unroll
          for (int m = 0; m < 2 * L + 1; ++m) b[L * L + m] += coef * t[m];
        });
      }
    });
  });
#pragma unroll
  for (int c = 0; c < DOUT; ++c) B[((size_t)n * DOUT + c) * K + k] = b[c];
}

template <int LOUT>
__global__ void f64_symcon_bwd_kernel(int N, int K, const int* __restrict__ species, const double* __restrict__ A,
                                      SymW64 w, const double* __restrict__ dB, double* __restrict__ dA) {
  constexpr int DOUT = (LOUT + 1) * (LOUT + 1);
  const int idx = blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= N * K) return;
  const int n = idx / K, k = idx % K, z = species[n];
  double a[16], da[16], gb[DOUT];
#pragma unroll
  for (int c = 0; c < 16; ++c) {
    a[c] = A[((size_t)n * 16 + c) * K + k];
    da[c] = 0.0;
  }
#pragma unroll
  for (int c = 0; c < DOUT; ++c) gb[c] = dB[((size_t)n * DOUT + c) * K + k];
  static_for<0, LOUT + 1>([&](auto LL) {
    constexpr int L = decltype(LL)::value;
    static_for<1, 4>([&](auto NUc) {
      constexpr int nu = decltype(NUc)::value;
      constexpr int ne = mt64::Trees<nu, L>::n;
      if constexpr (ne > 0) {
        const double* W = w.w[L][nu] + (size_t)z * ne * K + k;
        mt64::Trees<nu, L>::each([&](auto tree, int eta, double scale) {
          f64_tree_vjp<decltype(tree), L>(a, gb + L * L, W[(size_t)eta * K] * scale, da);
        });
      }
    });
  });
#pragma unroll
  for (int c = 0; c < 16; ++c) dA[((size_t)n * 16 + c) * K + k] = da[c];
}

// readouts, one thread per node. A layer below the last adds w . h[n][0][:]
// (hid == 0); the last layer adds w2 . silu(W1^T h[n][0][:]) and stores its
// gradient dE/dh[n][0][:] = W1 (w2 * silu'(.)) into dh0 (the backward's start).
__global__ void f64_readout_kernel(int N, int K, const double* __restrict__ h, int stride, const double* __restrict__ w,
                                   const double* __restrict__ w2, int hid, double* __restrict__ eps, int acc,
                                   double* __restrict__ dh0) {
  const int n = blockIdx.x * blockDim.x + threadIdx.x;
  if (n >= N) return;
  const double* hr = h + (size_t)n * stride;
  double e = 0.0;
  if (hid == 0) {
    for (int k = 0; k < K; ++k) e += w[k] * hr[k];
  } else {
    double zc[16];
    for (int j = 0; j < hid; ++j) {
      double z = 0.0;
      for (int k = 0; k < K; ++k) z += w[k * hid + j] * hr[k];
      zc[j] = z;
      e += w2[j] * silu64(z);
    }
    if (dh0)
      for (int k = 0; k < K; ++k) {
        double g = 0.0;
        for (int j = 0; j < hid; ++j) g += w[k * hid + j] * (w2[j] * silu64_grad(zc[j]));
        dh0[(size_t)n * K + k] = g;
      }
  }
  eps[n] = acc ? eps[n] + e : e;
}

// dst[n][0][k] += w[k] (a lower layer's readout gradient)
__global__ void f64_add_readout_grad_kernel(int N, int K, int stride, const double* __restrict__ w,
                                            double* __restrict__ dst) {
  const size_t idx = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= (size_t)N * K) return;
  dst[(idx / K) * stride + idx % K] += w[idx % K];
}

// h0[n][0][k] = W_embed[z_n][k]
__global__ void f64_embed_kernel(int N, int K, const int* __restrict__ species, const double* __restrict__ W,
                                 double* __restrict__ h0) {
  const size_t idx = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= (size_t)N * K) return;
  h0[idx] = W[(size_t)species[idx / K] * K + idx % K];
}

// g_e = dE/dd_e from dE/dY and dE/d(rb) by forward-mode differentiation
// (FP64 dual numbers) of the closed forms
__global__ void f64_edge_vjp_kernel(int E, const double* __restrict__ pos, const int* __restrict__ snd,
                                    const int* __restrict__ rcv, const double4* __restrict__ shift, double rc, int p,
                                    int nb, const double* __restrict__ dY, const double* __restrict__ de,
                                    double4* __restrict__ g) {
  using D3 = Dual3<double>;
  const int e = blockIdx.x * blockDim.x + threadIdx.x;
  if (e >= E) return;
  const int s = snd[e], r = rcv[e];
  const double4 sh = shift[e];
  const D3 dx((pos[3 * s + 0] - pos[3 * r + 0]) + sh.x, 1.0, 0.0, 0.0);
  const D3 dyv((pos[3 * s + 1] - pos[3 * r + 1]) + sh.y, 0.0, 1.0, 0.0);
  const D3 dz((pos[3 * s + 2] - pos[3 * r + 2]) + sh.z, 0.0, 0.0, 1.0);
  const D3 rr = dsqrt(dx * dx + dyv * dyv + dz * dz);
  if (!(rr.v > 0.0) || !isfinite(rr.v)) {
    g[e] = make_double4(0.0, 0.0, 0.0, 0.0);
    return;
  }
  const D3 inv = D3(1.0) / rr;
  D3 y[16];
  sh16<D3>(dx * inv, dyv * inv, dz * inv, y);
  double gx = 0.0, gy = 0.0, gz = 0.0;
  for (int m = 1; m < 16; ++m) {
    const double w = dY[(size_t)e * 16 + m];
    gx += w * y[m].x;
    gy += w * y[m].y;
    gz += w * y[m].z;
  }
  D3 eb[16];
  bessel_env<D3>(rr, rc, p, nb, eb);
  for (int n = 0; n < nb; ++n) {
    const double w = de[(size_t)e * nb + n];
    gx += w * eb[n].x;
    gy += w * eb[n].y;
    gz += w * eb[n].z;
  }
  g[e] = make_double4(gx, gy, gz, 0.0);
}

// F_i = sum_{e: rcv_e = i} g_e - sum_{e: snd_e = i} g_e (fixed order)
__global__ void f64_forces_kernel(int N, const int* __restrict__ rcv_off, const int* __restrict__ snd_off,
                                  const int* __restrict__ snd_perm, const double4* __restrict__ g,
                                  double* __restrict__ F) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= N) return;
  double fx = 0.0, fy = 0.0, fz = 0.0;
  for (int e = rcv_off[i]; e < rcv_off[i + 1]; ++e) {
    fx += g[e].x;
    fy += g[e].y;
    fz += g[e].z;
  }
  for (int q = snd_off[i]; q < snd_off[i + 1]; ++q) {
    const double4 v = g[snd_perm[q]];
    fx -= v.x;
    fy -= v.y;
    fz -= v.z;
  }
  F[3 * i + 0] = fx;
  F[3 * i + 1] = fy;
  F[3 * i + 2] = fz;
}

// E_g = sum of eps over the graph's atoms, in order
__global__ void f64_graph_energy_kernel(int G, const int* __restrict__ graph_off, const double* __restrict__ eps,
                                        double* __restrict__ E) {
  const int gi = blockIdx.x * blockDim.x + threadIdx.x;
  if (gi >= G) return;
  double acc = 0.0;
  for (int n = graph_off[gi]; n < graph_off[gi + 1]; ++n) acc += eps[n];
  E[gi] = acc;
}

// sigma_g[a][b] = inv_vol_g sum over the graph's edges of d_e[a] g_e[b]
__global__ void f64_stress_kernel(int G, const int* __restrict__ graph_off, const int* __restrict__ rcv_off,
                                  const double* __restrict__ pos, const int* __restrict__ snd,
                                  const int* __restrict__ rcv, const double4* __restrict__ shift,
                                  const double4* __restrict__ g, const double* __restrict__ inv_vol,
                                  double* __restrict__ stress) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= 9 * G) return;
  const int gi = i / 9, a = (i % 9) / 3, b = i % 3;
  double acc = 0.0;
  for (int e = rcv_off[graph_off[gi]]; e < rcv_off[graph_off[gi + 1]]; ++e) {
    const int s = snd[e], r = rcv[e];
    const double4 sh = shift[e];
    const double sv[3] = {sh.x, sh.y, sh.z};
    const double d = (pos[3 * s + a] - pos[3 * r + a]) + sv[a];
    const double4 gv = g[e];
    const double gg[3] = {gv.x, gv.y, gv.z};
    acc += d * gg[b];
  }
  stress[i] = acc * inv_vol[gi];
}

// dst = src (FP32 -> FP64), n values
__global__ void f64_widen_kernel(size_t n, const float* __restrict__ src, double* __restrict__ dst) {
  for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (size_t)gridDim.x * blockDim.x)
    dst[i] = (double)src[i];
}

unsigned blocks_for(size_t n, int t = 256) { return (unsigned)((n + t - 1) / t); }

}  // namespace

void f64_widen(hipStream_t s, size_t n, const float* src, double* dst) {
  if (n) f64_widen_kernel<<<std::min<size_t>(blocks_for(n), 4096), 256, 0, s>>>(n, src, dst);
}
void f64_geom(hipStream_t s, int E, const double* pos, const int* snd, const int* rcv, const double4* shift,
              double rc, int p, int nb, double* Y, double* rb, int* status) {
  if (E > 0) f64_geom_kernel<<<blocks_for(E), 256, 0, s>>>(E, pos, snd, rcv, shift, rc, p, nb, Y, rb, status);
}
void f64_radial_fwd(hipStream_t s, int E, int nb, const double* rb, const double* W0, const double* W1,
                    const double* W2, double* z1, double* z2, double* z3) {
  if (E > 0) f64_radial_fwd_kernel<<<E, 64, 0, s>>>(nb, rb, W0, W1, W2, z1, z2, z3);
}
void f64_radial_bwd(hipStream_t s, int E, int nb, const double* W0, const double* W1, const double* W2,
                    const double* z1, const double* z2, const double* z3, const double* da3, double* de, int acc) {
  if (E > 0) f64_radial_bwd_kernel<<<E, 64, 0, s>>>(nb, W0, W1, W2, z1, z2, z3, da3, de, acc);
}
bool f64_tp_fwd(hipStream_t s, int lh, int N, int K, const int* rcv_off, const int* snd, const double* z3,
                const double* W3, const double* Y, const double* h, double inv_c, double* At) {
  if (N <= 0) return true;
  const unsigned nb = blocks_for((size_t)N * K, 64);
  switch (lh) {
    case 0: f64_tp_fwd_kernel<0><<<nb, 64, 0, s>>>(N, K, rcv_off, snd, z3, W3, Y, h, inv_c, At); return true;
    case 1: f64_tp_fwd_kernel<1><<<nb, 64, 0, s>>>(N, K, rcv_off, snd, z3, W3, Y, h, inv_c, At); return true;
    case 2: f64_tp_fwd_kernel<2><<<nb, 64, 0, s>>>(N, K, rcv_off, snd, z3, W3, Y, h, inv_c, At); return true;
  }
  return false;
}
bool f64_tp_bwd(hipStream_t s, int lh, int E, int K, const int* snd, const int* rcv, const double* z3,
                const double* W3, const double* Y, const double* h, const double* dAt, double inv_c, double* dY,
                int accY, double* da3, double* Q) {
  if (E <= 0) return true;
  const unsigned nb = blocks_for(E, 64);
  switch (lh) {
    case 0: f64_tp_bwd_kernel<0><<<nb, 64, 0, s>>>(E, K, snd, rcv, z3, W3, Y, h, dAt, inv_c, dY, accY, da3, Q); return true;
    case 1: f64_tp_bwd_kernel<1><<<nb, 64, 0, s>>>(E, K, snd, rcv, z3, W3, Y, h, dAt, inv_c, dY, accY, da3, Q); return true;
    case 2: f64_tp_bwd_kernel<2><<<nb, 64, 0, s>>>(E, K, snd, rcv, z3, W3, Y, h, dAt, inv_c, dY, accY, da3, Q); return true;
  }
  return false;
}
void f64_sender_sum(hipStream_t s, int N, int C, int K, const int* snd_off, const int* snd_perm, const double* Q,
                    double* out) {
  if (N > 0) f64_sender_sum_kernel<<<blocks_for((size_t)N * C * K), 256, 0, s>>>(N, C, K, snd_off, snd_perm, Q, out);
}
void f64_linear(hipStream_t s, int N, int K, const Lin64& L, const int* species, const double* W, const double* x,
                double* y, const double* res) {
  if (N > 0 && L.cout > 0)
    f64_linear_kernel<<<blocks_for((size_t)N * L.cout * K), 256, 0, s>>>(N, K, L, species, W, x, y, res);
}
bool f64_symcon_fwd(hipStream_t s, int lout, int N, int K, const int* species, const double* A, const SymW64& w,
                    double* B) {
  if (N <= 0) return true;
  const unsigned nb = blocks_for((size_t)N * K, 64);
  switch (lout) {
    case 0: f64_symcon_fwd_kernel<0><<<nb, 64, 0, s>>>(N, K, species, A, w, B); return true;
    case 1: f64_symcon_fwd_kernel<1><<<nb, 64, 0, s>>>(N, K, species, A, w, B); return true;
    case 2: f64_symcon_fwd_kernel<2><<<nb, 64, 0, s>>>(N, K, species, A, w, B); return true;
  }
  return false;
}
bool f64_symcon_bwd(hipStream_t s, int lout, int N, int K, const int* species, const double* A, const SymW64& w,
                    const double* dB, double* dA) {
  if (N <= 0) return true;
  const unsigned nb = blocks_for((size_t)N * K, 64);
  switch (lout) {
    case 0: f64_symcon_bwd_kernel<0><<<nb, 64, 0, s>>>(N, K, species, A, w, dB, dA); return true;
    case 1: f64_symcon_bwd_kernel<1><<<nb, 64, 0, s>>>(N, K, species, A, w, dB, dA); return true;
    case 2: f64_symcon_bwd_kernel<2><<<nb, 64, 0, s>>>(N, K, species, A, w, dB, dA); return true;
  }
  return false;
}
void f64_readout(hipStream_t s, int N, int K, const double* h, int stride, const double* w, const double* w2,
                 int hid, double* eps, int acc, double* dh0) {
  if (N > 0) f64_readout_kernel<<<blocks_for(N), 256, 0, s>>>(N, K, h, stride, w, w2, hid, eps, acc, dh0);
}
void f64_add_readout_grad(hipStream_t s, int N, int K, int stride, const double* w, double* dst) {
  if (N > 0) f64_add_readout_grad_kernel<<<blocks_for((size_t)N * K), 256, 0, s>>>(N, K, stride, w, dst);
}
void f64_embed(hipStream_t s, int N, int K, const int* species, const double* W, double* h0) {
  if (N > 0) f64_embed_kernel<<<blocks_for((size_t)N * K), 256, 0, s>>>(N, K, species, W, h0);
}
void f64_edge_vjp(hipStream_t s, int E, const double* pos, const int* snd, const int* rcv, const double4* shift,
                  double rc, int p, int nb, const double* dY, const double* de, double4* g) {
  if (E > 0) f64_edge_vjp_kernel<<<blocks_for(E), 256, 0, s>>>(E, pos, snd, rcv, shift, rc, p, nb, dY, de, g);
}
void f64_forces(hipStream_t s, int N, const int* rcv_off, const int* snd_off, const int* snd_perm, const double4* g,
                double* F) {
  if (N > 0) f64_forces_kernel<<<blocks_for(N), 256, 0, s>>>(N, rcv_off, snd_off, snd_perm, g, F);
}
void f64_graph_energy(hipStream_t s, int G, const int* graph_off, const double* eps, double* E) {
  if (G > 0) f64_graph_energy_kernel<<<blocks_for(G), 256, 0, s>>>(G, graph_off, eps, E);
}
void f64_stress(hipStream_t s, int G, const int* graph_off, const int* rcv_off, const double* pos, const int* snd,
                const int* rcv, const double4* shift, const double4* g, const double* inv_vol, double* stress) {
  if (G > 0)
    f64_stress_kernel<<<blocks_for((size_t)9 * G), 256, 0, s>>>(G, graph_off, rcv_off, pos, snd, rcv, shift, g,
                                                                inv_vol, stress);
}

}  // namespace mace
