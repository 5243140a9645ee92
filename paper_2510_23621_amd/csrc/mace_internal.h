// Internal declarations shared by the kernel files and the host runtime of
// the MACE layer library (gfx950). Not part of the public C ABI.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace mace {

// Device status bits, OR-ed into one word of the workspace by the kernels
// that detect the condition and read back by mace_graph_check.
constexpr int kStatusNonFinite = 1;    // an edge vector with a NaN or infinite component
constexpr int kStatusZeroLength = 2;   // an edge of length 0 (coincident atoms)

constexpr int kMaxTerms = 48;
constexpr int kMaxGroups = 24;
constexpr int kLinTileNodes = 16;   // nodes per MFMA tile of the channel-mixing linear
constexpr int kLinQuad = 4;         // node tiles (one per wave) per block of the linear
constexpr int kLinQuadWide = 8;     // the same for the wide 16-bit launches on large graphs
constexpr int kLinQuadWideMinQuads = 256;   // kLinQuad blocks from which a 16-bit handle also groups by kLinQuadWide

// ----------------------------------------------------------------- numerics
// e^(-x) on the hardware base-2 exponential (v_exp_f32, about 1 ulp): the
// exponent -x log2(e) is carried as t + err, with log2(e) split into an FP32
// head and its tail (Cody and Waite) and the rounding error of the head product
// recovered by a fused multiply-add; then 2^(t + err) = 2^t (1 + err ln 2) to
// first order. The argument is clamped at x >= -88, where e^88 still fits FP32.
__device__ __forceinline__ float exp_neg(float x) {
  constexpr float kLog2e = 1.44269502162933349609375f;   // log2(e) rounded to FP32
  constexpr float kLog2eTail = 1.925963033500011e-08f;    // log2(e) - kLog2e
  constexpr float kLn2 = 0.693147180559945309f;
  x = fmaxf(x, -88.f);
  const float t = -x * kLog2e;
  float err = __builtin_fmaf(-x, kLog2e, -t);
  err = __builtin_fmaf(-x, kLog2eTail, err);
  const float p = __builtin_amdgcn_exp2f(t);
  return __builtin_fmaf(p, err * kLn2, p);
}

// 1 / d for d >= 1: v_rcp_f32 and one Newton step
__device__ __forceinline__ float recip_ge1(float d) {
  const float r = __builtin_amdgcn_rcpf(d);
  return __builtin_fmaf(r, __builtin_fmaf(-d, r, 1.f), r);
}

// SiLU and its derivative; as accurate as the same formulas with the FP32
// library exponential and IEEE division (2e-7 relative for SiLU, 1e-6
// absolute for the derivative, whose own cancellation dominates), in about
// a third of the instructions.
__device__ __forceinline__ float silu(float x) { return x * recip_ge1(1.f + exp_neg(x)); }
__device__ __forceinline__ float silu_grad(float x) {
  const float s = recip_ge1(1.f + exp_neg(x));
  return s * (1.f + x * (1.f - s));
}

// Round-to-nearest-even float -> bfloat16 -> float (inputs of BF16 linears).
__host__ __device__ __forceinline__ float bf16_round(float x) {
  uint32_t u;
  __builtin_memcpy(&u, &x, 4);
  if ((u & 0x7f800000u) == 0x7f800000u) {           // inf / nan: truncate, keep nan quiet
    u &= 0xffff0000u;
    if ((u & 0x007f0000u) == 0 && (x != x)) u |= 0x00400000u;
  } else {
    u += 0x7fffu + ((u >> 16) & 1u);
    u &= 0xffff0000u;
  }
  float r;
  __builtin_memcpy(&r, &u, 4);
  return r;
}

// bfloat16 bits of x rounded to nearest even (MFMA operands)
__host__ __device__ __forceinline__ unsigned short bf16_bits(float x) {
  const float r = bf16_round(x);
  unsigned int u;
  __builtin_memcpy(&u, &r, 4);
  return (unsigned short)(u >> 16);
}

// Split-BF16 operands (FP32-accurate products on the BF16 MFMA pipe): a pair of
// FP32 values x is carried as three packed bfloat16 words p0, p1, p2 with
// p0 = bf16(x), p1 = bf16(x - p0), p2 = bf16(x - p0 - p1) per element (each
// difference exact in FP32); v_cvt_pk_bf16_f32 rounds a pair to nearest even
// and packs it (first value in the low half), shifts and masks unpack it.
typedef float f2v __attribute__((ext_vector_type(2)));
typedef __bf16 bf2v __attribute__((ext_vector_type(2)));
__device__ __forceinline__ unsigned bf16_pack2(f2v x) { return __builtin_bit_cast(unsigned, __builtin_convertvector(x, bf2v)); }
__device__ __forceinline__ f2v bf16_unpack2(unsigned w) {
  return f2v{__builtin_bit_cast(float, w << 16), __builtin_bit_cast(float, w & 0xffff0000u)};
}
__device__ __forceinline__ void split3_pair(f2v x, unsigned& p0, unsigned& p1, unsigned& p2) {
  p0 = bf16_pack2(x);
  const f2v r1 = x - bf16_unpack2(p0);
  p1 = bf16_pack2(r1);
  p2 = bf16_pack2(r1 - bf16_unpack2(p1));
}

// Round-to-nearest-even float -> IEEE binary16 -> float (FP16-linear mode);
// magnitudes beyond the binary16 range become infinite.
__host__ __device__ __forceinline__ float fp16_round(float x) { return (float)(_Float16)x; }

// Inputs and weights of the channel-mixing linears: lowp 0 keeps FP32, 1
// rounds to bfloat16, 2 to binary16.
__host__ __device__ __forceinline__ float lowp_round(float x, int lowp) {
  return lowp == 1 ? bf16_round(x) : (lowp == 2 ? fp16_round(x) : x);
}

// Forward-mode dual number carrying d/d(vx, vy, vz) of an edge vector.
template <class S>
struct Dual3 {
  S v, x, y, z;
  __host__ __device__ Dual3() : v(0), x(0), y(0), z(0) {}
  __host__ __device__ Dual3(S a) : v(a), x(0), y(0), z(0) {}
  __host__ __device__ Dual3(S a, S b, S c, S d) : v(a), x(b), y(c), z(d) {}
};
template <class S>
__host__ __device__ __forceinline__ Dual3<S> operator+(Dual3<S> a, Dual3<S> b) {
  return Dual3<S>(a.v + b.v, a.x + b.x, a.y + b.y, a.z + b.z);
}
template <class S>
__host__ __device__ __forceinline__ Dual3<S> operator-(Dual3<S> a, Dual3<S> b) {
  return Dual3<S>(a.v - b.v, a.x - b.x, a.y - b.y, a.z - b.z);
}
template <class S>
__host__ __device__ __forceinline__ Dual3<S> operator*(Dual3<S> a, Dual3<S> b) {
  return Dual3<S>(a.v * b.v, a.x * b.v + a.v * b.x, a.y * b.v + a.v * b.y, a.z * b.v + a.v * b.z);
}
template <class S>
__host__ __device__ __forceinline__ Dual3<S> operator*(S s, Dual3<S> a) {
  return Dual3<S>(s * a.v, s * a.x, s * a.y, s * a.z);
}
template <class S>
__host__ __device__ __forceinline__ Dual3<S> operator*(Dual3<S> a, S s) { return s * a; }
template <class S>
__host__ __device__ __forceinline__ Dual3<S> operator+(Dual3<S> a, S s) { return Dual3<S>(a.v + s, a.x, a.y, a.z); }
template <class S>
__host__ __device__ __forceinline__ Dual3<S> operator-(Dual3<S> a, S s) { return Dual3<S>(a.v - s, a.x, a.y, a.z); }
template <class S>
__host__ __device__ __forceinline__ Dual3<S> operator-(S s, Dual3<S> a) { return Dual3<S>(s - a.v, -a.x, -a.y, -a.z); }
template <class S>
__host__ __device__ __forceinline__ Dual3<S> operator/(Dual3<S> a, Dual3<S> b) {
  S ib = S(1) / b.v;
  S q = a.v * ib;
  return Dual3<S>(q, (a.x - q * b.x) * ib, (a.y - q * b.y) * ib, (a.z - q * b.z) * ib);
}
template <class S>
__host__ __device__ __forceinline__ Dual3<S> dsqrt(Dual3<S> a) {
  S s = sqrt(a.v);
  S h = S(0.5) / s;
  return Dual3<S>(s, a.x * h, a.y * h, a.z * h);
}
__host__ __device__ __forceinline__ double dsqrt(double a) { return sqrt(a); }
__host__ __device__ __forceinline__ void dsincos(double a, double* s, double* c) { sincos(a, s, c); }
template <class S>
__host__ __device__ __forceinline__ void dsincos(Dual3<S> a, Dual3<S>* s, Dual3<S>* c) {
  S sv, cv;
  dsincos(a.v, &sv, &cv);
  *s = Dual3<S>(sv, cv * a.x, cv * a.y, cv * a.z);
  *c = Dual3<S>(cv, -sv * a.x, -sv * a.y, -sv * a.z);
}
__host__ __device__ __forceinline__ bool lt(double a, double b) { return a < b; }
template <class S>
__host__ __device__ __forceinline__ bool lt(Dual3<S> a, double b) { return a.v < b; }

template <class T> struct ScalarOf { using type = T; };
template <class S> struct ScalarOf<Dual3<S>> { using type = S; };

// Real spherical harmonics l <= 3 of a unit vector, component normalised
// (sum_m Y_lm^2 = 2l+1), m = -l..l with m<0 ~ sin, m>0 ~ cos, no
// Condon-Shortley phase. Closed forms of
//   Y_lm = sqrt(2l+1) sqrt((l-|m|)!/(l+|m|)!) c_m P_l^(|m|)(z) T_m(x, y).
template <class T>
__host__ __device__ __forceinline__ void sh16(T x, T y, T z, T* Y) {
  using S = typename ScalarOf<T>::type;
  const S s3 = S(1.7320508075688772);
  const S s15 = S(3.8729833462074170);
  const S s5h = S(1.1180339887498949);     // sqrt(5)/2
  const S s15h = S(1.9364916731037085);    // sqrt(15)/2
  const S c31 = S(0.5400617248673217);     // sqrt(7)/sqrt(6)/2
  const S c32 = S(5.1234753829797990);     // sqrt(105)/2
  const S c33 = S(2.0916500663351889);     // sqrt(35/8)
  const S s7h = S(1.3228756555322954);     // sqrt(7)/2
  T x2 = x * x, y2 = y * y, z2 = z * z;
  Y[0] = T(S(1));
  Y[1] = s3 * y;
  Y[2] = s3 * z;
  Y[3] = s3 * x;
  Y[4] = s15 * (x * y);
  Y[5] = s15 * (y * z);
  Y[6] = s5h * (S(3) * z2 - S(1));
  Y[7] = s15 * (x * z);
  Y[8] = s15h * (x2 - y2);
  T p31 = c31 * (S(15) * z2 - S(3));
  T t3c = x * (x2 - S(3) * y2);              // Re (x+iy)^3
  T t3s = y * (S(3) * x2 - y2);              // Im (x+iy)^3
  Y[9] = c33 * t3s;
  Y[10] = (S(2) * c32) * ((x * y) * z);
  Y[11] = p31 * y;
  Y[12] = s7h * (z * (S(5) * z2 - S(3)));
  Y[13] = p31 * x;
  Y[14] = c32 * (z * (x2 - y2));
  Y[15] = c33 * t3c;
}

// Bessel radial basis times the polynomial cutoff envelope:
//   e_n(r) = sqrt(2/rc) sin(n pi r / rc) / r * u(r/rc),  n = 1..nb,
//   u(x) = 1 - (p+1)(p+2)/2 x^p + p(p+2) x^(p+1) - p(p+1)/2 x^(p+2), x < 1,
// evaluated as u(x) = (1-x)^3 sum_{j<p} (j+1)(j+2)/2 x^j (the same polynomial,
// free of the cancellation the expanded form suffers near the cutoff), and
// sin(n theta) from one sine and cosine of theta = pi r / rc by the three-term
// recurrence sin((n+1) theta) = 2 cos(theta) sin(n theta) - sin((n-1) theta)
// (in FP64 within 1.1e-14 of the direct values for n <= 16, theta in (0, pi);
// on dual numbers it carries the derivatives with it).
template <class T>
__host__ __device__ __forceinline__ void bessel_env(T r, double rc, int p, int nb, T* e) {
  using S = typename ScalarOf<T>::type;
  const S pi = S(3.14159265358979323846);
  T xr = r * S(1.0 / rc);
  T q = T(S(0.5 * p * (p + 1)));
  for (int j = p - 2; j >= 0; --j) q = q * xr + S(0.5 * (j + 1) * (j + 2));
  T om = S(1) - xr;
  T env = (om * om) * (om * q);
  if (!lt(xr, 1.0)) env = T(S(0));
  T pre = (S(sqrt(2.0 / rc)) * env) / r;
  T s1, c1;
  dsincos(r * S(pi / rc), &s1, &c1);
  const T c2 = S(2) * c1;
  T sp = T(S(0)), sn = s1;   // sin((n-1) theta), sin(n theta) for n = 1
  for (int n = 0; n < nb; ++n) {
    e[n] = pre * sn;
    const T nx = c2 * sn - sp;
    sp = sn;
    sn = nx;
  }
}

// g = dE/dd of edge e from dE/dY (dy[16]) and dE/de (de[nb]), by forward-mode
// differentiation (FP64 dual numbers) of the same closed forms with respect to
// the three components of d.
__device__ __forceinline__ float4 edge_geometry_vjp(int e, const float* __restrict__ pos,
                                                    const int* __restrict__ snd, const int* __restrict__ rcv,
                                                    const double4* __restrict__ shift, double rc, int p, int nb,
                                                    const float* dy, const float* de) {
  using D3 = Dual3<double>;
  const int s = snd[e], r = rcv[e];
  const double4 sh = shift[e];
  const D3 dx(((double)pos[3 * s + 0] - (double)pos[3 * r + 0]) + sh.x, 1.0, 0.0, 0.0);
  const D3 dyv(((double)pos[3 * s + 1] - (double)pos[3 * r + 1]) + sh.y, 0.0, 1.0, 0.0);
  const D3 dz(((double)pos[3 * s + 2] - (double)pos[3 * r + 2]) + sh.z, 0.0, 0.0, 1.0);
  const D3 rr = dsqrt(dx * dx + dyv * dyv + dz * dz);
  const D3 inv = D3(1.0) / rr;
  D3 y[16];
  sh16<D3>(dx * inv, dyv * inv, dz * inv, y);
  double gx = 0.0, gy = 0.0, gz = 0.0;
  for (int m = 1; m < 16; ++m) {
    gx += (double)dy[m] * y[m].x;
    gy += (double)dy[m] * y[m].y;
    gz += (double)dy[m] * y[m].z;
  }
  // radial basis: the terms of bessel_env, each added as it is formed (no
  // array indexed by the run-time basis size, which would live in scratch)
  const D3 xr = rr * (1.0 / rc);
  D3 q = D3(0.5 * p * (p + 1));
  for (int j = p - 2; j >= 0; --j) q = q * xr + 0.5 * (j + 1) * (j + 2);
  const D3 om = D3(1.0) - xr;
  D3 env = (om * om) * (om * q);
  if (!lt(xr, 1.0)) env = D3(0.0);
  const D3 pre = (sqrt(2.0 / rc) * env) / rr;
  const double pi = 3.14159265358979323846;
  D3 s1, c1;
  dsincos(rr * (pi / rc), &s1, &c1);
  const D3 c2 = 2.0 * c1;
  D3 sp = D3(0.0), sn = s1;   // the recurrence of bessel_env
  for (int n = 0; n < nb; ++n) {
    const D3 en = pre * sn;
    const double w = de[n];
    gx += w * en.x;
    gy += w * en.y;
    gz += w * en.z;
    const D3 nx = c2 * sn - sp;
    sp = sn;
    sn = nx;
  }
  return make_float4((float)gx, (float)gy, (float)gz, 0.f);
}

// Geometry of edge e in FP64, rounded to FP32 once: d = (x_snd - x_rcv) +
// shift, r = |d|, u = d / r; Y[16] (real harmonics of u) and eb[nb] (radial
// basis times envelope). The periodic shift and the difference of wrapped
// positions would otherwise carry FP32 rounding into every edge.
// Returns the edge's device status bits: kStatusNonFinite when d is not
// finite, kStatusZeroLength when r = 0 (coincident atoms); 0 otherwise.
__device__ __forceinline__ int edge_geometry(int e, const float* __restrict__ pos, const int* __restrict__ snd,
                                             const int* __restrict__ rcv, const double4* __restrict__ shift,
                                             double rc, int p, int nb, float* yout, float* ebout) {
  const int s = snd[e], r = rcv[e];
  const double4 sh = shift[e];
  const double dx = ((double)pos[3 * s + 0] - (double)pos[3 * r + 0]) + sh.x;
  const double dy = ((double)pos[3 * s + 1] - (double)pos[3 * r + 1]) + sh.y;
  const double dz = ((double)pos[3 * s + 2] - (double)pos[3 * r + 2]) + sh.z;
  const double rr = sqrt(dx * dx + dy * dy + dz * dz);
  const double inv = 1.0 / rr;
  double y[16];
  sh16<double>(dx * inv, dy * inv, dz * inv, y);
  for (int m = 0; m < 16; ++m) yout[m] = (float)y[m];
  double eb[16];
  bessel_env<double>(rr, rc, p, nb, eb);
  for (int n = 0; n < nb; ++n) ebout[n] = (float)eb[n];
  return !isfinite(rr) ? kStatusNonFinite : (rr == 0.0 ? kStatusZeroLength : 0);
}

// One halving step of a 64-lane reduce-scatter over v[0 .. 2 N_): lanes with
// bit XOR set keep the upper half, the others the lower half, each adding the
// partner lane's copy of the half it keeps.
template <int N_, int XOR>
__device__ __forceinline__ void halve(float* v, int lane) {
  const bool hi = lane & XOR;
#pragma unroll
  for (int q = 0; q < N_; ++q) {
    const float send = hi ? v[q] : v[q + N_];
    const float keep = hi ? v[q + N_] : v[q];
    v[q] = keep + __shfl_xor(send, XOR);
  }
}

// Sum of v[0..15] over the 64 lanes of the wave: afterwards every lane l holds
// the total of index (l >> 2) & 15 (fixed butterfly order).
__device__ __forceinline__ float wave_reduce_scatter16(float* v, int lane) {
  halve<8, 32>(v, lane);
  halve<4, 16>(v, lane);
  halve<2, 8>(v, lane);
  halve<1, 4>(v, lane);
  float t = v[0];
  t += __shfl_xor(t, 2);
  t += __shfl_xor(t, 1);
  return t;
}

// --------------------------------------------------------------- launchers
struct LinTerm {
  int in_c0;          // first input component of this term
  int src;            // 0: input x, 1: input x2
  int species;        // weights depend on the node's species (stride w_sstride)
  int64_t w_off;      // float offset of the K x K weight (species 0)
};
struct LinGroup {
  int out_c0, ncomp;  // output components [out_c0, out_c0 + ncomp)
  int t0, t1;         // terms [t0, t1) accumulate into this output
  int dst;            // 0: output y, 1: output y2
};
struct LinPlan {
  int n_groups = 0, n_terms = 0;
  LinGroup g[kMaxGroups];
  LinTerm t[kMaxTerms];
  int64_t w_sstride = 0;    // float stride between species blocks
  int cin = 0, cout = 0;    // components per node of x / y
  int cin2 = 0, cout2 = 0;  // components per node of x2 / y2
};

// One output component of one group: the unit of blockIdx.y of the linear.
struct LinGC {
  unsigned char g, c;
};
constexpr int kMaxLinGC = 96;
// What a linear launch reads besides its LinArgs. Kept in device memory
// (written once at graph setup) rather than passed by value: at about 1.4 KB
// it would make every wave fetch its plan from the kernel-argument segment.
struct LinLaunch {
  LinPlan plan;
  LinGC gc[kMaxLinGC];
  int n_gc = 0;
};
// host copy (grid shape) and device copy (read by the kernel) of one plan
struct LinPlanRef {
  LinLaunch host;
  const LinLaunch* dev = nullptr;
};
LinLaunch make_lin_launch(const LinPlan& plan);

struct LinArgs {
  const float* x;           // [N][cin][K]
  float* y;                 // [N][cout][K]
  const float* x2;          // [N][cin2][K] (terms with src 1) or null
  float* y2;                // [N][cout2][K] (groups with dst 1) or null
  const float* residual;    // [N][cout][K] or null, added to every comp written to y
  const float* w;           // weight base (FP32, row-major [in][out])
  const float* wt;          // the same blob with every K x K block transposed ([out][in])
  const unsigned short* wbf;  // same tensors in the low precision (bf16 or binary16 bits), each K x K block packed [K/8][K][8]
  const int* quad_node;     // [n_quads][kLinQuad][16]: node of MFMA row r of wave w of a block, -1 for none
                            // (a block's nodes are up to kLinQuad tiles of 16 nodes of one species)
  const int* quad_species;  // [n_quads]
  int n_quads;
  // the same grouping with kLinQuadWide tiles per block ([n_quads8][kLinQuadWide][16]),
  // taken by the wide 16-bit launches when n_quads8 > 0
  const int* quad_node8;
  const int* quad_species8;
  int n_quads8;
  int K;                    // channels per component of y (and of x unless KI is set)
  int KI;                   // channels per component of x (0: K)
  int accumulate;           // y += instead of y =
  int lowp;                 // 0: FP32; round x and w to 1: bfloat16, 2: binary16 before multiplying
  const float* bias0;       // [K] or null: rounded like the weights and added last to component 0 of y
};

// Three channel-mixing linears in a row on the 16 components of the first
// layer (the 16-bit modes at K = 128 with a 128-wide factorised contraction):
// stage s multiplies by the weight block of the output's l at st[s].w_off[l]
// (+ species * w_sstride), FP32 (panel from wt, stored [out][in]) or 16-bit
// (panel from wbf, packed [K/8][K][8]).
struct ChainStage {
  int64_t w_off[4];
  int64_t w_sstride;   // 0: the same weights for every species
  int lowp;            // 0: FP32 operands; 1, 2: bfloat16, binary16 (inputs rounded)
};
struct ChainArgs {
  const float* x;              // [N][16][128]
  float* y;                    // [N][16][128]
  const float* wt;
  const unsigned short* wbf;
  const int* quad_node;        // as LinArgs (kLinQuad tiles per block, or kLinQuadWide when n_quads8 > 0)
  const int* quad_species;
  int n_quads;
  int n_quads8;                // > 0: quad_node / quad_species hold the kLinQuadWide grouping
  int lowp;                    // the 16-bit format of the 16-bit stages
  ChainStage st[3];
};
void launch_linear_chain3(hipStream_t s, const ChainArgs& a);

constexpr int kMaxRadialLayers = 4;
// hidden-layer weights (W0 of the layer, W1 and W2 follow it) and a3 outputs
// of up to kMaxRadialLayers interaction layers
struct RadialSet {
  const float* W[kMaxRadialLayers];
  float* a3[kMaxRadialLayers];
  // where set, the layer's a3 is written as its three bfloat16 parts instead,
  // [E][3][64] (part q of edge e at a3x + (3 e + q) 64): the split-BF16 edge
  // products then read them rather than splitting a3 per channel tile
  unsigned short* a3x[kMaxRadialLayers];
  int n;
  int rnd;   // precision study: rounding of every hidden layer's input and weights (0 none, 1 bf16, 2 fp16)
};
// first interaction layer in factorised form (U, gU: [N][16][64 S], S <= 4)
void launch_l0_gather(hipStream_t s, int N, int S, const int* rcv_off, const int* snd_z, const float* a3,
                      const float* Y, int rb, float* U);
void launch_l0_edge_bwd(hipStream_t s, int N, int S, const int* rcv_off, const int* snd_z, const float* a3,
                        const float* Y, const float* gU, int rb, float* da3, float* dY);
constexpr int kL0MaxSpecies = 4;
void launch_edge_prologue(hipStream_t s, int E, const float* pos, const int* snd, const int* rcv,
                          const double4* shift, double rc, int p, int nb, float* Y, float* rbf,
                          const RadialSet& rs, int* status);
// F from the per-edge g; the same launch writes the per-graph energies E from
// the node energies eps (as launch_graph_energy).
void launch_forces(hipStream_t s, int N, const int* rcv_off, const int* snd_off, const int* snd_perm,
                   const float4* g, float* F, int G, const int* graph_off, const float* eps, double* E);
void launch_radial_bwd(hipStream_t s, int E, const float* rbf, int nb, const float* W, const float* da3p,
                       const float* dYp, int n_part, float* dY, float* de, int accumulate, int rnd);
// Stress of every graph from the edge gradients g: per-chunk FP64 partials
// (chunks [beg, end) of at most kStressChunk edges of one graph, graph gi's
// chunks at chunk_off[gi] .. chunk_off[gi + 1]), then their ordered sum.
constexpr int kStressChunk = 8192;
void launch_stress(hipStream_t s, int G, int n_chunks, const int2* chunks, const int* chunk_off, const float* pos,
                   const int* snd, const int* rcv, const double4* shift, const float4* g, const double* inv_vol,
                   double* part, double* stress);
void launch_edge_vjp(hipStream_t s, int E, const float* pos, const int* snd, const int* rcv, const double4* shift,
                     double rc, int p, int nb, const float* dY, const float* de, float4* g);
// Edge-product launchers: radial 0 FP32, 1 BF16, 2 split BF16 (FP32-accurate),
// 3 split BF16 with a3 pre-split (l_h = 1); tp_round 0/1/2 none/bf16/fp16.
// They return false, enqueuing nothing, for an (l_h, radial mode) without an
// instance (tpr_supported is false).
bool tpr_supported(int lh_max, int radial_mode);
bool launch_tpr_fwd(hipStream_t s, int lh_max, int N, int K, const int* rcv_off, const int* snd,
                    const int* src_map, const float* a3, const float* W3, const float* Y, const float* h,
                    float inv_c, float* At, int radial_mode, int tp_round);
// As launch_tpr_fwd. The FP32-accurate l_h = 2 backward needs Q (false otherwise).
bool launch_tpr_bwd(hipStream_t s, int lh_max, int N, int K, int E, const int* rcv_off, const int* snd,
                    const int* src_map, const float* a3, const float* W3, const float* Y, const float* h,
                    float inv_c, const float* dAt, float* dYp, float* Q, float* da3p, int radial_mode,
                    int tp_round);
void launch_sender_sum(hipStream_t s, int N, int C, int K, const int* snd_off, const int* snd_perm,
                       const float* Q, float* out);
// ---- FP64 debug precision (k_fp64.hip)
// A channel-mixing linear as blocks of components: term t maps input
// components cx[t] .. cx[t] + nc[t] - 1 to output components cy[t] .. with
// the K x K weights at woff[t] (row-major [in][out]; per species, K K apart,
// when spec[t]); transpose applies W^T (the backward).
constexpr int kMaxLin64Terms = 32;
struct Lin64 {
  int n_terms = 0, cin = 0, cout = 0, transpose = 0;
  int cx[kMaxLin64Terms], cy[kMaxLin64Terms], nc[kMaxLin64Terms], spec[kMaxLin64Terms];
  long long woff[kMaxLin64Terms];
};
struct SymW64 {
  const double* w[4][4];    // [L][nu] -> [S][n_eta][K] or null
};
void f64_widen(hipStream_t s, size_t n, const float* src, double* dst);
void f64_geom(hipStream_t s, int E, const double* pos, const int* snd, const int* rcv, const double4* shift,
              double rc, int p, int nb, double* Y, double* rb, int* status);
void f64_radial_fwd(hipStream_t s, int E, int nb, const double* rb, const double* W0, const double* W1,
                    const double* W2, double* z1, double* z2, double* z3);
void f64_radial_bwd(hipStream_t s, int E, int nb, const double* W0, const double* W1, const double* W2,
                    const double* z1, const double* z2, const double* z3, const double* da3, double* de, int acc);
bool f64_tp_fwd(hipStream_t s, int lh, int N, int K, const int* rcv_off, const int* snd, const double* z3,
                const double* W3, const double* Y, const double* h, double inv_c, double* At);
bool f64_tp_bwd(hipStream_t s, int lh, int E, int K, const int* snd, const int* rcv, const double* z3,
                const double* W3, const double* Y, const double* h, const double* dAt, double inv_c, double* dY,
                int accY, double* da3, double* Q);
void f64_sender_sum(hipStream_t s, int N, int C, int K, const int* snd_off, const int* snd_perm, const double* Q,
                    double* out);
void f64_linear(hipStream_t s, int N, int K, const Lin64& L, const int* species, const double* W, const double* x,
                double* y, const double* res);
bool f64_symcon_fwd(hipStream_t s, int lout, int N, int K, const int* species, const double* A, const SymW64& w,
                    double* B);
bool f64_symcon_bwd(hipStream_t s, int lout, int N, int K, const int* species, const double* A, const SymW64& w,
                    const double* dB, double* dA);
void f64_readout(hipStream_t s, int N, int K, const double* h, int stride, const double* w, const double* w2,
                 int hid, double* eps, int acc, double* dh0);
void f64_add_readout_grad(hipStream_t s, int N, int K, int stride, const double* w, double* dst);
void f64_embed(hipStream_t s, int N, int K, const int* species, const double* W, double* h0);
void f64_edge_vjp(hipStream_t s, int E, const double* pos, const int* snd, const int* rcv, const double4* shift,
                  double rc, int p, int nb, const double* dY, const double* de, double4* g);
void f64_forces(hipStream_t s, int N, const int* rcv_off, const int* snd_off, const int* snd_perm, const double4* g,
                double* F);
void f64_graph_energy(hipStream_t s, int G, const int* graph_off, const double* eps, double* E);
void f64_stress(hipStream_t s, int G, const int* graph_off, const int* rcv_off, const double* pos, const int* snd,
                const int* rcv, const double4* shift, const double4* g, const double* inv_vol, double* stress);

struct SymW {
  const float* w[4][4];     // [L][nu] -> [S][n_eta][K] or null
};
void launch_symcon_fwd(hipStream_t s, int lout_max, int N, int K, const int* species, const float* A,
                       SymW w, float* B, int rnd);
void launch_symcon_bwd(hipStream_t s, int lout_max, int N, int K, const int* species, const float* A,
                       SymW w, const float* dB, float* dA, int rnd);
void launch_linear(hipStream_t s, const LinPlanRef& plan, const LinArgs& a);
// Algorithmic work of one linear launch over N nodes: flops = 2 K^2 per
// (node, term component); bytes = every distinct input component and weight
// block read once, every output component written once (read too when
// accumulating or adding the residual).
void linear_work(const LinPlan& p, const LinArgs& a, int64_t N, int n_species, double* flops, double* bytes);
// Linear readouts (sum_k h[n][0][k] w[k]) of layers below the last, evaluated
// together with the last layer's
constexpr int kMaxReadoutLin = 4;
struct ReadoutLin {
  const float* h[kMaxReadoutLin];   // [N][stride] layer outputs
  const float* w[kMaxReadoutLin];   // [K] readout weights
  int stride[kMaxReadoutLin];
  int n;
};
// eps[n] = (eps[n] if accumulate) + the linear readouts in order + the MLP
// readout of h (null: none), added left to right. dh: for the MLP readout, also
// store its gradient dE/dh[n][0][k] there (null: not wanted).
void launch_readout_fwd(hipStream_t s, int N, int K, const ReadoutLin& lin, const float* h, int h_stride,
                        const float* w1, const float* w2, int hidden, int lowp, int accumulate, float* eps,
                        float* dh);
void launch_graph_energy(hipStream_t s, int G, const int* graph_off, const float* eps, double* E);
void launch_species_table(hipStream_t s, int S, int K, const float* emb, const float* wup, int lowp,
                          float* table);
void launch_round(hipStream_t s, float* dst, const float* src, size_t n, int rnd);   // no-op for rnd = 0

}  // namespace mace
