// Node-level kernels: the channel-mixing linears (linear_up, path-merging
// linear, species-dependent linears, product-basis linear and their
// transposes), readouts, per-graph energy sums, the layer-0 species table.
#include <algorithm>
#include <set>
#include <utility>

#include "mace_internal.h"
#include "static_loops.h"

namespace mace {

// Channel-mixing linear on MFMA. A block of kLinQuad waves owns up to four
// 16-node tiles of one species (one per wave, the 16 MFMA rows), one output
// component of one group and up to 32 output channels (kLinCt = 2 column tiles
// of 16; blockIdx.z picks which 32). For every term of the group the block
// stages the term's weight panel (32 output columns x K inputs, stored [col][k]) in LDS
// once for its four tiles; each wave reads its A operand straight from memory
// as float4 rows and its B operand from LDS as 16-byte reads.
// FP32: v_mfma_f32_16x16x4_f32 with A[l%16][l/16], B[l/16][l%16]; the K-long
// reduction runs in the order k = 16 q + 4 s + c (s = l/16 the MFMA's k slot,
// c the float4 component), so a lane's A values for four MFMAs are one float4.
// BF16 / FP16 (inputs and weights rounded to nearest even, FP32 accumulation):
// v_mfma_f32_16x16x32_bf16 / _f16 with A[l%16][8(l/16)+i], B[8(l/16)+i][l%16];
// the weights come pre-packed as [K/8][K][8] 16-bit values, i.e. 16-byte runs
// along k.
// Result register r of lane l holds D[4(l/16)+r][l%16].
typedef float f4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf8 __attribute__((ext_vector_type(8)));
typedef _Float16 h8 __attribute__((ext_vector_type(8)));
typedef unsigned short us8 __attribute__((ext_vector_type(8)));

// eight values as MFMA operand bits, two per packed hardware conversion,
// rounded to nearest even (for finite values the bits of bf16_bits, or of a
// conversion to _Float16 one value at a time)
template <int LP>
__device__ __forceinline__ us8 lowp_bits8(f4 lo, f4 hi) {
  typedef unsigned u4_ __attribute__((ext_vector_type(4)));
  typedef _Float16 h2_ __attribute__((ext_vector_type(2)));
  auto pack = [](f2v x) -> unsigned {
    if constexpr (LP == 1) return bf16_pack2(x);
    else return __builtin_bit_cast(unsigned, __builtin_convertvector(x, h2_));
  };
  const u4_ w = {pack(f2v{lo[0], lo[1]}), pack(f2v{lo[2], lo[3]}), pack(f2v{hi[0], hi[1]}), pack(f2v{hi[2], hi[3]})};
  return __builtin_bit_cast(us8, w);
}

// Column tiles of 16 per block. Four by default (measured at 1,536 and 36,864
// atoms: 4 beats 2, most in the 16-bit modes); at K = 128 all eight when the
// launch still has kLinWideGrid blocks, so that each input row is read by one
// block only (36,864 atoms: FP32 linears 4.24 -> 3.64 ms per step; at 1,536
// atoms, 384 blocks, eight was slower).
constexpr int kLinCt = 4;
constexpr int kLinCtWide = 8;
constexpr int kLinWideGrid = 2048;
constexpr int kLinSmallGrid = 512;   // blocks below which a square linear takes one column tile per block

// LP: 0 FP32, 1 BF16, 2 FP16 (the 16-bit paths share everything but the
// rounding and the MFMA instruction). K channels per output component, KI per
// input component (KI != K only on the FP32 path). CT column tiles of 16
// per block: kLinCt, or 1 for launches too small to fill the chip otherwise.
// KH: the FP32 panel staged in KH parts of the k range, one after the other
// (LDS and the registers of the panel in flight divided by KH, the same k
// order, so the same result bit for bit), for more waves per SIMD.
template <int K, int KI, int LP, int CT, int QD = kLinQuad, int KH = 1>
__global__ void __launch_bounds__(64 * QD) __attribute__((amdgpu_waves_per_eu(KH > 1 ? 3 : 1)))
linear_kernel(const LinLaunch* __restrict__ Lp, LinArgs a) {
  constexpr int kLinQuad = QD;   // node tiles (waves) of this block
  const int* quad_node = QD == mace::kLinQuad ? a.quad_node : a.quad_node8;
  const int* quad_species = QD == mace::kLinQuad ? a.quad_species : a.quad_species8;
  constexpr bool BF16 = LP != 0;   // any 16-bit path
  const LinLaunch& L = *Lp;
  static_assert(KI % 32 == 0 && K % 16 == 0, "KI is a multiple of 32, K of 16");
  static_assert(kLinTileNodes == 16, "a node tile is the 16 rows of one MFMA");
  static_assert(!BF16 || KI == K, "16-bit linears are square");
  static_assert(KH == 1 || (!BF16 && (KI / KH) % 16 == 0), "k halves on the FP32 path only");
  constexpr int KIH = KI / KH;   // k range of one staged panel
  constexpr int PF = KIH + 4;    // FP32 panel row pitch in floats (4 mod 32: conflict-free 16-byte reads)
  constexpr int PB = KI + 8;   // 16-bit panel row pitch in elements (68 dwords at K = 128)
  constexpr int kPanel = BF16 ? (16 * CT * PB + 1) / 2 : 16 * CT * PF;
  __shared__ __align__(16) float sB[kPanel];
  unsigned short* sBb = reinterpret_cast<unsigned short*>(sB);
  const LinGC gcx = L.gc[blockIdx.y];
  const LinGroup grp = L.plan.g[gcx.g];
  const int c = gcx.c;
  const int ct0 = blockIdx.z * CT;
  constexpr int nct = K / 16;
  const int ncol = min(16 * CT, K - 16 * ct0);   // valid panel columns (K = 32 or 96: the last 64 are partial)
  const int tid = threadIdx.x, l = tid & 63, w = tid >> 6;
  const int quad = blockIdx.x;
  const int z = quad_species[quad];
  const int64_t zstride = (int64_t)z * L.plan.w_sstride;
  // A rows: node of MFMA row l%16 (a row without a node reads node 0 and is
  // zeroed; a spare wave has none and stores nothing)
  const int row_node = quad_node[((size_t)quad * kLinQuad + w) * kLinTileNodes + (l & 15)];
  const int node = max(row_node, 0);
  const float keep = row_node >= 0 ? 1.f : 0.f;
  f4 acc[CT];
#pragma unroll
  for (int j = 0; j < CT; ++j) acc[j] = f4{0.f, 0.f, 0.f, 0.f};
  // Terms are software-pipelined: the next term's A rows and weight panel are
  // requested into registers while the current term's MFMAs run.
  constexpr int kPanelVec = BF16 ? 16 * CT * (K / 8) : 16 * CT * (KIH / 4);   // 16-byte vectors per panel
  constexpr int kPanelPer = (kPanelVec + 64 * kLinQuad - 1) / (64 * kLinQuad);   // per thread
  f4 av[BF16 ? 1 : KIH / 16];
  us8 ab[BF16 ? KI / 32 : 1];
  f4 pv[BF16 ? 1 : kPanelPer];
  us8 pb[BF16 ? kPanelPer : 1];
  auto load_term = [&](int tm, int kh) {
    const LinTerm term = L.plan.t[tm];
    const int64_t zoff = term.species ? zstride : 0;
    const float* xrow = term.src ? a.x2 + ((size_t)node * L.plan.cin2 + term.in_c0 + c) * KI
                                 : a.x + ((size_t)node * L.plan.cin + term.in_c0 + c) * KI;
    if constexpr (!BF16) {
#pragma unroll
      for (int q = 0; q < KIH / 16; ++q)
        av[q] = *reinterpret_cast<const f4*>(xrow + KIH * kh + 16 * q + 4 * (l >> 4)) * keep;
      // panel row = output column n: the transposed blob holds W^T[n][0..KI) contiguous
      const float* Wt = a.wt + term.w_off + zoff;
#pragma unroll
      for (int u = 0; u < kPanelPer; ++u) {
        const int idx = min(tid + 64 * kLinQuad * u, kPanelVec - 1);
        const int col = idx / (KIH / 4), k4 = idx % (KIH / 4);
        const int n = 16 * ct0 + min(col, ncol - 1);
        pv[u] = *reinterpret_cast<const f4*>(Wt + (size_t)n * KI + KIH * kh + 4 * k4);
      }
    } else {
#pragma unroll
      for (int ks = 0; ks < K / 32; ++ks) {
        const f4 lo = *reinterpret_cast<const f4*>(xrow + 32 * ks + 8 * (l >> 4)) * keep;
        const f4 hi = *reinterpret_cast<const f4*>(xrow + 32 * ks + 8 * (l >> 4) + 4) * keep;
        ab[ks] = lowp_bits8<LP>(lo, hi);
      }
      // packed [K/8][K][8]: 8 consecutive k of output column n are 16 contiguous bytes
      const unsigned short* Wp = a.wbf + term.w_off + zoff;
#pragma unroll
      for (int u = 0; u < kPanelPer; ++u) {
        const int idx = min(tid + 64 * kLinQuad * u, kPanelVec - 1);
        const int col = idx / (K / 8), kc = idx % (K / 8);
        const int n = 16 * ct0 + min(col, ncol - 1);
        pb[u] = *reinterpret_cast<const us8*>(Wp + ((size_t)kc * K + n) * 8);
      }
    }
  };
  if (grp.t0 < grp.t1) load_term(grp.t0, 0);
  for (int st = KH * grp.t0; st < KH * grp.t1; ++st) {
    __syncthreads();   // the previous step's MFMAs have read the panel (steps: term, k half)
#pragma unroll
    for (int u = 0; u < kPanelPer; ++u) {
      const int idx = tid + 64 * kLinQuad * u;
      if (idx < kPanelVec) {
        if constexpr (!BF16) {
          const int col = idx / (KIH / 4), k4 = idx % (KIH / 4);
          *reinterpret_cast<f4*>(sB + col * PF + 4 * k4) = pv[u];
        } else {
          const int col = idx / (K / 8), kc = idx % (K / 8);
          *reinterpret_cast<us8*>(sBb + col * PB + 8 * kc) = pb[u];
        }
      }
    }
    __syncthreads();
    f4 avc[BF16 ? 1 : KIH / 16];
    us8 abc[BF16 ? KI / 32 : 1];
    if constexpr (!BF16) {
#pragma unroll
      for (int q = 0; q < KIH / 16; ++q) avc[q] = av[q];
    } else {
#pragma unroll
      for (int ks = 0; ks < KI / 32; ++ks) abc[ks] = ab[ks];
    }
    if (st + 1 < KH * grp.t1) load_term((st + 1) / KH, (st + 1) % KH);   // in flight during this step's MFMAs
    if constexpr (!BF16) {
#pragma unroll
      for (int q = 0; q < KIH / 16; ++q)
#pragma unroll
        for (int j = 0; j < CT; ++j) {
          const f4 b = *reinterpret_cast<const f4*>(sB + (16 * j + (l & 15)) * PF + 16 * q + 4 * (l >> 4));
#pragma unroll
          for (int cc = 0; cc < 4; ++cc) acc[j] = __builtin_amdgcn_mfma_f32_16x16x4f32(avc[q][cc], b[cc], acc[j], 0, 0, 0);
        }
    } else {
#pragma unroll
      for (int ks = 0; ks < K / 32; ++ks)
#pragma unroll
        for (int j = 0; j < CT; ++j) {
          const us8 b = *reinterpret_cast<const us8*>(sBb + (16 * j + (l & 15)) * PB + 32 * ks + 8 * (l >> 4));
          if constexpr (LP == 1)
            acc[j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf8, abc[ks]), __builtin_bit_cast(bf8, b),
                                                             acc[j], 0, 0, 0);
          else
            acc[j] = __builtin_amdgcn_mfma_f32_16x16x32_f16(__builtin_bit_cast(h8, abc[ks]), __builtin_bit_cast(h8, b),
                                                            acc[j], 0, 0, 0);
        }
    }
  }
  int out_node[4];   // node of result row 4 (l / 16) + r, -1 for none
#pragma unroll
  for (int r = 0; r < 4; ++r) out_node[r] = __shfl(row_node, 4 * (l >> 4) + r);
  float* y = grp.dst ? a.y2 : a.y;
  const int cout = grp.dst ? L.plan.cout2 : L.plan.cout;
  const float* residual = grp.dst ? nullptr : a.residual;
#pragma unroll
  for (int j = 0; j < CT; ++j) {
    const int ct = ct0 + j;
    if (ct >= nct) continue;
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      if (out_node[r] < 0) continue;
      const size_t o = ((size_t)out_node[r] * cout + grp.out_c0 + c) * K + 16 * ct + (l & 15);
      float v = acc[j][r];
      if (residual) v += residual[o];
      if (a.accumulate) v += y[o];
      if (a.bias0 && grp.out_c0 + c == 0 && !grp.dst) v += lowp_round(a.bias0[16 * ct + (l & 15)], a.lowp);
      y[o] = v;
    }
  }
}

// Three linears in a row on one component, in one launch (the 16-bit modes'
// first layer: the FP32 contraction U -> At, then the 16-bit path-merging and
// species linears; backward, their transposes in reverse order). A block owns
// up to four 16-node tiles of one species, one of the 16 components and all
// 128 output columns. Each stage multiplies exactly as linear_kernel does
// (same operand layouts, the same k order, inputs of a 16-bit stage rounded
// from their FP32 values) and leaves its FP32 result in the wave's LDS rows,
// which the next stage reads as linear_kernel reads its input rows: the
// output equals that of three linear_kernel launches bit for bit, without the
// two intermediate arrays going through HBM.
template <int LP, int QD>
__global__ void __launch_bounds__(64 * QD) linear_chain3_kernel(ChainArgs a) {
  constexpr int kLinQuad = QD;   // node tiles (waves) of this block
  constexpr int K = 128, CT = 8;
  constexpr int PF = 64 + 4;    // FP32 panel pitch: a 64-wide half of the k range (4 mod 32)
  constexpr int PB = K + 8;     // 16-bit panel pitch (elements)
  constexpr int PT = K + 4;     // stage output row pitch (floats)
  constexpr int kPanelF = 16 * CT * PF;
  constexpr int kPanelB = (16 * CT * PB + 1) / 2;
  constexpr int kPanel = kPanelF > kPanelB ? kPanelF : kPanelB;
  __shared__ __align__(16) float sB[kPanel];
  __shared__ __align__(16) float sT[kLinQuad * 16 * PT];
  unsigned short* sBb = reinterpret_cast<unsigned short*>(sB);
  const int c = blockIdx.y;                        // component l^2 + m
  const int lc = (c >= 1) + (c >= 4) + (c >= 9);   // its l
  const int tid = threadIdx.x, l = tid & 63, w = tid >> 6;
  const int quad = blockIdx.x;
  const int z = a.quad_species[quad];
  const int row_node = a.quad_node[((size_t)quad * kLinQuad + w) * kLinTileNodes + (l & 15)];
  const int node = max(row_node, 0);
  const float keep = row_node >= 0 ? 1.f : 0.f;
  float* T = sT + w * 16 * PT;
  f4 acc[CT];
  static_for<0, 3>([&](auto S) {
    constexpr int st = decltype(S)::value;
    const ChainStage& cs = a.st[st];
    const int64_t woff = cs.w_off[lc] + (int64_t)z * cs.w_sstride;
    // input row of MFMA row l%16: the launch input for the first stage, the
    // previous stage's result (this wave's LDS rows) after it
    const float* xrow = st == 0 ? a.x + ((size_t)node * 16 + c) * K : T + (l & 15) * PT;
    const float xk = st == 0 ? keep : 1.f;
#pragma unroll
    for (int j = 0; j < CT; ++j) acc[j] = f4{0.f, 0.f, 0.f, 0.f};
    if (cs.lowp == 0) {
      // FP32: k = 16 q + 4 s + cc as in linear_kernel, the panel in two halves of k
#pragma unroll
      for (int kh = 0; kh < 2; ++kh) {
        __syncthreads();   // every wave is done with the previous panel
        for (int idx = tid; idx < 16 * CT * 16; idx += 64 * kLinQuad) {
          const int col = idx >> 4, k4 = idx & 15;
          *reinterpret_cast<f4*>(sB + col * PF + 4 * k4) =
              *reinterpret_cast<const f4*>(a.wt + woff + (size_t)col * K + 64 * kh + 4 * k4);
        }
        __syncthreads();
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const f4 av = *reinterpret_cast<const f4*>(xrow + 64 * kh + 16 * q + 4 * (l >> 4)) * xk;
#pragma unroll
          for (int j = 0; j < CT; ++j) {
            const f4 b = *reinterpret_cast<const f4*>(sB + (16 * j + (l & 15)) * PF + 16 * q + 4 * (l >> 4));
#pragma unroll
            for (int cc = 0; cc < 4; ++cc) acc[j] = __builtin_amdgcn_mfma_f32_16x16x4f32(av[cc], b[cc], acc[j], 0, 0, 0);
          }
        }
      }
    } else {
      __syncthreads();
      for (int idx = tid; idx < 16 * CT * (K / 8); idx += 64 * kLinQuad) {
        const int col = idx / (K / 8), kc = idx % (K / 8);
        *reinterpret_cast<us8*>(sBb + col * PB + 8 * kc) = *reinterpret_cast<const us8*>(a.wbf + woff + ((size_t)kc * K + col) * 8);
      }
      __syncthreads();
#pragma unroll
      for (int ks = 0; ks < K / 32; ++ks) {
        const f4 lo = *reinterpret_cast<const f4*>(xrow + 32 * ks + 8 * (l >> 4)) * xk;
        const f4 hi = *reinterpret_cast<const f4*>(xrow + 32 * ks + 8 * (l >> 4) + 4) * xk;
        const us8 v = lowp_bits8<LP>(lo, hi);
#pragma unroll
        for (int j = 0; j < CT; ++j) {
          const us8 b = *reinterpret_cast<const us8*>(sBb + (16 * j + (l & 15)) * PB + 32 * ks + 8 * (l >> 4));
          if constexpr (LP == 1)
            acc[j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf8, v), __builtin_bit_cast(bf8, b), acc[j], 0, 0, 0);
          else
            acc[j] = __builtin_amdgcn_mfma_f32_16x16x32_f16(__builtin_bit_cast(h8, v), __builtin_bit_cast(h8, b), acc[j], 0, 0, 0);
        }
      }
    }
    if constexpr (st < 2) {
      // the result into this wave's rows (its input reads are done: the
      // products that used them come first); LDS operations of a wave
      // complete in order, and the barriers keep the compiler's order
      __asm__ volatile("" ::: "memory");
      __builtin_amdgcn_wave_barrier();
#pragma unroll
      for (int j = 0; j < CT; ++j)
#pragma unroll
        for (int r = 0; r < 4; ++r) T[(4 * (l >> 4) + r) * PT + 16 * j + (l & 15)] = acc[j][r];
      __asm__ volatile("" ::: "memory");
      __builtin_amdgcn_wave_barrier();
    }
  });
  int out_node[4];   // node of result row 4 (l / 16) + r, -1 for none
#pragma unroll
  for (int r = 0; r < 4; ++r) out_node[r] = __shfl(row_node, 4 * (l >> 4) + r);
#pragma unroll
  for (int j = 0; j < CT; ++j)
#pragma unroll
    for (int r = 0; r < 4; ++r)
      if (out_node[r] >= 0) a.y[((size_t)out_node[r] * 16 + c) * K + 16 * j + (l & 15)] = acc[j][r];
}

void launch_linear_chain3(hipStream_t s, const ChainArgs& a) {
  if (a.n_quads <= 0) return;
  if (a.n_quads8 > 0) {
    dim3 grid(a.n_quads8, 16), block(64 * kLinQuadWide);
    if (a.lowp == 2) linear_chain3_kernel<2, kLinQuadWide><<<grid, block, 0, s>>>(a);
    else linear_chain3_kernel<1, kLinQuadWide><<<grid, block, 0, s>>>(a);
    return;
  }
  dim3 grid(a.n_quads, 16), block(64 * kLinQuad);
  if (a.lowp == 2) linear_chain3_kernel<2, kLinQuad><<<grid, block, 0, s>>>(a);
  else linear_chain3_kernel<1, kLinQuad><<<grid, block, 0, s>>>(a);
}

LinLaunch make_lin_launch(const LinPlan& plan) {
  LinLaunch L;
  L.plan = plan;
  int n = 0;
  for (int g = 0; g < plan.n_groups; ++g)
    for (int c = 0; c < plan.g[g].ncomp && n < kMaxLinGC; ++c) {
      L.gc[n].g = (unsigned char)g;
      L.gc[n].c = (unsigned char)c;
      ++n;
    }
  L.n_gc = n;
  // Blocks run in blockIdx.y-major order. Where every group has one term
  // (a transposed path-merging linear: several outputs read each input
  // component), order the (group, component) units by the input component
  // they read, so that the blocks reading one input row run one after
  // another and find it in L2 instead of HBM.
  bool single = plan.n_groups > 0;
  for (int g = 0; g < plan.n_groups; ++g) single = single && plan.g[g].t1 - plan.g[g].t0 == 1;
  if (single) {
    auto key = [&](const LinGC& u) {
      const LinTerm& t = plan.t[plan.g[u.g].t0];
      return t.src * 4096 + t.in_c0 + u.c;
    };
    std::stable_sort(L.gc, L.gc + n, [&](const LinGC& a, const LinGC& b) { return key(a) < key(b); });
  }
  return L;
}

void linear_work(const LinPlan& p, const LinArgs& a, int64_t N, int n_species, double* flops, double* bytes) {
  const double K = a.K, KI = a.KI > 0 ? a.KI : a.K;
  const double row = (double)N * K * 4.0, row_in = (double)N * KI * 4.0;
  const double wbytes = KI * K * (a.lowp ? 2.0 : 4.0);
  std::set<std::pair<int, int>> in_comp;
  std::set<std::pair<int64_t, int>> wblk;
  double f = 0.0, b = 0.0;
  for (int gi = 0; gi < p.n_groups; ++gi) {
    const LinGroup& g = p.g[gi];
    for (int ti = g.t0; ti < g.t1; ++ti) {
      const LinTerm& t = p.t[ti];
      f += 2.0 * KI * K * (double)N * g.ncomp;
      for (int c = 0; c < g.ncomp; ++c) in_comp.insert({t.src, t.in_c0 + c});
      wblk.insert({t.w_off, t.species});
    }
    const bool resid = a.residual && g.dst == 0;
    b += g.ncomp * row * (1.0 + (a.accumulate ? 1.0 : 0.0) + (resid ? 1.0 : 0.0));
  }
  b += in_comp.size() * row_in;
  for (const auto& w : wblk) b += wbytes * (w.second ? n_species : 1);
  *flops = f;
  *bytes = b;
}

void launch_linear(hipStream_t s, const LinPlanRef& P, const LinArgs& a) {
  if (a.n_quads <= 0 || P.host.plan.n_groups <= 0 || !P.dev) return;
  const LinLaunch* L = P.dev;
  const int halves = (a.K / 16 + kLinCt - 1) / kLinCt;
  dim3 grid(a.n_quads, P.host.n_gc, halves), block(64 * kLinQuad);
  const int KI0 = a.KI > 0 ? a.KI : a.K;
  if (a.K == 128 && KI0 <= 128 && (int64_t)a.n_quads * P.host.n_gc >= kLinWideGrid) {
    // wide blocks: all 128 output columns, each input row read once
    dim3 gw(a.n_quads, P.host.n_gc, 1);
    if (KI0 != a.K) {
      if (a.lowp) return;
      switch (KI0) {
        case 32: linear_kernel<128, 32, 0, kLinCtWide><<<gw, block, 0, s>>>(L, a); break;
        case 64: linear_kernel<128, 64, 0, kLinCtWide><<<gw, block, 0, s>>>(L, a); break;
        case 96: linear_kernel<128, 96, 0, kLinCtWide><<<gw, block, 0, s>>>(L, a); break;
      }
      return;
    }
    if (a.lowp && a.n_quads8 > 0) {
      // large graphs, 16-bit operands: eight node tiles per block, so that each
      // staged weight panel serves twice the rows (36,864 atoms: BF16 linears
      // 2.94 -> 2.28 ms per step; FP32 unchanged, smaller graphs slower)
      dim3 g8(a.n_quads8, P.host.n_gc, 1), b8(64 * kLinQuadWide);
      if (a.lowp == 1) linear_kernel<128, 128, 1, kLinCtWide, kLinQuadWide><<<g8, b8, 0, s>>>(L, a);
      else linear_kernel<128, 128, 2, kLinCtWide, kLinQuadWide><<<g8, b8, 0, s>>>(L, a);
      return;
    }
    if (a.lowp == 1) linear_kernel<128, 128, 1, kLinCtWide><<<gw, block, 0, s>>>(L, a);
    else if (a.lowp == 2) linear_kernel<128, 128, 2, kLinCtWide><<<gw, block, 0, s>>>(L, a);
    // FP32: the panel in four k quarters (17 KB of LDS, 94 registers, five
    // waves per SIMD instead of two; 36,864 atoms: 3.58 -> 3.05 ms per step)
    else linear_kernel<128, 128, 0, kLinCtWide, kLinQuad, 4><<<gw, block, 0, s>>>(L, a);
    return;
  }
  if (KI0 == a.K && (int64_t)a.n_quads * P.host.n_gc * halves < kLinSmallGrid) {
    // small launch: one column tile per block, kLinCt times the blocks
    dim3 g1(a.n_quads, P.host.n_gc, a.K / 16);
    auto sq1 = [&](auto KK) {
      constexpr int k = decltype(KK)::value;
      if (a.lowp == 1) linear_kernel<k, k, 1, 1><<<g1, block, 0, s>>>(L, a);
      else if (a.lowp == 2) linear_kernel<k, k, 2, 1><<<g1, block, 0, s>>>(L, a);
      else linear_kernel<k, k, 0, 1><<<g1, block, 0, s>>>(L, a);
    };
    switch (a.K) {
      case 32: sq1(std::integral_constant<int, 32>{}); break;
      case 64: sq1(std::integral_constant<int, 64>{}); break;
      case 96: sq1(std::integral_constant<int, 96>{}); break;
      case 128: sq1(std::integral_constant<int, 128>{}); break;
    }
    return;
  }
  const int KI = a.KI > 0 ? a.KI : a.K;
  if (KI != a.K) {   // FP32 only: the factorised first-layer contraction and its transpose
    if (a.lowp) return;
    auto go = [&](auto KO, auto KIN) {
      linear_kernel<decltype(KO)::value, decltype(KIN)::value, 0, kLinCt><<<grid, block, 0, s>>>(L, a);
    };
    auto in_w = [&](auto KO) {
      switch (KI) {
        case 32: go(KO, std::integral_constant<int, 32>{}); break;
        case 64: go(KO, std::integral_constant<int, 64>{}); break;
        case 96: go(KO, std::integral_constant<int, 96>{}); break;
        case 128: go(KO, std::integral_constant<int, 128>{}); break;
        case 192: go(KO, std::integral_constant<int, 192>{}); break;
        case 256: go(KO, std::integral_constant<int, 256>{}); break;
      }
    };
    switch (a.K) {
      case 32: in_w(std::integral_constant<int, 32>{}); break;
      case 64: in_w(std::integral_constant<int, 64>{}); break;
      case 96: in_w(std::integral_constant<int, 96>{}); break;
      case 128: in_w(std::integral_constant<int, 128>{}); break;
      case 192: in_w(std::integral_constant<int, 192>{}); break;
      case 256: in_w(std::integral_constant<int, 256>{}); break;
    }
    return;
  }
#define MACE_LIN(KK)                                                            \
  case KK:                                                                     \
    if (a.lowp == 1) linear_kernel<KK, KK, 1, kLinCt><<<grid, block, 0, s>>>(L, a);    \
    else if (a.lowp == 2) linear_kernel<KK, KK, 2, kLinCt><<<grid, block, 0, s>>>(L, a); \
    else linear_kernel<KK, KK, 0, kLinCt><<<grid, block, 0, s>>>(L, a);                \
    break;
  switch (a.K) {
    MACE_LIN(32)
    MACE_LIN(64)
    MACE_LIN(96)
    MACE_LIN(128)
  }
#undef MACE_LIN
}

// ---------------------------------------------------------------- readouts
// One wave per node (4 per block). Non-last layers: eps[n] (+)= sum_k h[n][0][k] w[k].
// Last layer: eps[n] (+)= sum_j w2[j] silu(z_j), z_j = sum_k h[n][0][k] W1[k][j]
// (hidden <= 16): lane j + 16 q forms the part of z_j over the q-th quarter of
// the channels, xor-butterflies sum the quarters and then the hidden units, in
// a fixed order.
constexpr int kReadoutNodes = 4;

constexpr int kReadoutHiddenMax = 16;

// z_j of the last-layer readout, in every lane whose hidden index is j (each
// lane's loads are issued together, then summed in k order). sw1: W1 in LDS,
// already rounded, row pitch hp.
template <int K>
__device__ __forceinline__ float readout_hidden_z(const float* __restrict__ hrow, const float* sw1, int hp,
                                                  int hidden, int lowp, int lane) {
  const int j = lane & 15, q = lane >> 4;
  constexpr int kq = K / 4;
  float hv[kq], wv[kq];
#pragma unroll
  for (int i = 0; i < kq; ++i) {
    hv[i] = j < hidden ? hrow[q * kq + i] : 0.f;
    wv[i] = j < hidden ? sw1[(q * kq + i) * hp + j] : 0.f;
  }
  float z = 0.f;
#pragma unroll
  for (int i = 0; i < kq; ++i) z += lowp_round(hv[i], lowp) * wv[i];
  z += __shfl_xor(z, 16);
  z += __shfl_xor(z, 32);
  return z;
}

// dE/dh[n][0][k] = sum_j W1[k][j] w2[j] silu'(z_j) of the last-layer readout,
// stored to drow (the energy reaches the last layer's output, a single scalar
// component, only through this readout)
template <int K>
__device__ __forceinline__ void readout_mlp_grad(float z, const float* sw1, int hp, const float* __restrict__ w2,
                                                 int hidden, int lowp, int lane, float* __restrict__ drow) {
  const int j = lane & 15;
  const float gz = j < hidden ? lowp_round(lowp_round(w2[j], lowp) * silu_grad(z), lowp) : 0.f;
  float gs[kReadoutHiddenMax];
#pragma unroll
  for (int jj = 0; jj < kReadoutHiddenMax; ++jj) gs[jj] = __shfl(gz, jj);
#pragma unroll
  for (int r = 0; r < (K + 63) / 64; ++r) {
    const int k = lane + 64 * r;
    if (k < K) {
      float wv[kReadoutHiddenMax];
#pragma unroll
      for (int jj = 0; jj < kReadoutHiddenMax; ++jj) wv[jj] = jj < hidden ? sw1[k * hp + jj] : 0.f;
      float acc = 0.f;
#pragma unroll
      for (int jj = 0; jj < kReadoutHiddenMax; ++jj)
        if (jj < hidden) acc += gs[jj] * wv[jj];
      drow[k] = acc;
    }
  }
}

// sum_k h[k] w[k] of a linear readout, in every lane (fixed order: strided
// partial sums, then an xor-butterfly)
template <int K>
__device__ __forceinline__ float readout_linear(const float* __restrict__ hrow, const float* __restrict__ w, int lowp,
                                                int lane) {
  float v = 0.f;
#pragma unroll
  for (int r = 0; r < (K + 63) / 64; ++r) {
    const int k = lane + 64 * r;
    if (k < K) v += lowp_round(hrow[k], lowp) * lowp_round(w[k], lowp);
  }
#pragma unroll
  for (int m = 32; m > 0; m >>= 1) v += __shfl_xor(v, m);
  return v;
}

// eps[n] = (prior) + lin readout 0 + lin readout 1 + ... + MLP readout, added
// left to right: the prior is eps[n] itself when accumulate is set, and the MLP
// readout (h non-null, the last layer) reads h. dh (MLP readout only, null
// otherwise): its gradient is stored there as well, so that the backward pass
// starts from it.
template <int K>
__global__ void __launch_bounds__(64 * kReadoutNodes) readout_fwd_kernel(int N, ReadoutLin lin,
                                                                         const float* __restrict__ h, int h_stride,
                                                                         const float* __restrict__ w1,
                                                                         const float* __restrict__ w2, int hidden,
                                                                         int lowp, int accumulate,
                                                                         float* __restrict__ eps,
                                                                         float* __restrict__ dh) {
  const int n = blockIdx.x * kReadoutNodes + (threadIdx.x >> 6), lane = threadIdx.x & 63;
  // W1 rounded into LDS, row pitch hidden + 1 (the gradient's lanes run over k)
  __shared__ float sw1[K * (kReadoutHiddenMax + 1)];
  const int hp = hidden + 1;
  if (h) {
    for (int idx = threadIdx.x; idx < K * hidden; idx += blockDim.x)
      sw1[(idx / hidden) * hp + idx % hidden] = lowp_round(w1[idx], lowp);
    __syncthreads();
  }
  if (n >= N) return;
  bool have = accumulate != 0;
  float v = have ? eps[n] : 0.f;
  for (int i = 0; i < lin.n; ++i) {
    const float r = readout_linear<K>(lin.h[i] + (size_t)n * lin.stride[i], lin.w[i], lowp, lane);
    v = have ? v + r : r;
    have = true;
  }
  if (h) {
    const float z = readout_hidden_z<K>(h + (size_t)n * h_stride, sw1, hp, hidden, lowp, lane);
    const int j = lane & 15;
    float r = j < hidden ? lowp_round(silu(z), lowp) * lowp_round(w2[j], lowp) : 0.f;
#pragma unroll
    for (int m = 8; m > 0; m >>= 1) r += __shfl_xor(r, m);
    v = have ? v + r : r;
    if (dh) readout_mlp_grad<K>(z, sw1, hp, w2, hidden, lowp, lane, dh + (size_t)n * h_stride);
  }
  if (lane == 0) eps[n] = v;
}

// table[z][k] = sum_k' emb[z][k'] Wup[k'][k]: layer-0 features depend only on
// species. Accumulated in FP64 (one rounding, once per graph setup): a
// rounding error here is shared by every atom of the species.
__global__ void species_table_kernel(int S, int K, const float* __restrict__ emb, const float* __restrict__ wup,
                                     int lowp, float* __restrict__ table) {
  const int idx = blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= S * K) return;
  const int z = idx / K, k = idx % K;
  double acc = 0.0;
  for (int kk = 0; kk < K; ++kk) {
    float x = emb[(size_t)z * K + kk], w = wup[(size_t)kk * K + k];
    if (lowp) {
      x = lowp_round(x, lowp);
      w = lowp_round(w, lowp);
    }
    acc += (double)x * (double)w;
  }
  table[idx] = (float)acc;
}

void launch_readout_fwd(hipStream_t s, int N, int K, const ReadoutLin& lin, const float* h, int h_stride,
                        const float* w1, const float* w2, int hidden, int lowp, int accumulate, float* eps,
                        float* dh) {
  if (N <= 0 || (lin.n == 0 && !h)) return;
  const dim3 grid((N + kReadoutNodes - 1) / kReadoutNodes), block(64 * kReadoutNodes);
  float* dhx = h ? dh : nullptr;
  switch (K) {
    case 32: readout_fwd_kernel<32><<<grid, block, 0, s>>>(N, lin, h, h_stride, w1, w2, hidden, lowp, accumulate, eps, dhx); break;
    case 64: readout_fwd_kernel<64><<<grid, block, 0, s>>>(N, lin, h, h_stride, w1, w2, hidden, lowp, accumulate, eps, dhx); break;
    case 96: readout_fwd_kernel<96><<<grid, block, 0, s>>>(N, lin, h, h_stride, w1, w2, hidden, lowp, accumulate, eps, dhx); break;
    case 128: readout_fwd_kernel<128><<<grid, block, 0, s>>>(N, lin, h, h_stride, w1, w2, hidden, lowp, accumulate, eps, dhx); break;
  }
}
void launch_species_table(hipStream_t s, int S, int K, const float* emb, const float* wup, int lowp, float* table) {
  species_table_kernel<<<(S * K + 127) / 128, 128, 0, s>>>(S, K, emb, wup, lowp, table);
}

}  // namespace mace
