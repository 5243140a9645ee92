// Device neighbour list for the graph problem statement: sender j -> receiver
// i with image shift S is an edge iff
//   0 < (d_x^2 + d_y^2) + d_z^2 < r_c^2,  d = (x_j - x_i) + ((S_0 a_0 + S_1 a_1) + S_2 a_2),
// evaluated in FP64 with this operation order and no fused multiply-adds (the
// same expression as the host list, so both produce the same edge set), every
// periodic image enumerated, graphs never joined, output sorted by
// (receiver, sender, S_0, S_1, S_2).
//
// Method (hashed cell list):
//  1. every atom of a periodic graph is wrapped into its cell, x = x_w + n.cell
//     with n = floor(fractional coordinates); the wrapped fractional
//     coordinates lie in [0, 1), so images S' with |S'_a| <= floor(r_c |b_a| + 1)
//     (b_a the reciprocal row) cover every pair within r_c;
//  2. every image p = x_w + S'.cell of every atom (a candidate) is binned in
//     Cartesian cubes of edge r_c + 1e-6, the cube (with the graph) hashed into
//     a power-of-two slot table; a counting sort groups candidates by slot;
//  3. one thread per receiver visits the 27 cubes around it, keeps the
//     candidates of its own graph and cube, converts S' to the shift of the
//     given (unwrapped) positions, S = S' - n_j + n_i, and applies the exact
//     test above; a first pass counts, a scan gives each receiver its output
//     segment, a second pass writes it and sorts it by (sender, S).
// Binning only selects candidates; the cube edge exceeds r_c, so no pair
// within r_c is missed, and every edge passes the exact FP64 test.
#pragma clang fp contract(off)

#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdint>
#include <cstring>
#include <mutex>
#include <vector>

#include "../../include/mace.h"

namespace {

struct NlGraph {
  double cell[9];   // rows = lattice vectors; zero without periodicity
  double inv[9];    // cell^-1: fractional coordinate a = x . column a
  int periodic;
  int nr[3];        // wrapped-image range per lattice direction
  int a0, a1;       // atoms [a0, a1)
  int nimg;         // images per atom, prod (2 nr_a + 1)
  int pad;
  int64_t c0;       // first candidate of the graph
};

constexpr int kNlThreads = 256;
constexpr int kScanPerThread = 16;
constexpr int kScanTile = kNlThreads * kScanPerThread;
constexpr double kCoordLimit = 1e9;   // |coordinate| bound (keeps cube indices in int32)
constexpr int kFlagNonFinite = 1, kFlagRange = 2;

__device__ __forceinline__ int graph_of(const NlGraph* gs, int G, int atom) {
  int lo = 0, hi = G - 1;
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (gs[mid].a0 <= atom) lo = mid;
    else hi = mid - 1;
  }
  return lo;
}

__device__ __forceinline__ int graph_of_cand(const NlGraph* gs, int G, int64_t c) {
  int lo = 0, hi = G - 1;
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (gs[mid].c0 <= c) lo = mid;
    else hi = mid - 1;
  }
  return lo;
}

__device__ __forceinline__ uint32_t slot_of(int g, int bx, int by, int bz, uint32_t mask) {
  uint64_t h = (uint64_t)(uint32_t)g;
  h = h * 0x100000001B3ull + (uint32_t)bx;
  h = h * 0x100000001B3ull + (uint32_t)by;
  h = h * 0x100000001B3ull + (uint32_t)bz;
  h ^= h >> 33;   // splitmix64 finaliser
  h *= 0xFF51AFD7ED558CCDull;
  h ^= h >> 33;
  h *= 0xC4CEB9FE1A85EC53ull;
  h ^= h >> 33;
  return (uint32_t)h & mask;
}

__device__ __forceinline__ int cube(double p, double bs) { return (int)floor(p / bs); }

// Wrap atoms of periodic graphs into the cell; flag non-finite or huge coordinates.
__global__ void nl_wrap_kernel(int N, const double* __restrict__ pos, const NlGraph* __restrict__ gs, int G,
                               double* __restrict__ xw, int4* __restrict__ nsh, int* __restrict__ flags) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= N) return;
  const NlGraph& g = gs[graph_of(gs, G, i)];
  const double x[3] = {pos[3 * i], pos[3 * i + 1], pos[3 * i + 2]};
  int bad = 0;
  for (int c = 0; c < 3; ++c) {
    if (!isfinite(x[c])) bad |= kFlagNonFinite;
    else if (fabs(x[c]) > kCoordLimit) bad |= kFlagRange;
  }
  if (bad) atomicOr(flags, bad);
  int n[3] = {0, 0, 0};
  double w[3] = {x[0], x[1], x[2]};
  if (g.periodic && !bad) {
    for (int a = 0; a < 3; ++a) n[a] = (int)floor((x[0] * g.inv[0 * 3 + a] + x[1] * g.inv[1 * 3 + a]) + x[2] * g.inv[2 * 3 + a]);
    for (int c = 0; c < 3; ++c)
      w[c] = x[c] - (((double)n[0] * g.cell[0 * 3 + c] + (double)n[1] * g.cell[1 * 3 + c]) + (double)n[2] * g.cell[2 * 3 + c]);
  }
  for (int c = 0; c < 3; ++c) xw[3 * i + c] = bad ? 0.0 : w[c];
  nsh[i] = make_int4(n[0], n[1], n[2], bad);
}

// Candidates: image S' of atom j, its cube and slot; slot populations counted.
__global__ void nl_cand_kernel(int64_t C, const NlGraph* __restrict__ gs, int G, const double* __restrict__ xw,
                               double bs, uint32_t mask, int* __restrict__ cand_j, int4* __restrict__ cand_s,
                               int4* __restrict__ cand_b, int* __restrict__ slot_cnt) {
  const int64_t c = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (c >= C) return;
  const int gi = graph_of_cand(gs, G, c);
  const NlGraph& g = gs[gi];
  const int64_t local = c - g.c0;
  const int j = g.a0 + (int)(local / g.nimg);
  int s = (int)(local % g.nimg);
  const int w2 = 2 * g.nr[2] + 1, w1 = 2 * g.nr[1] + 1;
  const int s2 = s % w2 - g.nr[2];
  s /= w2;
  const int s1 = s % w1 - g.nr[1];
  const int s0 = s / w1 - g.nr[0];
  int b[3];
  for (int q = 0; q < 3; ++q) {
    const double p = xw[3 * j + q] + (((double)s0 * g.cell[0 * 3 + q] + (double)s1 * g.cell[1 * 3 + q]) +
                                      (double)s2 * g.cell[2 * 3 + q]);
    b[q] = cube(p, bs);
  }
  cand_j[c] = j;
  cand_s[c] = make_int4(s0, s1, s2, gi);
  cand_b[c] = make_int4(b[0], b[1], b[2], 0);
  atomicAdd(&slot_cnt[slot_of(gi, b[0], b[1], b[2], mask)], 1);
}

__global__ void nl_scatter_kernel(int64_t C, const int4* __restrict__ cand_s, const int4* __restrict__ cand_b,
                                  uint32_t mask, const int64_t* __restrict__ slot_off, int* __restrict__ slot_fill,
                                  int* __restrict__ order) {
  const int64_t c = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (c >= C) return;
  const int4 b = cand_b[c];
  const uint32_t slot = slot_of(cand_s[c].w, b.x, b.y, b.z, mask);
  order[slot_off[slot] + atomicAdd(&slot_fill[slot], 1)] = (int)c;
}

// Receiver pass, one wave per receiver: WRITE = false counts the edges of
// receiver i, WRITE = true writes them to [off_i, off_{i+1}) sorted by
// (sender, S). The candidates of the 27 cubes around the receiver form one
// index range (cube after cube, slot order within a cube) that the lanes
// take 64 at a time; an edge's place is the number of passing candidates
// before it (ballot prefix). The segment is sorted by rank (each edge's
// position = the number of keys below its own; keys are distinct) from a
// per-wave LDS copy, or, beyond kNlSortCap edges, by one lane in place.
constexpr int kNlWaves = 4;        // receivers per block
constexpr int kNlSortCap = 256;    // edges per receiver sorted through LDS

struct NlKey {
  int j, s0, s1, s2;
};

__device__ __forceinline__ bool key_lt(const NlKey& a, const NlKey& b) {
  if (a.j != b.j) return a.j < b.j;
  if (a.s0 != b.s0) return a.s0 < b.s0;
  if (a.s1 != b.s1) return a.s1 < b.s1;
  return a.s2 < b.s2;
}

template <bool WRITE>
__global__ void __launch_bounds__(64 * kNlWaves)
nl_receiver_kernel(int N, const double* __restrict__ pos, const NlGraph* __restrict__ gs, int G,
                   const double* __restrict__ xw, const int4* __restrict__ nsh, double bs, double rc2, uint32_t mask,
                   const int64_t* __restrict__ slot_off, const int* __restrict__ order,
                   const int* __restrict__ cand_j, const int4* __restrict__ cand_s, const int4* __restrict__ cand_b,
                   int* __restrict__ count, const int64_t* __restrict__ off, int32_t* __restrict__ sender,
                   int32_t* __restrict__ receiver, int32_t* __restrict__ shifts) {
  __shared__ int64_t s_first[kNlWaves][27];
  __shared__ int64_t s_end[kNlWaves][28];   // inclusive prefix of the cube ranges
  __shared__ int s_cube[kNlWaves][27][3];
  __shared__ NlKey s_key[WRITE ? kNlWaves : 1][WRITE ? kNlSortCap : 1];
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int i = blockIdx.x * kNlWaves + w;
  if (i >= N) return;   // whole wave; no block-wide barrier below
  const int gi = graph_of(gs, G, i);
  const NlGraph& g = gs[gi];
  const int4 ni = nsh[i];
  const int64_t base = WRITE ? off[i] : 0;
  const int64_t n_expect = WRITE ? off[i + 1] - off[i] : 0;
  if (WRITE && n_expect == 0) return;
  int64_t n = 0;
  if (!ni.w) {
    const double xi[3] = {pos[3 * i], pos[3 * i + 1], pos[3 * i + 2]};
    const int bi[3] = {cube(xw[3 * i], bs), cube(xw[3 * i + 1], bs), cube(xw[3 * i + 2], bs)};
    // lanes 0..26: one neighbouring cube each, its slot range, then the prefix
    int64_t len = 0;
    if (lane < 27) {
      const int bx = bi[0] + lane / 9 - 1, by = bi[1] + (lane / 3) % 3 - 1, bz = bi[2] + lane % 3 - 1;
      const uint32_t slot = slot_of(gi, bx, by, bz, mask);
      s_first[w][lane] = slot_off[slot];
      len = slot_off[slot + 1] - slot_off[slot];
      s_cube[w][lane][0] = bx;
      s_cube[w][lane][1] = by;
      s_cube[w][lane][2] = bz;
    }
    long long incl = len;
#pragma unroll
    for (int st = 1; st < 32; st <<= 1) {
      const long long v = __shfl_up(incl, st);
      if (lane >= st) incl += v;
    }
    if (lane < 27) s_end[w][lane] = incl;
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
    const int64_t total = s_end[w][26];
    for (int64_t q0 = 0; q0 < total; q0 += 64) {
      const int64_t q = q0 + lane;
      bool hit = false;
      int j = 0, S[3] = {0, 0, 0};
      if (q < total) {
        int c = 0;
        while (s_end[w][c] <= q) ++c;   // the cube whose range holds q
        const int64_t qs = s_first[w][c] + (q - (c ? s_end[w][c - 1] : 0));
        const int cidx = order[qs];
        const int4 cs = cand_s[cidx];
        const int4 cb = cand_b[cidx];
        if (cs.w == gi && cb.x == s_cube[w][c][0] && cb.y == s_cube[w][c][1] && cb.z == s_cube[w][c][2]) {
          j = cand_j[cidx];
          const int4 nj = nsh[j];
          if (!nj.w) {
            S[0] = cs.x - nj.x + ni.x;
            S[1] = cs.y - nj.y + ni.y;
            S[2] = cs.z - nj.z + ni.z;
            double d[3];
            for (int q3 = 0; q3 < 3; ++q3) {
              const double sv = g.periodic ? ((double)S[0] * g.cell[0 * 3 + q3] + (double)S[1] * g.cell[1 * 3 + q3]) +
                                                 (double)S[2] * g.cell[2 * 3 + q3]
                                           : 0.0;
              d[q3] = (pos[3 * j + q3] - xi[q3]) + sv;
            }
            const double r2 = (d[0] * d[0] + d[1] * d[1]) + d[2] * d[2];
            hit = r2 < rc2 && r2 > 0.0;
          }
        }
      }
      const uint64_t bal = __ballot(hit);
      if (WRITE && hit) {
        const int64_t at = n + __builtin_amdgcn_mbcnt_hi((uint32_t)(bal >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)bal, 0));
        if (n_expect <= kNlSortCap) {
          if (at < kNlSortCap) s_key[w][at] = NlKey{j, S[0], S[1], S[2]};
        } else {
          const int64_t e = base + at;
          sender[e] = j;
          shifts[3 * e] = S[0];
          shifts[3 * e + 1] = S[1];
          shifts[3 * e + 2] = S[2];
        }
      }
      n += __popcll(bal);
    }
  }
  if (!WRITE) {
    if (lane == 0) count[i] = (int)n;
    return;
  }
  if (n_expect <= kNlSortCap) {
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
    for (int a = lane; a < n_expect; a += 64) {
      const NlKey ka = s_key[w][a];
      int rank = 0;
      for (int b = 0; b < n_expect; ++b) rank += key_lt(s_key[w][b], ka);
      const int64_t e = base + rank;
      sender[e] = ka.j;
      receiver[e] = i;
      shifts[3 * e] = ka.s0;
      shifts[3 * e + 1] = ka.s1;
      shifts[3 * e + 2] = ka.s2;
    }
    return;
  }
  // long segment: insertion sort in place by lane 0, after every lane's
  // writes above are visible to it
  for (int64_t a = lane; a < n_expect; a += 64) receiver[base + a] = i;
  __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "workgroup");
  __builtin_amdgcn_wave_barrier();
  if (lane != 0) return;
  for (int64_t a = 1; a < n_expect; ++a) {
    const int64_t ea = base + a;
    const NlKey ka{sender[ea], shifts[3 * ea], shifts[3 * ea + 1], shifts[3 * ea + 2]};
    int64_t b = a - 1;
    while (b >= 0) {
      const int64_t eb = base + b;
      const NlKey kb{sender[eb], shifts[3 * eb], shifts[3 * eb + 1], shifts[3 * eb + 2]};
      if (!key_lt(ka, kb)) break;
      sender[eb + 1] = kb.j;
      shifts[3 * (eb + 1)] = kb.s0;
      shifts[3 * (eb + 1) + 1] = kb.s1;
      shifts[3 * (eb + 1) + 2] = kb.s2;
      --b;
    }
    const int64_t ed = base + b + 1;
    sender[ed] = ka.j;
    shifts[3 * ed] = ka.s0;
    shifts[3 * ed + 1] = ka.s1;
    shifts[3 * ed + 2] = ka.s2;
  }
}

// Exclusive scan of n int32 counts into out[0..n] (out[n] = total), int64.
// Tile pass (kScanTile elements per block, tile totals to bsum), one-block
// pass over the tile totals, then the tile offsets added.
__device__ __forceinline__ int64_t block_exclusive_scan(int64_t v, int64_t* sh, int64_t* total) {
  const int t = threadIdx.x;
  sh[t] = v;
  __syncthreads();
  for (int st = 1; st < kNlThreads; st <<= 1) {
    const int64_t add = t >= st ? sh[t - st] : 0;
    __syncthreads();
    sh[t] += add;
    __syncthreads();
  }
  const int64_t incl = sh[t];
  *total = sh[kNlThreads - 1];
  __syncthreads();
  return incl - v;
}

__global__ void __launch_bounds__(kNlThreads) nl_scan_tile_kernel(int64_t n, const int* __restrict__ in,
                                                                    int64_t* __restrict__ out,
                                                                    int64_t* __restrict__ bsum) {
  __shared__ int64_t sh[kNlThreads];
  const int64_t t0 = (int64_t)blockIdx.x * kScanTile + (int64_t)threadIdx.x * kScanPerThread;
  int64_t s = 0;
  for (int u = 0; u < kScanPerThread; ++u)
    if (t0 + u < n) s += in[t0 + u];
  int64_t total;
  int64_t run = block_exclusive_scan(s, sh, &total);
  for (int u = 0; u < kScanPerThread; ++u)
    if (t0 + u < n) {
      out[t0 + u] = run;
      run += in[t0 + u];
    }
  if (threadIdx.x == 0) bsum[blockIdx.x] = total;
}

__global__ void __launch_bounds__(kNlThreads) nl_scan_top_kernel(int nb, int64_t* __restrict__ bsum) {
  __shared__ int64_t sh[kNlThreads];
  int64_t carry = 0;
  for (int c0 = 0; c0 < nb; c0 += kNlThreads) {
    const int idx = c0 + threadIdx.x;
    const int64_t v = idx < nb ? bsum[idx] : 0;
    int64_t total;
    const int64_t ex = block_exclusive_scan(v, sh, &total);
    if (idx < nb) bsum[idx] = carry + ex;
    carry += total;
  }
  if (threadIdx.x == 0) bsum[nb] = carry;
}

__global__ void nl_scan_add_kernel(int64_t n, int64_t* __restrict__ out, const int64_t* __restrict__ bsum,
                                   int nb) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) out[i] += bsum[i / kScanTile];
  if (i == 0) out[n] = bsum[nb];
}

void scan(hipStream_t s, int64_t n, const int* in, int64_t* out, int64_t* bsum) {
  const int nb = (int)((n + kScanTile - 1) / kScanTile);
  if (nb > 0) nl_scan_tile_kernel<<<nb, kNlThreads, 0, s>>>(n, in, out, bsum);
  nl_scan_top_kernel<<<1, kNlThreads, 0, s>>>(nb, bsum);
  const int64_t blocks = std::max<int64_t>(1, (n + kNlThreads - 1) / kNlThreads);
  nl_scan_add_kernel<<<(unsigned)blocks, kNlThreads, 0, s>>>(n, out, bsum, nb);
}

bool invert3(const double* c, double* inv) {
  const double det = c[0] * (c[4] * c[8] - c[5] * c[7]) - c[1] * (c[3] * c[8] - c[5] * c[6]) +
                     c[2] * (c[3] * c[7] - c[4] * c[6]);
  if (!(std::fabs(det) > 0) || !std::isfinite(det)) return false;
  inv[0] = (c[4] * c[8] - c[5] * c[7]) / det;
  inv[1] = (c[2] * c[7] - c[1] * c[8]) / det;
  inv[2] = (c[1] * c[5] - c[2] * c[4]) / det;
  inv[3] = (c[5] * c[6] - c[3] * c[8]) / det;
  inv[4] = (c[0] * c[8] - c[2] * c[6]) / det;
  inv[5] = (c[2] * c[3] - c[0] * c[5]) / det;
  inv[6] = (c[3] * c[7] - c[4] * c[6]) / det;
  inv[7] = (c[1] * c[6] - c[0] * c[7]) / det;
  inv[8] = (c[0] * c[4] - c[1] * c[3]) / det;
  return true;
}

// a[0 .. na) = 0, b[0 .. nb) = 0, c[0] = 0: the counters a list starts from
// (a kernel rather than memsets, so that a captured call replays correctly)
__global__ void nl_zero_kernel(int* __restrict__ a, uint32_t na, int* __restrict__ b, uint32_t nb,
                               int* __restrict__ c) {
  const uint32_t stride = gridDim.x * blockDim.x;
  for (uint32_t i = blockIdx.x * blockDim.x + threadIdx.x; i < na; i += stride) a[i] = 0;
  for (uint32_t i = blockIdx.x * blockDim.x + threadIdx.x; i < nb; i += stride) b[i] = 0;
  if (blockIdx.x == 0 && threadIdx.x == 0) c[0] = 0;
}

constexpr int64_t kMaxCandidates = int64_t(1) << 30;

// Host plan: per-graph records, candidate count, slot table size and the
// workspace layout (256-byte aligned pieces).
struct NlPlan {
  std::vector<NlGraph> gs;
  int64_t C = 0;
  uint32_t n_slots = 0;
  size_t o_gs, o_xw, o_nsh, o_cj, o_cs, o_cb, o_scnt, o_sfill, o_soff, o_order, o_rcnt, o_roff, o_bsum, o_flags,
      bytes;
};

mace_status plan_nl(int64_t N, const double* cells, const int32_t* goff, int32_t G, double r_cut, NlPlan& p) {
  if (N < 0 || N > (int64_t(1) << 30) || !(r_cut > 0) || !std::isfinite(r_cut) || G < 1) return MACE_EINVAL;
  if (!goff && G != 1) return MACE_EINVAL;
  p.gs.assign(G, NlGraph{});
  int64_t C = 0;
  for (int g = 0; g < G; ++g) {
    NlGraph& r = p.gs[g];
    std::memset(&r, 0, sizeof(r));
    r.a0 = goff ? goff[g] : 0;
    r.a1 = goff ? goff[g + 1] : (int)N;
    if (r.a0 < 0 || r.a1 < r.a0 || r.a1 > N || (g == 0 && r.a0 != 0)) return MACE_ERANGE;
    if (g > 0 && r.a0 != p.gs[g - 1].a1) return MACE_ERANGE;
    int64_t nimg = 1;
    if (cells) {
      r.periodic = 1;
      std::memcpy(r.cell, cells + 9 * g, sizeof(r.cell));
      if (!invert3(r.cell, r.inv)) return MACE_EINVAL;
      for (int a = 0; a < 3; ++a) {
        const double bn = std::sqrt(r.inv[0 * 3 + a] * r.inv[0 * 3 + a] + r.inv[1 * 3 + a] * r.inv[1 * 3 + a] +
                                    r.inv[2 * 3 + a] * r.inv[2 * 3 + a]);
        const double m = std::floor(r_cut * bn + 1.0 + 1e-6);
        if (!(m < 1e4)) return MACE_EUNSUPPORTED;
        r.nr[a] = (int)m;
        nimg *= 2 * r.nr[a] + 1;
      }
    }
    if (nimg > kMaxCandidates) return MACE_EUNSUPPORTED;
    r.nimg = (int)nimg;
    r.c0 = C;
    C += (int64_t)(r.a1 - r.a0) * nimg;
    if (C > kMaxCandidates) return MACE_EUNSUPPORTED;
  }
  if (!goff && p.gs[0].a1 != N) return MACE_ERANGE;
  if (p.gs[G - 1].a1 != N) return MACE_ERANGE;
  p.C = C;
  uint32_t ns = 1024;
  while ((int64_t)ns < 2 * C) ns <<= 1;
  p.n_slots = ns;
  size_t o = 0;
  auto take = [&](size_t bytes) {
    const size_t at = o;
    o += (bytes + 255) & ~size_t(255);
    return at;
  };
  const size_t n1 = (size_t)std::max<int64_t>(N, 1), c1 = (size_t)std::max<int64_t>(C, 1);
  p.o_gs = take(sizeof(NlGraph) * G);
  p.o_xw = take(sizeof(double) * 3 * n1);
  p.o_nsh = take(sizeof(int4) * n1);
  p.o_cj = take(sizeof(int) * c1);
  p.o_cs = take(sizeof(int4) * c1);
  p.o_cb = take(sizeof(int4) * c1);
  p.o_scnt = take(sizeof(int) * ns);
  p.o_sfill = take(sizeof(int) * ns);
  p.o_soff = take(sizeof(int64_t) * (ns + 1));
  p.o_order = take(sizeof(int) * c1);
  p.o_rcnt = take(sizeof(int) * n1);
  p.o_roff = take(sizeof(int64_t) * (n1 + 1));
  const int64_t tiles = (std::max<int64_t>(ns, n1) + kScanTile - 1) / kScanTile;
  p.o_bsum = take(sizeof(int64_t) * (tiles + 1));
  p.o_flags = take(sizeof(int));
  p.bytes = o;
  return MACE_OK;
}

}  // namespace

extern "C" size_t mace_neighbor_workspace_bytes(int64_t n_atoms, const double* cells, const int32_t* graph_offsets,
                                                int32_t n_graphs, double r_cut) {
  NlPlan p;
  if (plan_nl(n_atoms, cells, graph_offsets, n_graphs, r_cut, p) != MACE_OK) return 0;
  return p.bytes;
}

namespace {

// The list built in the device buffer w (at least p.bytes), planned by plan_nl.
mace_status nl_run(const NlPlan& p, int64_t n_atoms, const double* positions, int32_t n_graphs, double r_cut,
                   int64_t max_edges, int32_t* sender, int32_t* receiver, int32_t* shifts, int64_t* n_edges,
                   void* workspace, void* stream) {
  *n_edges = 0;
  if (n_atoms == 0) return MACE_OK;
  hipStream_t s = (hipStream_t)stream;
  char* w = reinterpret_cast<char*>(workspace);
  auto* gs = reinterpret_cast<NlGraph*>(w + p.o_gs);
  auto* xw = reinterpret_cast<double*>(w + p.o_xw);
  auto* nsh = reinterpret_cast<int4*>(w + p.o_nsh);
  auto* cj = reinterpret_cast<int*>(w + p.o_cj);
  auto* cs = reinterpret_cast<int4*>(w + p.o_cs);
  auto* cb = reinterpret_cast<int4*>(w + p.o_cb);
  auto* scnt = reinterpret_cast<int*>(w + p.o_scnt);
  auto* sfill = reinterpret_cast<int*>(w + p.o_sfill);
  auto* soff = reinterpret_cast<int64_t*>(w + p.o_soff);
  auto* order = reinterpret_cast<int*>(w + p.o_order);
  auto* rcnt = reinterpret_cast<int*>(w + p.o_rcnt);
  auto* roff = reinterpret_cast<int64_t*>(w + p.o_roff);
  auto* bsum = reinterpret_cast<int64_t*>(w + p.o_bsum);
  auto* flags = reinterpret_cast<int*>(w + p.o_flags);
  const int N = (int)n_atoms, G = n_graphs;
  const double bs = r_cut + 1e-6, rc2 = r_cut * r_cut;
  const uint32_t mask = p.n_slots - 1;
  hipError_t err = hipMemcpyAsync(gs, p.gs.data(), sizeof(NlGraph) * G, hipMemcpyHostToDevice, s);
  if (err != hipSuccess) {
    (void)hipStreamSynchronize(s);   // the plan's host copy must outlive the upload
    return MACE_EHIP;
  }
  nl_zero_kernel<<<std::min<unsigned>(1024, (p.n_slots + kNlThreads - 1) / kNlThreads), kNlThreads, 0, s>>>(
      scnt, p.n_slots, sfill, p.n_slots, flags);
  const unsigned nblk = (unsigned)((N + kNlThreads - 1) / kNlThreads);
  const unsigned cblk = (unsigned)((p.C + kNlThreads - 1) / kNlThreads);
  nl_wrap_kernel<<<nblk, kNlThreads, 0, s>>>(N, positions, gs, G, xw, nsh, flags);
  if (p.C > 0) {
    nl_cand_kernel<<<cblk, kNlThreads, 0, s>>>(p.C, gs, G, xw, bs, mask, cj, cs, cb, scnt);
  }
  scan(s, p.n_slots, scnt, soff, bsum);
  if (p.C > 0) nl_scatter_kernel<<<cblk, kNlThreads, 0, s>>>(p.C, cs, cb, mask, soff, sfill, order);
  const unsigned rblk = (unsigned)((N + kNlWaves - 1) / kNlWaves);
  nl_receiver_kernel<false><<<rblk, 64 * kNlWaves, 0, s>>>(N, positions, gs, G, xw, nsh, bs, rc2, mask, soff, order, cj,
                                                         cs, cb, rcnt, nullptr, nullptr, nullptr, nullptr);
  scan(s, N, rcnt, roff, bsum);
  int64_t total = 0;
  int hflags = 0;
  err = hipGetLastError();
  if (err == hipSuccess) err = hipMemcpyAsync(&total, roff + N, sizeof(int64_t), hipMemcpyDeviceToHost, s);
  if (err == hipSuccess) err = hipMemcpyAsync(&hflags, flags, sizeof(int), hipMemcpyDeviceToHost, s);
  const hipError_t serr = hipStreamSynchronize(s);
  if (err == hipSuccess) err = serr;
  if (err != hipSuccess) return MACE_EHIP;
  if (hflags & kFlagNonFinite) return MACE_ENONFINITE;
  if (hflags & kFlagRange) return MACE_ERANGE;
  *n_edges = total;
  if (total > max_edges) return MACE_ENOSPACE;
  if (total > 0)
    nl_receiver_kernel<true><<<rblk, 64 * kNlWaves, 0, s>>>(N, positions, gs, G, xw, nsh, bs, rc2, mask, soff, order,
                                                          cj, cs, cb, nullptr, roff, sender, receiver, shifts);
  return hipGetLastError() == hipSuccess ? MACE_OK : MACE_EHIP;
}

}  // namespace

extern "C" mace_status mace_neighbor_list_device(int64_t n_atoms, const double* positions, const double* cells,
                                                 const int32_t* graph_offsets, int32_t n_graphs, double r_cut,
                                                 int64_t max_edges, int32_t* sender, int32_t* receiver,
                                                 int32_t* shifts, int64_t* n_edges, void* workspace,
                                                 size_t workspace_bytes, void* stream) {
  if (!n_edges || (n_atoms > 0 && !positions) || max_edges < 0) return MACE_EINVAL;
  NlPlan p;
  mace_status st = plan_nl(n_atoms, cells, graph_offsets, n_graphs, r_cut, p);
  if (st != MACE_OK) return st;
  if (!workspace || workspace_bytes < p.bytes) return MACE_ENOSPACE;
  if (max_edges > 0 && (!sender || !receiver || !shifts)) return MACE_EINVAL;
  return nl_run(p, n_atoms, positions, n_graphs, r_cut, max_edges, sender, receiver, shifts, n_edges, workspace,
                stream);
}

// ---- the same list without a workspace argument: a file-scope device array
// serves as the workspace. Every GPU holds its own copy until the process
// ends; host code addresses it only through the pointer hipGetSymbolAddress
// returns for the current device (the array's name on the host is not a
// device address).
constexpr size_t kNlScratchBytes = MACE_NEIGHBOR_SCRATCH_BYTES;
static __device__ __align__(256) unsigned char scratch[kNlScratchBytes];

namespace {
constexpr int kMaxScratchDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxScratchDevices] = {};

// this device's scratch, looked up once per device
void* device_scratch() {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxScratchDevices) return nullptr;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* ptr = nullptr;
    if (hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch)) != hipSuccess || !ptr) return nullptr;
    g_scratch_ptr[dev] = ptr;
  }
  return g_scratch_ptr[dev];
}
}  // namespace

extern "C" mace_status mace_neighbor_list_device_noalloc(int64_t n_atoms, const double* positions,
                                                         const double* cells, const int32_t* graph_offsets,
                                                         int32_t n_graphs, double r_cut, int64_t max_edges,
                                                         int32_t* sender, int32_t* receiver, int32_t* shifts,
                                                         int64_t* n_edges, void* stream) {
  if (!n_edges || (n_atoms > 0 && !positions) || max_edges < 0) return MACE_EINVAL;
  NlPlan p;
  mace_status st = plan_nl(n_atoms, cells, graph_offsets, n_graphs, r_cut, p);
  if (st != MACE_OK) return st;
  if (p.bytes > kNlScratchBytes) return MACE_ENOSPACE;
  if (max_edges > 0 && (!sender || !receiver || !shifts)) return MACE_EINVAL;
  void* w = device_scratch();
  if (!w) return MACE_EHIP;
  return nl_run(p, n_atoms, positions, n_graphs, r_cut, max_edges, sender, receiver, shifts, n_edges, w, stream);
}
