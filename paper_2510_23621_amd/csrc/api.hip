// Host runtime of the MACE layer library: argument checks, model and layer
// plans, workspace carving, graph setup (CSR by receiver, sender lists,
// species tiles, image shift vectors), the host neighbour list, and the
// launch sequences of the energy forward pass and the force backward pass.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstring>
#include <map>
#include <string>
#include <tuple>
#include <vector>

#include "../../include/mace.h"
#include "mace_internal.h"
#include "so3_tables.hpp"

using namespace mace;

namespace {

struct Tensor {
  std::string name;
  std::vector<int64_t> shape;
  int64_t fan_in;
  int64_t offset;  // floats
  int64_t size() const {
    int64_t n = 1;
    for (auto d : shape) n *= d;
    return n;
  }
};

struct LayerPlan {
  int t = 0;
  bool last = false;
  std::vector<int> in_ls, out_ls;
  std::vector<so3h::Path> paths;
  int P = 0, mid = 0, din = 0, dout = 0, lh_max = 0, lout_max = 0;
  std::vector<int> path_off;
};

struct Model {
  mace_model_desc d{};
  int dh = 0;  // hidden components
  std::vector<LayerPlan> layers;
  std::vector<Tensor> tensors;
  std::map<std::string, int64_t> off;
  int64_t total = 0;       // floats of the weight blob
  int64_t comb_off = 0;    // after the blob: layer-0 path-merging x species weights [4][S][K][K]
  int l0_ki = 0;           // channels of the factorised first layer's U (64 S), 0 when S > kL0MaxSpecies
  int64_t l0_off = 0;      // after those: its weights [4][S][l0_ki][K] (transposed copy [4][S][K][l0_ki])
  int64_t total_ext = 0;   // blob + combined weights (FP32 copies only)
  int max_P = 0, max_mid = 0, max_din = 0, max_dout = 0;
};

int n_eta(int nu, int L) {
  static std::map<std::pair<int, int>, int> cache;
  auto key = std::make_pair(nu, L);
  auto it = cache.find(key);
  if (it != cache.end()) return it->second;
  int n = (int)so3h::select_trees(nu, L, (L % 2) ? -1 : 1).size();
  cache[key] = n;
  return n;
}

mace_status build_model(const mace_model_desc* desc, Model& m) {
  if (!desc) return MACE_EINVAL;
  const mace_model_desc& d = *desc;
  if (d.n_species < 1 || d.n_layers < 1 || d.n_layers > MACE_MAX_LAYERS || !(d.r_cut > 0) || !(d.c_norm > 0) ||
      d.envelope_p < 1)
    return MACE_EINVAL;
  if (d.sh_lmax != 3 || d.correlation != 3 || d.n_bessel < 1 || d.n_bessel > 16 || d.radial_hidden[0] != 64 ||
      d.radial_hidden[1] != 64 || d.radial_hidden[2] != 64 || d.readout_hidden < 1 || d.readout_hidden > 16 ||
      !(d.K == 32 || d.K == 64 || d.K == 96 || d.K == 128))
    return MACE_EUNSUPPORTED;
  // per layer 0..2, non-increasing: every output irrep of a layer after the
  // first is also an input irrep, so the residual species linear covers it
  for (int t = 0; t + 1 < d.n_layers; ++t)
    if (d.hidden_lmax[t] < 0 || d.hidden_lmax[t] > 2 || (t > 0 && d.hidden_lmax[t] > d.hidden_lmax[t - 1]))
      return MACE_EUNSUPPORTED;
  m.d = d;
  // the largest hidden feature width (components per channel) between layers
  m.dh = 1;
  for (int t = 0; t + 1 < d.n_layers; ++t) m.dh = std::max(m.dh, (d.hidden_lmax[t] + 1) * (d.hidden_lmax[t] + 1));
  const int64_t S = d.n_species, K = d.K;
  int64_t o = 0;
  auto add = [&](const std::string& name, std::vector<int64_t> shape, int64_t fan) {
    Tensor t{name, shape, fan, o};
    o += t.size();
    m.off[name] = t.offset;
    m.tensors.push_back(t);
  };
  add("embed", {S, K}, S);
  for (int t = 0; t < d.n_layers; ++t) {
    LayerPlan L;
    L.t = t;
    L.last = (t == d.n_layers - 1);
    if (t == 0) L.in_ls = {0};
    else for (int l = 0; l <= d.hidden_lmax[t - 1]; ++l) L.in_ls.push_back(l);
    if (L.last) L.out_ls = {0};
    else for (int l = 0; l <= d.hidden_lmax[t]; ++l) L.out_ls.push_back(l);
    L.lh_max = L.in_ls.back();
    L.lout_max = L.out_ls.back();
    L.paths = so3h::tp_paths(L.lh_max, d.sh_lmax);
    L.P = (int)L.paths.size();
    for (auto& p : L.paths) {
      L.path_off.push_back(L.mid);
      L.mid += 2 * p.lo + 1;
    }
    L.din = (L.lh_max + 1) * (L.lh_max + 1);
    L.dout = (L.lout_max + 1) * (L.lout_max + 1);
    std::string pre = std::to_string(t) + ".";
    for (int l : L.in_ls) add(pre + "up." + std::to_string(l), {K, K}, K);
    const int64_t h[4] = {d.n_bessel, 64, 64, 64};
    for (int i = 0; i < 3; ++i) add(pre + "radial." + std::to_string(i), {h[i], h[i + 1]}, h[i]);
    add(pre + "radial.3", {64, (int64_t)L.P * K}, 64);
    for (int p = 0; p < L.P; ++p) {
      int nin = 0;
      for (auto& q : L.paths) nin += (q.lo == L.paths[p].lo);
      add(pre + "linear." + std::to_string(p), {K, K}, nin * K);
    }
    if (t == 0) {
      for (int l = 0; l <= d.sh_lmax; ++l) add(pre + "skip." + std::to_string(l), {S, K, K}, K);
    } else {
      for (int Lo : L.out_ls)
        if (std::find(L.in_ls.begin(), L.in_ls.end(), Lo) != L.in_ls.end())
          add(pre + "skip." + std::to_string(Lo), {S, K, K}, K);
    }
    for (int Lo : L.out_ls)
      for (int nu = 1; nu <= d.correlation; ++nu) {
        int ne = n_eta(nu, Lo);
        if (ne) add(pre + "symc." + std::to_string(Lo) + "." + std::to_string(nu), {S, ne, K}, ne);
      }
    for (int Lo : L.out_ls) add(pre + "prod." + std::to_string(Lo), {K, K}, K);
    if (!L.last) {
      add(pre + "readout", {K}, K);
    } else {
      add(pre + "readout.0", {K, d.readout_hidden}, K);
      add(pre + "readout.1", {d.readout_hidden}, d.readout_hidden);
    }
    m.max_P = std::max(m.max_P, L.P);
    m.max_mid = std::max(m.max_mid, L.mid);
    m.max_din = std::max(m.max_din, L.din);
    m.max_dout = std::max(m.max_dout, L.dout);
    m.layers.push_back(L);
  }
  m.total = o;
  m.comb_off = o;
  m.l0_ki = S <= kL0MaxSpecies ? 64 * (int)S : 0;
  m.l0_off = o + 4 * S * K * K;
  m.total_ext = m.l0_off + 4 * S * (int64_t)m.l0_ki * K;
  return MACE_OK;
}

// ------------------------------------------------------------ workspace
struct Carver {
  char* base;
  size_t used = 0;
  template <class T>
  T* take(size_t count) {
    used = (used + 255) & ~size_t(255);
    T* p = base ? reinterpret_cast<T*>(base + used) : nullptr;
    used += count * sizeof(T);
    return p;
  }
};

struct Buffers {
  float *w = nullptr, *wT = nullptr, *sp_table = nullptr, *sp_round = nullptr;   // (rounded copy: precision study)
  float* w_round = nullptr;   // precision study: rounded copies of the last radial layers' weights
  unsigned short *wbf = nullptr, *wbfT = nullptr;   // 16-bit K-packed copies (BF16- / FP16-linear modes)
  int *species = nullptr, *snd = nullptr, *rcv = nullptr, *rcv_off = nullptr, *snd_off = nullptr,
      *snd_perm = nullptr, *graph_off = nullptr, *quad_node = nullptr, *quad_species = nullptr,
      *quad_node8 = nullptr, *quad_species8 = nullptr;
  double4* shift = nullptr;
  float *Y = nullptr, *rbf = nullptr;
  std::vector<float*> a3;   // per layer: [E][64] last radial hidden layer
  std::vector<unsigned short*> a3x;   // per layer: its three bfloat16 parts [E][3][64] (split-BF16 products)
  std::vector<float*> A, hin, ht;
  float *hlast = nullptr, *sc = nullptr, *At = nullptr, *Apre = nullptr, *B = nullptr;
  // backward
  float *dh0 = nullptr, *dh1 = nullptr, *dB = nullptr, *dA = nullptr, *dApre = nullptr, *dAt = nullptr,
        *dY = nullptr, *de = nullptr, *Q = nullptr, *dht = nullptr;
  float *da3p = nullptr, *dYp = nullptr;   // per-channel-tile partials [K/16][E][64], [K/16][E][16]
  float *U0 = nullptr, *gU0 = nullptr;     // factorised first layer: U and dE/dU, [N][16][l0_ki]
  int* snd_z = nullptr;                    // [E] species of each edge's sender
  float4* g = nullptr;
  double* inv_vol = nullptr;      // [G] 1/|det cell|, or 1 without cells
  int2* stress_chunks = nullptr;  // [n_stress_chunks] edge ranges of the stress reduction
  int* stress_chunk_off = nullptr;   // [G + 1] first chunk of each graph
  double* stress_part = nullptr;  // [n_stress_chunks][9] partial sums
  int* status = nullptr;          // device status word (kStatus* bits)
  LinLaunch* lin_dev = nullptr;   // 6 plans per layer + 6
};

int64_t n_tiles_bound(int64_t N, int S) { return (N + kLinTileNodes - 1) / kLinTileNodes + S; }
// every graph has at least one chunk; a graph of n edges has ceil(n / kStressChunk)
int64_t stress_chunk_bound(int64_t E, int G) { return G + E / kStressChunk + 1; }

void carve(const Model& m, int64_t N, int64_t E, int G, Carver& c, Buffers& b) {
  const int64_t K = m.d.K, S = m.d.n_species, T = m.d.n_layers;
  const int nb = m.d.n_bessel;
  b.w = c.take<float>(m.total_ext);
  b.wT = c.take<float>(m.total_ext);
  b.wbf = c.take<unsigned short>(m.total);
  b.wbfT = c.take<unsigned short>(m.total);
  b.sp_table = c.take<float>(S * K);
  b.sp_round = c.take<float>(S * K);
  b.w_round = c.take<float>(m.total_ext);
  b.species = c.take<int>(N);
  b.snd = c.take<int>(std::max<int64_t>(E, 1));
  b.rcv = c.take<int>(std::max<int64_t>(E, 1));
  b.rcv_off = c.take<int>(N + 1);
  b.snd_off = c.take<int>(N + 1);
  b.snd_perm = c.take<int>(std::max<int64_t>(E, 1));
  b.graph_off = c.take<int>(G + 1);
  const int64_t nt = n_tiles_bound(N, (int)S);   // also bounds the number of quads
  b.quad_node = c.take<int>(nt * kLinQuad * kLinTileNodes);
  b.quad_species = c.take<int>(nt);
  b.quad_node8 = c.take<int>(nt * kLinQuadWide * kLinTileNodes);
  b.quad_species8 = c.take<int>(nt);
  b.shift = c.take<double4>(std::max<int64_t>(E, 1));
  b.Y = c.take<float>(std::max<int64_t>(E, 1) * 16);
  b.rbf = c.take<float>(std::max<int64_t>(E, 1) * nb);
  b.a3.resize(T);
  b.a3x.resize(T);
  b.A.resize(T);
  b.hin.assign(T, nullptr);
  b.ht.assign(T, nullptr);
  for (int t = 0; t < T; ++t) {
    const LayerPlan& L = m.layers[t];
    b.a3[t] = c.take<float>(std::max<int64_t>(E, 1) * 64);
    b.a3x[t] = c.take<unsigned short>(std::max<int64_t>(E, 1) * 3 * 64);
    b.A[t] = c.take<float>(N * 16 * K);
    if (t > 0) {
      b.hin[t] = c.take<float>(N * L.din * K);
      b.ht[t] = c.take<float>(N * L.din * K);
    }
  }
  b.hlast = c.take<float>(N * K);
  b.sc = c.take<float>(N * m.max_dout * K);
  b.At = c.take<float>(N * m.max_mid * K);
  b.Apre = c.take<float>(N * 16 * K);
  b.B = c.take<float>(N * m.max_dout * K);
  const int64_t dmax = std::max<int64_t>(m.dh, 1);
  b.dh0 = c.take<float>(N * dmax * K);
  b.dh1 = c.take<float>(N * dmax * K);
  b.dB = c.take<float>(N * m.max_dout * K);
  b.dA = c.take<float>(N * 16 * K);
  b.dApre = c.take<float>(N * 16 * K);
  b.dAt = c.take<float>(N * m.max_mid * K);
  b.dY = c.take<float>(std::max<int64_t>(E, 1) * 16);
  b.da3p = c.take<float>((K / 16) * std::max<int64_t>(E, 1) * 64);
  b.dYp = c.take<float>((K / 16) * std::max<int64_t>(E, 1) * 16);
  b.de = c.take<float>(std::max<int64_t>(E, 1) * nb);
  b.Q = c.take<float>(std::max<int64_t>(E, 1) * m.max_din * K);
  b.dht = c.take<float>(N * m.max_din * K);
  b.g = c.take<float4>(std::max<int64_t>(E, 1));
  b.inv_vol = c.take<double>(G);
  const int64_t n_sc = stress_chunk_bound(E, G);
  b.stress_chunks = c.take<int2>(n_sc);
  b.stress_chunk_off = c.take<int>(G + 1);
  b.stress_part = c.take<double>(n_sc * 9);
  b.lin_dev = c.take<LinLaunch>(6 * T + 6);
  b.snd_z = c.take<int>(std::max<int64_t>(E, 1));
  if (m.l0_ki) {
    b.U0 = c.take<float>(N * 16 * m.l0_ki);
    b.gU0 = c.take<float>(N * 16 * m.l0_ki);
  }
  b.status = c.take<int>(64);
}

// Buffers of the FP64 debug precision (carved after the FP32 ones, for
// MACE_FP64 handles only).
struct Buffers64 {
  double* w = nullptr;                          // the weight blob in FP64
  double *Y = nullptr, *rb = nullptr;           // [E][16], [E][nb]
  std::vector<double*> z;                       // per layer 3 x [E][64]: radial pre-activations
  std::vector<double*> h;                       // h^t, t = 0..T: [N][d_t][K]
  std::vector<double*> A;                       // per layer [N][16][K]
  std::vector<double*> ht;                      // per layer: sender features W h^t [N][din][K]
  double *sc = nullptr, *At = nullptr, *Apre = nullptr, *B = nullptr;
  double *dh0 = nullptr, *dh1 = nullptr, *dB = nullptr, *dA = nullptr, *dApre = nullptr, *dAt = nullptr,
         *dht = nullptr, *dY = nullptr, *de = nullptr, *da3 = nullptr, *Q = nullptr;
  double4* g = nullptr;                         // [E] dE/dd
};

void carve64(const Model& m, int64_t N, int64_t E, Carver& c, Buffers64& b) {
  const int64_t K = m.d.K, T = m.d.n_layers, E1 = std::max<int64_t>(E, 1);
  b.w = c.take<double>(m.total);
  b.Y = c.take<double>(E1 * 16);
  b.rb = c.take<double>(E1 * m.d.n_bessel);
  b.z.assign(3 * T, nullptr);
  for (auto& z : b.z) z = c.take<double>(E1 * 64);
  b.h.assign(T + 1, nullptr);
  b.h[0] = c.take<double>(N * K);
  for (int t = 0; t < T; ++t) b.h[t + 1] = c.take<double>(N * m.layers[t].dout * K);
  b.A.assign(T, nullptr);
  for (auto& a : b.A) a = c.take<double>(N * 16 * K);
  const int64_t dmax = std::max<int64_t>(m.max_din, m.max_dout);
  b.ht.assign(T, nullptr);
  for (int t = 0; t < T; ++t) b.ht[t] = c.take<double>(N * m.layers[t].din * K);
  b.sc = c.take<double>(N * m.max_dout * K);
  b.At = c.take<double>(N * m.max_mid * K);
  b.Apre = c.take<double>(N * 16 * K);
  b.B = c.take<double>(N * m.max_dout * K);
  b.dh0 = c.take<double>(N * dmax * K);
  b.dh1 = c.take<double>(N * dmax * K);
  b.dB = c.take<double>(N * m.max_dout * K);
  b.dA = c.take<double>(N * 16 * K);
  b.dApre = c.take<double>(N * 16 * K);
  b.dAt = c.take<double>(N * m.max_mid * K);
  b.dht = c.take<double>(N * m.max_din * K);
  b.dY = c.take<double>(E1 * 16);
  b.de = c.take<double>(E1 * m.d.n_bessel);
  b.da3 = c.take<double>(E1 * 64);
  b.Q = c.take<double>(E1 * m.max_din * K);
  b.g = c.take<double4>(E1);
}

}  // namespace

enum KernelId {
  KID_EDGE_FEATURES = 0, KID_TP_FWD, KID_LINEAR, KID_SYMCON_FWD, KID_READOUT,
  KID_TP_BWD, KID_RADIAL_BWD, KID_SYMCON_BWD, KID_SENDER_SUM, KID_EDGE_BWD, KID_FORCES, KID_GRAPH_ENERGY,
  KID_L0_GATHER, KID_L0_BWD, KID_COUNT
};
const char* kKernelNames[KID_COUNT] = {
  "edge_prologue_kernel", "tpr_fwd_kernel", "linear_kernel", "symcon_fwd_kernel",
  "readout_kernel", "tpr_bwd_kernel", "radial_bwd_kernel", "symcon_bwd_kernel", "sender_sum_kernel",
  "edge_vjp_kernel", "forces_kernel", "graph_energy_kernel", "l0_gather_kernel",
  "l0_edge_bwd_kernel"};
constexpr int kProfPairs = 4096;

struct mace_graph {
  // profiling: events around every launch of one kernel class
  int prof_kernel = -1;
  std::vector<hipEvent_t> prof_ev;   // 2 * kProfPairs
  int prof_used = 0;
  int64_t prof_dropped = 0;
  double prof_flops = 0.0, prof_bytes = 0.0;   // algorithmic work of the profiled launches
  Model m;
  Buffers b;
  Buffers64 b64;   // MACE_FP64 handles only
  int64_t N = 0, E = 0;
  int G = 1;
  int n_tiles = 0, n_quads = 0;
  int n_quads8 = 0;   // blocks of the kLinQuadWide grouping (16-bit modes, large graphs), 0: not used
  int n_stress_chunks = 0;
  mace_precision prec = MACE_FP32;
  // linear plans per layer (host copy for the grid, device copy for the kernel)
  std::vector<LinPlanRef> upskip, upskipT, lin, linT, prod, prodT;
  LinPlanRef skip0, skip0T, comb0, comb0T;
  // first layer in factorised form: U -> A (FP32; composed with the
  // path-merging and species linears) or U -> At (16-bit modes), and transposes
  LinPlanRef l0f, l0fT;
  bool l0_fact = false;
  bool radial_split = true;   // FP32 last radial layer on split-BF16 MFMA (mace_fp32_products)
  // precision study: operand rounding of the edge product / contraction / radial MLP
  int tp_round = 0, sc_round = 0, rad_round = 0;
  bool l0_chain = true;     // 16-bit modes: the first layer's linears fused (mace_debug_fused_linears bit 0)
  bool wide_tiles = true;   // 16-bit modes, large graphs: eight node tiles per wide linear block (bit 1)
};

namespace {

struct ProfScope {
  mace_graph* h;
  hipStream_t s;
  bool on;
  int slot;
  ProfScope(mace_graph* h_, int kid, hipStream_t s_) : h(h_), s(s_), on(false), slot(0) {
    if (h->prof_kernel != kid) return;
    if (h->prof_used >= kProfPairs) {
      h->prof_dropped++;
      return;
    }
    slot = h->prof_used++;
    on = true;
    hipEventRecord(h->prof_ev[2 * slot], s);
  }
  ~ProfScope() {
    if (on) hipEventRecord(h->prof_ev[2 * slot + 1], s);
  }
};
#define PROF(kid) ProfScope _prof_##__LINE__(h, kid, s)

// The first layer runs in factorised form where it has fewer multiply-adds:
// per node 16 x 64 S x K (U to the message) against per edge 64 x P K (the
// last radial layer), i.e. when the mean degree exceeds about 4 S (with a
// margin for the per-edge passes of both forms).
bool l0_auto(const Model& m, int64_t N, int64_t E) {
  return m.l0_ki > 0 && E >= 3 * (int64_t)m.d.n_species * N;
}

// The edge products of layer t run their last radial layer on split-BF16
// operands, and both read a3 as the three parts the prologue writes (radial
// mode 3; the edge-lane backwards, l_h = 1 and 2), or split it per tile (2).
bool layer_factorised(const mace_graph* h, int t) {
  return t == 0 && h->l0_fact && !h->tp_round && !h->rad_round;
}
bool a3_presplit(const mace_graph* h, int t) {
  return h->radial_split && h->prec != MACE_BF16_RADIAL && h->m.layers[t].lh_max >= 1 && !layer_factorised(h, t);
}
int radial_mode(const mace_graph* h, int t) {
  return h->prec == MACE_BF16_RADIAL ? 1 : (!h->radial_split ? 0 : (a3_presplit(h, t) ? 3 : 2));
}

// Every edge product the handle's settings will launch has a kernel instance
// (checked before anything is enqueued; the launchers check again).
bool launchable(const mace_graph* h) {
  for (int t = 0; t < h->m.d.n_layers; ++t)
    if (!layer_factorised(h, t) && !tpr_supported(h->m.layers[t].lh_max, radial_mode(h, t))) return false;
  return true;
}

// A linear launch, bracketed for profiling; while the linear class is
// selected its algorithmic work is summed too.
void run_linear(mace_graph* h, hipStream_t s, const LinPlanRef& P, const LinArgs& a) {
  ProfScope ps(h, KID_LINEAR, s);
  if (ps.on && a.n_quads > 0 && P.host.plan.n_groups > 0) {
    double f = 0.0, b = 0.0;
    linear_work(P.host.plan, a, h->N, h->m.d.n_species, &f, &b);
    h->prof_flops += f;
    h->prof_bytes += b;
  }
  launch_linear(s, P, a);
}

mace_status hip_ok(hipError_t e) { return e == hipSuccess ? MACE_OK : MACE_EHIP; }

// rounding mode of the channel-mixing linears: 0 FP32, 1 bfloat16, 2 binary16
int lowp_mode(mace_precision p) {
  return (p == MACE_BF16_LINEAR || p == MACE_BF16_RADIAL) ? 1 : (p == MACE_FP16_LINEAR ? 2 : 0);
}

// The 16-bit modes' factorised first layer runs its three linears (the FP32
// contraction, then the 16-bit path-merging and species linears; backward,
// their transposes) as one launch each way where the shapes allow it:
// K = 128, a 128-wide contraction (two species) and plans of one term per l
// whose input component is the output component.
bool chain_stage_of(const LinPlanRef& P, int lowp, ChainStage* cs) {
  const LinPlan& p = P.host.plan;
  if (p.n_groups != 4 || p.cin != 16 || p.cout != 16) return false;
  int species = -1;
  for (int gi = 0; gi < 4; ++gi) {
    const LinGroup& G = p.g[gi];
    if (G.out_c0 != gi * gi || G.ncomp != 2 * gi + 1 || G.t1 - G.t0 != 1 || G.dst) return false;
    const LinTerm& t = p.t[G.t0];
    if (t.in_c0 != G.out_c0 || t.src) return false;
    if (species >= 0 && species != t.species) return false;
    species = t.species;
    cs->w_off[gi] = t.w_off;
  }
  cs->w_sstride = species ? p.w_sstride : 0;
  cs->lowp = lowp;
  return true;
}

bool run_l0_chain(mace_graph* h, hipStream_t s, bool backward) {
  const Model& m = h->m;
  const int lowp = lowp_mode(h->prec);
  if (!h->l0_chain || !lowp || m.d.K != 128 || m.l0_ki != 128 || m.layers[0].mid != 16) return false;
  Buffers& b = h->b;
  ChainArgs a;
  const LinPlanRef* P[3];
  if (!backward) {
    a.x = b.U0;
    a.y = b.A[0];
    a.wt = b.wT;
    a.wbf = b.wbf;
    P[0] = &h->l0f;
    P[1] = &h->lin[0];
    P[2] = &h->skip0;
  } else {
    a.x = b.dA;
    a.y = b.gU0;
    a.wt = b.w;
    a.wbf = b.wbfT;
    P[0] = &h->skip0T;
    P[1] = &h->linT[0];
    P[2] = &h->l0fT;
  }
  const int fp32_stage = backward ? 2 : 0;
  for (int q = 0; q < 3; ++q)
    if (!chain_stage_of(*P[q], q == fp32_stage ? 0 : lowp, &a.st[q])) return false;
  const bool eight = h->wide_tiles && h->n_quads8 > 0;
  a.n_quads = h->n_quads;
  a.n_quads8 = eight ? h->n_quads8 : 0;
  a.quad_node = eight ? b.quad_node8 : b.quad_node;
  a.quad_species = eight ? b.quad_species8 : b.quad_species;
  a.lowp = lowp;
  ProfScope ps(h, KID_LINEAR, s);
  if (ps.on && a.n_quads > 0) {
    // algorithmic work: three K x K products per node and component; the
    // input and output rows once, and each stage's weight blocks
    const double K = m.d.K, N = (double)h->N, S = m.d.n_species;
    h->prof_flops += 3.0 * 2.0 * K * K * N * 16.0;
    double wb = 0.0;
    for (int q = 0; q < 3; ++q) wb += 4.0 * K * K * (a.st[q].lowp ? 2.0 : 4.0) * (a.st[q].w_sstride ? S : 1.0);
    h->prof_bytes += 2.0 * N * 16.0 * K * 4.0 + wb;
  }
  launch_linear_chain3(s, a);
  return true;
}

LinPlan plan_single_per_l(const std::vector<int>& ls, const std::string& pre, const Model& m, int cin, int cout,
                          bool species) {
  LinPlan p;
  p.cin = cin;
  p.cout = cout;
  p.w_sstride = (int64_t)m.d.K * m.d.K;
  for (int l : ls) {
    LinGroup g{l * l, 2 * l + 1, p.n_terms, p.n_terms + 1, 0};
    p.t[p.n_terms++] = LinTerm{l * l, 0, species ? 1 : 0, m.off.at(pre + std::to_string(l))};
    p.g[p.n_groups++] = g;
  }
  return p;
}

void make_plans(mace_graph* h) {
  const Model& m = h->m;
  const int T = m.d.n_layers;
  h->upskip.resize(T); h->upskipT.resize(T); h->lin.resize(T); h->linT.resize(T);
  h->prod.resize(T); h->prodT.resize(T);
  const int64_t KK = (int64_t)m.d.K * m.d.K;
  for (int t = 0; t < T; ++t) {
    const LayerPlan& L = m.layers[t];
    const std::string pre = std::to_string(t) + ".";
    std::vector<int> both;   // l in the layer's input and output irreps: residual species linear
    for (int Lo : L.out_ls)
      if (std::find(L.in_ls.begin(), L.in_ls.end(), Lo) != L.in_ls.end()) both.push_back(Lo);
    // forward, t >= 1: linear_up (hin -> ht) and the residual species linear
    // (hin -> sc) read the same input: one launch, two outputs
    {
      LinPlan p;
      p.cin = L.din;
      p.cout = L.din;
      p.cout2 = L.dout;
      p.w_sstride = KK;
      for (int l : L.in_ls) {
        p.g[p.n_groups++] = LinGroup{l * l, 2 * l + 1, p.n_terms, p.n_terms + 1, 0};
        p.t[p.n_terms++] = LinTerm{l * l, 0, 0, m.off.at(pre + "up." + std::to_string(l))};
      }
      if (t > 0)
        for (int l : both) {
          p.g[p.n_groups++] = LinGroup{l * l, 2 * l + 1, p.n_terms, p.n_terms + 1, 1};
          p.t[p.n_terms++] = LinTerm{l * l, 0, 1, m.off.at(pre + "skip." + std::to_string(l))};
        }
      h->upskip[t].host = make_lin_launch(p);
    }
    // backward, t >= 1: dh^t = dE/dht upT + dE/dsc skipT, one output, two inputs
    {
      LinPlan p;
      p.cin = L.din;    // x = dE/dht
      p.cin2 = L.dout;  // x2 = dE/dsc (the gradient of this layer's output)
      p.cout = L.din;
      p.w_sstride = KK;
      for (int l : L.in_ls) {
        const int t0 = p.n_terms;
        p.t[p.n_terms++] = LinTerm{l * l, 0, 0, m.off.at(pre + "up." + std::to_string(l))};
        if (t > 0 && std::find(both.begin(), both.end(), l) != both.end())
          p.t[p.n_terms++] = LinTerm{l * l, 1, 1, m.off.at(pre + "skip." + std::to_string(l))};
        p.g[p.n_groups++] = LinGroup{l * l, 2 * l + 1, t0, p.n_terms, 0};
      }
      h->upskipT[t].host = make_lin_launch(p);
    }
    // path-merging linear: output l collects every path with l_out = l
    LinPlan lp;
    lp.cin = L.mid;
    lp.cout = 16;
    for (int l = 0; l <= 3; ++l) {
      LinGroup g{l * l, 2 * l + 1, lp.n_terms, lp.n_terms, 0};
      for (int p = 0; p < L.P; ++p)
        if (L.paths[p].lo == l)
          lp.t[lp.n_terms++] = LinTerm{L.path_off[p], 0, 0, m.off.at(pre + "linear." + std::to_string(p))};
      g.t1 = lp.n_terms;
      lp.g[lp.n_groups++] = g;
    }
    h->lin[t].host = make_lin_launch(lp);
    LinPlan lt;
    lt.cin = 16;
    lt.cout = L.mid;
    for (int p = 0; p < L.P; ++p) {
      int lo = L.paths[p].lo;
      lt.g[lt.n_groups++] = LinGroup{L.path_off[p], 2 * lo + 1, lt.n_terms, lt.n_terms + 1, 0};
      lt.t[lt.n_terms++] = LinTerm{lo * lo, 0, 0, m.off.at(pre + "linear." + std::to_string(p))};
    }
    h->linT[t].host = make_lin_launch(lt);
    h->prod[t].host = make_lin_launch(plan_single_per_l(L.out_ls, pre + "prod.", m, L.dout, L.dout, false));
    h->prodT[t] = h->prod[t];
  }
  h->skip0.host = make_lin_launch(plan_single_per_l({0, 1, 2, 3}, "0.skip.", m, 16, 16, true));
  h->skip0T = h->skip0;
  // FP32: layer 0's path-merging linear followed by its species linear is one
  // species linear with the product weights (one path per l_out at layer 0)
  {
    LinPlan p;
    p.cin = m.layers[0].mid;
    p.cout = 16;
    p.w_sstride = KK;
    for (int l = 0; l <= 3; ++l) {
      p.g[p.n_groups++] = LinGroup{l * l, 2 * l + 1, p.n_terms, p.n_terms + 1, 0};
      p.t[p.n_terms++] = LinTerm{l * l, 0, 1, m.comb_off + (int64_t)l * m.d.n_species * KK};
    }
    h->comb0.host = make_lin_launch(p);
    p.cin = 16;
    p.cout = m.layers[0].mid;
    h->comb0T.host = make_lin_launch(p);
  }
  // factorised first layer: one term per l on components l^2 .. l^2 + 2l; the
  // weights depend on the receiver's species where they include its species linear
  if (m.l0_ki) {
    const bool composed = lowp_mode(h->prec) == 0;
    LinPlan p;
    p.cin = 16;
    p.cout = 16;
    p.w_sstride = (int64_t)m.l0_ki * m.d.K;
    for (int l = 0; l <= 3; ++l) {
      p.g[p.n_groups++] = LinGroup{l * l, 2 * l + 1, p.n_terms, p.n_terms + 1, 0};
      p.t[p.n_terms++] = LinTerm{l * l, 0, composed ? 1 : 0, m.l0_off + (int64_t)l * m.d.n_species * p.w_sstride};
    }
    h->l0f.host = make_lin_launch(p);
    h->l0fT = h->l0f;
  }
}

// copy every plan to the device buffer carved for them; the kernels read it there
hipError_t upload_plans(mace_graph* h, hipStream_t s) {
  const int T = h->m.d.n_layers;
  std::vector<LinPlanRef*> refs;
  for (int t = 0; t < T; ++t)
    for (auto* v : {&h->upskip, &h->upskipT, &h->lin, &h->linT, &h->prod, &h->prodT})
      refs.push_back(&(*v)[t]);
  for (auto* r : {&h->skip0, &h->skip0T, &h->comb0, &h->comb0T, &h->l0f, &h->l0fT}) refs.push_back(r);
  std::vector<LinLaunch> host(refs.size());
  for (size_t q = 0; q < refs.size(); ++q) {
    host[q] = refs[q]->host;
    refs[q]->dev = h->b.lin_dev + q;
  }
  hipError_t e = hipMemcpyAsync(h->b.lin_dev, host.data(), host.size() * sizeof(LinLaunch), hipMemcpyHostToDevice, s);
  if (e != hipSuccess) return e;
  return hipStreamSynchronize(s);
}

LinArgs largs(mace_graph* h, const float* x, float* y, const float* residual, bool transposed, int accumulate,
              const float* x2 = nullptr, float* y2 = nullptr) {
  LinArgs a;
  a.x = x;
  a.y = y;
  a.x2 = x2;
  a.y2 = y2;
  a.residual = residual;
  a.w = transposed ? h->b.wT : h->b.w;
  a.wt = transposed ? h->b.w : h->b.wT;
  a.wbf = transposed ? h->b.wbfT : h->b.wbf;
  a.quad_node = h->b.quad_node;
  a.quad_species = h->b.quad_species;
  a.n_quads = h->n_quads;
  a.quad_node8 = h->b.quad_node8;
  a.quad_species8 = h->b.quad_species8;
  a.n_quads8 = h->wide_tiles ? h->n_quads8 : 0;
  a.K = h->m.d.K;
  a.KI = 0;
  a.accumulate = accumulate;
  a.lowp = lowp_mode(h->prec);
  a.bias0 = nullptr;
  return a;
}

// the factorised first layer's contraction (FP32 in every mode): U (l0_ki
// channels) -> K channels, or its transpose
LinArgs largs_l0(mace_graph* h, const float* x, float* y, bool transposed) {
  LinArgs a = largs(h, x, y, nullptr, transposed, 0);
  a.lowp = 0;
  a.K = transposed ? h->m.l0_ki : h->m.d.K;
  a.KI = transposed ? h->m.d.K : h->m.l0_ki;
  return a;
}

SymW symw(mace_graph* h, int t) {
  SymW w;
  std::memset(&w, 0, sizeof(w));
  const LayerPlan& L = h->m.layers[t];
  for (int Lo : L.out_ls)
    for (int nu = 1; nu <= 3; ++nu) {
      auto it = h->m.off.find(std::to_string(t) + ".symc." + std::to_string(Lo) + "." + std::to_string(nu));
      if (it != h->m.off.end()) w.w[Lo][nu] = h->b.w + it->second;
    }
  return w;
}

// Forward pass; keeps every intermediate the backward pass reads.
// seed_grad: the last layer's readout also stores the backward pass's
// starting gradient (dE/dh of the last layer's output, in b.dh0).
void run_forward(mace_graph* h, hipStream_t s, const float* pos, float* eps, bool seed_grad) {
  const Model& m = h->m;
  Buffers& b = h->b;
  const int N = (int)h->N, E = (int)h->E, K = m.d.K;
  const int lowp = lowp_mode(h->prec);
  {
    PROF(KID_EDGE_FEATURES);
    // geometry and the radial hidden layers of every interaction layer, in
    // launches of up to kMaxRadialLayers layers
    for (int t0 = 0; t0 < m.d.n_layers; t0 += kMaxRadialLayers) {
      RadialSet rs;
      rs.n = std::min(kMaxRadialLayers, m.d.n_layers - t0);
      rs.rnd = h->rad_round;
      for (int q = 0; q < rs.n; ++q) {
        rs.W[q] = b.w + m.off.at(std::to_string(t0 + q) + ".radial.0");
        rs.a3[q] = b.a3[t0 + q];
        rs.a3x[q] = a3_presplit(h, t0 + q) ? b.a3x[t0 + q] : nullptr;
      }
      // (a later chunk recomputes the same Y and rbf)
      launch_edge_prologue(s, E, pos, b.snd, b.rcv, b.shift, m.d.r_cut, m.d.envelope_p, m.d.n_bessel, b.Y, b.rbf,
                           rs, b.status);
    }
  }
  if (h->rad_round) {
    // precision study: the last radial layer (inside the edge products) reads rounded weights
    for (int t = 0; t < m.d.n_layers; ++t) {
      const int64_t o = m.off.at(std::to_string(t) + ".radial.3");
      launch_round(s, b.w_round + o, b.w + o, (size_t)64 * m.layers[t].P * K, h->rad_round);
    }
  }
  const float* wr3 = h->rad_round ? b.w_round : b.w;
  if (h->tp_round) {
    // precision study: the edge products read rounded harmonics and sender features
    launch_round(s, b.Y, b.Y, (size_t)E * 16, h->tp_round);
    launch_round(s, b.sp_round, b.sp_table, (size_t)m.d.n_species * K, h->tp_round);
  }
  const float inv_c = (float)(1.0 / m.d.c_norm);
  ReadoutLin ro{};   // linear readouts not yet evaluated
  int ro_acc = 0;     // eps already holds earlier readouts
  for (int t = 0; t < m.d.n_layers; ++t) {
    const LayerPlan& L = m.layers[t];
    const std::string pre = std::to_string(t) + ".";
    if (layer_factorised(h, t)) {
      // factorised first layer: U per receiver, then one contraction (FP32
      // mode: straight to A; 16-bit modes: to At, then their own linears)
      {
        PROF(KID_L0_GATHER);
        launch_l0_gather(s, N, m.d.n_species, b.rcv_off, b.snd_z, b.a3[0], b.Y, h->prec == MACE_BF16_RADIAL, b.U0);
      }
      if (!lowp) {
        run_linear(h, s, h->l0f, largs_l0(h, b.U0, b.A[0], false));
      } else if (!run_l0_chain(h, s, false)) {
        run_linear(h, s, h->l0f, largs_l0(h, b.U0, b.At, false));
        run_linear(h, s, h->lin[0], largs(h, b.At, b.Apre, nullptr, false, 0));
        run_linear(h, s, h->skip0, largs(h, b.Apre, b.A[0], nullptr, false, 0));
      }
    } else {
      // edge product with the sender features: the species table at layer 0,
      // linear_up of h^t (with the residual species linear) after it
      const float* src = h->tp_round ? b.sp_round : b.sp_table;
      const int* src_map = b.species;
      if (t > 0) {
        run_linear(h, s, h->upskip[t], largs(h, b.hin[t], b.ht[t], nullptr, false, 0, nullptr, b.sc));
        launch_round(s, b.ht[t], b.ht[t], (size_t)N * L.din * K, h->tp_round);
        src = b.ht[t];
        src_map = nullptr;
      }
      {
        PROF(KID_TP_FWD);
        const float* a3t = a3_presplit(h, t) ? reinterpret_cast<const float*>(b.a3x[t]) : b.a3[t];
        (void)launch_tpr_fwd(s, L.lh_max, N, K, b.rcv_off, b.snd, src_map, a3t, wr3 + m.off.at(pre + "radial.3"),
                       b.Y, src, inv_c, b.At, radial_mode(h, t), h->tp_round);
      }
      if (t == 0 && !lowp) {
        run_linear(h, s, h->comb0, largs(h, b.At, b.A[t], nullptr, false, 0));
      } else if (t == 0) {   // 16-bit linears: each linear rounds its own inputs and weights
        run_linear(h, s, h->lin[t], largs(h, b.At, b.Apre, nullptr, false, 0));
        run_linear(h, s, h->skip0, largs(h, b.Apre, b.A[t], nullptr, false, 0));
      } else {
        run_linear(h, s, h->lin[t], largs(h, b.At, b.A[t], nullptr, false, 0));
      }
    }
    {
      PROF(KID_SYMCON_FWD);
      launch_symcon_fwd(s, L.lout_max, N, K, b.species, b.A[t], symw(h, t), b.B, h->sc_round);
    }
    float* hout = L.last ? b.hlast : b.hin[t + 1];
    {
      run_linear(h, s, h->prod[t], largs(h, b.B, hout, t > 0 ? b.sc : nullptr, false, 0));
    }
    if (!L.last) {
      // evaluated with the last layer's readout (or earlier, kMaxReadoutLin at a time)
      if (ro.n == kMaxReadoutLin) {
        PROF(KID_READOUT);
        launch_readout_fwd(s, N, K, ro, nullptr, 0, nullptr, nullptr, 0, lowp, ro_acc, eps, nullptr);
        ro_acc = 1;
        ro.n = 0;
      }
      ro.h[ro.n] = hout;
      ro.w[ro.n] = b.w + m.off.at(pre + "readout");
      ro.stride[ro.n] = L.dout * K;
      ++ro.n;
    } else {
      PROF(KID_READOUT);
      launch_readout_fwd(s, N, K, ro, hout, L.dout * K, b.w + m.off.at(pre + "readout.0"),
                         b.w + m.off.at(pre + "readout.1"), m.d.readout_hidden, lowp, ro_acc, eps,
                         seed_grad ? b.dh0 : nullptr);
    }
  }
}

// Ends with the forces F and, in the same launch, the per-graph energies
// graph_e of the node energies eps.
void run_backward(mace_graph* h, hipStream_t s, const float* pos, float* F, const float* eps, double* graph_e) {
  const Model& m = h->m;
  Buffers& b = h->b;
  const int N = (int)h->N, E = (int)h->E, K = m.d.K, T = m.d.n_layers;
  const int lowp = lowp_mode(h->prec);
  const float inv_c = (float)(1.0 / m.d.c_norm);
  float* dnext = b.dh0;
  float* dprev = b.dh1;
  for (int t = T - 1; t >= 0; --t) {
    const LayerPlan& L = m.layers[t];
    const std::string pre = std::to_string(t) + ".";
    float* hout = L.last ? b.hlast : b.hin[t + 1];
    // dnext already holds dE/d(output of layer t): for the last layer (one
    // scalar component) its forward readout stored it; for a layer below the
    // last, the transposed linear that wrote dnext added that layer's readout
    // gradient (the readout weights) in its epilogue.
    {
      run_linear(h, s, h->prodT[t], largs(h, dnext, b.dB, nullptr, true, 0));
    }
    {
      PROF(KID_SYMCON_BWD);
      launch_symcon_bwd(s, L.lout_max, N, K, b.species, b.A[t], symw(h, t), b.dB, b.dA, h->sc_round);
    }
    const bool fact = layer_factorised(h, t);
    // dE/dAt (the transposes of the linears after the edge product); the
    // factorised first layer ends in dE/dU instead
    const float* dApre = b.dA;
    const bool chained = fact && lowp && run_l0_chain(h, s, true);   // dE/dA -> dE/dU in one launch
    if (t == 0 && lowp && !chained) {   // 16-bit modes: each linear's own transpose
      run_linear(h, s, h->skip0T, largs(h, b.dA, b.dApre, nullptr, true, 0));
      dApre = b.dApre;
    }
    if (!chained) {
      if (fact && !lowp) {
        run_linear(h, s, h->l0fT, largs_l0(h, b.dA, b.gU0, true));
      } else if (t == 0 && !lowp) {
        run_linear(h, s, h->comb0T, largs(h, b.dA, b.dAt, nullptr, true, 0));
      } else {
        run_linear(h, s, h->linT[t], largs(h, dApre, b.dAt, nullptr, true, 0));
        if (fact) run_linear(h, s, h->l0fT, largs_l0(h, b.dAt, b.gU0, true));
      }
    }
    int n_part = K / 16;
    if (fact) {
      // dE/da3 and dE/dY per edge, whole (one partial each)
      PROF(KID_L0_BWD);
      launch_l0_edge_bwd(s, N, m.d.n_species, b.rcv_off, b.snd_z, b.a3[0], b.Y, b.gU0, h->prec == MACE_BF16_RADIAL,
                         b.da3p, b.dYp);
      n_part = 1;
    } else {
      const float* src = t == 0 ? (h->tp_round ? b.sp_round : b.sp_table) : b.ht[t];
      const int* src_map = t == 0 ? b.species : nullptr;
      PROF(KID_TP_BWD);
      (void)launch_tpr_bwd(s, L.lh_max, N, K, E, b.rcv_off, b.snd, src_map,
                     a3_presplit(h, t) ? reinterpret_cast<const float*>(b.a3x[t]) : b.a3[t],
                     (h->rad_round ? b.w_round : b.w) + m.off.at(pre + "radial.3"),
                     b.Y, src, inv_c, b.dAt, b.dYp, t > 0 ? b.Q : nullptr, b.da3p, radial_mode(h, t), h->tp_round);
    }
    // The edge backward wrote Q and the partials (about 390 MB at K = 128,
    // more than the last-level cache holds); the sender sum reads Q first
    // (measured faster than the radial backward first).
    if (t > 0) {
      PROF(KID_SENDER_SUM);
      launch_sender_sum(s, N, L.din, K, b.snd_off, b.snd_perm, b.Q, b.dht);
    }
    {
      PROF(KID_RADIAL_BWD);
      launch_radial_bwd(s, E, b.rbf, m.d.n_bessel, b.w + m.off.at(pre + "radial.0"), b.da3p, b.dYp, n_part,
                        b.dY, b.de, t < T - 1, h->rad_round);
    }
    if (t > 0) {
      {
        LinArgs la = largs(h, b.dht, dprev, nullptr, true, 0, dnext);
        la.bias0 = b.w + m.off.at(std::to_string(t - 1) + ".readout");   // layer t - 1 is not the last
        run_linear(h, s, h->upskipT[t], la);
      }
      std::swap(dnext, dprev);
    }
  }
  {
    PROF(KID_EDGE_BWD);
    launch_edge_vjp(s, E, pos, b.snd, b.rcv, b.shift, m.d.r_cut, m.d.envelope_p, m.d.n_bessel, b.dY, b.de, b.g);
  }
  {
    PROF(KID_FORCES);
    launch_forces(s, N, b.rcv_off, b.snd_off, b.snd_perm, b.g, F, h->G, b.graph_off, eps, graph_e);
  }
}

// ---------------------------------------------------------------- FP64 debug precision
// The same model in FP64 on simple kernels (k_fp64.hip), every layer in
// per-edge form; positions, node energies and forces are FP64.

// a linear of blocks of components (see Lin64); spec for the species-dependent ones
struct Lin64Builder {
  Lin64 L;
  Lin64Builder(int cin, int cout, bool transpose) {
    std::memset(&L, 0, sizeof(L));
    L.cin = cin;
    L.cout = cout;
    L.transpose = transpose;
  }
  Lin64Builder& add(int cx, int cy, int nc, int64_t woff, bool spec) {
    const int t = L.n_terms++;
    L.cx[t] = cx;
    L.cy[t] = cy;
    L.nc[t] = nc;
    L.woff[t] = woff;
    L.spec[t] = spec;
    return *this;
  }
};

SymW64 symw64(const mace_graph* h, int t) {
  SymW64 w;
  std::memset(&w, 0, sizeof(w));
  for (int Lo : h->m.layers[t].out_ls)
    for (int nu = 1; nu <= 3; ++nu) {
      auto it = h->m.off.find(std::to_string(t) + ".symc." + std::to_string(Lo) + "." + std::to_string(nu));
      if (it != h->m.off.end()) w.w[Lo][nu] = h->b64.w + it->second;
    }
  return w;
}

bool f64_supported(const mace_graph* h) {
  if (h->m.d.n_layers > 8 || h->m.d.n_bessel > 16) return false;
  for (const LayerPlan& L : h->m.layers)
    if (L.lh_max > 2 || L.lout_max > 2 || (int)L.paths.size() > kMaxLin64Terms) return false;
  return true;
}

void run_forward64(mace_graph* h, hipStream_t s, const double* pos, double* eps, bool seed_grad) {
  const Model& m = h->m;
  Buffers& b = h->b;
  Buffers64& d = h->b64;
  const int N = (int)h->N, E = (int)h->E, K = m.d.K, nb = m.d.n_bessel;
  const double* W = d.w;
  f64_geom(s, E, pos, b.snd, b.rcv, b.shift, m.d.r_cut, m.d.envelope_p, nb, d.Y, d.rb, b.status);
  f64_embed(s, N, K, b.species, W + m.off.at("embed"), d.h[0]);
  const double inv_c = 1.0 / m.d.c_norm;
  for (int t = 0; t < m.d.n_layers; ++t) {
    const LayerPlan& L = m.layers[t];
    const std::string pre = std::to_string(t) + ".";
    double** z = d.z.data() + 3 * t;
    f64_radial_fwd(s, E, nb, d.rb, W + m.off.at(pre + "radial.0"), W + m.off.at(pre + "radial.1"),
                   W + m.off.at(pre + "radial.2"), z[0], z[1], z[2]);
    // linear_up, and the residual species linear of the layers above the first
    Lin64Builder up(L.din, L.din, false);
    for (int l : L.in_ls) up.add(l * l, l * l, 2 * l + 1, m.off.at(pre + "up." + std::to_string(l)), false);
    f64_linear(s, N, K, up.L, b.species, W, d.h[t], d.ht[t], nullptr);
    const double* sc = nullptr;
    if (t > 0) {
      Lin64Builder sk(L.din, L.dout, false);
      for (int Lo : L.out_ls)
        if (std::find(L.in_ls.begin(), L.in_ls.end(), Lo) != L.in_ls.end())
          sk.add(Lo * Lo, Lo * Lo, 2 * Lo + 1, m.off.at(pre + "skip." + std::to_string(Lo)), true);
      f64_linear(s, N, K, sk.L, b.species, W, d.h[t], d.sc, nullptr);
      sc = d.sc;
    }
    f64_tp_fwd(s, L.lh_max, N, K, b.rcv_off, b.snd, z[2], W + m.off.at(pre + "radial.3"), d.Y, d.ht[t], inv_c,
               d.At);
    // path-merging linear (at the first layer followed by the species linear)
    Lin64Builder lin(L.mid, 16, false);
    for (int q = 0; q < L.P; ++q) {
      const int lo = L.paths[q].lo;
      lin.add(L.path_off[q], lo * lo, 2 * lo + 1, m.off.at(pre + "linear." + std::to_string(q)), false);
    }
    if (t == 0) {
      f64_linear(s, N, K, lin.L, b.species, W, d.At, d.Apre, nullptr);
      Lin64Builder sk0(16, 16, false);
      for (int l = 0; l <= 3; ++l) sk0.add(l * l, l * l, 2 * l + 1, m.off.at(pre + "skip." + std::to_string(l)), true);
      f64_linear(s, N, K, sk0.L, b.species, W, d.Apre, d.A[t], nullptr);
    } else {
      f64_linear(s, N, K, lin.L, b.species, W, d.At, d.A[t], nullptr);
    }
    f64_symcon_fwd(s, L.lout_max, N, K, b.species, d.A[t], symw64(h, t), d.B);
    Lin64Builder prod(L.dout, L.dout, false);
    for (int Lo : L.out_ls) prod.add(Lo * Lo, Lo * Lo, 2 * Lo + 1, m.off.at(pre + "prod." + std::to_string(Lo)), false);
    f64_linear(s, N, K, prod.L, b.species, W, d.B, d.h[t + 1], sc);
    if (!L.last)
      f64_readout(s, N, K, d.h[t + 1], L.dout * K, W + m.off.at(pre + "readout"), nullptr, 0, eps, t > 0, nullptr);
    else
      f64_readout(s, N, K, d.h[t + 1], L.dout * K, W + m.off.at(pre + "readout.0"), W + m.off.at(pre + "readout.1"),
                  m.d.readout_hidden, eps, t > 0, seed_grad ? d.dh0 : nullptr);
  }
}

void run_backward64(mace_graph* h, hipStream_t s, const double* pos, double* F) {
  const Model& m = h->m;
  Buffers& b = h->b;
  Buffers64& d = h->b64;
  const int N = (int)h->N, E = (int)h->E, K = m.d.K, nb = m.d.n_bessel, T = m.d.n_layers;
  const double* W = d.w;
  const double inv_c = 1.0 / m.d.c_norm;
  double* dnext = d.dh0;   // dE/dh^{t+1}; the last readout seeded it
  double* dprev = d.dh1;
  for (int t = T - 1; t >= 0; --t) {
    const LayerPlan& L = m.layers[t];
    const std::string pre = std::to_string(t) + ".";
    double** z = d.z.data() + 3 * t;
    if (!L.last) f64_add_readout_grad(s, N, K, L.dout * K, W + m.off.at(pre + "readout"), dnext);
    Lin64Builder prodT(L.dout, L.dout, true);
    for (int Lo : L.out_ls) prodT.add(Lo * Lo, Lo * Lo, 2 * Lo + 1, m.off.at(pre + "prod." + std::to_string(Lo)), false);
    f64_linear(s, N, K, prodT.L, b.species, W, dnext, d.dB, nullptr);
    f64_symcon_bwd(s, L.lout_max, N, K, b.species, d.A[t], symw64(h, t), d.dB, d.dA);
    const double* dA = d.dA;
    if (t == 0) {
      Lin64Builder sk0T(16, 16, true);
      for (int l = 0; l <= 3; ++l) sk0T.add(l * l, l * l, 2 * l + 1, m.off.at(pre + "skip." + std::to_string(l)), true);
      f64_linear(s, N, K, sk0T.L, b.species, W, d.dA, d.dApre, nullptr);
      dA = d.dApre;
    }
    Lin64Builder linT(16, L.mid, true);
    for (int q = 0; q < L.P; ++q) {
      const int lo = L.paths[q].lo;
      linT.add(lo * lo, L.path_off[q], 2 * lo + 1, m.off.at(pre + "linear." + std::to_string(q)), false);
    }
    f64_linear(s, N, K, linT.L, b.species, W, dA, d.dAt, nullptr);
    f64_tp_bwd(s, L.lh_max, E, K, b.snd, b.rcv, z[2], W + m.off.at(pre + "radial.3"), d.Y, d.ht[t], d.dAt, inv_c,
               d.dY, t < T - 1, d.da3, t > 0 ? d.Q : nullptr);
    f64_radial_bwd(s, E, nb, W + m.off.at(pre + "radial.0"), W + m.off.at(pre + "radial.1"),
                   W + m.off.at(pre + "radial.2"), z[0], z[1], z[2], d.da3, d.de, t < T - 1);
    if (t > 0) {
      // dE/dh^t: through linear_up (the sender sum of the per-edge gradients)
      // and through the residual species linear
      f64_sender_sum(s, N, L.din, K, b.snd_off, b.snd_perm, d.Q, d.dht);
      Lin64Builder upT(L.din, L.din, true);
      for (int l : L.in_ls) upT.add(l * l, l * l, 2 * l + 1, m.off.at(pre + "up." + std::to_string(l)), false);
      f64_linear(s, N, K, upT.L, b.species, W, d.dht, dprev, nullptr);
      Lin64Builder skT(L.dout, L.din, true);
      for (int Lo : L.out_ls)
        if (std::find(L.in_ls.begin(), L.in_ls.end(), Lo) != L.in_ls.end())
          skT.add(Lo * Lo, Lo * Lo, 2 * Lo + 1, m.off.at(pre + "skip." + std::to_string(Lo)), true);
      f64_linear(s, N, K, skT.L, b.species, W, dnext, dprev, dprev);
      std::swap(dnext, dprev);
    }
  }
  f64_edge_vjp(s, E, pos, b.snd, b.rcv, b.shift, m.d.r_cut, m.d.envelope_p, nb, d.dY, d.de, d.g);
  f64_forces(s, N, b.rcv_off, b.snd_off, b.snd_perm, d.g, F);
}

}  // namespace

// ================================================================== C ABI
extern "C" {

const char* mace_status_string(mace_status s) {
  switch (s) {
    case MACE_OK: return "ok";
    case MACE_EINVAL: return "invalid argument";
    case MACE_ERANGE: return "index out of range or edges not sorted by receiver";
    case MACE_ENOSPACE: return "workspace or output capacity too small";
    case MACE_EHIP: return "HIP runtime error";
    case MACE_ENONFINITE: return "non-finite input";
    case MACE_ESTATE: return "invalid handle state";
    case MACE_EUNSUPPORTED: return "model shape not supported by the kernels";
  }
  return "unknown status";
}

mace_status mace_weight_layout(const mace_model_desc* desc, int32_t max_tensors, int64_t* sizes, int64_t* fan_in,
                               char* names, int32_t name_len, int32_t* n_tensors, int64_t* total_floats) {
  Model m;
  mace_status st = build_model(desc, m);
  if (st != MACE_OK) return st;
  if (n_tensors) *n_tensors = (int32_t)m.tensors.size();
  if (total_floats) *total_floats = m.total;
  if ((int)m.tensors.size() > max_tensors) return MACE_ENOSPACE;
  for (size_t i = 0; i < m.tensors.size(); ++i) {
    if (sizes) sizes[i] = m.tensors[i].size();
    if (fan_in) fan_in[i] = m.tensors[i].fan_in;
    if (names && name_len > 0) {
      char* dst = names + (size_t)i * name_len;
      size_t n = std::min<size_t>(m.tensors[i].name.size(), (size_t)name_len - 1);
      std::memcpy(dst, m.tensors[i].name.data(), n);
      dst[n] = 0;
    }
  }
  return MACE_OK;
}

size_t mace_workspace_bytes(const mace_model_desc* desc, int64_t n_atoms, int64_t n_edges, int32_t n_graphs,
                            mace_precision prec) {
  Model m;
  if (build_model(desc, m) != MACE_OK || n_atoms < 1 || n_edges < 0 || n_graphs < 1) return 0;
  Carver c{nullptr};
  Buffers b;
  carve(m, n_atoms, n_edges, n_graphs, c, b);
  if (prec == MACE_FP64) {
    Buffers64 b64;
    carve64(m, n_atoms, n_edges, c, b64);
  }
  return c.used + 256;
}

mace_status mace_graph_setup(const mace_model_desc* desc, const float* weights, int64_t weight_floats,
                             int64_t n_atoms, const int32_t* species, int64_t n_edges, const int32_t* edge_index,
                             const int32_t* unit_shifts, const double* cells, const int32_t* graph_of_atom,
                             int32_t n_graphs, mace_precision prec, void* workspace, size_t workspace_bytes,
                             void* stream, mace_graph** out) {
  if (!out) return MACE_EINVAL;
  *out = nullptr;
  Model m;
  mace_status st = build_model(desc, m);
  if (st != MACE_OK) return st;
  if (!weights || !species || !workspace || n_atoms < 1 || n_edges < 0 || n_graphs < 1) return MACE_EINVAL;
  if (n_edges > 0 && !edge_index) return MACE_EINVAL;
  if (prec != MACE_FP32 && prec != MACE_BF16_LINEAR && prec != MACE_FP16_LINEAR && prec != MACE_BF16_RADIAL &&
      prec != MACE_FP64)
    return MACE_EINVAL;
  if (weight_floats != m.total) return MACE_EINVAL;
  if (n_atoms > (1LL << 30) || n_edges > (1LL << 31) - 1) return MACE_EUNSUPPORTED;
  if (!graph_of_atom && n_graphs != 1) return MACE_EINVAL;
  if (unit_shifts && !cells) return MACE_EINVAL;
  if (mace_workspace_bytes(desc, n_atoms, n_edges, n_graphs, prec) > workspace_bytes) return MACE_ENOSPACE;
  hipStream_t s = (hipStream_t)stream;
  const int64_t N = n_atoms, E = n_edges, K = m.d.K, S = m.d.n_species;
  const int G = n_graphs;

  // --- host copies of the graph description
  std::vector<int32_t> hs(N), he(2 * E), hsh(unit_shifts ? 3 * E : 0), hg(N, 0);
  std::vector<double> hc(cells ? 9 * G : 0);
  std::vector<float> hw(m.total);
  auto cp = [&](void* dst, const void* src, size_t bytes) {
    return bytes ? hipMemcpyAsync(dst, src, bytes, hipMemcpyDeviceToHost, s) : hipSuccess;
  };
  if (cp(hs.data(), species, N * 4) != hipSuccess || cp(he.data(), edge_index, 2 * E * 4) != hipSuccess ||
      (unit_shifts && cp(hsh.data(), unit_shifts, 3 * E * 4) != hipSuccess) ||
      (cells && cp(hc.data(), cells, 9 * G * 8) != hipSuccess) ||
      (graph_of_atom && cp(hg.data(), graph_of_atom, N * 4) != hipSuccess) ||
      cp(hw.data(), weights, m.total * 4) != hipSuccess || hipStreamSynchronize(s) != hipSuccess)
    return MACE_EHIP;

  // --- validation
  for (int64_t i = 0; i < N; ++i) {
    if (hs[i] < 0 || hs[i] >= S) return MACE_ERANGE;
    if (hg[i] < 0 || hg[i] >= G || (i > 0 && hg[i] < hg[i - 1])) return MACE_ERANGE;
  }
  const int32_t* hsnd = he.data();
  const int32_t* hrcv = he.data() + E;
  for (int64_t e = 0; e < E; ++e) {
    if (hsnd[e] < 0 || hsnd[e] >= N || hrcv[e] < 0 || hrcv[e] >= N) return MACE_ERANGE;
    if (e > 0 && hrcv[e] < hrcv[e - 1]) return MACE_ERANGE;
    if (hg[hsnd[e]] != hg[hrcv[e]]) return MACE_ERANGE;
    bool zero_shift = !unit_shifts || (hsh[3 * e] == 0 && hsh[3 * e + 1] == 0 && hsh[3 * e + 2] == 0);
    if (hsnd[e] == hrcv[e] && zero_shift) return MACE_ERANGE;
  }
  for (float v : hw)
    if (!std::isfinite(v)) return MACE_ENONFINITE;

  // --- derived topology
  std::vector<int32_t> rcv_off(N + 1, 0), snd_off(N + 1, 0), snd_perm(E), goff(G + 1, 0);
  for (int64_t e = 0; e < E; ++e) {
    rcv_off[hrcv[e] + 1]++;
    snd_off[hsnd[e] + 1]++;
  }
  for (int64_t i = 0; i < N; ++i) {
    rcv_off[i + 1] += rcv_off[i];
    snd_off[i + 1] += snd_off[i];
  }
  {
    std::vector<int32_t> fillp(snd_off.begin(), snd_off.end() - 1);
    for (int64_t e = 0; e < E; ++e) snd_perm[fillp[hsnd[e]]++] = (int32_t)e;  // increasing e per sender
  }
  for (int64_t i = 0; i < N; ++i) goff[hg[i] + 1]++;
  for (int gi = 0; gi < G; ++gi) goff[gi + 1] += goff[gi];
  std::vector<double4> shv(std::max<int64_t>(E, 1), make_double4(0, 0, 0, 0));
  if (unit_shifts) {
    for (int64_t e = 0; e < E; ++e) {
      const double* c = hc.data() + 9 * hg[hrcv[e]];
      double S0 = hsh[3 * e], S1 = hsh[3 * e + 1], S2 = hsh[3 * e + 2];
      double v[3];
      for (int a = 0; a < 3; ++a) v[a] = ((S0 * c[a]) + (S1 * c[3 + a])) + (S2 * c[6 + a]);
      shv[e] = make_double4(v[0], v[1], v[2], 0.0);
    }
  }
  // nodes grouped by species, tiles of <= kLinTileNodes nodes of one species
  std::vector<int32_t> order, tstart, tcount, tspec;
  for (int z = 0; z < S; ++z) {
    int64_t first = (int64_t)order.size();
    for (int64_t i = 0; i < N; ++i)
      if (hs[i] == z) order.push_back((int32_t)i);
    for (int64_t q = first; q < (int64_t)order.size(); q += kLinTileNodes) {
      tstart.push_back((int32_t)q);
      tcount.push_back((int32_t)std::min<int64_t>(kLinTileNodes, (int64_t)order.size() - q));
      tspec.push_back(z);
    }
  }
  // transposed copy of every K x K block (backward linears) and of the last
  // radial layer [64][P*K] -> [P*K][64] (radial-MLP backward)
  std::vector<float> hwT(hw);
  for (auto& t : m.tensors) {
    const auto& sh = t.shape;
    if (t.name.size() > 9 && t.name.compare(t.name.size() - 9, 9, ".radial.3") == 0) {
      const int64_t rows = sh[0], cols = sh[1];
      for (int64_t r = 0; r < rows; ++r)
        for (int64_t c2 = 0; c2 < cols; ++c2) hwT[t.offset + c2 * rows + r] = hw[t.offset + r * cols + c2];
      continue;
    }
    if (sh.size() >= 2 && sh[sh.size() - 1] == K && sh[sh.size() - 2] == K) {
      int64_t blocks = t.size() / (K * K);
      for (int64_t q = 0; q < blocks; ++q) {
        const float* src = hw.data() + t.offset + q * K * K;
        float* dst = hwT.data() + t.offset + q * K * K;
        for (int64_t r = 0; r < K; ++r)
          for (int64_t c2 = 0; c2 < K; ++c2) dst[c2 * K + r] = src[r * K + c2];
      }
    }
  }

  // layer 0: path-merging weight of the path into l_out = l times the species
  // weight of l, W_comb[l][z] = W_lin[p(l)] W_skip[l][z] (FP64 sums, one rounding),
  // and its transpose, after the blob
  hw.resize(m.total_ext, 0.f);
  hwT.resize(m.total_ext, 0.f);
  {
    const LayerPlan& L0 = m.layers[0];
    for (int l = 0; l <= 3; ++l) {
      int p = -1;
      for (int q = 0; q < L0.P; ++q)
        if (L0.paths[q].lo == l) p = q;
      const float* wl = hw.data() + m.off.at("0.linear." + std::to_string(p));
      for (int64_t z = 0; z < S; ++z) {
        const float* ws = hw.data() + m.off.at("0.skip." + std::to_string(l)) + z * K * K;
        const int64_t base = m.comb_off + ((int64_t)l * S + z) * K * K;
        for (int64_t k = 0; k < K; ++k)
          for (int64_t n = 0; n < K; ++n) {
            double acc = 0.0;
            for (int64_t j = 0; j < K; ++j) acc += (double)wl[k * K + j] * (double)ws[j * K + n];
            hw[base + k * K + n] = (float)acc;
            hwT[base + n * K + k] = (float)acc;
          }
      }
    }
  }

  // factorised first layer (S <= kL0MaxSpecies): U (64 S channels per
  // component) to the layer's message, with c = l^2 + m, p(l) the path
  // (0, l, l), table[s][k] = sum_k' emb[s][k'] Wup[k'][k] (the mode's rounding
  // of emb and Wup, unrounded FP64 sums):
  //   Wf[l][s, j][k] = inv_c W3[j][p(l) K + k] table[s][k]     (U -> At)
  // and in FP32 mode composed with the path-merging and species linears,
  //   Wtot[l][z][s, j][k] = sum_k' Wf[l][s, j][k'] (W_lin[p(l)] W_skip[l][z])[k'][k]   (U -> A)
  // FP64 throughout, one rounding; stored [l][z][s, j][k] (16-bit modes: z = 0
  // only) and transposed [l][z][k][s, j].
  if (m.l0_ki) {
    const LayerPlan& L0 = m.layers[0];
    const int lowp = lowp_mode(prec);
    const int64_t KI = m.l0_ki, PK = (int64_t)L0.P * K;
    const double inv_c = 1.0 / m.d.c_norm;
    std::vector<double> tab(S * K, 0.0);
    const float* emb = hw.data() + m.off.at("embed");
    const float* wup = hw.data() + m.off.at("0.up.0");
    for (int64_t z = 0; z < S; ++z)
      for (int64_t k = 0; k < K; ++k) {
        double acc = 0.0;
        for (int64_t q = 0; q < K; ++q)
          acc += (double)lowp_round(emb[z * K + q], lowp) * (double)lowp_round(wup[q * K + k], lowp);
        tab[z * K + k] = acc;
      }
    const float* w3 = hw.data() + m.off.at("0.radial.3");
    std::vector<double> wf(KI * K), M(K * K);
    for (int l = 0; l <= 3; ++l) {
      int p = -1;
      for (int q = 0; q < L0.P; ++q)
        if (L0.paths[q].lo == l) p = q;
      for (int64_t sj = 0; sj < KI; ++sj) {
        const int64_t sp = sj / 64, j = sj % 64;
        for (int64_t k = 0; k < K; ++k) {
          double w = w3[j * PK + p * K + k];
          if (prec == MACE_BF16_RADIAL) w = bf16_round((float)w);
          wf[sj * K + k] = inv_c * w * tab[sp * K + k];
        }
      }
      const int nz = lowp ? 1 : (int)S;
      for (int z = 0; z < nz; ++z) {
        const int64_t base = m.l0_off + ((int64_t)l * S + z) * KI * K;
        if (lowp) {
          for (int64_t sj = 0; sj < KI; ++sj)
            for (int64_t k = 0; k < K; ++k) {
              hw[base + sj * K + k] = (float)wf[sj * K + k];
              hwT[base + k * KI + sj] = (float)wf[sj * K + k];
            }
          continue;
        }
        const float* wl = hw.data() + m.off.at("0.linear." + std::to_string(p));
        const float* ws = hw.data() + m.off.at("0.skip." + std::to_string(l)) + (int64_t)z * K * K;
        for (int64_t a = 0; a < K; ++a)
          for (int64_t n = 0; n < K; ++n) {
            double acc = 0.0;
            for (int64_t q = 0; q < K; ++q) acc += (double)wl[a * K + q] * (double)ws[q * K + n];
            M[a * K + n] = acc;
          }
        for (int64_t sj = 0; sj < KI; ++sj)
          for (int64_t n = 0; n < K; ++n) {
            double acc = 0.0;
            for (int64_t q = 0; q < K; ++q) acc += wf[sj * K + q] * M[q * K + n];
            hw[base + sj * K + n] = (float)acc;
            hwT[base + n * KI + sj] = (float)acc;
          }
      }
    }
  }

  // 16-bit copies (bf16 or binary16, by mode) of every K x K block, packed
  // [K/8][K][8] (element (k, n) at ((k/8) K + n) 8 + k%8) for the MFMA B
  // operand of the 16-bit linears
  std::vector<uint16_t> hbf(m.total, 0), hbfT(m.total, 0);
  auto to_bf16 = [](float x) -> uint16_t {
    uint32_t u;
    std::memcpy(&u, &x, 4);
    u += 0x7fffu + ((u >> 16) & 1u);
    return (uint16_t)(u >> 16);
  };
  auto to_16 = [&](float x) -> uint16_t {
    if (prec != MACE_FP16_LINEAR) return to_bf16(x);
    const _Float16 hx = (_Float16)x;   // round to nearest even, overflow to infinity
    uint16_t u;
    std::memcpy(&u, &hx, 2);
    return u;
  };
  for (auto& t : m.tensors) {
    const auto& sh = t.shape;
    if (!(sh.size() >= 2 && sh[sh.size() - 1] == K && sh[sh.size() - 2] == K)) continue;
    const int64_t blocks = t.size() / (K * K);
    for (int64_t q = 0; q < blocks; ++q) {
      const int64_t base = t.offset + q * K * K;
      for (int64_t k = 0; k < K; ++k)
        for (int64_t n = 0; n < K; ++n) {
          const int64_t dst = base + ((k / 8) * K + n) * 8 + (k % 8);
          hbf[dst] = to_16(hw[base + k * K + n]);
          hbfT[dst] = to_16(hwT[base + k * K + n]);
        }
    }
  }

  auto* h = new mace_graph();
  h->m = m;
  h->N = N;
  h->E = E;
  h->G = G;
  h->prec = prec;
  h->n_tiles = (int)tstart.size();
  // runs of up to kLinQuad consecutive tiles of one species (one linear block each)
  std::vector<int32_t> qtile, qcount;
  for (int t = 0; t < h->n_tiles;) {
    int n = 1;
    while (n < kLinQuad && t + n < h->n_tiles && tspec[t + n] == tspec[t]) ++n;
    qtile.push_back(t);
    qcount.push_back(n);
    t += n;
  }
  h->n_quads = (int)qtile.size();
  std::vector<int32_t> qnode((size_t)h->n_quads * kLinQuad * kLinTileNodes, -1), qspec(h->n_quads);
  for (int q = 0; q < h->n_quads; ++q) {
    qspec[q] = tspec[qtile[q]];
    for (int w = 0; w < qcount[q]; ++w) {
      const int t = qtile[q] + w;
      for (int r = 0; r < tcount[t]; ++r) qnode[((size_t)q * kLinQuad + w) * kLinTileNodes + r] = order[tstart[t] + r];
    }
  }
  // 16-bit modes on large graphs: the same tiles in runs of up to kLinQuadWide
  // (the wide 16-bit linears and the fused first-layer linears take them)
  std::vector<int32_t> qnode8, qspec8;
  if (lowp_mode(prec) && h->n_quads >= kLinQuadWideMinQuads) {
    for (int t = 0; t < h->n_tiles;) {
      int n = 1;
      while (n < kLinQuadWide && t + n < h->n_tiles && tspec[t + n] == tspec[t]) ++n;
      const size_t q = qspec8.size();
      qspec8.push_back(tspec[t]);
      qnode8.resize((q + 1) * kLinQuadWide * kLinTileNodes, -1);
      for (int w = 0; w < n; ++w)
        for (int r = 0; r < tcount[t + w]; ++r)
          qnode8[(q * kLinQuadWide + w) * kLinTileNodes + r] = order[tstart[t + w] + r];
      t += n;
    }
    h->n_quads8 = (int)qspec8.size();
  }
  // the buffers are carved from the workspace base rounded up to 256 bytes
  // (mace_workspace_bytes includes that slack)
  Carver c{reinterpret_cast<char*>((reinterpret_cast<uintptr_t>(workspace) + 255) & ~uintptr_t(255))};
  carve(h->m, N, E, G, c, h->b);
  if (prec == MACE_FP64) carve64(h->m, N, E, c, h->b64);
  Buffers& b = h->b;
  auto up = [&](void* dst, const void* src, size_t bytes) {
    return bytes ? hipMemcpyAsync(dst, src, bytes, hipMemcpyHostToDevice, s) : hipSuccess;
  };
  hipError_t err = hipSuccess;
  auto chk = [&](hipError_t e) { if (e != hipSuccess && err == hipSuccess) err = e; };
  chk(up(b.w, hw.data(), m.total_ext * 4));
  chk(up(b.wT, hwT.data(), m.total_ext * 4));
  chk(up(b.wbf, hbf.data(), m.total * 2));
  chk(up(b.wbfT, hbfT.data(), m.total * 2));
  chk(up(b.species, hs.data(), N * 4));
  chk(up(b.snd, hsnd, E * 4));
  chk(up(b.rcv, hrcv, E * 4));
  chk(up(b.rcv_off, rcv_off.data(), (N + 1) * 4));
  chk(up(b.snd_off, snd_off.data(), (N + 1) * 4));
  chk(up(b.snd_perm, snd_perm.data(), E * 4));
  std::vector<int32_t> snd_z(std::max<int64_t>(E, 1), 0);
  for (int64_t e = 0; e < E; ++e) snd_z[e] = hs[hsnd[e]];
  chk(up(b.snd_z, snd_z.data(), E * 4));
  chk(up(b.graph_off, goff.data(), (G + 1) * 4));
  std::vector<double> inv_vol(G, 1.0);
  if (cells)
    for (int gi = 0; gi < G; ++gi) {
      const double* c = hc.data() + 9 * gi;
      const double det = c[0] * (c[4] * c[8] - c[5] * c[7]) - c[1] * (c[3] * c[8] - c[5] * c[6]) +
                         c[2] * (c[3] * c[7] - c[4] * c[6]);
      inv_vol[gi] = det != 0.0 ? 1.0 / std::fabs(det) : 0.0;
    }
  chk(up(b.inv_vol, inv_vol.data(), G * 8));
  {
    std::vector<int2> sch;
    std::vector<int32_t> sco(G + 1, 0);
    for (int gi = 0; gi < G; ++gi) {
      const int e0 = rcv_off[goff[gi]], e1 = rcv_off[goff[gi + 1]];
      sco[gi] = (int32_t)sch.size();
      int e = e0;
      do {
        const int ee = std::min(e1, e + kStressChunk);
        sch.push_back(make_int2(e, ee));
        e = ee;
      } while (e < e1);
    }
    sco[G] = (int32_t)sch.size();
    h->n_stress_chunks = (int)sch.size();
    chk(up(b.stress_chunks, sch.data(), sch.size() * sizeof(int2)));
    chk(up(b.stress_chunk_off, sco.data(), (G + 1) * 4));
  }
  chk(up(b.quad_node, qnode.data(), qnode.size() * 4));
  chk(up(b.quad_species, qspec.data(), qspec.size() * 4));
  chk(up(b.quad_node8, qnode8.data(), qnode8.size() * 4));
  chk(up(b.quad_species8, qspec8.data(), qspec8.size() * 4));
  chk(up(b.shift, shv.data(), E * sizeof(double4)));
  chk(hipMemsetAsync(b.status, 0, sizeof(int), s));
  launch_species_table(s, (int)S, (int)K, b.w + m.off.at("embed"), b.w + m.off.at("0.up.0"),
                       lowp_mode(prec), b.sp_table);
  if (prec == MACE_FP64) f64_widen(s, (size_t)m.total, b.w, h->b64.w);
  chk(hipGetLastError());
  chk(hipStreamSynchronize(s));  // host vectors go out of scope below
  if (err != hipSuccess) {
    delete h;
    return MACE_EHIP;
  }
  h->l0_fact = l0_auto(h->m, N, E);
  make_plans(h);
  if (upload_plans(h, s) != hipSuccess) {
    delete h;
    return MACE_EHIP;
  }
  *out = h;
  return MACE_OK;
}

mace_status mace_forward_energy(mace_graph* g, const void* positions, void* node_energy, double* graph_energy,
                                void* stream) {
  if (!g || !positions || !node_energy || !graph_energy) return MACE_EINVAL;
  hipStream_t s = (hipStream_t)stream;
  if (g->prec == MACE_FP64) {
    if (!f64_supported(g)) return MACE_EUNSUPPORTED;
    run_forward64(g, s, static_cast<const double*>(positions), static_cast<double*>(node_energy), false);
    f64_graph_energy(s, g->G, g->b.graph_off, static_cast<const double*>(node_energy), graph_energy);
    return hip_ok(hipGetLastError());
  }
  if (!launchable(g)) return MACE_EUNSUPPORTED;
  run_forward(g, s, static_cast<const float*>(positions), static_cast<float*>(node_energy), false);
  {
    mace_graph* h = g;
    PROF(KID_GRAPH_ENERGY);
    launch_graph_energy(s, g->G, g->b.graph_off, static_cast<const float*>(node_energy), graph_energy);
  }
  return hip_ok(hipGetLastError());
}

mace_status mace_forces(mace_graph* g, const void* positions, void* node_energy, double* graph_energy,
                        void* forces, void* stream) {
  if (!g || !positions || !node_energy || !graph_energy || !forces) return MACE_EINVAL;
  hipStream_t s = (hipStream_t)stream;
  if (g->prec == MACE_FP64) {
    if (!f64_supported(g)) return MACE_EUNSUPPORTED;
    const double* pos = static_cast<const double*>(positions);
    run_forward64(g, s, pos, static_cast<double*>(node_energy), true);
    run_backward64(g, s, pos, static_cast<double*>(forces));
    f64_graph_energy(s, g->G, g->b.graph_off, static_cast<const double*>(node_energy), graph_energy);
    return hip_ok(hipGetLastError());
  }
  if (!launchable(g)) return MACE_EUNSUPPORTED;
  const float* pos = static_cast<const float*>(positions);
  run_forward(g, s, pos, static_cast<float*>(node_energy), true);
  run_backward(g, s, pos, static_cast<float*>(forces), static_cast<const float*>(node_energy), graph_energy);
  return hip_ok(hipGetLastError());
}

mace_status mace_forces_stress(mace_graph* g, const void* positions, void* node_energy, double* graph_energy,
                               void* forces, double* stress, void* stream) {
  if (!g || !positions || !node_energy || !graph_energy || !forces || !stress) return MACE_EINVAL;
  mace_status st = mace_forces(g, positions, node_energy, graph_energy, forces, stream);
  if (st != MACE_OK) return st;
  hipStream_t s = (hipStream_t)stream;
  if (g->prec == MACE_FP64) {
    f64_stress(s, g->G, g->b.graph_off, g->b.rcv_off, static_cast<const double*>(positions), g->b.snd, g->b.rcv,
               g->b.shift, g->b64.g, g->b.inv_vol, stress);
    return hip_ok(hipGetLastError());
  }
  {
    mace_graph* h = g;
    PROF(KID_FORCES);
    launch_stress(s, g->G, g->n_stress_chunks, g->b.stress_chunks, g->b.stress_chunk_off,
                  static_cast<const float*>(positions), g->b.snd,
                  g->b.rcv, g->b.shift, g->b.g, g->b.inv_vol, g->b.stress_part, stress);
  }
  return hip_ok(hipGetLastError());
}

mace_status mace_graph_check(mace_graph* g, int32_t* device_flags, void* stream) {
  if (!g) return MACE_EINVAL;
  hipStream_t s = (hipStream_t)stream;
  int flags = 0;
  if (hipMemcpyAsync(&flags, g->b.status, sizeof(int), hipMemcpyDeviceToHost, s) != hipSuccess ||
      hipMemsetAsync(g->b.status, 0, sizeof(int), s) != hipSuccess || hipStreamSynchronize(s) != hipSuccess)
    return MACE_EHIP;
  if (device_flags) *device_flags = flags;
  if (flags & kStatusNonFinite) return MACE_ENONFINITE;
  if (flags & kStatusZeroLength) return MACE_ERANGE;
  return MACE_OK;
}

void mace_graph_destroy(mace_graph* g) {
  if (!g) return;
  for (auto e : g->prof_ev) hipEventDestroy(e);
  delete g;
}

mace_status mace_layer0_form(mace_graph* g, int32_t request, int32_t* in_use) {
  if (!g || request > MACE_L0_FACTORED) return MACE_EINVAL;
  if (g->prec == MACE_FP64) {   // every layer in per-edge form
    if (request == MACE_L0_FACTORED) return MACE_EUNSUPPORTED;
    if (in_use) *in_use = MACE_L0_EDGE;
    return MACE_OK;
  }
  if (request == MACE_L0_FACTORED && !g->m.l0_ki) return MACE_EUNSUPPORTED;
  if (request == MACE_L0_AUTO) g->l0_fact = l0_auto(g->m, g->N, g->E);
  else if (request == MACE_L0_EDGE) g->l0_fact = false;
  else if (request == MACE_L0_FACTORED) g->l0_fact = true;
  // the form the next calls will run: the precision study's edge-product and
  // radial-MLP rounding force the per-edge form whatever was requested
  if (in_use) *in_use = layer_factorised(g, 0) ? MACE_L0_FACTORED : MACE_L0_EDGE;
  return MACE_OK;
}

mace_status mace_debug_fused_linears(mace_graph* g, int32_t request, int32_t* in_use) {
  if (!g || request > 3) return MACE_EINVAL;
  if (request >= 0) {
    g->l0_chain = (request & 1) != 0;
    g->wide_tiles = (request & 2) != 0;
  }
  if (in_use) {
    const Model& m = g->m;
    ChainStage cs;
    const bool chain = g->l0_chain && lowp_mode(g->prec) && m.d.K == 128 && m.l0_ki == 128 &&
                       m.layers[0].mid == 16 && layer_factorised(g, 0) && chain_stage_of(g->l0f, 0, &cs) &&
                       chain_stage_of(g->lin[0], 1, &cs) && chain_stage_of(g->skip0, 1, &cs);
    const bool eight = g->wide_tiles && g->n_quads8 > 0 && m.d.K == 128;
    *in_use = (chain ? 1 : 0) | (eight ? 2 : 0);
  }
  return MACE_OK;
}

mace_status mace_fp32_products(mace_graph* g, int32_t request, int32_t* in_use) {
  if (!g || (g->prec == MACE_FP64 && request >= 0)) return MACE_EINVAL;
  if (request >= 0) {
    if (g->prec == MACE_BF16_RADIAL || (request != MACE_PRODUCTS_FP32 && request != MACE_PRODUCTS_SPLIT_BF16))
      return MACE_EINVAL;
    g->radial_split = request == MACE_PRODUCTS_SPLIT_BF16;
  }
  if (in_use) *in_use = g->prec == MACE_BF16_RADIAL ? 1 : (g->radial_split ? MACE_PRODUCTS_SPLIT_BF16 : MACE_PRODUCTS_FP32);
  return MACE_OK;
}

mace_status mace_block_rounding(mace_graph* g, int32_t block, int32_t format, int32_t* in_use) {
  if (!g || (block != MACE_BLOCK_EDGE_PRODUCT && block != MACE_BLOCK_SYMMETRIC_CONTRACTION &&
             block != MACE_BLOCK_RADIAL_MLP) || format > 2 || (g->prec == MACE_FP64 && format > 0))
    return MACE_EINVAL;
  int& r = block == MACE_BLOCK_EDGE_PRODUCT ? g->tp_round
                                            : (block == MACE_BLOCK_SYMMETRIC_CONTRACTION ? g->sc_round : g->rad_round);
  if (format >= 0) r = format;
  if (in_use) *in_use = r;
  return MACE_OK;
}

mace_status mace_profile_select(mace_graph* g, int32_t kernel) {
  if (!g || kernel < -1 || kernel >= KID_COUNT) return MACE_EINVAL;
  if (kernel >= 0 && g->prof_ev.empty()) {
    g->prof_ev.resize(2 * kProfPairs);
    for (auto& e : g->prof_ev)
      if (hipEventCreate(&e) != hipSuccess) return MACE_EHIP;
  }
  g->prof_kernel = kernel;
  g->prof_used = 0;
  g->prof_dropped = 0;
  g->prof_flops = g->prof_bytes = 0.0;
  return MACE_OK;
}

mace_status mace_profile_work(mace_graph* g, double* flops, double* bytes) {
  if (!g || !flops || !bytes) return MACE_EINVAL;
  *flops = g->prof_flops;
  *bytes = g->prof_bytes;
  return MACE_OK;
}

mace_status mace_profile_read(mace_graph* g, double* total_ms, int64_t* launches) {
  if (!g || !total_ms || !launches) return MACE_EINVAL;
  double tot = 0.0;
  for (int i = 0; i < g->prof_used; ++i) {
    if (hipEventSynchronize(g->prof_ev[2 * i + 1]) != hipSuccess) return MACE_EHIP;
    float ms = 0.f;
    if (hipEventElapsedTime(&ms, g->prof_ev[2 * i], g->prof_ev[2 * i + 1]) != hipSuccess) return MACE_EHIP;
    tot += ms;
  }
  *total_ms = tot;
  *launches = g->prof_used;
  g->prof_used = 0;
  return g->prof_dropped ? MACE_ENOSPACE : MACE_OK;
}

const char* mace_kernel_name(int32_t kernel) {
  return (kernel >= 0 && kernel < KID_COUNT) ? kKernelNames[kernel] : "";
}

mace_status mace_debug_real_cg(int32_t l1, int32_t l2, int32_t l3, double* out) {
  if (!out || l1 < 0 || l2 < 0 || l3 < std::abs(l1 - l2) || l3 > l1 + l2 || l1 > 8 || l2 > 8) return MACE_EINVAL;
  auto C = so3h::real_cg(l1, l2, l3);
  std::copy(C.v.begin(), C.v.end(), out);
  return MACE_OK;
}

mace_status mace_debug_trees(int32_t nu, int32_t L, int32_t parity, int32_t max_trees, int32_t* trees,
                             double* scales, int32_t* n_trees) {
  if (nu < 1 || nu > 3 || L < 0 || L > 6 || (parity != 1 && parity != -1) || !n_trees) return MACE_EINVAL;
  auto sel = so3h::select_trees(nu, L, parity);
  *n_trees = (int32_t)sel.size();
  if ((int)sel.size() > max_trees) return MACE_ENOSPACE;
  for (size_t i = 0; i < sel.size(); ++i) {
    if (trees) {
      trees[4 * i + 0] = sel[i].l1;
      trees[4 * i + 1] = sel[i].l2;
      trees[4 * i + 2] = sel[i].l3;
      trees[4 * i + 3] = sel[i].l12;
    }
    if (scales) scales[i] = sel[i].scale;
  }
  return MACE_OK;
}

mace_status mace_debug_edge_features(int64_t n, const float* vec, double r_cut, int32_t envelope_p, int32_t n_bessel,
                                     float* Y, float* rbf) {
  if (n < 0 || !vec || !Y || !rbf || n_bessel < 1 || n_bessel > 16 || !(r_cut > 0)) return MACE_EINVAL;
  for (int64_t e = 0; e < n; ++e) {
    double dx = vec[3 * e], dy = vec[3 * e + 1], dz = vec[3 * e + 2];
    double rr = sqrt(dx * dx + dy * dy + dz * dz);
    double inv = 1.0 / rr;
    double y[16], eb[16];
    sh16<double>(dx * inv, dy * inv, dz * inv, y);
    bessel_env<double>(rr, r_cut, envelope_p, n_bessel, eb);
    for (int q = 0; q < 16; ++q) Y[16 * e + q] = (float)y[q];
    for (int q = 0; q < n_bessel; ++q) rbf[e * n_bessel + q] = (float)eb[q];
  }
  return MACE_OK;
}

}  // extern "C"
