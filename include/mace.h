/* mace.h -- C ABI of the MI355X (gfx950) MACE layer library.
 *
 * Computes, for a batch of atomic graphs, per-atom energies eps_i, per-graph
 * energies E_g = sum_{i in g} eps_i and forces F_i = -dE/dr_i of a MACE model
 * (arXiv 2510.23621: graph problem statement; two-body edge embedding,
 * Eq. 26; product basis, Eq. 27; message/update/readout paragraph; energy and
 * force equations; architecture table of the appendix).  Inputs follow the
 * problem statement: species, positions, directed edges j -> i within the
 * cutoff with their periodic image shifts, and model weights.
 *
 * Pointers marked (dev) are device memory owned by the caller; pointers
 * marked (host) are host memory owned by the caller.  The library never
 * allocates or frees device memory: every buffer it needs is carved from
 * the caller's workspace.  Entry points taking a stream enqueue on it.
 *
 * Errors: every entry point validates its arguments synchronously and
 * returns a mace_status; nothing is enqueued when it returns an error.
 */
#ifndef MACE_H_
#define MACE_H_

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  MACE_OK = 0,
  MACE_EINVAL = -1,       /* null pointer, bad size, inconsistent arguments */
  MACE_ERANGE = -2,       /* index or species out of range, unsorted edges */
  MACE_ENOSPACE = -3,     /* workspace or output capacity too small */
  MACE_EHIP = -4,         /* a HIP runtime call failed */
  MACE_ENONFINITE = -5,   /* non-finite input detected */
  MACE_ESTATE = -6,       /* handle in a state that does not allow the call */
  MACE_EUNSUPPORTED = -7  /* model shape outside what the kernels implement */
} mace_status;

typedef enum {
  MACE_FP32 = 0,          /* every step in FP32 */
  MACE_BF16_LINEAR = 1,   /* channel-mixing linears with BF16 inputs and weights,
                             FP32 accumulation; everything else FP32 */
  MACE_FP16_LINEAR = 2,   /* the same with IEEE binary16 (round to nearest even;
                             an input or weight beyond 65504 becomes infinite and
                             the outputs then hold non-finite values) */
  MACE_BF16_RADIAL = 3,   /* MACE_BF16_LINEAR, and the last layer of the radial
                             MLP (the P*K-wide one) on BF16 operands with FP32
                             accumulation: R = bf16(a3) bf16(W) forward and
                             dE/da3 = bf16(dE/dR) bf16(W)^T backward */
  MACE_FP64 = 4           /* debug precision: every step in FP64 on the vector
                             units (plain kernels, not tuned for speed), every
                             layer in per-edge form; positions, node energies
                             and forces are FP64 (the FP64 baseline every
                             precision arm of the paper is measured against) */
} mace_precision;

#define MACE_MAX_LAYERS 8

/* Model hyper-parameters (host).  Supported: sh_lmax = 3, correlation = 3,
 * 1 <= n_bessel <= 16, radial_hidden = {64, 64, 64}, 1 <= readout_hidden <= 16,
 * 0 <= hidden_lmax[t] <= 2 and non-increasing in t, K in {32, 64, 96, 128},
 * 1 <= n_layers <= MACE_MAX_LAYERS (other values: MACE_EUNSUPPORTED, or
 * MACE_EINVAL for n_layers).  Layer t's input irreps are 0e for t = 0 and
 * 0e+...+l for l = hidden_lmax[t - 1] after it (the architecture table's
 * hidden irreps, alternating parity); its output irreps are those of
 * hidden_lmax[t], and 0e for the last layer. */
typedef struct mace_model_desc {
  int32_t n_species;       /* S */
  int32_t K;               /* channels */
  int32_t n_layers;        /* interaction layers T */
  int32_t sh_lmax;         /* edge harmonics l <= sh_lmax */
  int32_t correlation;     /* nu <= correlation */
  int32_t n_bessel;        /* radial basis size */
  int32_t envelope_p;      /* polynomial envelope exponent */
  int32_t radial_hidden[3];
  int32_t readout_hidden;  /* hidden width of the last readout MLP */
  int32_t hidden_lmax[MACE_MAX_LAYERS];  /* [t]: lmax of the features leaving layer t, for
                                            t < n_layers - 1; later entries are ignored */
  double r_cut;            /* cutoff radius (A) */
  double c_norm;           /* neighbour-sum normalisation constant */
} mace_model_desc;

typedef struct mace_graph mace_graph;  /* opaque handle (host metadata) */

/* Layout of the FP32 weight blob: tensor t occupies sizes[t] floats, in
 * this order: "embed" [S][K]; then per layer t: "t.up.l" [K][K] per input l;
 * "t.radial.0..3" ([nb][64], [64][64], [64][64], [64][P*K], path-major);
 * "t.linear.p" [K][K] per edge-product path p; species linears "t.skip.l"
 * [S][K][K]; symmetric-contraction weights "t.symc.L.nu" [S][n_eta][K];
 * "t.prod.L" [K][K]; readout "t.readout" [K] (non-last layers) or
 * "t.readout.0" [K][16], "t.readout.1" [16] (last layer).  Every matrix is
 * row-major [in][out].  fan_in[t] is the fan-in used for N(0,1)/sqrt(fan_in)
 * initialisation.  sizes, fan_in (host) of capacity max_tensors; names
 * (host, may be NULL) of capacity max_tensors * name_len, each entry
 * NUL-terminated.  Returns MACE_ENOSPACE (with *n_tensors set) when the
 * capacity is too small. */
mace_status mace_weight_layout(const mace_model_desc* desc, int32_t max_tensors, int64_t* sizes,
                               int64_t* fan_in, char* names, int32_t name_len, int32_t* n_tensors,
                               int64_t* total_floats);

/* Bytes of device workspace a graph of this size needs. 0 on invalid input. */
size_t mace_workspace_bytes(const mace_model_desc* desc, int64_t n_atoms, int64_t n_edges, int32_t n_graphs,
                            mace_precision prec);

/* Neighbour list (host, FP64 cell list) of the graph problem statement:
 * edge j -> i with shift S is kept iff 0 < |(x_j - x_i) + S.cell|^2 < r_cut^2,
 * every periodic image enumerated, atoms of different graphs never joined,
 * sorted by (receiver, sender, S).  positions (host) [N][3]; cells (host)
 * [G][3][3] rows = lattice vectors, or NULL (no periodicity);
 * graph_of_atom (host) [N] nondecreasing or NULL.  Outputs (host) of
 * capacity max_edges: sender [E], receiver [E], shifts [E][3].  When the
 * capacity is too small returns MACE_ENOSPACE with *n_edges = the count. */
mace_status mace_neighbor_list(int64_t n_atoms, const double* positions, const double* cells,
                               const int32_t* graph_of_atom, int32_t n_graphs, double r_cut, int64_t max_edges,
                               int32_t* sender, int32_t* receiver, int32_t* shifts, int64_t* n_edges);

/* The same neighbour list built on the device (FP64 hashed cell list; the
 * same cutoff expression, evaluated without fused multiply-adds, so the
 * output equals mace_neighbor_list's element for element).  positions (dev)
 * [N][3] FP64, |coordinates| <= 1e9; cells (host) [G][3][3] rows = lattice
 * vectors, or NULL; graph_offsets (host) [G+1] (atoms of graph g are
 * [off[g], off[g+1]), off[0] = 0, off[G] = N) or NULL for one graph.
 * Outputs (dev) of capacity max_edges: sender [E], receiver [E], shifts
 * [E][3], sorted by (receiver, sender, S).  workspace (dev) of at least
 * mace_neighbor_workspace_bytes.  Waits for the stream once, to read the
 * edge count into *n_edges (host); the outputs are then written by work
 * enqueued on stream.  MACE_ENOSPACE (with *n_edges = the count, outputs
 * untouched) when max_edges is too small; MACE_ENONFINITE / MACE_ERANGE for
 * non-finite / out-of-bound coordinates; MACE_EUNSUPPORTED beyond 2^30
 * periodic-image candidates. */
size_t mace_neighbor_workspace_bytes(int64_t n_atoms, const double* cells, const int32_t* graph_offsets,
                                     int32_t n_graphs, double r_cut);
mace_status mace_neighbor_list_device(int64_t n_atoms, const double* positions, const double* cells,
                                      const int32_t* graph_offsets, int32_t n_graphs, double r_cut,
                                      int64_t max_edges, int32_t* sender, int32_t* receiver, int32_t* shifts,
                                      int64_t* n_edges, void* workspace, size_t workspace_bytes, void* stream);

/* For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid allocation): the same
 * list as mace_neighbor_list_device, same arguments and results, without the
 * workspace argument.  Its kernels use a file-scope device array of
 * MACE_NEIGHBOR_SCRATCH_BYTES bytes instead, which every GPU the library runs
 * on holds until the process ends (enough for 36,864 periodic atoms at a
 * 6 A cutoff).  Calls no allocating routine.  Returns MACE_ENOSPACE, with
 * nothing enqueued, when the list would need more than that
 * (mace_neighbor_workspace_bytes > MACE_NEIGHBOR_SCRATCH_BYTES).  Every call
 * on one GPU shares that GPU's array: calls that overlap on one GPU (other
 * streams, other host threads) race and must be serialised by the caller.
 * Each call clears what its kernels need zeroed. */
#define MACE_NEIGHBOR_SCRATCH_BYTES ((size_t)80 << 20)
mace_status mace_neighbor_list_device_noalloc(int64_t n_atoms, const double* positions, const double* cells,
                                              const int32_t* graph_offsets, int32_t n_graphs, double r_cut,
                                              int64_t max_edges, int32_t* sender, int32_t* receiver, int32_t* shifts,
                                              int64_t* n_edges, void* stream);

/* Validate and pack a graph and the weights into the workspace.
 * Paper: "Graph representation of atomic configurations" (atoms are nodes
 * with coordinates r_i and species z_i, edges join atoms within the cutoff;
 * here every periodic image within the cutoff is an edge of its own) and the
 * architecture-breakdown table of the appendix (the weights).
 * weights (dev) FP32 blob in mace_weight_layout order; species (dev) [N] in
 * 0..S-1; edge_index (dev) [2][E]: row 0 senders j, row 1 receivers i,
 * receivers nondecreasing; unit_shifts (dev) [E][3] or NULL (no
 * periodicity); cells (dev) [G][3][3] FP64 or NULL; graph_of_atom (dev) [N]
 * nondecreasing or NULL (one graph); workspace (dev) of at least
 * mace_workspace_bytes.  Synchronises the stream (setup is not on the hot
 * path).  After it returns the caller may free weights, species,
 * edge_index, unit_shifts, cells and graph_of_atom. */
mace_status mace_graph_setup(const mace_model_desc* desc, const float* weights, int64_t weight_floats,
                             int64_t n_atoms, const int32_t* species, int64_t n_edges, const int32_t* edge_index,
                             const int32_t* unit_shifts, const double* cells, const int32_t* graph_of_atom,
                             int32_t n_graphs, mace_precision prec, void* workspace, size_t workspace_bytes,
                             void* stream, mace_graph** out);

/* Positions, node energies and forces are FP32 (float) for every precision
 * but MACE_FP64, where they are FP64 (double); per-graph energies and the
 * stress are FP64 always.
 *
 * Energies.  Paper: "Higher-order Message Passing in MACE" -- the two-body
 * edge embedding (Eq. 26), the node-local product basis (Eq. 27), the message
 * over correlation orders, the linear update with residual and the readouts;
 * and the energy equation of "MACE inference: energy and forces", eps_i from
 * the invariant features, E = sum_i eps_i (here per graph, summed in FP64 in
 * a fixed order).  positions (dev) [N][3]; node_energy (dev) [N];
 * graph_energy (dev) [G] FP64.  No host synchronisation, no allocation.
 * MACE_EUNSUPPORTED (nothing enqueued) if the handle's settings select an
 * edge-product instance that is not built. */
mace_status mace_forward_energy(mace_graph* g, const void* positions, void* node_energy, double* graph_energy,
                                void* stream);

/* Energies and forces.  Paper: the force equation of "MACE inference:
 * energy and forces", F_i = -dE/dr_i = -sum_j d eps_j / d r_i, evaluated by
 * the reverse pass of every step of mace_forward_energy (a hand-written
 * vector-Jacobian product, deterministic: no floating-point atomics).  As
 * mace_forward_energy plus forces (dev) [N][3]. */
mace_status mace_forces(mace_graph* g, const void* positions, void* node_energy, double* graph_energy,
                        void* forces, void* stream);

/* Energies, forces and the stress of every graph.  Paper: the NPT
 * observables of "Precision-loss metrics" monitor the pressure p(t) of a
 * periodic box, p = -tr(sigma)/3; sigma itself is not defined there. stress (dev) [G][3][3] FP64 row-major:
 * sigma_g[a][b] = (1/V_g) dE_g/d(epsilon_ab) for a homogeneous strain acting
 * on row vectors, x -> x (I + epsilon), applied to the graph's positions and
 * cell rows; equivalently (1/V_g) sum over the graph's edges of d_e[a] g_e[b]
 * with d_e the edge vector and g_e = dE/dd_e. V_g = |det cell_g|; for a
 * handle set up without cells V = 1 (the bare strain derivative). Summed in
 * FP64 in a fixed order (bitwise reproducible). Other arguments and behaviour
 * as mace_forces. */
mace_status mace_forces_stress(mace_graph* g, const void* positions, void* node_energy, double* graph_energy,
                               void* forces, double* stress, void* stream);

/* How the first interaction layer forms its message.  Its sender features
 * depend on the species only (the embedding through linear_up) and its paths
 * are (0, l, l), whose coupling is the identity, so Eq. 26 summed over a
 * receiver's edges factorises: U[i][c][s][j] = sum over the edges into i
 * from atoms of species s of a3[e][j] Y[e][c] (a3 the last hidden layer of
 * the radial MLP, c = l^2 + m), then one node-level contraction of U with the
 * last radial layer and the species table (in MACE_FP32, composed with the
 * path-merging and species linears that follow it, in FP64 at setup).
 *   MACE_L0_EDGE:     the per-edge product, as every other layer;
 *   MACE_L0_FACTORED: the factorised form (S <= 4 only, else MACE_EUNSUPPORTED);
 *   MACE_L0_AUTO:     setup's choice, factorised when S <= 4 and E >= 3 S N.
 * Both forms compute the same function and differ only in FP32 rounding
 * order.  request < 0 only queries; *in_use (host, may be NULL) receives
 * MACE_L0_EDGE or MACE_L0_FACTORED.  Takes effect for calls enqueued after
 * it returns; no device work. */
typedef enum { MACE_L0_AUTO = 0, MACE_L0_EDGE = 1, MACE_L0_FACTORED = 2 } mace_l0_form;
mace_status mace_layer0_form(mace_graph* g, int32_t request, int32_t* in_use);

/* Operands of the P*K-wide last radial layer (formed inside the edge-product
 * kernels of the layers in per-edge form) in the modes other than
 * MACE_BF16_RADIAL.  (The channel-mixing linears stay on FP32 MFMA: split
 * products were measured slower there, where the MFMA is not the bound.)
 *   MACE_PRODUCTS_FP32:       FP32 MFMA (v_mfma_f32_16x16x4_f32);
 *   MACE_PRODUCTS_SPLIT_BF16: every FP32 operand x carried as x0 + x1 + x2,
 *     the bfloat16 roundings of x, x - x0 and x - x0 - x1 (together exact),
 *     and each product formed from the six partial products down to
 *     relative size 2^-18 on BF16 MFMA with FP32 accumulation: as accurate
 *     as FP32 products (the dropped terms are below 2^-26 relative), at a
 *     fraction of the FP32 MFMA time.  The default.
 * request < 0 only queries; *in_use (host, may be NULL) receives the setting
 * (MACE_BF16_RADIAL handles report 1 and refuse a change with MACE_EINVAL).
 * Takes effect for calls enqueued after it returns; no device work. */
typedef enum { MACE_PRODUCTS_FP32 = 0, MACE_PRODUCTS_SPLIT_BF16 = 2 } mace_fp32_products_kind;
mace_status mace_fp32_products(mace_graph* g, int32_t request, int32_t* in_use);

/* Per-block precision study (the paper's per-block low-precision experiments,
 * run on the whole model): the operands of one block are rounded to nearest
 * even as they are loaded, all arithmetic and sums staying FP32, on top of
 * the handle's precision mode.
 *   block MACE_BLOCK_EDGE_PRODUCT: the sender features, the harmonics and the
 *     radial weights R of every edge product (the CG constants stay FP32);
 *     the first layer then runs in per-edge form (its factorised form never
 *     forms R);
 *   block MACE_BLOCK_SYMMETRIC_CONTRACTION: A and the contraction weights (the
 *     coupling constants stay FP32);
 *   block MACE_BLOCK_RADIAL_MLP: the input and the weights of every layer of
 *     the radial MLP (the radial basis, each SiLU output, W0..W3); the first
 *     layer then runs in per-edge form.
 *   format 0 none (the default), 1 bfloat16, 2 IEEE binary16 (magnitudes
 *     beyond 65504 become infinite); format < 0 only queries.
 * Gradients pass through the rounding unchanged.  *in_use (host, may be
 * NULL) receives the setting.  Takes effect for calls enqueued after it
 * returns; no device work. */
typedef enum {
  MACE_BLOCK_EDGE_PRODUCT = 0,
  MACE_BLOCK_SYMMETRIC_CONTRACTION = 1,
  MACE_BLOCK_RADIAL_MLP = 2
} mace_block;
mace_status mace_block_rounding(mace_graph* g, int32_t block, int32_t format, int32_t* in_use);

/* Device-detected errors of the calls enqueued since setup or the previous
 * check: the edge kernels OR status bits into a word of the workspace,
 * 1 = an edge vector with a non-finite component (NaN or infinite
 * positions), 2 = an edge of length zero (coincident atoms).  After such a
 * call the outputs are undefined but the handle stays valid.  Enqueues a
 * read and a reset of the word on stream, waits for the stream, stores the
 * bits in *device_flags (host, may be NULL) and returns MACE_ENONFINITE if
 * flag 1 is set, else MACE_ERANGE if flag 2 is set, else MACE_OK. */
mace_status mace_graph_check(mace_graph* g, int32_t* device_flags, void* stream);

/* Releases the host handle (the workspace stays the caller's). */
void mace_graph_destroy(mace_graph* g);

const char* mace_status_string(mace_status s);

/* Kernel timing (profiling aid, host): while kernel class `kernel` is
 * selected (0 <= kernel < number of classes; -1 = none), every launch of
 * that class made by mace_forward_energy / mace_forces is bracketed by a
 * pair of HIP events recorded on the call's stream (at most 4096 launches
 * between reads).  mace_profile_read waits for those events and returns the
 * summed kernel milliseconds and the launch count since the last select or
 * read; MACE_ENOSPACE if launches were dropped.  mace_kernel_name gives the
 * class's kernel symbol stem ("" when out of range). */
mace_status mace_profile_select(mace_graph* g, int32_t kernel);
mace_status mace_profile_read(mace_graph* g, double* total_ms, int64_t* launches);
const char* mace_kernel_name(int32_t kernel);
/* Algorithmic work of the selected class's launches since the last select
 * (host outputs; not reset by mace_profile_read).  Summed for the linear
 * class only (0 for the others): flops = 2 K^2 per node and weight term
 * component; bytes = each distinct input component, output component and
 * weight block moved once (outputs read too when accumulated into or when a
 * residual is added; 16-bit weights count 2 bytes). */
mace_status mace_profile_work(mace_graph* g, double* flops, double* bytes);

/* Test switch (host) for callers that check the 16-bit modes' linear
 * layouts against the plain ones, which they equal bit for bit. Bit 0: with
 * K = 128 and a 128-wide factorised contraction, the first layer's
 * contraction, path-merging and species linears (and their transposes) run
 * as one launch each way instead of three. Bit 1: on graphs of at least 256
 * blocks of four 16-node tiles, the wide 16-bit linears take eight tiles per
 * block. request 3 (both, the default) to 0 (neither) sets them, < 0 only
 * queries; *in_use (host, may be NULL) = the bits in effect for this
 * handle's mode, shapes and first-layer form. MACE_EINVAL for a NULL handle
 * or a request above 3. */
mace_status mace_debug_fused_linears(mace_graph* g, int32_t request, int32_t* in_use);

/* Table export for checking the library's couplings (host). */
/* real CG C^{l3}_{l1 l2}[m1][m2][m3] into out (host) [(2l1+1)(2l2+1)(2l3+1)] */
mace_status mace_debug_real_cg(int32_t l1, int32_t l2, int32_t l3, double* out);
/* coupling trees kept for (nu, L, parity): trees (host) [max][4] = (l1, l2, l3, l12), scales (host) [max] */
mace_status mace_debug_trees(int32_t nu, int32_t L, int32_t parity, int32_t max_trees, int32_t* trees,
                             double* scales, int32_t* n_trees);
/* harmonics and radial basis of the kernels, evaluated on the host:
 * vec (host) [n][3] edge vectors -> Y (host) [n][16], rbf (host) [n][n_bessel] */
mace_status mace_debug_edge_features(int64_t n, const float* vec, double r_cut, int32_t envelope_p,
                                     int32_t n_bessel, float* Y, float* rbf);

#ifdef __cplusplus
}
#endif

#endif /* MACE_H_ */
