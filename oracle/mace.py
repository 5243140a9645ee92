"""Plain FP64 MACE energy and forces on the CPU (oracle).

Follows the paper's model section: the graph problem statement, the two-body
edge embedding A (Eq. 26), the product basis B (Eq. 27), the message as a
weighted sum over correlation orders and couplings, the linear update with a
residual, the readouts, E = sum_i eps_i and F_i = -dE/dr_i; and the module
and parameter table of the architecture-breakdown appendix (ScaleShiftMACE:
embedding, radial embedding, harmonics, Interactions[0] = non-residual block
with a species-dependent linear on the message, Interactions[t>=1] = residual
block, product-basis linears, linear readout then a 128->16->1 MLP readout).

Readings where the paper is silent, ambiguous or garbled (each one fixed
here and followed identically by the HIP library, which is written
separately):

R1  Harmonics, CG couplings, U basis: see ``oracle.so3``.
R2  Path set of the edge product: (l_h, l_Y, l_out) with l_h over the hidden
    irreps entering the layer, l_Y = 0..3, l_out = 0..3, l_h+l_Y+l_out even
    (natural parity), sorted lexicographically; the coupling is
    C^{l_out}_{l_h l_Y}: hidden feature first, harmonic second.  Reproduces
    the appendix's 4 / 10 paths and 16x / 40x mid dimensions.
R3  Edge vector d = r_sender + shift - r_receiver.
R4  Radial basis: e_n(r) = sqrt(2/rc) sin(n pi r/rc)/r * u(r/rc), n = 1..8,
    polynomial envelope u(x) = 1 - (p+1)(p+2)/2 x^p + p(p+2) x^(p+1)
    - p(p+1)/2 x^(p+2) for x < 1, else 0, with p = 5 (the text's value; the
    appendix config lists 6).
R5  Radial MLP [8, 64, 64, 64, P*K], bias-free, plain SiLU between layers.
R6  Neighbour sum divided by a model constant c_norm.
R7  Layer 0 applies the species-dependent linear to the message after the
    path-merging linear (no residual); layers t >= 1 add a species-dependent
    linear of h^t (residual) to the product linear's output.
R8  The product basis of the last layer outputs scalars only.
R9  Readouts act on the scalars of h^{t+1}: a K->1 linear for t < T-1, and
    K->16->SiLU->1 for the last layer, all bias-free.  E0 = 0, scale 1,
    shift 0.
R10 Every linear is y_k = sum_k' W[k', k] x_k'; weights are N(0,1)/sqrt(fan_in)
    (fan_in of a species-dependent linear = K; of a path-merging linear =
    number of paths into that l times K; of a product-basis weight block =
    number of couplings eta for that (nu, L)).
R11 BF16-linear mode (emulation): inputs and weights of the channel-mixing
    linears (linear_up, path-merging linear, species linears, product linear,
    readout linears) rounded to bfloat16 (round to nearest even); all sums
    and every other step in FP64. FP16-linear mode: the same with IEEE
    binary16 (round to nearest even, overflow to infinity).
R12 Stress: the NPT metrics paragraph takes the pressure as -tr(sigma)/3 and
    does not define sigma. Here sigma = (1/V) dE/d(epsilon) for a homogeneous
    strain acting on row vectors, x -> x (I + epsilon), on positions and cell
    rows alike; V = |det cell|, or 1 for a graph without a cell.
R13 BF16-radial mode (emulation): BF16-linear, and the last product of the
    radial MLP takes bfloat16-rounded inputs and weights.
    In both 16-bit emulations autograd differentiates the rounding as a cast:
    the gradient that flows back into a rounded operand is itself rounded to
    the same format (after the FP64 transposed product), whereas the library
    rounds the incoming gradient before its transposed product. Both are
    16-bit backward passes; they differ by rounding order only.
"""
from __future__ import annotations

import math
from dataclasses import dataclass, field

import numpy as np
import torch

from . import so3
from .neighbors import neighbor_list

DT = torch.float64


@dataclass(frozen=True)
class ModelDesc:
    n_species: int
    K: int
    hidden_lmax: int | tuple    # lmax of the hidden irreps leaving non-last layers (one, or one per layer)
    r_cut: float
    c_norm: float
    n_layers: int = 2
    sh_lmax: int = 3
    correlation: int = 3
    n_bessel: int = 8
    envelope_p: int = 5
    radial_hidden: tuple = (64, 64, 64)
    readout_hidden: int = 16


def hidden_lmax_of(d: ModelDesc, t: int) -> int:
    """lmax of the hidden irreps leaving layer t (t < n_layers - 1)."""
    return d.hidden_lmax if isinstance(d.hidden_lmax, int) else int(d.hidden_lmax[t])


def layer_in_ls(d: ModelDesc, t: int):
    return [0] if t == 0 else list(range(hidden_lmax_of(d, t - 1) + 1))


def layer_out_ls(d: ModelDesc, t: int):
    return [0] if t == d.n_layers - 1 else list(range(hidden_lmax_of(d, t) + 1))


def tp_paths(d: ModelDesc, t: int):
    """Edge tensor-product paths (l_h, l_Y, l_out), reading R2."""
    paths = []
    for lh in layer_in_ls(d, t):
        for ly in range(d.sh_lmax + 1):
            for lo in range(abs(lh - ly), min(lh + ly, d.sh_lmax) + 1):
                if (lh + ly + lo) % 2 == 0:
                    paths.append((lh, ly, lo))
    return paths


def weight_layout(d: ModelDesc):
    """[(name, shape, fan_in)] in blob order."""
    S, K = d.n_species, d.K
    lay = [("embed", (S, K), S)]
    for t in range(d.n_layers):
        in_ls, out_ls = layer_in_ls(d, t), layer_out_ls(d, t)
        paths = tp_paths(d, t)
        P = len(paths)
        for l in in_ls:
            lay.append((f"{t}.up.{l}", (K, K), K))
        h = (d.n_bessel,) + tuple(d.radial_hidden)
        for i in range(len(h) - 1):
            lay.append((f"{t}.radial.{i}", (h[i], h[i + 1]), h[i]))
        lay.append((f"{t}.radial.{len(h) - 1}", (h[-1], P * K), h[-1]))
        for p, (lh, ly, lo) in enumerate(paths):
            n_in = sum(1 for q in paths if q[2] == lo)
            lay.append((f"{t}.linear.{p}", (K, K), n_in * K))
        if t == 0:
            for l in range(d.sh_lmax + 1):
                lay.append((f"{t}.skip.{l}", (S, K, K), K))
        else:
            for L in out_ls:
                if L in in_ls:
                    lay.append((f"{t}.skip.{L}", (S, K, K), K))
        for L in out_ls:
            for nu in range(1, d.correlation + 1):
                ne = so3.n_eta(nu, L)
                if ne:
                    lay.append((f"{t}.symc.{L}.{nu}", (S, ne, K), ne))
        for L in out_ls:
            lay.append((f"{t}.prod.{L}", (K, K), K))
        if t < d.n_layers - 1:
            lay.append((f"{t}.readout", (K,), K))
        else:
            lay.append((f"{t}.readout.0", (K, d.readout_hidden), K))
            lay.append((f"{t}.readout.1", (d.readout_hidden,), d.readout_hidden))
    return lay


def unpack_weights(d: ModelDesc, blob: np.ndarray):
    out, o = {}, 0
    for name, shape, _ in weight_layout(d):
        n = int(np.prod(shape))
        out[name] = torch.from_numpy(np.asarray(blob[o:o + n], dtype=np.float64).reshape(shape).copy())
        o += n
    if o != len(blob):
        raise ValueError(f"weight blob has {len(blob)} floats, layout needs {o}")
    return out


# --------------------------------------------------------------------------
# per-edge features (Eq. 26 ingredients)
# --------------------------------------------------------------------------

def envelope(x: torch.Tensor, p: int) -> torch.Tensor:
    """Polynomial cutoff envelope, reading R4."""
    v = (1.0 - (p + 1) * (p + 2) / 2.0 * x ** p + p * (p + 2) * x ** (p + 1)
         - p * (p + 1) / 2.0 * x ** (p + 2))
    return torch.where(x < 1.0, v, torch.zeros_like(x))


def bessel_basis(r: torch.Tensor, r_cut: float, n_basis: int, p: int) -> torch.Tensor:
    """e_n(r), n = 1..n_basis, reading R4 -> [E, n_basis]."""
    n = torch.arange(1, n_basis + 1, dtype=r.dtype)
    b = math.sqrt(2.0 / r_cut) * torch.sin(n[None, :] * math.pi * r[:, None] / r_cut) / r[:, None]
    return b * envelope(r / r_cut, p)[:, None]


def silu(x):
    return x * torch.sigmoid(x)


def radial_mlp(e: torch.Tensor, W: dict, t: int, n_hidden: int, bf16_last: bool = False,
               rnd=None) -> torch.Tensor:
    """Reading R5: e @ W0 -> SiLU -> ... -> @ W_last (with bf16_last, the last
    product takes bfloat16-rounded inputs and weights, R13). rnd (a rounding
    from _rounding: the per-block precision study's radial-MLP block) rounds
    the input and the weights of every layer, the basis e included."""
    r = rnd if rnd is not None else (lambda x: x)
    h = e
    for i in range(n_hidden):
        h = silu(r(h) @ r(W[f"{t}.radial.{i}"]))
    Wl = W[f"{t}.radial.{n_hidden}"]
    if bf16_last:
        return _round_bf16(r(h)) @ _round_bf16(r(Wl))
    return r(h) @ r(Wl)


# --------------------------------------------------------------------------
# model
# --------------------------------------------------------------------------

def _round_bf16(x: torch.Tensor) -> torch.Tensor:
    return x.to(torch.bfloat16).to(DT)


def _round_fp16(x: torch.Tensor) -> torch.Tensor:
    return x.to(torch.float16).to(DT)


def _rounding(fmt):
    """Operand rounding of one block for the per-block precision study:
    None (FP64), "bf16" or "fp16" (round to nearest even; the arithmetic and
    every sum stay FP64). Gradients pass through the rounding unchanged
    (x + (round(x) - x) with the difference held constant: the value is
    round(x) exactly, the derivative 1)."""
    if fmt is None:
        return lambda x: x
    r = {"bf16": _round_bf16, "fp16": _round_fp16}[fmt]
    return lambda x: x + (r(x) - x).detach()


class _Lin:
    """Channel-mixing linear y = x @ W with optional BF16 or FP16 emulation
    of its inputs and weights (R11)."""

    def __init__(self, bf16: bool, fp16: bool = False):
        assert not (bf16 and fp16)
        self.round = _round_bf16 if bf16 else (_round_fp16 if fp16 else None)

    def __call__(self, x, W):
        if self.round is not None:
            return self.round(x) @ self.round(W)
        return x @ W

    def species(self, x, W, z):
        """x [N, c, K], W [S, K, K], z [N]: y[n] = x[n] @ W[z[n]]."""
        Wz = W[z]
        if self.round is not None:
            return torch.bmm(self.round(x), self.round(Wz))
        return torch.bmm(x, Wz)


def symmetric_contraction(A: torch.Tensor, W: dict, t: int, L: int, z: torch.Tensor,
                          correlation: int, chunk: int = 64, rnd=None) -> torch.Tensor:
    """Eq. 27 + message: B_{n,k,M} = sum_nu sum_eta W^{nu}_{z_n,L}[eta,k]
    sum_{a_1..a_nu} U^{nu,L}_eta[M, a_1..a_nu] prod_xi A_{n,k,a_xi}.

    A: [N, 16, K] -> [N, 2L+1, K].  Dense U, node chunks to bound memory.
    rnd: optional rounding of the operands A and W (the U constants are not
    rounded).
    """
    rnd = rnd or (lambda x: x)
    A = rnd(A)
    N, ncomp, K = A.shape
    outs = []
    Us = {}
    for nu in range(1, correlation + 1):
        _trees, us = so3.u_basis(nu, L)
        if us:
            Us[nu] = torch.from_numpy(np.stack(us).reshape(len(us) * (2 * L + 1), -1))
    for c0 in range(0, N, chunk):
        a = A[c0:c0 + chunk].transpose(1, 2)                  # [n, K, 16]
        n = a.shape[0]
        zc = z[c0:c0 + chunk]
        acc = torch.zeros(n, K, 2 * L + 1, dtype=DT)
        mono = None
        for nu in range(1, correlation + 1):
            mono = a if nu == 1 else (mono[..., :, None] * a[..., None, :]).reshape(n, K, -1)
            if nu not in Us:
                continue
            ne = Us[nu].shape[0] // (2 * L + 1)
            Bnu = (mono @ Us[nu].T).reshape(n, K, ne, 2 * L + 1)   # [n,K,eta,M]
            w = rnd(W[f"{t}.symc.{L}.{nu}"][zc])                     # [n, eta, K]
            acc = acc + torch.einsum("nkem,nek->nkm", Bnu, w)
        outs.append(acc.transpose(1, 2))
    return torch.cat(outs, dim=0)


@dataclass
class Graph:
    sender: torch.Tensor
    receiver: torch.Tensor
    shift_vec: torch.Tensor     # [E,3] float64 (S . cell)
    species: torch.Tensor
    graph_of_atom: torch.Tensor
    n_graphs: int


def build_graph(system, d: ModelDesc) -> Graph:
    s, r, S = neighbor_list(system.positions, d.r_cut, system.cells, system.graph_of_atom)
    if system.cells is not None and len(s):
        g = system.graph_of_atom[r]
        cells = np.asarray(system.cells, dtype=np.float64)[g]          # [E,3,3]
        Sf = S.astype(np.float64)
        sv = ((Sf[:, 0:1] * cells[:, 0]) + (Sf[:, 1:2] * cells[:, 1])) + (Sf[:, 2:3] * cells[:, 2])
    else:
        sv = np.zeros((len(s), 3))
    return Graph(torch.from_numpy(s), torch.from_numpy(r), torch.from_numpy(sv),
                 torch.from_numpy(np.asarray(system.species, dtype=np.int64)),
                 torch.from_numpy(np.asarray(system.graph_of_atom, dtype=np.int64)),
                 int(system.n_graphs))


def _edge_features(d: ModelDesc, graph: Graph, pos: torch.Tensor, sl=slice(None)):
    """Y [e,16] and the radial basis [e, n_basis] of the edges in slice sl
    (graph problem statement; reading R3 for the edge vector)."""
    snd, rcv = graph.sender[sl], graph.receiver[sl]
    vec = pos[snd] + graph.shift_vec[sl] - pos[rcv]                      # R3
    r = torch.sqrt((vec * vec).sum(-1))
    u = vec / r[:, None]
    Y = so3.sh_all(u, d.sh_lmax)                                         # [e,16]
    rb = bessel_basis(r, d.r_cut, d.n_bessel, d.envelope_p)              # [e,8]
    return Y, rb


def _edge_messages(d: ModelDesc, W: dict, t: int, ht: dict, snd: torch.Tensor, Y: torch.Tensor,
                   rb: torch.Tensor, bf16_radial: bool = False, rtp=None, rrad=None):
    """Eq. 26 before the neighbour sum, per path p = (l_h, l_Y, l_out):
    m[e, m3, k] = R[e, p, k] sum_{m1, m2} C[m1, m2, m3] ht[s_e, m1, k] Y[e, m2]
    for the edges whose senders, harmonics and radial basis are given.
    Returns a list over paths of [e, 2 l_out + 1, K]."""
    rtp = rtp or (lambda x: x)
    paths = tp_paths(d, t)
    R = rtp(radial_mlp(rb, W, t, len(d.radial_hidden), bf16_radial, rnd=rrad).reshape(-1, len(paths), d.K))
    out = []
    for p, (lh, ly, lo) in enumerate(paths):
        C = torch.from_numpy(so3.real_cg(lh, ly, lo))
        hs = rtp(ht[lh][snd])                                             # [e, 2lh+1, K]
        Yl = rtp(Y[:, ly * ly: ly * ly + 2 * ly + 1])                     # [e, 2ly+1]
        out.append(torch.einsum("abc,eak,eb->eck", C, hs, Yl) * R[:, p, None, :])
    return out


def _linear_up(d: ModelDesc, W: dict, t: int, h: dict, lin) -> dict:
    """Eq. 26's sender features W h^t, per l of the layer's input."""
    return {l: lin(h[l], W[f"{t}.up.{l}"]) for l in layer_in_ls(d, t)}


def _node_update(d: ModelDesc, W: dict, t: int, At: list, h: dict, z: torch.Tensor, lin, rsc=None):
    """Everything of layer t after the neighbour sum, node by node: the
    path-merging linear, the species linear (layer 0) or residual (t >= 1,
    R7), the product basis (Eq. 27) with its weights, the product linear and
    the layer's readout. At: per path [n, 2 l_out + 1, K], already divided
    by c_norm; h: the layer's input features. Returns (h^{t+1}, eps_t [n])."""
    in_ls, out_ls = layer_in_ls(d, t), layer_out_ls(d, t)
    paths = tp_paths(d, t)
    K = d.K
    n = z.shape[0]
    sc = {}
    if t > 0:
        for L in out_ls:
            if L in in_ls:
                sc[L] = lin.species(h[L], W[f"{t}.skip.{L}"], z)
    A = []
    for l in range(d.sh_lmax + 1):
        acc = torch.zeros(n, 2 * l + 1, K, dtype=DT)
        for p, (_, _, lo) in enumerate(paths):
            if lo == l:
                acc = acc + lin(At[p], W[f"{t}.linear.{p}"])
        A.append(acc)
    if t == 0:                                                             # R7
        A = [lin.species(A[l], W[f"{t}.skip.{l}"], z) for l in range(d.sh_lmax + 1)]
    Afull = torch.cat(A, dim=1)                                            # [n,16,K]
    hn = {}
    for L in out_ls:
        B = symmetric_contraction(Afull, W, t, L, z, d.correlation, rnd=rsc)
        hn[L] = lin(B, W[f"{t}.prod.{L}"])
        if L in sc:
            hn[L] = hn[L] + sc[L]
    s0 = hn[0][:, 0, :]                                                    # [n,K]
    if t < d.n_layers - 1:
        e_t = lin(s0, W[f"{t}.readout"][:, None])[:, 0]
    else:
        hid = silu(lin(s0, W[f"{t}.readout.0"]))
        e_t = lin(hid, W[f"{t}.readout.1"][:, None])[:, 0]
    return hn, e_t, Afull


def node_energies(d: ModelDesc, W: dict, graph: Graph, pos: torch.Tensor,
                  bf16_linear: bool = False, edge_chunk: int = 1 << 16,
                  return_intermediates: bool = False, fp16_linear: bool = False, bf16_radial: bool = False,
                  tp_round=None, symcon_round=None, radial_round=None):
    """Per-atom energies eps_i [N] for positions pos [N,3] (float64).

    tp_round / symcon_round / radial_round ("bf16", "fp16" or None) round the
    operands of one block for the per-block precision study: the edge
    product's sender features, harmonics and radial weights (not the CG
    constants), the symmetric contraction's A and weights (not U), or every
    radial-MLP layer's input and weights."""
    lin = _Lin(bf16_linear, fp16_linear)
    rtp, rsc, rrad = _rounding(tp_round), _rounding(symcon_round), _rounding(radial_round)
    z = graph.species
    N = pos.shape[0]
    K = d.K
    snd, rcv = graph.sender, graph.receiver
    E = len(snd)
    Y, rb = _edge_features(d, graph, pos)
    inter = {"Y": Y, "rbf": rb}

    # node embedding: linear on one-hot species
    h = {0: W["embed"][z][:, None, :]}                                   # {l: [N, 2l+1, K]}
    eps = torch.zeros(N, dtype=DT)
    for t in range(d.n_layers):
        paths = tp_paths(d, t)
        ht = _linear_up(d, W, t, h, lin)                                  # linear_up
        At = [torch.zeros(N, 2 * lo + 1, K, dtype=DT) for (_, _, lo) in paths]
        for e0 in range(0, E, edge_chunk):
            sl = slice(e0, e0 + edge_chunk)
            msg = _edge_messages(d, W, t, ht, snd[sl], Y[sl], rb[sl], bf16_radial, rtp, rrad)
            for p in range(len(paths)):
                At[p] = At[p].index_add(0, rcv[sl], msg[p])
        At = [a / d.c_norm for a in At]                                   # R6
        hn, e_t, Afull = _node_update(d, W, t, At, h, z, lin, rsc)
        eps = eps + e_t
        if return_intermediates:
            inter[f"{t}.A"] = Afull
            inter[f"{t}.h"] = hn
        h = hn
    if return_intermediates:
        return eps, inter
    return eps


def energy_forces_chunked(d: ModelDesc, blob: np.ndarray, system, graph: Graph | None = None,
                          bf16_linear: bool = False, fp16_linear: bool = False, edge_chunk: int = 1 << 15,
                          node_chunk: int = 256):
    """Energies and forces of large graphs in bounded memory, by a two-pass
    vector-Jacobian product over edge and node chunks.

    The neighbour sum of Eq. 26 is linear in the edge messages, so with
    g_t = dE/dAt_t known at the nodes, the gradient reaching edge e is
    g_t[r_e] / c_norm and the edges can be back-propagated chunk by chunk;
    every step after the neighbour sum acts node by node, so its backward
    runs in node chunks. Pass 1 (no gradients) evaluates the model as
    node_energies does and keeps each layer's input h^t and summed messages
    At_t. Pass 2 walks the layers from the last: the node-level backward
    of layer t gives dE/dAt_t and the direct part of dE/dh^t (residual);
    the edge chunks, recomputed with gradients, give dE/dpos (through the
    harmonics and the radial basis) and dE/d(W h^t) at the senders, which
    linear_up carries back to h^t and on to layer t-1. F = -dE/dpos
    (force equation). Same arithmetic as energy_forces up to summation
    order. Returns dict(eps, energy, forces, graph)."""
    W = unpack_weights(d, blob)
    if graph is None:
        graph = build_graph(system, d)
    lin = _Lin(bf16_linear, fp16_linear)
    z = graph.species
    snd, rcv = graph.sender, graph.receiver
    N, E, K = len(z), len(snd), d.K
    pos0 = torch.tensor(system.positions, dtype=DT)
    echunks = [slice(e0, min(e0 + edge_chunk, E)) for e0 in range(0, E, edge_chunk)]
    nchunks = [slice(n0, min(n0 + node_chunk, N)) for n0 in range(0, N, node_chunk)]

    def node_slice(At, h, sl):
        return [a[sl] for a in At], {l: v[sl] for l, v in h.items()}

    # pass 1: forward, no gradients
    hs, Ats = [], []
    eps = torch.zeros(N, dtype=DT)
    with torch.no_grad():
        h = {0: W["embed"][z][:, None, :]}
        for t in range(d.n_layers):
            paths = tp_paths(d, t)
            ht = _linear_up(d, W, t, h, lin)
            At = [torch.zeros(N, 2 * lo + 1, K, dtype=DT) for (_, _, lo) in paths]
            for sl in echunks:
                Y, rb = _edge_features(d, graph, pos0, sl)
                msg = _edge_messages(d, W, t, ht, snd[sl], Y, rb)
                for p in range(len(paths)):
                    At[p].index_add_(0, rcv[sl], msg[p])
            At = [a / d.c_norm for a in At]
            hn = {l: [] for l in layer_out_ls(d, t)}
            for sl in nchunks:
                a_s, h_s = node_slice(At, h, sl)
                hn_s, e_s, _ = _node_update(d, W, t, a_s, h_s, z[sl], lin)
                for l in hn:
                    hn[l].append(hn_s[l])
                eps[sl] += e_s
            hs.append(h)
            Ats.append(At)
            h = {l: torch.cat(v, dim=0) for l, v in hn.items()}

    # pass 2: backward, last layer first
    pos = pos0.clone().requires_grad_(True)
    g_next = None                                                         # dE/dh^{t+1}
    for t in reversed(range(d.n_layers)):
        paths = tp_paths(d, t)
        in_ls = layer_in_ls(d, t)
        h = hs[t]
        gAt = [torch.zeros_like(a) for a in Ats[t]]
        gh = {l: torch.zeros_like(h[l]) for l in in_ls}
        for sl in nchunks:
            a_s, h_s = node_slice(Ats[t], h, sl)
            a_s = [a.clone().requires_grad_(True) for a in a_s]
            h_s = {l: v.clone().requires_grad_(True) for l, v in h_s.items()}
            hn_s, e_s, _ = _node_update(d, W, t, a_s, h_s, z[sl], lin)
            L = e_s.sum()
            if g_next is not None:
                for l, v in hn_s.items():
                    L = L + (v * g_next[l][sl]).sum()
            leaves = a_s + [h_s[l] for l in in_ls]
            grads = torch.autograd.grad(L, leaves, allow_unused=True)
            for p in range(len(paths)):
                if grads[p] is not None:
                    gAt[p][sl] = grads[p]
            for j, l in enumerate(in_ls):
                if grads[len(paths) + j] is not None:
                    gh[l][sl] = grads[len(paths) + j]
        # the edge chunks: messages recomputed with gradients, contracted with
        # dE/dAt at their receivers (the adjoint of the neighbour sum)
        h_leaf = {l: h[l].clone().requires_grad_(True) for l in in_ls}
        ht = _linear_up(d, W, t, h_leaf, lin)
        ht_leaf = {l: v.detach().clone().requires_grad_(True) for l, v in ht.items()}
        for sl in echunks:
            Y, rb = _edge_features(d, graph, pos, sl)
            msg = _edge_messages(d, W, t, ht_leaf, snd[sl], Y, rb)
            r_s = rcv[sl]
            L = sum((msg[p] * gAt[p][r_s]).sum() for p in range(len(paths))) / d.c_norm
            L.backward()
        if t > 0:
            gup = torch.autograd.grad([ht[l] for l in in_ls], [h_leaf[l] for l in in_ls],
                                      grad_outputs=[ht_leaf[l].grad for l in in_ls], allow_unused=True)
            g_next = {l: gh[l] + (gup[j] if gup[j] is not None else 0.0) for j, l in enumerate(in_ls)}
    F = -pos.grad if pos.grad is not None else torch.zeros_like(pos0)
    Eg = torch.zeros(graph.n_graphs, dtype=DT).index_add(0, graph.graph_of_atom, eps)
    return {"eps": eps.numpy(), "energy": Eg.numpy(), "forces": F.detach().numpy(), "graph": graph}


def contraction_order_shares(d: ModelDesc, blob: np.ndarray, system, graph: Graph | None = None,
                             node_chunk: int = 256):
    """Share of each correlation order nu in the product basis of Eq. 27,
    share[t][L][nu] = sum |B_nu| / sum_nu' sum |B_nu'| over nodes, channels
    and components, B_nu being the nu-th term of the sum over correlation
    orders (weights of the other orders set to zero). A parity case that
    claims to exercise Eq. 27 beyond nu = 1 needs every share to be
    non-negligible."""
    W = unpack_weights(d, blob)
    if graph is None:
        graph = build_graph(system, d)
    z = graph.species
    N = len(z)
    pos = torch.tensor(system.positions, dtype=DT)
    with torch.no_grad():
        _, inter = node_energies(d, W, graph, pos, return_intermediates=True)
    out = {}
    for t in range(d.n_layers):
        A = inter[f"{t}.A"]
        out[t] = {}
        for L in layer_out_ls(d, t):
            tot = {}
            for nu in range(1, d.correlation + 1):
                if not so3.n_eta(nu, L):
                    continue
                Wn = dict(W)
                for mu in range(1, d.correlation + 1):
                    if mu != nu and so3.n_eta(mu, L):
                        Wn[f"{t}.symc.{L}.{mu}"] = torch.zeros_like(W[f"{t}.symc.{L}.{mu}"])
                s = 0.0
                for n0 in range(0, N, node_chunk):
                    sl = slice(n0, n0 + node_chunk)
                    s += float(symmetric_contraction(A[sl], Wn, t, L, z[sl], d.correlation).abs().sum())
                tot[nu] = s
            S = sum(tot.values())
            out[t][L] = {nu: v / S for nu, v in tot.items()}
    return out


def graph_energies(eps: torch.Tensor, graph: Graph) -> torch.Tensor:
    return torch.zeros(graph.n_graphs, dtype=DT).index_add(0, graph.graph_of_atom, eps)


def energy_forces(d: ModelDesc, blob: np.ndarray, system, graph: Graph | None = None,
                  bf16_linear: bool = False, forces: bool = True, fp16_linear: bool = False,
                  bf16_radial: bool = False, tp_round=None, symcon_round=None, radial_round=None):
    """Returns dict(eps [N], energy [G], forces [N,3] or None, graph)."""
    W = unpack_weights(d, blob)
    if graph is None:
        graph = build_graph(system, d)
    pos = torch.tensor(system.positions, dtype=DT, requires_grad=forces)
    eps = node_energies(d, W, graph, pos, bf16_linear=bf16_linear, fp16_linear=fp16_linear,
                        bf16_radial=bf16_radial, tp_round=tp_round, symcon_round=symcon_round,
                        radial_round=radial_round)
    Eg = graph_energies(eps, graph)
    F = None
    if forces:
        # F = -dE/dr; with no edge at all E does not depend on r and F = 0
        g = None
        if Eg.requires_grad:
            (g,) = torch.autograd.grad(Eg.sum(), pos, allow_unused=True)
        F = -g if g is not None else torch.zeros_like(pos)
    return {"eps": eps.detach().numpy(), "energy": Eg.detach().numpy(),
            "forces": None if F is None else F.numpy(), "graph": graph}


def stress(d: ModelDesc, blob: np.ndarray, system, graph: Graph | None = None,
           bf16_linear: bool = False, fp16_linear: bool = False, bf16_radial: bool = False):
    """Stress of every graph, sigma_g = (1/V_g) dE_g/d(epsilon_g) [G,3,3].

    The pressure of the NPT metrics paragraph is p = -tr(sigma)/3. A
    homogeneous strain epsilon acts on row vectors, x -> x (I + epsilon), on
    the positions of the graph's atoms and on the rows of its cell (so every
    periodic shift S.cell transforms the same way); the derivative is taken
    at epsilon = 0 by autograd. V_g = |det cell_g|; a graph without a cell
    gets V = 1, i.e. the bare strain derivative.
    """
    W = unpack_weights(d, blob)
    if graph is None:
        graph = build_graph(system, d)
    G = graph.n_graphs
    strain = torch.zeros(G, 3, 3, dtype=DT, requires_grad=True)
    Fm = torch.eye(3, dtype=DT)[None] + strain                           # [G,3,3]
    pos0 = torch.tensor(system.positions, dtype=DT)
    pos = torch.einsum("na,nab->nb", pos0, Fm[graph.graph_of_atom])
    g_edge = graph.graph_of_atom[graph.receiver]
    shifted = Graph(graph.sender, graph.receiver, torch.einsum("ea,eab->eb", graph.shift_vec, Fm[g_edge]),
                    graph.species, graph.graph_of_atom, graph.n_graphs)
    eps = node_energies(d, W, shifted, pos, bf16_linear=bf16_linear, fp16_linear=fp16_linear,
                        bf16_radial=bf16_radial)
    Eg = graph_energies(eps, graph)
    dE = None
    if Eg.requires_grad:
        (dE,) = torch.autograd.grad(Eg.sum(), strain, allow_unused=True)
    dE = torch.zeros(G, 3, 3, dtype=DT) if dE is None else dE.detach()
    if system.cells is not None:
        vol = torch.tensor([abs(np.linalg.det(np.asarray(c, dtype=np.float64))) for c in system.cells], dtype=DT)
    else:
        vol = torch.ones(G, dtype=DT)
    return (dE / vol[:, None, None]).numpy()

