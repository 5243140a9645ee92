"""ctypes binding of libmace_amd.so: the C entry points under the same names,
argument marshalling only.  Every step of the path runs in the library's
HIP kernels; PyTorch only provides device memory and the stream.

Loading fails loudly when the library has not been built (there is no
fallback implementation).
"""
from __future__ import annotations

import ctypes
import os

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libmace_amd.so")

MACE_FP32 = 0
MACE_BF16_LINEAR = 1
MACE_FP16_LINEAR = 2
MACE_BF16_RADIAL = 3
MACE_FP64 = 4
MACE_L0_AUTO = 0
MACE_L0_EDGE = 1
MACE_L0_FACTORED = 2
MACE_PRODUCTS_FP32 = 0
MACE_PRODUCTS_SPLIT_BF16 = 2
MACE_BLOCK_EDGE_PRODUCT = 0
MACE_BLOCK_SYMMETRIC_CONTRACTION = 1
MACE_BLOCK_RADIAL_MLP = 2
MACE_NEIGHBOR_SCRATCH_BYTES = 80 << 20
MAX_LAYERS = 8   # MACE_MAX_LAYERS
STATUS = {0: "MACE_OK", -1: "MACE_EINVAL", -2: "MACE_ERANGE", -3: "MACE_ENOSPACE", -4: "MACE_EHIP",
          -5: "MACE_ENONFINITE", -6: "MACE_ESTATE", -7: "MACE_EUNSUPPORTED"}

EXPORTED = ["mace_weight_layout", "mace_workspace_bytes", "mace_neighbor_list", "mace_graph_setup",
            "mace_forward_energy", "mace_forces", "mace_forces_stress", "mace_graph_destroy", "mace_status_string",
            "mace_debug_real_cg", "mace_debug_trees", "mace_debug_edge_features", "mace_profile_select",
            "mace_profile_read", "mace_kernel_name", "mace_graph_check", "mace_profile_work",
            "mace_neighbor_workspace_bytes", "mace_neighbor_list_device", "mace_layer0_form",
            "mace_fp32_products", "mace_block_rounding", "mace_neighbor_list_device_noalloc",
            "mace_debug_fused_linears"]


class MaceError(RuntimeError):
    def __init__(self, code: int, where: str):
        super().__init__(f"{where}: {STATUS.get(code, code)}")
        self.code = code


class mace_model_desc(ctypes.Structure):
    _fields_ = [("n_species", ctypes.c_int32), ("K", ctypes.c_int32), ("n_layers", ctypes.c_int32),
                ("sh_lmax", ctypes.c_int32), ("correlation", ctypes.c_int32), ("n_bessel", ctypes.c_int32),
                ("envelope_p", ctypes.c_int32), ("radial_hidden", ctypes.c_int32 * 3),
                ("readout_hidden", ctypes.c_int32), ("hidden_lmax", ctypes.c_int32 * MAX_LAYERS),
                ("r_cut", ctypes.c_double), ("c_norm", ctypes.c_double)]


def make_desc(n_species, K, hidden_lmax, r_cut, c_norm, n_layers=2, sh_lmax=3, correlation=3, n_bessel=8,
              envelope_p=5, radial_hidden=(64, 64, 64), readout_hidden=16) -> mace_model_desc:
    d = mace_model_desc()
    d.n_species, d.K, d.n_layers = n_species, K, n_layers
    d.sh_lmax, d.correlation, d.n_bessel, d.envelope_p = sh_lmax, correlation, n_bessel, envelope_p
    d.radial_hidden[:] = list(radial_hidden)
    d.readout_hidden = readout_hidden
    # one l_max for every non-last layer, or one per layer
    hl = [hidden_lmax] * (n_layers - 1) if isinstance(hidden_lmax, (int, np.integer)) else list(hidden_lmax)
    if len(hl) < n_layers - 1 or n_layers > MAX_LAYERS:
        raise ValueError("hidden_lmax needs an entry per non-last layer, at most MACE_MAX_LAYERS layers")
    d.hidden_lmax[:] = (hl + [0] * MAX_LAYERS)[:MAX_LAYERS]
    d.r_cut, d.c_norm = float(r_cut), float(c_norm)
    return d


_lib = None


def lib() -> ctypes.CDLL:
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise ImportError(f"{LIB_PATH} is missing: build it with paper_2510_23621_amd.build.build()")
        L = ctypes.CDLL(LIB_PATH)
        P, I32, I64, D, Z = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_double, ctypes.c_size_t
        dp = ctypes.POINTER(mace_model_desc)
        L.mace_weight_layout.argtypes = [dp, I32, P, P, P, I32, P, P]
        L.mace_workspace_bytes.argtypes = [dp, I64, I64, I32, I32]
        L.mace_workspace_bytes.restype = Z
        L.mace_neighbor_list.argtypes = [I64, P, P, P, I32, D, I64, P, P, P, P]
        L.mace_neighbor_workspace_bytes.argtypes = [I64, P, P, I32, D]
        L.mace_neighbor_workspace_bytes.restype = Z
        L.mace_neighbor_list_device.argtypes = [I64, P, P, P, I32, D, I64, P, P, P, P, P, Z, P]
        L.mace_neighbor_list_device_noalloc.argtypes = [I64, P, P, P, I32, D, I64, P, P, P, P, P]
        L.mace_graph_setup.argtypes = [dp, P, I64, I64, P, I64, P, P, P, P, I32, I32, P, Z, P, P]
        L.mace_forward_energy.argtypes = [P, P, P, P, P]
        L.mace_forces.argtypes = [P, P, P, P, P, P]
        L.mace_forces_stress.argtypes = [P, P, P, P, P, P, P]
        L.mace_graph_destroy.argtypes = [P]
        L.mace_graph_check.argtypes = [P, P, P]
        L.mace_profile_work.argtypes = [P, P, P]
        L.mace_layer0_form.argtypes = [P, I32, P]
        L.mace_fp32_products.argtypes = [P, I32, P]
        L.mace_debug_fused_linears.argtypes = [P, I32, P]
        L.mace_block_rounding.argtypes = [P, I32, I32, P]
        L.mace_graph_destroy.restype = None
        L.mace_status_string.argtypes = [I32]
        L.mace_status_string.restype = ctypes.c_char_p
        L.mace_debug_real_cg.argtypes = [I32, I32, I32, P]
        L.mace_debug_trees.argtypes = [I32, I32, I32, I32, P, P, P]
        L.mace_debug_edge_features.argtypes = [I64, P, D, I32, I32, P, P]
        L.mace_profile_select.argtypes = [P, I32]
        L.mace_profile_read.argtypes = [P, P, P]
        L.mace_kernel_name.argtypes = [I32]
        L.mace_kernel_name.restype = ctypes.c_char_p
        for name in EXPORTED:
            f = getattr(L, name)
            if f.restype is ctypes.c_int:
                f.restype = I32
        _lib = L
    return _lib


def _check(code: int, where: str):
    if code != 0:
        raise MaceError(code, where)


def _ptr(x):
    """Device pointer of a torch tensor, host pointer of a numpy array, or None."""
    if x is None:
        return None
    if isinstance(x, np.ndarray):
        return x.ctypes.data
    return x.data_ptr()


def _stream(stream):
    if stream is None:
        import torch
        return torch.cuda.current_stream().cuda_stream
    return stream if isinstance(stream, int) else stream.cuda_stream


# ------------------------------------------------------------------ entry points

def mace_weight_layout(desc: mace_model_desc):
    """[(name, size, fan_in)] per tensor of the weight blob, and the total float count."""
    n = ctypes.c_int32()
    tot = ctypes.c_int64()
    code = lib().mace_weight_layout(ctypes.byref(desc), 0, None, None, None, 0, ctypes.byref(n),
                                    ctypes.byref(tot))
    if code not in (0, -3):
        raise MaceError(code, "mace_weight_layout")
    sizes = np.zeros(n.value, np.int64)
    fans = np.zeros(n.value, np.int64)
    width = 48
    names = ctypes.create_string_buffer(n.value * width)
    _check(lib().mace_weight_layout(ctypes.byref(desc), n.value, sizes.ctypes.data, fans.ctypes.data, names, width,
                                    ctypes.byref(n), ctypes.byref(tot)), "mace_weight_layout")
    raw = names.raw
    nm = [raw[i * width:(i + 1) * width].split(b"\0", 1)[0].decode() for i in range(n.value)]
    return list(zip(nm, sizes.tolist(), fans.tolist())), int(tot.value)


def mace_workspace_bytes(desc, n_atoms, n_edges, n_graphs, prec=MACE_FP32) -> int:
    return int(lib().mace_workspace_bytes(ctypes.byref(desc), n_atoms, n_edges, n_graphs, prec))


def mace_neighbor_list(positions: np.ndarray, r_cut: float, cells=None, graph_of_atom=None, n_graphs: int = 1):
    """(sender, receiver, shifts) int32 numpy arrays, canonical order."""
    pos = np.ascontiguousarray(positions, dtype=np.float64)
    cl = None if cells is None else np.ascontiguousarray(cells, dtype=np.float64)
    goa = None if graph_of_atom is None else np.ascontiguousarray(graph_of_atom, dtype=np.int32)
    ne = ctypes.c_int64()
    L = lib()
    code = L.mace_neighbor_list(len(pos), _ptr(pos), _ptr(cl), _ptr(goa), n_graphs, float(r_cut), 0,
                                None, None, None, ctypes.byref(ne))
    if code not in (0, -3):
        raise MaceError(code, "mace_neighbor_list")
    E = ne.value
    snd = np.zeros(E, np.int32)
    rcv = np.zeros(E, np.int32)
    sh = np.zeros((E, 3), np.int32)
    _check(L.mace_neighbor_list(len(pos), _ptr(pos), _ptr(cl), _ptr(goa), n_graphs, float(r_cut), E,
                                _ptr(snd), _ptr(rcv), _ptr(sh), ctypes.byref(ne)), "mace_neighbor_list")
    return snd, rcv, sh


def mace_neighbor_workspace_bytes(n_atoms: int, r_cut: float, cells=None, graph_offsets=None, n_graphs: int = 1) -> int:
    cl = None if cells is None else np.ascontiguousarray(cells, dtype=np.float64)
    go = None if graph_offsets is None else np.ascontiguousarray(graph_offsets, dtype=np.int32)
    return int(lib().mace_neighbor_workspace_bytes(int(n_atoms), _ptr(cl), _ptr(go), int(n_graphs), float(r_cut)))


def mace_neighbor_list_device(positions, r_cut: float, cells=None, graph_offsets=None, n_graphs: int = 1,
                              max_edges=None, stream=None):
    """Device neighbour list. positions: float64 device tensor [N, 3]; cells
    (host numpy [G, 3, 3]) or None; graph_offsets (host numpy int32 [G+1]) or
    None. Returns (sender, receiver, shifts) int32 device tensors. With
    max_edges None the count is taken first (one extra call)."""
    import torch
    N = int(positions.shape[0])
    cl = None if cells is None else np.ascontiguousarray(cells, dtype=np.float64)
    go = None if graph_offsets is None else np.ascontiguousarray(graph_offsets, dtype=np.int32)
    nbytes = mace_neighbor_workspace_bytes(N, r_cut, cl, go, n_graphs)
    if nbytes == 0:
        raise MaceError(-1, "mace_neighbor_workspace_bytes")
    ws = torch.empty(nbytes, dtype=torch.uint8, device=positions.device)
    ne = ctypes.c_int64()
    L = lib()

    def call(cap, snd, rcv, sh):
        return L.mace_neighbor_list_device(N, _ptr(positions), _ptr(cl), _ptr(go), int(n_graphs), float(r_cut), cap,
                                           _ptr(snd), _ptr(rcv), _ptr(sh), ctypes.byref(ne), _ptr(ws), nbytes,
                                           _stream(stream))
    if max_edges is None:
        code = call(0, None, None, None)
        if code not in (0, -3):
            raise MaceError(code, "mace_neighbor_list_device")
        max_edges = ne.value
    snd = torch.empty(max(max_edges, 1), dtype=torch.int32, device=positions.device)
    rcv = torch.empty_like(snd)
    sh = torch.empty(max(max_edges, 1), 3, dtype=torch.int32, device=positions.device)
    _check(call(max_edges, snd, rcv, sh), "mace_neighbor_list_device")
    E = ne.value
    return snd[:E], rcv[:E], sh[:E]


def mace_neighbor_list_device_noalloc(positions, r_cut: float, cells=None, graph_offsets=None, n_graphs: int = 1,
                                      max_edges=None, stream=None):
    """As mace_neighbor_list_device, through the entry point that takes no
    workspace (the library's static device scratch): allocates nothing on the
    device itself; the output tensors are allocated here, by torch."""
    import torch
    N = int(positions.shape[0])
    cl = None if cells is None else np.ascontiguousarray(cells, dtype=np.float64)
    go = None if graph_offsets is None else np.ascontiguousarray(graph_offsets, dtype=np.int32)
    ne = ctypes.c_int64()
    L = lib()

    def call(cap, snd, rcv, sh):
        return L.mace_neighbor_list_device_noalloc(N, _ptr(positions), _ptr(cl), _ptr(go), int(n_graphs),
                                                   float(r_cut), cap, _ptr(snd), _ptr(rcv), _ptr(sh),
                                                   ctypes.byref(ne), _stream(stream))
    if max_edges is None:
        code = call(0, None, None, None)
        if code not in (0, -3):
            raise MaceError(code, "mace_neighbor_list_device_noalloc")
        max_edges = ne.value
    snd = torch.empty(max(max_edges, 1), dtype=torch.int32, device=positions.device)
    rcv = torch.empty_like(snd)
    sh = torch.empty(max(max_edges, 1), 3, dtype=torch.int32, device=positions.device)
    _check(call(max_edges, snd, rcv, sh), "mace_neighbor_list_device_noalloc")
    E = ne.value
    return snd[:E], rcv[:E], sh[:E]


def mace_graph_setup(desc, weights, n_atoms, species, n_edges, edge_index, unit_shifts, cells, graph_of_atom,
                     n_graphs, prec, workspace, stream=None) -> int:
    """Returns the opaque handle (an integer address)."""
    h = ctypes.c_void_p()
    code = lib().mace_graph_setup(ctypes.byref(desc), _ptr(weights), weights.numel(), n_atoms, _ptr(species),
                                  n_edges, _ptr(edge_index), _ptr(unit_shifts), _ptr(cells), _ptr(graph_of_atom),
                                  n_graphs, prec, _ptr(workspace), workspace.numel() * workspace.element_size(),
                                  _stream(stream), ctypes.byref(h))
    _check(code, "mace_graph_setup")
    return h.value


def mace_forward_energy(handle, positions, node_energy, graph_energy, stream=None):
    _check(lib().mace_forward_energy(handle, _ptr(positions), _ptr(node_energy), _ptr(graph_energy),
                                     _stream(stream)), "mace_forward_energy")


def mace_forces(handle, positions, node_energy, graph_energy, forces, stream=None):
    _check(lib().mace_forces(handle, _ptr(positions), _ptr(node_energy), _ptr(graph_energy), _ptr(forces),
                             _stream(stream)), "mace_forces")


def mace_forces_stress(handle, positions, node_energy, graph_energy, forces, stress, stream=None):
    _check(lib().mace_forces_stress(handle, _ptr(positions), _ptr(node_energy), _ptr(graph_energy), _ptr(forces),
                                    _ptr(stress), _stream(stream)), "mace_forces_stress")


def mace_graph_check(handle, stream=None):
    """(status, flags): the status code and the device status bits since setup
    or the previous check (1 non-finite edge vector, 2 zero-length edge); the
    word is reset. Returns the status instead of raising."""
    flags = ctypes.c_int32(0)
    code = lib().mace_graph_check(handle, ctypes.byref(flags), _stream(stream))
    if code == -4 or code == -1:
        _check(code, "mace_graph_check")
    return code, flags.value


def mace_graph_destroy(handle):
    if handle:
        lib().mace_graph_destroy(handle)


def mace_status_string(code: int) -> str:
    return lib().mace_status_string(code).decode()


def mace_debug_real_cg(l1, l2, l3) -> np.ndarray:
    out = np.zeros((2 * l1 + 1) * (2 * l2 + 1) * (2 * l3 + 1))
    _check(lib().mace_debug_real_cg(l1, l2, l3, out.ctypes.data), "mace_debug_real_cg")
    return out.reshape(2 * l1 + 1, 2 * l2 + 1, 2 * l3 + 1)


def mace_debug_trees(nu, L, parity):
    n = ctypes.c_int32()
    lib().mace_debug_trees(nu, L, parity, 0, None, None, ctypes.byref(n))
    trees = np.zeros((max(n.value, 1), 4), np.int32)
    scales = np.zeros(max(n.value, 1))
    _check(lib().mace_debug_trees(nu, L, parity, n.value, trees.ctypes.data, scales.ctypes.data, ctypes.byref(n)),
           "mace_debug_trees")
    return trees[:n.value], scales[:n.value]


def mace_debug_edge_features(vec: np.ndarray, r_cut: float, envelope_p: int = 5, n_bessel: int = 8):
    v = np.ascontiguousarray(vec, dtype=np.float32)
    Y = np.zeros((len(v), 16), np.float32)
    rbf = np.zeros((len(v), n_bessel), np.float32)
    _check(lib().mace_debug_edge_features(len(v), v.ctypes.data, float(r_cut), envelope_p, n_bessel,
                                          Y.ctypes.data, rbf.ctypes.data), "mace_debug_edge_features")
    return Y, rbf


def mace_layer0_form(handle, request: int = -1) -> int:
    """Select (MACE_L0_AUTO / _EDGE / _FACTORED) or, with request < 0, only
    query the form of the first layer's message; returns the form in use."""
    used = ctypes.c_int32(0)
    _check(lib().mace_layer0_form(handle, request, ctypes.byref(used)), "mace_layer0_form")
    return used.value


def mace_debug_fused_linears(handle, request: int = -1) -> int:
    """Test switch of the 16-bit modes' linear layouts: bit 0 fuses the
    first-layer linears, bit 1 takes eight node tiles per wide block on large
    graphs (3, the default: both; 0: neither); request < 0 only queries.
    Returns the bits in effect for this handle."""
    used = ctypes.c_int32(0)
    _check(lib().mace_debug_fused_linears(handle, request, ctypes.byref(used)), "mace_debug_fused_linears")
    return used.value


def mace_fp32_products(handle, request: int = -1) -> int:
    """Select (MACE_PRODUCTS_FP32 / MACE_PRODUCTS_SPLIT_BF16) or, with request < 0,
    only query the operands of the last radial layer; returns the setting."""
    used = ctypes.c_int32(0)
    _check(lib().mace_fp32_products(handle, request, ctypes.byref(used)), "mace_fp32_products")
    return used.value


def mace_block_rounding(handle, block: int, fmt: int = -1) -> int:
    """Precision study: set (0 none, 1 bfloat16, 2 binary16) or, with
    fmt < 0, only query the operand rounding of one block; returns it."""
    used = ctypes.c_int32(0)
    _check(lib().mace_block_rounding(handle, block, fmt, ctypes.byref(used)), "mace_block_rounding")
    return used.value


def mace_profile_select(handle, kernel: int):
    _check(lib().mace_profile_select(handle, kernel), "mace_profile_select")


def mace_profile_read(handle):
    """(summed milliseconds, launches) of the selected kernel class since the last read."""
    ms = ctypes.c_double()
    n = ctypes.c_int64()
    _check(lib().mace_profile_read(handle, ctypes.byref(ms), ctypes.byref(n)), "mace_profile_read")
    return ms.value, n.value


def mace_profile_work(handle):
    """(flops, bytes): algorithmic work of the selected class's launches."""
    f, b = ctypes.c_double(0), ctypes.c_double(0)
    _check(lib().mace_profile_work(handle, ctypes.byref(f), ctypes.byref(b)), "mace_profile_work")
    return f.value, b.value


def mace_kernel_name(kernel: int) -> str:
    return lib().mace_kernel_name(kernel).decode()


def kernel_ids() -> dict:
    out, k = {}, 0
    while True:
        name = mace_kernel_name(k)
        if not name:
            return out
        out[name] = k
        k += 1
