"""Throughput of MACE energy + forces on one MI355X through the C ABI.

One step = one mace_forces call (energy forward + force backward, every
kernel of the path) over periodic water, 1536 atoms (512 H2O, 1 g/cm^3,
cutoff 5 A, ~54 neighbours per atom), K = 128, hidden 128x0e+128x1o,
correlation 3, 2 layers; synthetic positions and N(0,1)/sqrt(fan_in) weights.
Inputs are resident in HBM before the timed region.

Prints one JSON line: atoms/s (value), edges/s, ms per step, the roofline
of the dominant kernel (measured with HIP events on the library's stream
over the timed region), and the FP64 CPU oracle timed on a bounded sample.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0
FP32_MFMA_PEAK_TFLOPS = 157.3
BF16_MFMA_PEAK_TFLOPS = 2500.0
KERNEL_SOURCES = {"edge_prologue_kernel": "k_radial.hip", "radial_bwd_kernel": "k_radial.hip",
                  "tpr_fwd_kernel": "k_tpr.hip", "tpr_bwd_kernel": "k_tpr.hip", "linear_kernel": "k_node.hip",
                  "l0_gather_kernel": "k_layer0.hip", "l0_edge_bwd_kernel": "k_layer0.hip"}
# kernel classes whose roofline is the FP32 MFMA peak (dense contractions);
# the others are priced against HBM bandwidth
MFMA_BOUND = ("edge_prologue_kernel", "radial_bwd_kernel", "tpr_fwd_kernel", "tpr_bwd_kernel")
# (l0_gather_kernel and l0_edge_bwd_kernel are priced against HBM bandwidth)


def source_hash(kname):
    import hashlib
    src = os.path.join(ROOT, "paper_2510_23621_amd", "csrc", KERNEL_SOURCES.get(kname, "api.hip"))
    h = hashlib.sha256()
    for f in (src, os.path.join(ROOT, "paper_2510_23621_amd", "csrc", "mace_internal.h")):
        with open(f, "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


def measured_traffic(kname, workload):
    """HBM bytes per launch of `kname` from the committed PMC summary
    (FETCH_SIZE + WRITE_SIZE, copy-calibrated), or None when absent or taken
    on a different version of the kernel's source."""
    path = os.path.join(ROOT, "profiles", "traffic.json")
    if not os.path.exists(path):
        return None
    with open(path) as fh:
        rec = json.load(fh).get(workload, {}).get(kname)
    if not rec or rec.get("source_hash") != source_hash(kname):
        return None
    return rec["bytes_per_launch"]


def kernel_work(name, model, N, E, l0_factored=False, n_species=2, presplit=False):
    """Algorithmic (bytes, flops) of every launch of kernel class `name` in
    one step, summed.  Bytes count each compulsory HBM read/write once; flops
    of the MFMA-bound classes count the dense contractions only (the radial
    MLP layers, including the last one formed inside the tensor-product
    kernels), not the Clebsch-Gordan arithmetic on the vector ALUs.  With
    the first layer in factorised form its message comes from the l0_*
    kernels and its radial backward reads one partial.  With presplit
    (split-BF16 products), a3 of the per-edge l_h = 1 layers is stored as its
    three bfloat16 parts, 384 bytes per edge instead of 256."""
    K, nb, layers = model["K"], model["n_bessel"], model["layers"]
    n_ct = K // 16
    ki = 64 * n_species
    tot_b = tot_f = 0.0
    for t, L in enumerate(layers):
        P, mid, din = L["P"], L["mid"], L["din"]
        fact = l0_factored and t == 0
        a3b = 384 if (presplit and din == 4 and not fact) else 256
        if fact and name in ("tpr_fwd_kernel", "tpr_bwd_kernel"):
            continue
        if name == "l0_gather_kernel" and fact:      # a3, Y, sender species in; U out
            tot_b += E * (256 + 64 + 4) + (N + 1) * 4 + N * 16 * ki * 4
            tot_f += E * 2 * 64 * 16
        elif name == "l0_edge_bwd_kernel" and fact:  # gU, a3, Y, sender species in; dE/da3, dE/dY out
            tot_b += N * 16 * ki * 4 + E * (256 + 64 + 4) + E * (256 + 64)
            tot_f += E * 2 * 2 * 64 * 16
        elif name == "tpr_fwd_kernel":
            tot_b += E * (a3b + 64 + 4) + N * (din + mid) * K * 4 + (N + 1) * 4 + 64 * P * K * 4
            tot_f += E * 2 * 64 * P * K
        elif name == "tpr_bwd_kernel":
            q = din * K * 4 if t > 0 else 0
            tot_b += E * (a3b + 64 + 4 + n_ct * (64 + 256) + q) + N * (din + mid) * K * 4 + 64 * P * K * 4
            tot_f += E * 2 * 2 * 64 * P * K
        elif name == "edge_prologue_kernel":      # geometry once, hidden layers of every layer
            tot_b += E * ((12 + 8 + 32 + 64 + nb * 4) if t == 0 else 0) + E * a3b   # a3
            tot_f += E * 2 * (nb * 64 + 2 * 64 * 64)
        elif name == "radial_bwd_kernel":
            acc = t < len(layers) - 1          # de and dY accumulate into the later layer's values
            parts = 1 if fact else n_ct
            tot_b += E * (nb * 4 + parts * (256 + 64) + 64 * (1 + acc) + nb * 4 * (1 + acc))
            tot_f += E * 2 * (3 * nb * 64 + 6 * 64 * 64)   # hidden layers again, then their VJP
    return tot_b, tot_f


def linear_roofline(B, g, pos, stream, steps, prec, kid):
    """The channel-mixing linears (every linear_kernel launch of a step):
    algorithmic flops and bytes (summed by the library from the launch plans)
    over their HIP-event time, against the MFMA peak of the mode's operand
    type and against HBM bandwidth."""
    eps, Eg, F = g.outputs(True)
    B.mace_profile_select(g.handle, kid)
    for _ in range(steps):
        B.mace_forces(g.handle, pos, eps, Eg, F, stream)
    ms, launches = B.mace_profile_read(g.handle)
    flops, byts = B.mace_profile_work(g.handle)
    B.mace_profile_select(g.handle, -1)
    peak = FP32_MFMA_PEAK_TFLOPS if prec == B.MACE_FP32 else BF16_MFMA_PEAK_TFLOPS
    tfl = flops / (ms * 1e-3) / 1e12
    gbs = byts / (ms * 1e-3) / 1e9
    return {"launches_per_step": launches / steps, "avg_launch_ms": round(ms / max(launches, 1), 5),
            "ms_per_step": round(ms / steps, 4), "flops_per_step": int(flops / steps),
            "bytes_per_step": int(byts / steps), "achieved_tflops": round(tfl, 2),
            "mfma_peak_tflops": peak, "mfma_frac": round(tfl / peak, 4),
            "achieved_gbs": round(gbs, 1), "hbm_frac": round(gbs / HBM_PEAK_GBS, 4)}


def cpu_baseline(params, seconds_hint=15.0, max_reps=10):
    """FP64 oracle E+F on a 64-molecule periodic water box with the same
    model (a bounded sample of the workload; atoms/s scales with atoms),
    repeated until about `seconds_hint` seconds of CPU work."""
    import torch

    import synth
    from oracle import mace
    torch.set_num_threads(os.cpu_count() or 1)
    sysm = synth.water_box(64, seed=11)
    d = mace.ModelDesc(**params)
    blob = synth.weight_blob(mace.weight_layout(d), 0)
    graph = mace.build_graph(sysm, d)
    t0 = time.perf_counter()
    reps = 0
    while reps < max_reps and (reps == 0 or time.perf_counter() - t0 < seconds_hint):
        mace.energy_forces(d, blob, sysm, graph=graph)
        reps += 1
    per = (time.perf_counter() - t0) / reps
    return {"value": sysm.n_atoms / per, "unit": "atoms/s", "cores": torch.get_num_threads(), "kind": "oracle",
            "sample": f"FP64 oracle energy+forces, periodic water 64 H2O ({sysm.n_atoms} atoms, "
                      f"{len(graph.sender)} edges), same model; {reps} evaluation(s), {per:.2f} s each"}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=100)
    ap.add_argument("--warmup", type=int, default=100)
    ap.add_argument("--config", type=int, default=1)
    ap.add_argument("--prec", choices=["fp32", "bf16", "fp16", "bf16radial"], default="fp32")
    ap.add_argument("--kernel", default="auto", help="kernel class whose roofline is reported")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--only-main", action="store_true",
                    help="only the timed steps of the selected mode (for kernel traces): no per-call spread, "
                         "linear roofline, forward-only, other modes or neighbour list")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="only copy 1 GiB three times (reference kernel for scaling HBM counters)")
    args = ap.parse_args()
    if args.copy_calibration:
        import torch
        x = torch.ones(2 ** 28, dtype=torch.float32, device="cuda")
        y = torch.empty_like(x)
        for _ in range(3):
            y.copy_(x)
        torch.cuda.synchronize()
        print(json.dumps({"copy_calibration_bytes": x.numel() * 4, "repeats": 3}), flush=True)
        return
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print(f"bench.py runs on one GPU only (asked for {max(args.gpus, world)}): the library has no multi-GPU path",
              file=sys.stderr)
        sys.exit(2)

    import torch

    import synth
    from paper_2510_23621_amd import binding as B
    from paper_2510_23621_amd.graph import MaceGraph
    from synth.configs import CONFIGS, make_system, model_params

    cfg = args.config
    params = model_params(cfg)
    prec = {"fp32": B.MACE_FP32, "bf16": B.MACE_BF16_LINEAR, "fp16": B.MACE_FP16_LINEAR,
            "bf16radial": B.MACE_BF16_RADIAL}[args.prec]
    sysm = make_system(cfg, seed=0)
    desc = B.make_desc(**params)
    lay, _ = B.mace_weight_layout(desc)
    blob = synth.weight_blob([(n, (s,), f) for n, s, f in lay], 0)
    snd, rcv, sh = B.mace_neighbor_list(sysm.positions, params["r_cut"], sysm.cells, sysm.graph_of_atom,
                                        sysm.n_graphs)
    N, E = sysm.n_atoms, len(snd)
    periodic = sysm.cells is not None
    g = MaceGraph(desc, blob, sysm.species.astype(np.int32), np.stack([snd, rcv]).astype(np.int32),
                  sh if periodic else None, sysm.cells if periodic else None,
                  sysm.graph_of_atom.astype(np.int32) if sysm.n_graphs > 1 else None, sysm.n_graphs, prec)
    pos = torch.from_numpy(sysm.positions.astype(np.float32)).cuda()
    eps, Eg, F = g.outputs(True)
    stream = torch.cuda.current_stream()
    for _ in range(args.warmup):
        B.mace_forces(g.handle, pos, eps, Eg, F, stream)
    torch.cuda.synchronize()

    # dominant kernel: the class with the most time in one profiled step
    kids = B.kernel_ids()
    kname = args.kernel
    if kname == "auto":
        best, best_ms = None, -1.0
        for name, kid in kids.items():
            B.mace_profile_select(g.handle, kid)
            B.mace_forces(g.handle, pos, eps, Eg, F, stream)
            ms, _ = B.mace_profile_read(g.handle)
            if ms > best_ms:
                best, best_ms = name, ms
        kname = best
    B.mace_profile_select(g.handle, kids[kname])
    torch.cuda.synchronize()

    t0 = torch.cuda.Event(enable_timing=True)
    t1 = torch.cuda.Event(enable_timing=True)
    t0.record(stream)
    for _ in range(args.steps):
        B.mace_forces(g.handle, pos, eps, Eg, F, stream)
    t1.record(stream)
    torch.cuda.synchronize()
    total_ms = t0.elapsed_time(t1)
    k_ms, k_launches = B.mace_profile_read(g.handle)
    B.mace_profile_select(g.handle, -1)
    ms_step = total_ms / args.steps

    from paper_2510_23621_amd.csrc_info import layer_shapes
    model = layer_shapes(params)
    l0_factored = B.mace_layer0_form(g.handle, -1) == B.MACE_L0_FACTORED
    presplit = prec != B.MACE_BF16_RADIAL and B.mace_fp32_products(g.handle, -1) == B.MACE_PRODUCTS_SPLIT_BF16
    byts, flops = kernel_work(kname, model, N, E, l0_factored, params["n_species"], presplit)
    per_launch = k_launches / args.steps
    avg_launch_ms = k_ms / max(k_launches, 1)
    bytes_per_launch = byts / max(per_launch, 1)
    flops_per_launch = flops / max(per_launch, 1)
    gbs = bytes_per_launch / (avg_launch_ms * 1e-3) / 1e9
    tfl = flops_per_launch / (avg_launch_ms * 1e-3) / 1e12
    if kname in MFMA_BOUND:
        roof = {"bound": "mfma", "achieved": round(tfl, 3), "peak": FP32_MFMA_PEAK_TFLOPS, "unit": "TFLOP/s",
                "frac": round(tfl / FP32_MFMA_PEAK_TFLOPS, 4)}
        split = (kname in ("tpr_fwd_kernel", "tpr_bwd_kernel") and prec != B.MACE_BF16_RADIAL
                 and B.mace_fp32_products(g.handle, -1) == B.MACE_PRODUCTS_SPLIT_BF16
                 and (kname == "tpr_fwd_kernel" or params["hidden_lmax"] <= 1))
        if split:
            # FP32-accurate products as six BF16 MFMA products each: the flops
            # above are the FP32 products the algorithm needs; the BF16 MFMA
            # pipe executes six times as many
            roof.update({"operands": "split-bf16 (3 parts, 6 bf16 products per fp32 product, fp32 accumulation)",
                         "executed_bf16_tflops": round(6 * tfl, 2), "bf16_peak": BF16_MFMA_PEAK_TFLOPS,
                         "executed_frac_of_bf16_peak": round(6 * tfl / BF16_MFMA_PEAK_TFLOPS, 4)})
    else:
        roof = {"bound": "hbm", "achieved": round(gbs, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                "frac": round(gbs / HBM_PEAK_GBS, 4)}
    roof.update({"traffic": measured_traffic(kname, CONFIGS[cfg]["name"] + "_" + args.prec), "kernel": kname,
                 "avg_launch_ms": round(avg_launch_ms, 5),
                 "launches_per_step": per_launch, "algorithmic_bytes_per_launch": int(bytes_per_launch),
                 "algorithmic_flops_per_launch": int(flops_per_launch),
                 "kernel_share_of_step": round(k_ms / total_ms, 4)})

    if args.only_main:
        print(json.dumps({"metric": "atoms/s (timed steps only)", "value": round(N * args.steps / (total_ms * 1e-3), 1),
                          "ms_per_step": round(ms_step, 4), "roofline": roof,
                          "layer0_form": "factorised" if l0_factored else "per-edge"}), flush=True)
        g.close()
        return
    # outside the timed region: per-call spread, the linears' roofline, the
    # forward pass alone, and the other precision modes on the same workload
    evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(args.steps)]
    for a, b in evs:
        a.record(stream)
        B.mace_forces(g.handle, pos, eps, Eg, F, stream)
        b.record(stream)
    torch.cuda.synchronize()
    per_call = np.array([a.elapsed_time(b) for a, b in evs])
    linears = {prec: linear_roofline(B, g, pos, stream, args.steps, prec, kids["linear_kernel"])}
    f0 = torch.cuda.Event(enable_timing=True)
    f1 = torch.cuda.Event(enable_timing=True)
    for _ in range(args.warmup):
        B.mace_forward_energy(g.handle, pos, eps, Eg, stream)
    f0.record(stream)
    for _ in range(args.steps):
        B.mace_forward_energy(g.handle, pos, eps, Eg, stream)
    f1.record(stream)
    torch.cuda.synchronize()
    fwd_ms = f0.elapsed_time(f1) / args.steps
    others = {}
    for other, oname in ((B.MACE_FP32, "fp32"), (B.MACE_BF16_LINEAR, "bf16_linear"), (B.MACE_FP16_LINEAR, "fp16_linear"),
                         (B.MACE_BF16_RADIAL, "bf16_linear_and_radial")):
        if other == prec:
            continue
        g2 = MaceGraph(desc, blob, sysm.species.astype(np.int32), np.stack([snd, rcv]).astype(np.int32),
                       sh if periodic else None, sysm.cells if periodic else None,
                       sysm.graph_of_atom.astype(np.int32) if sysm.n_graphs > 1 else None, sysm.n_graphs, other)
        eps2, Eg2, F2 = g2.outputs(True)
        for _ in range(args.warmup):
            B.mace_forces(g2.handle, pos, eps2, Eg2, F2, stream)
        f0.record(stream)
        for _ in range(args.steps):
            B.mace_forces(g2.handle, pos, eps2, Eg2, F2, stream)
        f1.record(stream)
        torch.cuda.synchronize()
        other_ms = f0.elapsed_time(f1) / args.steps
        others[oname] = {"atoms_per_s": round(N / (other_ms * 1e-3), 1), "edges_per_s": round(E / (other_ms * 1e-3), 1),
                         "ms_per_step": round(other_ms, 4)}
        linears[other] = linear_roofline(B, g2, pos, stream, args.steps, other, kids["linear_kernel"])
        g2.close()

    # the device neighbour list of the same system (outside the timed region)
    dpos = torch.from_numpy(np.ascontiguousarray(sysm.positions, dtype=np.float64)).cuda()
    goff = None
    if sysm.n_graphs > 1:
        goff = np.concatenate([[0], np.cumsum(np.bincount(sysm.graph_of_atom, minlength=sysm.n_graphs))])
    nl_ms = []
    for _ in range(6):
        torch.cuda.synchronize()
        t_a = time.perf_counter()
        s_d, _, _ = B.mace_neighbor_list_device(dpos, params["r_cut"], sysm.cells, goff, sysm.n_graphs, max_edges=E)
        torch.cuda.synchronize()
        nl_ms.append((time.perf_counter() - t_a) * 1e3)
    t_a = time.perf_counter()
    B.mace_neighbor_list(sysm.positions, params["r_cut"], sysm.cells, sysm.graph_of_atom, sysm.n_graphs)
    host_nl_ms = (time.perf_counter() - t_a) * 1e3
    assert len(s_d) == E

    out = {
        "metric": "atoms/s and edges/s for MACE energy+forces (FP32, BF16-linear); % roofline",
        "value": round(N * args.steps / (total_ms * 1e-3), 1),
        "unit": "atoms/s",
        "edges_per_s": round(E * args.steps / (total_ms * 1e-3), 1),
        "n_gpus": 1, "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(ms_step, 4),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": {B.MACE_FP32: "f32", B.MACE_BF16_LINEAR: "f32+bf16-linear", B.MACE_FP16_LINEAR: "f32+f16-linear",
                  B.MACE_BF16_RADIAL: "f32+bf16-linear+bf16-radial"}[prec],
        "data": "synthetic",
        "config": {"workload": CONFIGS[cfg]["name"], "n_atoms": N, "n_edges": E, "K": params["K"],
                   "hidden_lmax": params["hidden_lmax"], "r_cut": params["r_cut"], "correlation": 3,
                   "layers": 2, "precision": args.prec,
                   "layer0_form": "factorised" if l0_factored else "per-edge"},
        "roofline": roof,
        "step_ms_p10_p50_p90": [round(float(np.percentile(per_call, q)), 4) for q in (10, 50, 90)],
        "forward_only": {"atoms_per_s": round(N / (fwd_ms * 1e-3), 1), "ms": round(fwd_ms, 4)},
        "other_precisions": others,
        "neighbor_list": {"device_ms_median": round(float(np.median(nl_ms[1:])), 3),
                          "host_ms": round(host_nl_ms, 2), "edges": E,
                          "note": "wall time of one call incl. workspace allocation and the edge-count read-back"},
        "linears": {name: linears[p] for p, name in ((B.MACE_FP32, "fp32"), (B.MACE_BF16_LINEAR, "bf16_linear"),
                                                      (B.MACE_FP16_LINEAR, "fp16_linear")) if p in linears},
    }
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(params)
    g.close()
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
