"""Throughput of MACE energy + forces on one MI355X through the C ABI.

One step = one mace_forces call (energy forward + force backward, every
kernel of the path) over periodic water, 36,864 atoms (12,288 H2O,
1 g/cm^3, cutoff 6 A, ~86 neighbours per atom), K = 128, hidden
128x0e+128x1o+128x2e, correlation 3, 2 layers; synthetic positions and
N(0,1)/sqrt(fan_in) weights.  Inputs are resident in HBM before the timed
region.  FP32 is the headline; the BF16- and FP16-linear arms and the
1,536-atom workload are reported beside it.

Prints one JSON line: atoms/s (value), edges/s, ms per step, the roofline
of the dominant kernel (its algorithmic work over its launch time, measured
with HIP events on the library's stream over the timed region), and the FP64
CPU oracle timed on a bounded sample of the same workload.
"""
from __future__ import annotations

import argparse
import json
import os
import platform
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0
FP32_MFMA_PEAK_TFLOPS = 157.3
# FP32 vector arithmetic without packed (two-wide) FP32 instructions, which
# this build does not emit: 256 CUs x 4 SIMDs x 16 lanes x 2 flop x 2.4 GHz
FP32_VALU_PEAK_TFLOPS = 78.6
BF16_MFMA_PEAK_TFLOPS = 2500.0
KERNEL_SOURCES = {"edge_prologue_kernel": "k_radial.hip", "radial_bwd_kernel": "k_radial.hip",
                  "tpr_fwd_kernel": "k_tpr.hip", "tpr_bwd_kernel": "k_tpr.hip", "linear_kernel": "k_node.hip",
                  "l0_gather_kernel": "k_layer0.hip", "l0_edge_bwd_kernel": "k_layer0.hip",
                  "sender_sum_kernel": "k_sender.hip"}
# the edge-product kernels: dense radial products (MFMA) plus the CG
# contraction (VALU); the other kernel classes are priced against HBM
EDGE_PRODUCT = ("tpr_fwd_kernel", "tpr_bwd_kernel")
METRIC = "atoms/s and edges/s for MACE energy+forces (FP32, BF16-linear); % roofline"
PREC_NAMES = {"fp32": "MACE_FP32", "bf16": "MACE_BF16_LINEAR", "fp16": "MACE_FP16_LINEAR",
              "bf16radial": "MACE_BF16_RADIAL", "fp64": "MACE_FP64"}


def source_hash(kname):
    import hashlib
    src = os.path.join(ROOT, "paper_2510_23621_amd", "csrc", KERNEL_SOURCES.get(kname, "api.hip"))
    h = hashlib.sha256()
    for f in (src, os.path.join(ROOT, "paper_2510_23621_amd", "csrc", "mace_internal.h")):
        with open(f, "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


def measured_traffic(kname, key):
    """HBM bytes per launch of `kname` from the committed PMC summary
    (FETCH_SIZE + WRITE_SIZE, copy-calibrated), or None when absent or taken
    on a different version of the kernel's source."""
    path = os.path.join(ROOT, "profiles", "traffic.json")
    if not os.path.exists(path):
        return None
    with open(path) as fh:
        rec = json.load(fh).get(key, {}).get(kname)
    if not rec or rec.get("source_hash") != source_hash(kname):
        return None
    return rec["bytes_per_launch"]


def edge_product_work(layer, K, E, N, backward):
    """Algorithmic work of one edge-product launch (one layer in per-edge
    form), per the cost model: per edge the last radial layer 2*64*P*K flop
    (dense, MFMA) and the CG contraction 2K(nnz + mid) flop (VALU), the
    backward twice the forward (R recomputed and dE/da3; the CG VJP).
    Compulsory HBM bytes of the fused form: E*16 + N*(D_in + mid)*K*4
    (doubled for the backward).  Returns (mfma_flops, valu_flops,
    compulsory_bytes)."""
    P, mid, din, nnz = layer["P"], layer["mid"], layer["din"], layer["nnz"]
    f = 2 if backward else 1
    return (f * E * 2 * 64 * P * K, f * E * 2 * K * (nnz + mid), f * (E * 16 + N * (din + mid) * K * 4))


def hbm_class_bytes(name, model, N, E, l0_factored, n_species, presplit):
    """Compulsory bytes of every launch of an HBM-priced kernel class in one
    step, summed: each input and output the kernel must move, once."""
    K, nb, layers = model["K"], model["n_bessel"], model["layers"]
    n_ct = K // 16
    ki = 64 * n_species
    tot = 0.0
    for t, L in enumerate(layers):
        mid, din = L["mid"], L["din"]
        fact = l0_factored and t == 0
        a3b = 384 if (presplit and din == 4 and not fact) else 256
        if name == "l0_gather_kernel" and fact:
            tot += E * (256 + 64 + 4) + (N + 1) * 4 + N * 16 * ki * 4
        elif name == "l0_edge_bwd_kernel" and fact:
            tot += N * 16 * ki * 4 + E * (256 + 64 + 4) + E * (256 + 64)
        elif name == "edge_prologue_kernel":
            tot += E * ((12 + 8 + 32 + 64 + nb * 4) if t == 0 else 0) + E * a3b
        elif name == "radial_bwd_kernel":
            acc = t < len(layers) - 1
            parts = 1 if fact else n_ct
            tot += E * (nb * 4 + parts * (256 + 64) + 64 * (1 + acc) + nb * 4 * (1 + acc))
        elif name == "sender_sum_kernel" and t > 0:
            tot += E * (din * K * 4 + 4) + N * din * K * 4
    return tot


def cpu_model():
    try:
        with open("/proc/cpuinfo") as fh:
            for line in fh:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return platform.processor() or "unknown"


def cpu_baseline(params, seconds_hint=15.0, max_reps=6):
    """FP64 oracle E+F on a 64-molecule periodic water box (192 atoms) with
    the workload's model and cutoff: a bounded sample of the workload (the
    oracle's cost is per edge and per node, so atoms/s carries over),
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
        mace.energy_forces_chunked(d, blob, sysm, graph=graph)
        reps += 1
    per = (time.perf_counter() - t0) / reps
    return {"value": round(sysm.n_atoms / per, 2), "unit": "atoms/s", "cores": torch.get_num_threads(),
            "kind": "oracle", "cpu": cpu_model(),
            "sample": f"FP64 oracle energy+forces (two-pass chunked VJP), periodic water 64 H2O "
                      f"({sysm.n_atoms} atoms, {len(graph.sender)} edges) with the workload's model and cutoff; "
                      f"{reps} evaluation(s), {per:.2f} s each"}


class Arm:
    """One workload and precision mode bound to the library."""

    def __init__(self, B, cfg, prec):
        import torch

        import synth
        from paper_2510_23621_amd.graph import MaceGraph
        from synth.configs import CONFIGS, make_system, model_params
        self.B, self.cfg, self.prec = B, cfg, prec
        self.name = CONFIGS[cfg]["name"]
        self.params = model_params(cfg)
        self.sysm = make_system(cfg, seed=0)
        desc = B.make_desc(**self.params)
        lay, _ = B.mace_weight_layout(desc)
        blob = synth.weight_blob([(n, (s,), f) for n, s, f in lay], 0)
        sysm = self.sysm
        snd, rcv, sh = B.mace_neighbor_list(sysm.positions, self.params["r_cut"], sysm.cells, sysm.graph_of_atom,
                                            sysm.n_graphs)
        self.N, self.E = sysm.n_atoms, len(snd)
        periodic = sysm.cells is not None
        self.g = MaceGraph(desc, blob, sysm.species.astype(np.int32), np.stack([snd, rcv]).astype(np.int32),
                           sh if periodic else None, sysm.cells if periodic else None,
                           sysm.graph_of_atom.astype(np.int32) if sysm.n_graphs > 1 else None, sysm.n_graphs, prec)
        self.pos = torch.from_numpy(sysm.positions).to(self.g.dtype).cuda()
        self.out = self.g.outputs(True)
        self.stream = torch.cuda.current_stream()

    def step(self):
        eps, Eg, F = self.out
        self.B.mace_forces(self.g.handle, self.pos, eps, Eg, F, self.stream)

    def timed(self, warmup, steps, kid=None):
        """ms per step over `steps` calls after `warmup`; with kid, the summed
        HIP-event time and launch count of that kernel class over the same calls."""
        import torch
        B = self.B
        for _ in range(warmup):
            self.step()
        torch.cuda.synchronize()
        if kid is not None:
            B.mace_profile_select(self.g.handle, kid)
        t0 = torch.cuda.Event(enable_timing=True)
        t1 = torch.cuda.Event(enable_timing=True)
        t0.record(self.stream)
        for _ in range(steps):
            self.step()
        t1.record(self.stream)
        torch.cuda.synchronize()
        k = None
        if kid is not None:
            k = B.mace_profile_read(self.g.handle)
            B.mace_profile_select(self.g.handle, -1)
        return t0.elapsed_time(t1) / steps, k

    def dominant_kernel(self):
        """The kernel class with the most time in one profiled step."""
        B = self.B
        best, best_ms = None, -1.0
        for name, kid in B.kernel_ids().items():
            B.mace_profile_select(self.g.handle, kid)
            self.step()
            ms, _ = B.mace_profile_read(self.g.handle)
            if ms > best_ms:
                best, best_ms = name, ms
        B.mace_profile_select(self.g.handle, -1)
        return best

    def linears(self, steps):
        """The channel-mixing linears (every linear_kernel launch of a step):
        algorithmic flops and bytes (summed by the library from the launch
        plans) over their HIP-event time, against the MFMA peak of the mode's
        operand type and against HBM bandwidth."""
        B = self.B
        B.mace_profile_select(self.g.handle, B.kernel_ids()["linear_kernel"])
        for _ in range(steps):
            self.step()
        ms, launches = B.mace_profile_read(self.g.handle)
        flops, byts = B.mace_profile_work(self.g.handle)
        B.mace_profile_select(self.g.handle, -1)
        peak = FP32_MFMA_PEAK_TFLOPS if self.prec == B.MACE_FP32 else BF16_MFMA_PEAK_TFLOPS
        tfl = flops / (ms * 1e-3) / 1e12
        gbs = byts / (ms * 1e-3) / 1e9
        return {"launches_per_step": launches / steps, "avg_launch_ms": round(ms / max(launches, 1), 5),
                "ms_per_step": round(ms / steps, 4), "flops_per_step": int(flops / steps),
                "bytes_per_step": int(byts / steps), "achieved_tflops": round(tfl, 2),
                "mfma_peak_tflops": peak, "mfma_frac": round(tfl / peak, 4),
                "achieved_gbs": round(gbs, 1), "hbm_frac": round(gbs / HBM_PEAK_GBS, 4)}

    def roofline(self, kname, k_ms, k_launches, steps, total_ms, traffic_key):
        from paper_2510_23621_amd.csrc_info import layer_shapes
        B = self.B
        model = layer_shapes(self.params)
        l0_factored = B.mace_layer0_form(self.g.handle, -1) == B.MACE_L0_FACTORED
        presplit = (self.prec != B.MACE_BF16_RADIAL
                    and B.mace_fp32_products(self.g.handle, -1) == B.MACE_PRODUCTS_SPLIT_BF16)
        per_launch = k_launches / steps
        avg_ms = k_ms / max(k_launches, 1)
        if kname in EDGE_PRODUCT:
            mf = vf = cb = 0.0
            for t, L in enumerate(model["layers"]):
                if l0_factored and t == 0:
                    continue
                a, b, c = edge_product_work(L, model["K"], self.E, self.N, kname == "tpr_bwd_kernel")
                mf, vf, cb = mf + a, vf + b, cb + c
            mf, vf, cb = mf / per_launch, vf / per_launch, cb / per_launch
            tfl = (mf + vf) / (avg_ms * 1e-3) / 1e12
            roof = {"bound": "mfma", "achieved": round(tfl, 3), "peak": FP32_MFMA_PEAK_TFLOPS, "unit": "TFLOP/s",
                    "frac": round(tfl / FP32_MFMA_PEAK_TFLOPS, 4),
                    "work": "per edge 2*64*P*K (radial layer, MFMA) + 2K(nnz+mid) (CG, VALU), x2 backward",
                    "mfma_flops_per_launch": int(mf), "valu_flops_per_launch": int(vf),
                    # MFMA and VALU issue do not overlap on a gfx950 SIMD: the
                    # ideal time is the sum of the two pipes' times at peak, the
                    # FP32-accurate radial products running as six BF16 MFMA
                    # products each (split operands) and the CG on FP32 VALU
                    "pipe_time_frac": round((6 * mf / (BF16_MFMA_PEAK_TFLOPS * 1e12)
                                             + vf / (FP32_VALU_PEAK_TFLOPS * 1e12)) / (avg_ms * 1e-3), 4),
                    "compulsory_bytes_per_launch": int(cb)}
        else:
            byts = hbm_class_bytes(kname, model, self.N, self.E, l0_factored, self.params["n_species"], presplit)
            byts /= max(per_launch, 1)
            gbs = byts / (avg_ms * 1e-3) / 1e9
            roof = {"bound": "hbm", "achieved": round(gbs, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                    "frac": round(gbs / HBM_PEAK_GBS, 4), "compulsory_bytes_per_launch": int(byts)}
        roof.update({"traffic": measured_traffic(kname, traffic_key), "kernel": kname,
                     "avg_launch_ms": round(avg_ms, 5), "launches_per_step": per_launch,
                     "kernel_share_of_step": round(k_ms / (total_ms * steps), 4)})
        return roof, l0_factored

    def close(self):
        self.g.close()


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=100)
    ap.add_argument("--warmup", type=int, default=100)
    ap.add_argument("--config", type=int, default=3)
    ap.add_argument("--prec", choices=list(PREC_NAMES), default="fp32")
    ap.add_argument("--kernel", default="auto", help="kernel class whose roofline is reported")
    ap.add_argument("--other-steps", type=int, default=30, help="timed steps of the other precision arms")
    ap.add_argument("--secondary-config", type=int, default=1, help="workload reported beside the main one (-1: none)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--only-main", action="store_true",
                    help="only the timed steps of the selected mode (for kernel traces and counters)")
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

    from paper_2510_23621_amd import binding as B

    prec = getattr(B, PREC_NAMES[args.prec])
    arm = Arm(B, args.config, prec)
    N, E = arm.N, arm.E
    for _ in range(min(args.warmup, 3)):
        arm.step()
    torch.cuda.synchronize()
    kname = arm.dominant_kernel() if args.kernel == "auto" else args.kernel
    ms_step, (k_ms, k_launches) = arm.timed(args.warmup, args.steps, B.kernel_ids()[kname])
    roof, l0_factored = arm.roofline(kname, k_ms, k_launches, args.steps, ms_step, f"{arm.name}_{args.prec}")
    if args.only_main:
        print(json.dumps({"metric": "atoms/s (timed steps only)", "value": round(N / (ms_step * 1e-3), 1),
                          "ms_per_step": round(ms_step, 4), "workload": arm.name, "roofline": roof}), flush=True)
        arm.close()
        return

    # outside the timed region: per-call spread, the forward pass alone, the
    # linears, the other precision modes and the secondary workload
    evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
           for _ in range(min(args.steps, 50))]
    for a, b in evs:
        a.record(arm.stream)
        arm.step()
        b.record(arm.stream)
    torch.cuda.synchronize()
    per_call = np.array([a.elapsed_time(b) for a, b in evs])
    eps, Eg, _ = arm.out
    f0 = torch.cuda.Event(enable_timing=True)
    f1 = torch.cuda.Event(enable_timing=True)
    f0.record(arm.stream)
    for _ in range(args.other_steps):
        B.mace_forward_energy(arm.g.handle, arm.pos, eps, Eg, arm.stream)
    f1.record(arm.stream)
    torch.cuda.synchronize()
    fwd_ms = f0.elapsed_time(f1) / args.other_steps
    linears = {args.prec: arm.linears(args.other_steps)}
    arm.close()
    del arm
    torch.cuda.empty_cache()

    others = {}
    for oname, pname in (("fp32", "fp32"), ("bf16_linear", "bf16"), ("fp16_linear", "fp16"),
                         ("bf16_linear_and_radial", "bf16radial")):
        if pname == args.prec:
            continue
        o = Arm(B, args.config, getattr(B, PREC_NAMES[pname]))
        oms, _ = o.timed(max(5, args.other_steps // 3), args.other_steps)
        others[oname] = {"atoms_per_s": round(N / (oms * 1e-3), 1), "edges_per_s": round(E / (oms * 1e-3), 1),
                         "ms_per_step": round(oms, 4)}
        if pname in ("fp32", "bf16", "fp16"):
            linears[pname] = o.linears(args.other_steps)
        o.close()
        del o
        torch.cuda.empty_cache()

    secondary = None
    if args.secondary_config >= 0 and args.secondary_config != args.config:
        secondary = {}
        for pname in ("fp32", "bf16", "fp64"):
            s = Arm(B, args.secondary_config, getattr(B, PREC_NAMES[pname]))
            if pname == "fp64":   # the debug precision: plain FP64 kernels, a few steps
                sms, _ = s.timed(1, 3)
                secondary[pname] = {"workload": s.name, "atoms_per_s": round(s.N / (sms * 1e-3), 1),
                                    "ms_per_step": round(sms, 3)}
            else:
                sk = s.dominant_kernel()
                sms, (sk_ms, sk_n) = s.timed(100, 100, B.kernel_ids()[sk])
                sroof, _ = s.roofline(sk, sk_ms, sk_n, 100, sms, f"{s.name}_{pname}")
                secondary[pname] = {"workload": s.name, "n_atoms": s.N, "n_edges": s.E,
                                    "atoms_per_s": round(s.N / (sms * 1e-3), 1),
                                    "edges_per_s": round(s.E / (sms * 1e-3), 1), "ms_per_step": round(sms, 4),
                                    "roofline": sroof}
            s.close()
            del s
            torch.cuda.empty_cache()

    out = {
        "metric": METRIC,
        "value": round(N / (ms_step * 1e-3), 1),
        "unit": "atoms/s",
        "edges_per_s": round(E / (ms_step * 1e-3), 1),
        "n_gpus": 1, "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(ms_step, 4),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": {"fp32": "f32", "bf16": "f32+bf16-linear", "fp16": "f32+f16-linear",
                  "bf16radial": "f32+bf16-linear+bf16-radial"}[args.prec],
        "data": "synthetic",
        "config": {"workload": CONFIG_NAME(args.config), "n_atoms": N, "n_edges": E},
        "roofline": roof,
        "layer0_form": "factorised" if l0_factored else "per-edge",
        "step_ms_p10_p50_p90": [round(float(np.percentile(per_call, q)), 4) for q in (10, 50, 90)],
        "forward_only": {"atoms_per_s": round(N / (fwd_ms * 1e-3), 1), "ms": round(fwd_ms, 4)},
        "other_precisions": others,
        "linears": linears,
        "secondary_workload": secondary,
    }
    if not args.no_cpu_baseline:
        from synth.configs import model_params
        out["cpu_baseline"] = cpu_baseline(model_params(args.config))
    print(json.dumps(out), flush=True)


def CONFIG_NAME(cfg):
    from synth.configs import CONFIGS
    return CONFIGS[cfg]["name"]


if __name__ == "__main__":
    main()
