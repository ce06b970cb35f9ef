#!/usr/bin/env python3
"""Throughput of PackMamba's packed hot path on one MI355X.

One step = causal conv1d forward -> selective scan forward (saving chunk states)
-> selective scan backward -> causal conv1d backward (its upstream gradient is
the scan's du), over one batch of the Mamba-1.4B layer shape: 8 packed rows of
4096 tokens, d_inner 4096, d_state 16, conv width 4, bf16 activations, fp32
state.  Inputs are resident in HBM before timing starts; every buffer, including
the workspaces, is allocated beforehand.  Prints one JSON line.

  python bench.py [--gpus 1] [--steps K] [--warmup W] [--config 2] [--no-cpu-baseline]
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "packed selective-scan+conv1d fwd+bwd tokens/s at Mamba-1.4B shape; % HBM peak"
HBM_PEAK = 8.0e12              # bytes/s
# VALU issue rate: 256 CUs x 4 SIMDs x 16 lanes x 2.4 GHz, one lane-op per slot
VALU_PEAK = 256 * 4 * 16 * 2.4e9
# Algorithmic VALU slots per (token, channel, state); v_exp_f32 issues at half rate (2 slots).
SLOTS_FWD = 6                  # Abar (mul + exp2), dt*B*u (mul), h (fma), y (fma)
SLOTS_BWD = 17                 # replay Abar, Bbar x, h; dh (mul + fma); sum dh B (fma);
#                                q = dh * Abar h_prev (2 mul); ddt (fma); dA (fma); dB, dC (mul + add each)
KERNEL_SOURCES = ("common.hpp", "scan_bwd.hip")


def minimal_bytes(Nb, Dn, L, N, W, s):
    """Bytes each op must move at least (inputs read once, outputs written once)."""
    E, T = Nb * Dn * L, Nb * L
    return {
        "conv_fwd": E * 2 * s + 4 * T + 4 * Dn * (W + 1),
        "scan_fwd": E * 4 * s + T * (2 * N * s + 4) + 4 * (Dn * N + 2 * Dn),
        "scan_bwd": E * 7 * s + T * (2 * N * s + 4 + 8 * N) + 8 * (Dn * N + 2 * Dn),
        "conv_bwd": E * 3 * s + 4 * T + 8 * Dn * (W + 1),
    }


def kernel_hash() -> str:
    h = hashlib.sha256()
    for f in KERNEL_SOURCES:
        with open(os.path.join(ROOT, "paper_2408_03865_amd", "csrc", f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


def stored_traffic():
    """HBM traffic of the dominant kernel from the last counter run, if its source is unchanged."""
    p = os.path.join(ROOT, "profiles", "scan_bwd_traffic.json")
    try:
        with open(p) as fh:
            t = json.load(fh)
    except (OSError, ValueError):
        return None
    return t if t.get("kernel_hash") == kernel_hash() else None


def cpu_baseline(d, cfg, rows):
    import oracle as O
    sl = slice(0, rows)
    x, dout, pos = d["x"][sl], d["dout"][sl], d["pos"][sl]
    t0 = time.perf_counter()
    u = O.conv1d_fwd(x, d["w"], d["bias"], pos, silu=True)
    args = dict(u=u, delta=d["delta"][sl], A=d["A"], B=d["B"][sl], C=d["C"][sl], D=d["D"],
                z=d["z"][sl], delta_bias=d["delta_bias"], delta_softplus=True, pos=pos)
    O.scan_fwd(**args)
    g = O.scan_bwd(**args, dout=dout)
    O.conv1d_bwd(x, d["w"], d["bias"], pos, g["du"], silu=True)
    dt = time.perf_counter() - t0
    tokens = rows * cfg.seqlen
    return {"value": tokens / dt, "unit": "tokens/s", "cores": O.num_threads(), "kind": "oracle",
            "sample": f"batch rows 0..{rows - 1} of the same workload ({tokens} tokens x {cfg.dim} "
                      f"channels), conv1d + selective scan forward and backward in fp64",
            "seconds": dt}


def main():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--config", default="2")
    ap.add_argument("--variant", default="paper", choices=["paper", "general"])
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-rows", type=int, default=8)
    ap.add_argument("--copy-probe", type=int, default=0, metavar="BYTES",
                    help="only copy BYTES with a plain device copy (calibrates HBM byte counters)")
    args = ap.parse_args()
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print(f"bench.py runs on one GPU only (got --gpus {args.gpus}, WORLD_SIZE {world}); "
              "this build has no multi-GPU path.", file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    if args.copy_probe:
        n = args.copy_probe // 4
        src = torch.ones(n, dtype=torch.float32, device="cuda:0")
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"copy_probe_bytes": n * 4, "dispatches": 3}))
        return

    import workloads as W
    from paper_2408_03865_amd import _lib

    if not os.path.exists(_lib.LIB_PATH):
        import __graft_entry__
        __graft_entry__.build()
    lib = _lib.load()
    dev = torch.device("cuda:0")
    cfg = W.config(args.config)
    Nb, Dn, L, N, Wd = cfg.batch, cfg.dim, cfg.seqlen, cfg.dstate, cfg.width
    code = _lib.BF16 if cfg.dtype == "bf16" else _lib.F32
    tdt = torch.bfloat16 if cfg.dtype == "bf16" else torch.float32
    s = 2 if cfg.dtype == "bf16" else 4

    print(f"# generating config {cfg.key} inputs {Nb}x{Dn}x{L}", file=sys.stderr, flush=True)
    d = W.make_inputs(cfg, variant=args.variant)

    def act(a):
        return torch.from_numpy(a).to(tdt).to(dev)

    def f32(a):
        return torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).to(dev)

    x, dl, z, B, C, dout = (act(d[k]) for k in ("x", "delta", "z", "B", "C", "dout"))
    A, D, dbias, w, bias = (f32(d[k]) for k in ("A", "D", "delta_bias", "w", "bias"))
    pos = torch.from_numpy(d["pos"]).to(dev)
    u = torch.empty_like(x)
    out = torch.empty_like(x)
    du, ddl, dz, dx = (torch.empty_like(x) for _ in range(4))
    dA, dD, ddb = torch.empty_like(A), torch.empty_like(D), torch.empty_like(dbias)
    dB = torch.empty((Nb, N, L), dtype=torch.float32, device=dev)
    dC = torch.empty_like(dB)
    dw, dcb = torch.empty_like(w), torch.empty_like(bias)
    nst = (L + _lib.STATE_STRIDE - 1) // _lib.STATE_STRIDE
    states = torch.empty((Nb, Dn, nst, N), dtype=torch.float32, device=dev)
    ws_scan = torch.empty(lib.packmamba_selective_scan_bwd_workspace_size(Nb, Dn, L, N), dtype=torch.uint8, device=dev)
    ws_fwd = torch.empty(max(1, lib.packmamba_selective_scan_fwd_workspace_size(Nb, Dn, L, N)), dtype=torch.uint8, device=dev)
    ws_conv = torch.empty(lib.packmamba_causal_conv1d_bwd_workspace_size(Nb, Dn, L, Wd), dtype=torch.uint8, device=dev)
    stream = torch.cuda.current_stream(dev)
    sp = stream.cuda_stream
    P = lambda t: t.data_ptr()  # noqa: E731

    def conv_fwd():
        _lib.check("conv_fwd", lib.packmamba_causal_conv1d_fwd(P(x), P(w), P(bias), P(pos), P(u), Nb, Dn, L, Wd, code, 1, sp))

    def scan_fwd():
        _lib.check("scan_fwd", lib.packmamba_selective_scan_fwd(
            P(u), P(dl), P(A), P(B), P(C), P(D), P(z), P(dbias), 1, P(pos), P(out), P(states),
            P(ws_fwd), ws_fwd.numel(), Nb, Dn, L, N, code, sp))

    def scan_bwd():
        _lib.check("scan_bwd", lib.packmamba_selective_scan_bwd(
            P(u), P(dl), P(A), P(B), P(C), P(D), P(z), P(dbias), 1, P(pos), P(dout), P(states),
            P(du), P(ddl), P(dA), P(dB), P(dC), P(dD), P(dz), P(ddb), P(ws_scan), ws_scan.numel(),
            Nb, Dn, L, N, code, sp))

    def conv_bwd():
        _lib.check("conv_bwd", lib.packmamba_causal_conv1d_bwd(
            P(x), P(w), P(bias), P(pos), P(du), P(dx), P(dw), P(dcb), P(ws_conv), ws_conv.numel(),
            Nb, Dn, L, Wd, code, 1, sp))

    ops = [("conv_fwd", conv_fwd), ("scan_fwd", scan_fwd), ("scan_bwd", scan_bwd), ("conv_bwd", conv_bwd)]

    def step():
        for _, f in ops:
            f()

    print("# warmup", file=sys.stderr, flush=True)
    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()

    # ---- timed region: exactly K steps ----
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    t_wall = time.perf_counter()
    e0.record(stream)
    for _ in range(args.steps):
        step()
    e1.record(stream)
    torch.cuda.synchronize()
    t_wall = time.perf_counter() - t_wall
    ms_step = e0.elapsed_time(e1) / args.steps
    print(f"# timed {args.steps} steps: {ms_step:.3f} ms/step (wall {t_wall / args.steps * 1e3:.3f})",
          file=sys.stderr, flush=True)

    # ---- per-op durations, HIP events on the launch stream ----
    evs = [[torch.cuda.Event(enable_timing=True) for _ in range(len(ops) + 1)] for _ in range(args.steps)]
    for it in range(args.steps):
        evs[it][0].record(stream)
        for i, (_, f) in enumerate(ops):
            f()
            evs[it][i + 1].record(stream)
    torch.cuda.synchronize()
    op_ms = {name: float(np.mean([evs[it][i].elapsed_time(evs[it][i + 1]) for it in range(args.steps)]))
             for i, (name, _) in enumerate(ops)}

    mb = minimal_bytes(Nb, Dn, L, N, Wd, s)
    total_bytes = sum(mb.values())
    tokens = Nb * L
    value = tokens / (ms_step * 1e-3)
    E = Nb * Dn * L
    bwd_s = op_ms["scan_bwd"] * 1e-3
    achieved = E * N * SLOTS_BWD / bwd_s / 1e12
    peak = VALU_PEAK / 1e12
    traffic = stored_traffic()
    roof = {
        "bound": "alu", "achieved": round(achieved, 3), "peak": round(peak, 3), "unit": "Tslot/s",
        "frac": round(achieved / peak, 4),
        "traffic": (traffic["bytes_per_launch"] if traffic else None),
        "kernel": "selective_scan_bwd (main kernel + two finalize kernels, one ABI call)",
        "duration_ms": round(op_ms["scan_bwd"], 4),
        "hbm_frac_of_minimal_bytes": round(mb["scan_bwd"] / bwd_s / HBM_PEAK, 4),
    }
    line = {
        "metric": METRIC, "value": round(value, 1), "unit": "tokens/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(ms_step, 4),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "f32",
        "data": "synthetic",
        "config": {
            "workload": f"{cfg.name} layer: {Nb} packed rows x {L} tokens, d_inner {Dn}, d_state {N}, "
                        f"conv width {Wd}, {cfg.dtype} activations, fp32 state; sequence lengths "
                        f"{cfg.lengths[0]}{tuple(cfg.lengths[1:])} packed sequentially",
            "batch": Nb, "seqlen": L, "dim": Dn, "dstate": N, "width": Wd, "storage": cfg.dtype,
            "sequences": int(len(d["lengths"])), "variant": args.variant,
        },
        "hbm_frac": round(total_bytes / (ms_step * 1e-3) / HBM_PEAK, 4),
        "minimal_bytes_per_step": int(total_bytes),
        "ops": {k: {"ms": round(v, 4), "minimal_GBps": round(mb[k] / (v * 1e-3) / 1e9, 1),
                    "hbm_frac": round(mb[k] / (v * 1e-3) / HBM_PEAK, 4)} for k, v in op_ms.items()},
        "scan_hbm_frac": round((mb["scan_fwd"] + mb["scan_bwd"]) /
                               ((op_ms["scan_fwd"] + op_ms["scan_bwd"]) * 1e-3) / HBM_PEAK, 4),
        "roofline": roof,
        "device": torch.cuda.get_device_name(0),
    }
    if not args.no_cpu_baseline:
        print("# cpu baseline (oracle)", file=sys.stderr, flush=True)
        line["cpu_baseline"] = cpu_baseline(d, cfg, args.cpu_rows)
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
