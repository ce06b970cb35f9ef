#!/usr/bin/env python3
"""Throughput of PackMamba's packed hot path on one MI355X.

One step = causal conv1d forward -> selective scan forward (saving chunk states)
-> selective scan backward -> causal conv1d backward (its upstream gradient is
the scan's du), over one batch of the Mamba-1.4B layer shape: 8 packed rows of
4096 tokens, d_inner 4096, d_state 16, conv width 4, bf16 activations, fp32
state.  Inputs are resident in HBM before timing starts; every buffer, including
the workspaces, is allocated beforehand.  Prints one JSON line.

At that shape the line also carries "comparison": the same real tokens through the
same kernels padded to the longest sequence (one sequence per row) and run one
sequence per call chain, with the packed path's speedup over each.

  python bench.py [--gpus 1] [--steps K] [--warmup W] [--config 2] [--variant paper|general]
                  [--no-cpu-baseline] [--no-compare]
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
KERNEL_SOURCES = ("common.hpp", "launch.hpp", "scan_bwd.hip")


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


def stored_traffic(shape):
    """HBM traffic of the dominant kernel from the last counter run, if its source is unchanged
    and the run measured this shape (batch, seqlen, dim, dstate, storage); else None."""
    p = os.path.join(ROOT, "profiles", "scan_bwd_traffic_mamba1.4b_step.json")
    try:
        with open(p) as fh:
            t = json.load(fh)
    except (OSError, ValueError):
        return None
    if t.get("kernel_hash") != kernel_hash() or t.get("shape") != shape:
        return None
    return t


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
            "cores_note": f"OpenMP threads the oracle ran with; {len(os.sched_getaffinity(0))} CPUs in the "
                          "process's affinity mask",
            "sample": f"batch rows 0..{rows - 1} of the same workload ({tokens} tokens x {cfg.dim} "
                      f"channels), conv1d + selective scan forward and backward in fp64",
            "seconds": dt}


class Chain:
    """Buffers and C-ABI calls of one step: conv fwd -> scan fwd (saving chunk states)
    -> scan bwd -> conv bwd (upstream gradient = the scan's du).  Every buffer,
    workspaces included, is allocated here, before any timing."""

    def __init__(self, lib, t, code, width, stream, states=False):
        """states: every row continues a sequence from another row (its first position
        index is not 0): initial states go in, final states come out, with gradients."""
        import torch
        from paper_2408_03865_amd import _lib
        self.lib, self.t, self.code, self.W, self.sp = lib, t, code, width, stream.cuda_stream
        x = t["x"]
        self.Nb, self.Dn, self.L = x.shape
        self.N = t["A"].shape[1]
        Nb, Dn, L, N, dev = self.Nb, self.Dn, self.L, self.N, x.device
        e = lambda: torch.empty_like(x)  # noqa: E731
        self.u, self.out, self.du, self.ddl, self.dz, self.dx = (e() for _ in range(6))
        self.dA, self.dD, self.ddb = (torch.empty_like(t[k]) for k in ("A", "D", "delta_bias"))
        self.dB = torch.empty((Nb, N, L), dtype=torch.float32, device=dev)
        self.dC = torch.empty_like(self.dB)
        self.dw, self.dcb = torch.empty_like(t["w"]), torch.empty_like(t["bias"])
        nsaved = lib.packmamba_selective_scan_fwd_saved_states_size(Nb, Dn, L, N) // 4
        self.states = torch.empty(nsaved, dtype=torch.float32, device=dev)

        def ws(n):
            return torch.empty(max(1, int(n)), dtype=torch.uint8, device=dev)
        self.ws_fwd = ws(lib.packmamba_selective_scan_fwd_workspace_size(Nb, Dn, L, N))
        self.ws_scan = ws(lib.packmamba_selective_scan_bwd_workspace_size(Nb, Dn, L, N))
        self.ws_conv = ws(lib.packmamba_causal_conv1d_bwd_workspace_size(Nb, Dn, L, width))
        self.st = {}
        if states:
            g = torch.Generator(device=dev).manual_seed(7)
            xs = lambda: torch.randn((Nb, Dn, width - 1), generator=g, device=dev).to(x.dtype)  # noqa: E731
            hs = lambda: torch.randn((Nb, Dn, N), generator=g, device=dev)  # noqa: E731
            self.st = {"xi": xs(), "xf": xs(), "dxf": xs(), "dxi": xs(), "h0": hs(), "hf": hs(),
                       "dhf": hs(), "dh0": hs()}

    def ops(self):
        from paper_2408_03865_amd import _lib
        lib, t, c, sp = self.lib, self.t, self.code, self.sp
        Nb, Dn, L, N, W = self.Nb, self.Dn, self.L, self.N, self.W
        P = lambda v: v.data_ptr()  # noqa: E731
        S = lambda k: self.st[k].data_ptr() if self.st else None  # noqa: E731

        def conv_fwd():
            _lib.check("conv_fwd", lib.packmamba_causal_conv1d_fwd(
                P(t["x"]), P(t["w"]), P(t["bias"]), P(t["pos"]), S("xi"), P(self.u), S("xf"), Nb, Dn, L, W,
                c, 1, sp))

        def scan_fwd():
            _lib.check("scan_fwd", lib.packmamba_selective_scan_fwd(
                P(self.u), P(t["delta"]), P(t["A"]), P(t["B"]), P(t["C"]), P(t["D"]), P(t["z"]),
                P(t["delta_bias"]), 1, P(t["pos"]), S("h0"), P(self.out), S("hf"), P(self.states),
                P(self.ws_fwd), self.ws_fwd.numel(), Nb, Dn, L, N, c, sp))

        def scan_bwd():
            _lib.check("scan_bwd", lib.packmamba_selective_scan_bwd(
                P(self.u), P(t["delta"]), P(t["A"]), P(t["B"]), P(t["C"]), P(t["D"]), P(t["z"]),
                P(t["delta_bias"]), 1, P(t["pos"]), S("h0"), P(t["dout"]), S("dhf"), P(self.states),
                P(self.du), P(self.ddl), P(self.dA), P(self.dB), P(self.dC), P(self.dD), P(self.dz),
                P(self.ddb), S("dh0"), P(self.ws_scan), self.ws_scan.numel(), Nb, Dn, L, N, c, sp))

        def conv_bwd():
            _lib.check("conv_bwd", lib.packmamba_causal_conv1d_bwd(
                P(t["x"]), P(t["w"]), P(t["bias"]), P(t["pos"]), S("xi"), P(self.du), S("dxf"), P(self.dx),
                P(self.dw), P(self.dcb), S("dxi"), P(self.ws_conv), self.ws_conv.numel(), Nb, Dn, L, W, c, 1,
                sp))

        return [("conv_fwd", conv_fwd), ("scan_fwd", scan_fwd), ("scan_bwd", scan_bwd),
                ("conv_bwd", conv_bwd)]


def sequences(pos):
    """(row, offset, length) of every packed sequence, from the position indices."""
    import numpy as np
    out = []
    for b in range(pos.shape[0]):
        st = np.flatnonzero(pos[b] == 0).tolist() + [pos.shape[1]]
        out += [(b, st[i], st[i + 1] - st[i]) for i in range(len(st) - 1)]
    return out


def time_steps(step_fn, stream, steps, warmup):
    import torch
    for _ in range(warmup):
        step_fn()
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record(stream)
    for _ in range(steps):
        step_fn()
    e1.record(stream)
    torch.cuda.synchronize()
    return e0.elapsed_time(e1) / steps


def cold_steps(step_fn, stream, steps, flush_bytes=1 << 29):
    """Median time of one step with the caches cold: before each step (outside its
    events) a fill of ``flush_bytes`` evicts the L2s and the 256 MB memory-side cache,
    so the step's inputs come from HBM even where the previous step left them cached."""
    import numpy as np
    import torch
    buf = torch.empty(flush_bytes // 4, dtype=torch.float32, device=stream.device)
    evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(steps)]
    for it, (e0, e1) in enumerate(evs):
        buf.fill_(float(it))
        e0.record(stream)
        step_fn()
        e1.record(stream)
    torch.cuda.synchronize()
    ms = [e0.elapsed_time(e1) for e0, e1 in evs]
    del buf
    return {"ms_per_step": round(float(np.median(ms)), 4), "flush_bytes": int(flush_bytes),
            "steps": steps}


def with_states(lib, tens, pos_host, code, width, stream, steps, warmup, packed_step):
    """The same step with every row continuing a sequence cut at the end of another row
    (its first sequence's position indices start at 100), initial states in, final
    states out, and their gradients: the state-passing path.  Timed alternately with
    the packed step (three rounds each, medians), so that both see the same memory and
    cache conditions."""
    import numpy as np
    import torch
    pos = pos_host.copy()
    for b in range(pos.shape[0]):
        st = np.flatnonzero(pos[b, 1:] == 0)
        n = int(st[0]) + 1 if st.size else pos.shape[1]
        pos[b, :n] += 100
    t = dict(tens, pos=torch.from_numpy(pos).to(tens["x"].device))
    ch = Chain(lib, t, code, width, stream, states=True)
    ops = [f for _, f in ch.ops()]
    packed, cont = [], []
    for _ in range(3):
        packed.append(time_steps(packed_step, stream, steps, warmup))
        cont.append(time_steps(lambda: [f() for f in ops], stream, steps, warmup))
    ms, ref = float(np.median(cont)), float(np.median(packed))
    return {"ms_per_step": round(ms, 4), "packed_ms_per_step": round(ref, 4),
            "overhead_vs_packed": round(ms / ref - 1.0, 4), "rows_continued": int(pos.shape[0])}


def packing_rates(law, seqlen, count=20000, seed=0):
    """Padding of the host packing plans (the library's C++ planner) on a stream of
    ``count`` lengths drawn from the workload's length law: the sequential seal, local
    greedy with windows of 64 and 1024 sequences, and cutting at the row end."""
    import numpy as np
    import paper_2408_03865_amd as P
    import workloads as W
    ln = W.draw_stream_lengths(law, np.random.default_rng(seed), count)
    out = {"sequences": count, "mean_length": round(float(ln.mean()), 1)}
    for name, policy, w in (("sequential", "sequential", 1), ("greedy64", "greedy", 64),
                            ("greedy1024", "greedy", 1024), ("cut", "cut", 1)):
        pieces, rows = P.pack_plan(ln, seqlen, policy, window=w)
        out[name] = round(P.padding_rate(pieces, rows, seqlen), 5)
    return out


def comparison(lib, tens, pos_host, code, width, stream, steps, warmup, packed_ms):
    """The same real tokens and kernels without packing: (a) padded, one sequence per row
    padded with zeros to the longest length, position indices 0..L-1 on every row; (b)
    single, one call chain per sequence.  Tokens/s counts real tokens only."""
    import torch
    seqs = sequences(pos_host)
    real = sum(n for _, _, n in seqs)
    lmax = max(n for _, _, n in seqs)
    dev = tens["x"].device

    def timed(step_fn):
        for _ in range(warmup):
            step_fn()
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        for _ in range(steps):
            step_fn()
        e1.record(stream)
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / steps

    res = {"sequences": len(seqs), "real_tokens": real}
    # (a) padded
    pt = {k: tens[k] for k in ("A", "D", "delta_bias", "w", "bias")}
    for k in ("x", "delta", "z", "B", "C", "dout"):
        src = tens[k]
        dst = torch.zeros((len(seqs), src.shape[1], lmax), dtype=src.dtype, device=dev)
        for i, (b, o, n) in enumerate(seqs):
            dst[i, :, :n] = src[b, :, o:o + n]
        pt[k] = dst
    pt["pos"] = torch.arange(lmax, dtype=torch.int32, device=dev).repeat(len(seqs), 1).contiguous()
    ch = Chain(lib, pt, code, width, stream)
    ops = [f for _, f in ch.ops()]
    ms = timed(lambda: [f() for f in ops])
    res["padded"] = {"rows": len(seqs), "seqlen": lmax, "ms_per_step": round(ms, 4),
                     "tokens_per_s": round(real / (ms * 1e-3), 1),
                     "padding_frac": round(1.0 - real / (len(seqs) * lmax), 4),
                     "packed_speedup": round(ms / packed_ms, 3)}
    del ch, ops, pt
    torch.cuda.empty_cache()
    # (b) single
    chains = []
    for b, o, n in seqs:
        st = {k: tens[k] for k in ("A", "D", "delta_bias", "w", "bias")}
        for k in ("x", "delta", "z", "B", "C", "dout"):
            st[k] = tens[k][b:b + 1, :, o:o + n].contiguous()
        st["pos"] = torch.arange(n, dtype=torch.int32, device=dev).reshape(1, n)
        chains.append(Chain(lib, st, code, width, stream))
    ops = [f for c in chains for _, f in c.ops()]
    ms = timed(lambda: [f() for f in ops])
    res["single"] = {"calls_per_step": len(ops), "ms_per_step": round(ms, 4),
                     "tokens_per_s": round(real / (ms * 1e-3), 1),
                     "packed_speedup": round(ms / packed_ms, 3)}
    return res


BLOCK_PHASES = {"norm": "other", "in_proj": "gemm", "conv": "conv", "x_proj": "gemm", "scan": "scan",
                "out_proj": "gemm", "out_proj_bwd": "gemm", "scan_bwd": "scan", "x_proj_bwd": "gemm",
                "conv_bwd": "conv", "in_proj_bwd": "gemm", "norm_bwd": "other"}


def block_bench(args, d=None):
    """One packed Mamba-1 block (Mamba-1.4B layer: d_model 2048, d_inner 4096, d_state 16,
    dt_rank 128, conv width 4, bf16), forward and backward, on the tokens of the 1.4B
    workload: packed, padded to the longest sequence, and one sequence per call.  The
    time per phase comes from events between the phases of each step."""
    import numpy as np
    import torch
    import workloads as W
    import paper_2408_03865_amd.block as BK

    dev = torch.device("cuda:0")
    stream = torch.cuda.current_stream(dev)
    cfg = W.config("2")
    Nb, L, Dn, N = cfg.batch, cfg.seqlen, cfg.dim, cfg.dstate
    dm, R, Wd = 2048, 128, cfg.width
    if d is None:
        d = W.make_inputs(cfg)
    g = torch.Generator(device=dev).manual_seed(0)
    bf = torch.bfloat16
    rn = lambda *sh: torch.randn(sh, generator=g, device=dev)  # noqa: E731
    p = {"norm_w": torch.ones(dm, device=dev), "W_in": (rn(2 * Dn, dm) / dm ** 0.5).to(bf),
         "conv_w": torch.from_numpy(d["w"]).to(dev), "conv_b": torch.zeros(Dn, device=dev),
         "W_x": (rn(R + 2 * N, Dn) / Dn ** 0.5).to(bf), "W_dt": (rn(Dn, R) / R ** 0.5).to(bf),
         "dt_bias": torch.from_numpy(d["delta_bias"]).to(dev), "A": torch.from_numpy(d["A"]).to(dev),
         "D": torch.ones(Dn, device=dev), "W_out": (rn(dm, Dn) / Dn ** 0.5).to(bf)}
    x = rn(Nb, dm, L).to(bf)
    dout = rn(Nb, dm, L).to(bf)
    pos = torch.from_numpy(d["pos"]).to(dev)

    def run(xx, dd, pp, marks=None):
        mk = None
        if marks is not None:
            def mk(name):
                e = torch.cuda.Event(enable_timing=True)
                e.record(stream)
                marks.append((name, e))
        out, ctx = BK.block_forward(xx, pp, p, mark=mk)
        BK.block_backward(dd, ctx, p, mark=mk)

    steps, warmup = args.steps, args.warmup
    ms = time_steps(lambda: run(x, dout, pos), stream, steps, warmup)
    # per-phase times, averaged over the steps
    phase = {k: 0.0 for k in BLOCK_PHASES}
    for _ in range(steps):
        marks = []
        run(x, dout, pos, marks)
        torch.cuda.synchronize()
        for (a, e0), (_, e1) in zip(marks, marks[1:]):
            if a in phase:
                phase[a] += e0.elapsed_time(e1) / steps
    cat = {}
    for k, v in phase.items():
        cat[BLOCK_PHASES[k]] = cat.get(BLOCK_PHASES[k], 0.0) + v
    tokens = Nb * L
    res = {"metric": "packed Mamba-1.4B block fwd+bwd tokens/s", "value": round(tokens / (ms * 1e-3), 1),
           "unit": "tokens/s", "ms_per_step": round(ms, 4), "steps": steps, "warmup": warmup,
           "dtype": "bf16", "data": "synthetic",
           "config": {"workload": "one Mamba-1.4B block: 8 packed rows x 4096 tokens, d_model 2048, d_inner 4096, "
                                  "d_state 16, dt_rank 128, conv width 4, bf16 activations and projection weights",
                      "batch": Nb, "seqlen": L},
           "phase_ms": {k: round(v, 4) for k, v in phase.items()},
           "class_ms": {k: round(v, 4) for k, v in cat.items()}}
    # same tokens, padded and single
    seqs = sequences(d["pos"])
    lmax = max(n for _, _, n in seqs)
    xp = torch.zeros((len(seqs), dm, lmax), dtype=bf, device=dev)
    dp = torch.zeros_like(xp)
    for i, (b, o, n) in enumerate(seqs):
        xp[i, :, :n] = x[b, :, o:o + n]
        dp[i, :, :n] = dout[b, :, o:o + n]
    pp = torch.arange(lmax, dtype=torch.int32, device=dev).repeat(len(seqs), 1).contiguous()
    msp = time_steps(lambda: run(xp, dp, pp), stream, 3, 1)
    phase_p = {k: 0.0 for k in BLOCK_PHASES}
    marks = []
    run(xp, dp, pp, marks)
    torch.cuda.synchronize()
    for (a, e0), (_, e1) in zip(marks, marks[1:]):
        if a in phase_p:
            phase_p[a] += e0.elapsed_time(e1)
    cat_p = {}
    for k, v in phase_p.items():
        cat_p[BLOCK_PHASES[k]] = cat_p.get(BLOCK_PHASES[k], 0.0) + v
    del xp, dp
    torch.cuda.empty_cache()
    singles = [(x[b:b + 1, :, o:o + n].contiguous(), dout[b:b + 1, :, o:o + n].contiguous(),
                torch.arange(n, dtype=torch.int32, device=dev)[None].contiguous()) for b, o, n in seqs]
    mss = time_steps(lambda: [run(a, b_, c) for a, b_, c in singles], stream, 3, 1)
    res["comparison"] = {
        "padded": {"rows": len(seqs), "seqlen": lmax, "ms_per_step": round(msp, 4),
                   "packed_speedup": round(msp / ms, 3),
                   "class_ms": {k: round(v, 4) for k, v in cat_p.items()},
                   "class_speedup": {k: round(cat_p[k] / cat[k], 3) for k in cat}},
        "single": {"calls_per_step": len(seqs), "ms_per_step": round(mss, 4),
                   "packed_speedup": round(mss / ms, 3)},
    }
    return res


def main():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    # 20 warm-up steps by default: the clocks settle only after tens of milliseconds of work
    # (5 left the short configs' timed steps up to 8% slow)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--config", default="2")
    ap.add_argument("--variant", default="paper", choices=["paper", "general"])
    ap.add_argument("--dtype", default=None, choices=["f32", "bf16"],
                    help="storage type of the activations, overriding the workload's (bf16 at the large shapes)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--block", action="store_true",
                    help="time one packed Mamba-1.4B block (projections, norm, conv, scan), fwd+bwd, "
                         "against padding and single-sequence calls, instead of the operator step")
    ap.add_argument("--no-compare", action="store_true",
                    help="skip the padded / single-sequence runs of the same tokens (Mamba-1.4B shape only)")
    ap.add_argument("--cpu-rows", type=int, default=8)
    ap.add_argument("--no-workloads", action="store_true",
                    help="at the Mamba-1.4B shape, skip the other workloads (configs 1, 3, 4a, 4b, fp32, random A)")
    ap.add_argument("--copy-probe", type=int, default=0, metavar="BYTES",
                    help="only copy BYTES with a plain device copy (calibrates HBM byte counters)")
    args = ap.parse_args()
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print(f"bench.py runs on one GPU only (got --gpus {args.gpus}, WORLD_SIZE {world}); "
              "the path is single-GPU; rows would be split across ranks, one process per GPU.", file=sys.stderr)
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

    if args.block:
        if not os.path.exists(_lib.LIB_PATH):
            import __graft_entry__
            __graft_entry__.build()
        print(json.dumps(block_bench(args)), flush=True)
        return
    if not os.path.exists(_lib.LIB_PATH):
        import __graft_entry__
        __graft_entry__.build()
    lib = _lib.load()
    dev = torch.device("cuda:0")
    stream = torch.cuda.current_stream(dev)
    cfg = W.config(args.config, **({"dtype": args.dtype} if args.dtype else {}))
    Nb, Dn, L, N, Wd = cfg.batch, cfg.dim, cfg.seqlen, cfg.dstate, cfg.width
    code = _lib.BF16 if cfg.dtype == "bf16" else _lib.F32

    head = run_workload(lib, cfg, args.variant, args.steps, args.warmup, stream, keep=True)
    print(f"# timed {args.steps} steps: median {head['ms_per_step']:.3f} ms/step, mean {head['mean_ms_per_step']:.3f}",
          file=sys.stderr, flush=True)
    d, tens, step = head.pop("_d"), head.pop("_tens"), head.pop("_step")
    op_ms = {k: v["ms"] for k, v in head["ops"].items()}

    cold = cold_steps(step, stream, args.steps)
    cold["tokens_per_s"] = round(Nb * L / (cold["ms_per_step"] * 1e-3), 1)

    mb = minimal_bytes(Nb, Dn, L, N, Wd, 2 if cfg.dtype == "bf16" else 4)
    E = Nb * Dn * L
    bwd_s = op_ms["scan_bwd"] * 1e-3
    achieved = E * N * SLOTS_BWD / bwd_s / 1e12
    peak = VALU_PEAK / 1e12
    traffic = stored_traffic({"batch": Nb, "seqlen": L, "dim": Dn, "dstate": N, "storage": cfg.dtype})
    roof = {
        # the dominant kernel is issue-bound (plain fp32 VALU arithmetic): its roofline is the
        # VALU issue rate; the metric's own roofline, HBM, is reported beside it
        "bound": "alu", "achieved": round(achieved, 3), "peak": round(peak, 3), "unit": "Tslot/s",
        "frac": round(achieved / peak, 4),
        "traffic": (traffic["bytes_per_launch"] if traffic else None),
        "traffic_source": ("replayed from the stored rocprofv3 FETCH_SIZE/WRITE_SIZE run "
                           "profiles/scan_bwd_traffic_mamba1.4b_step.json (same kernel source hash and shape), "
                           "not measured in this run" if traffic else None),
        "kernel": "selective_scan_bwd (main kernel + finalize kernels, one ABI call)",
        "duration_ms": round(op_ms["scan_bwd"], 4),
        "hbm": {"bound": "hbm", "achieved": round(mb["scan_bwd"] / bwd_s / 1e9, 1), "peak": HBM_PEAK / 1e9,
                "unit": "GB/s", "frac": round(mb["scan_bwd"] / bwd_s / HBM_PEAK, 4),
                "bytes_per_launch": int(mb["scan_bwd"])},
        "metric_roofline": "hbm (the metric's % of HBM peak: roofline.hbm.frac for this kernel, "
                           "hbm_frac / scan_hbm_frac for the step)",
    }
    line = {
        "metric": METRIC, "value": round(Nb * L / (head["ms_per_step"] * 1e-3), 1), "unit": "tokens/s",
        "n_gpus": 1, "steps": args.steps, "warmup": args.warmup, "ms_per_step": head["ms_per_step"],
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": cfg.dtype, "data": "synthetic",
        "config": head["config"],
        "mean_ms_per_step": head["mean_ms_per_step"],
        "timing": "ms_per_step and per-op ms are medians over the K timed steps (HIP events on the launch "
                  "stream after every ABI call); value = tokens / median step",
        "hbm_frac": head["hbm_frac"],
        "minimal_bytes_per_step": head["minimal_bytes_per_step"],
        "ops": head["ops"],
        "scan_hbm_frac": head["scan_hbm_frac"],
        "roofline": roof,
        "cold_cache": cold,
        "device": torch.cuda.get_device_name(0),
    }
    if args.config == "2" and not args.no_compare:
        print("# state passing: every row continues a sequence", file=sys.stderr, flush=True)
        line["state_passing"] = with_states(lib, tens, d["pos"], code, Wd, stream, steps=10, warmup=3,
                                            packed_step=step)
        print("# comparison: padded and single-sequence runs of the same tokens", file=sys.stderr, flush=True)
        line["comparison"] = comparison(lib, tens, d["pos"], code, Wd, stream, steps=5, warmup=2,
                                        packed_ms=head["ms_per_step"])
    if cfg.lengths[0] == "lognormal":
        line["packing_padding"] = packing_rates(cfg.lengths, L)
    cpu_d = d
    del tens, step
    torch.cuda.empty_cache()
    if args.config == "2" and not args.no_workloads:
        # every other workload, through the same step: the other layer shapes, the boundary
        # stress and long-row rows, fp32 activations, and random parameter values
        extra = {}
        for key, name, kw, var in (("1", "1", {}, "paper"), ("3", "3", {}, "paper"), ("4a", "4a", {}, "paper"),
                                   ("4b", "4b", {}, "paper"), ("2", "2-f32", {"dtype": "f32"}, "paper"),
                                   ("2", "2-general", {}, "general")):
            print(f"# workload {name}", file=sys.stderr, flush=True)
            r = run_workload(lib, W.config(key, **kw), var, args.steps, args.warmup, stream)
            r.pop("minimal_bytes_per_step")
            extra[name] = r
            torch.cuda.empty_cache()
        line["workloads"] = extra
        print("# packed Mamba-1.4B block", file=sys.stderr, flush=True)
        blk = block_bench(args, d=cpu_d if args.variant == "paper" and args.dtype in (None, "bf16") else None)
        blk.pop("metric", None)
        line["block"] = blk
        torch.cuda.empty_cache()
    if not args.no_cpu_baseline:
        print("# cpu baseline (oracle)", file=sys.stderr, flush=True)
        line["cpu_baseline"] = cpu_baseline(cpu_d, cfg, args.cpu_rows)
    print(json.dumps(line), flush=True)


def run_workload(lib, cfg, variant, steps, warmup, stream, keep=False):
    """Synthetic inputs of one workload on the device, K timed steps after W warm-ups, with
    a HIP event after every ABI call of every timed step: median step and per-op times,
    the minimal bytes of each op and the resulting fractions of the HBM peak."""
    import numpy as np
    import torch
    import workloads as W
    from paper_2408_03865_amd import _lib
    dev = stream.device
    Nb, Dn, L, N, Wd = cfg.batch, cfg.dim, cfg.seqlen, cfg.dstate, cfg.width
    code = _lib.BF16 if cfg.dtype == "bf16" else _lib.F32
    tdt = torch.bfloat16 if cfg.dtype == "bf16" else torch.float32
    s = 2 if cfg.dtype == "bf16" else 4
    print(f"# generating config {cfg.key} inputs {Nb}x{Dn}x{L} {cfg.dtype} {variant}", file=sys.stderr, flush=True)
    d = W.make_inputs(cfg, variant=variant)
    tens = {k: torch.from_numpy(d[k]).to(tdt).to(dev) for k in ("x", "delta", "z", "B", "C", "dout")}
    tens.update({k: torch.from_numpy(np.ascontiguousarray(d[k], dtype=np.float32)).to(dev)
                 for k in ("A", "D", "delta_bias", "w", "bias")})
    tens["pos"] = torch.from_numpy(d["pos"]).to(dev)
    chain = Chain(lib, tens, code, Wd, stream)
    ops = chain.ops()

    def step():
        for _, f in ops:
            f()

    for _ in range(warmup):
        step()
    torch.cuda.synchronize()
    # timed region: exactly K steps, with a HIP event on the launch stream after every op
    nops = len(ops)
    marks = [torch.cuda.Event(enable_timing=True) for _ in range(steps * nops + 1)]
    torch.cuda.synchronize()
    marks[0].record(stream)
    for it in range(steps):
        for i, (_, f) in enumerate(ops):
            f()
            marks[1 + it * nops + i].record(stream)
    torch.cuda.synchronize()
    total = marks[0].elapsed_time(marks[-1])
    per_step = [marks[it * nops].elapsed_time(marks[(it + 1) * nops]) for it in range(steps)]
    op_ms = {name: float(np.median([marks[it * nops + i].elapsed_time(marks[it * nops + i + 1])
                                    for it in range(steps)]))
             for i, (name, _) in enumerate(ops)}
    ms = float(np.median(per_step))
    mb = minimal_bytes(Nb, Dn, L, N, Wd, s)
    total_bytes = sum(mb.values())
    res = {
        "config": {
            "workload": f"{cfg.name} layer: {Nb} packed rows x {L} tokens, d_inner {Dn}, d_state {N}, "
                        f"conv width {Wd}, {cfg.dtype} activations, fp32 state; sequence lengths "
                        f"{cfg.lengths[0]}{tuple(cfg.lengths[1:])}",
            "batch": Nb, "seqlen": L, "dim": Dn, "dstate": N, "width": Wd, "storage": cfg.dtype,
            "arithmetic": "f32", "sequences": int(len(d["lengths"])), "variant": variant,
        },
        "ms_per_step": round(ms, 4),
        "mean_ms_per_step": round(total / steps, 4),
        "tokens_per_s": round(Nb * L / (ms * 1e-3), 1),
        "hbm_frac": round(total_bytes / (ms * 1e-3) / HBM_PEAK, 4),
        "minimal_bytes_per_step": int(total_bytes),
        "ops": {k: {"ms": round(v, 4), "minimal_GBps": round(mb[k] / (v * 1e-3) / 1e9, 1),
                    "hbm_frac": round(mb[k] / (v * 1e-3) / HBM_PEAK, 4)} for k, v in op_ms.items()},
        "scan_hbm_frac": round((mb["scan_fwd"] + mb["scan_bwd"]) /
                               ((op_ms["scan_fwd"] + op_ms["scan_bwd"]) * 1e-3) / HBM_PEAK, 4),
        "scan_bwd_alu_frac": round(Nb * Dn * L * N * SLOTS_BWD / (op_ms["scan_bwd"] * 1e-3) / VALU_PEAK, 4),
    }
    if keep:
        res.update(_d=d, _tens=tens, _step=step)
    else:
        del chain, ops, tens
    return res


if __name__ == "__main__":
    main()
