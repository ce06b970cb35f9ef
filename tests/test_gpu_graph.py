"""The C ABI under HIP graph capture: the whole step (conv fwd -> scan fwd saving states ->
scan bwd -> conv bwd) is captured once through torch's graph API (the calls run on the
capture stream; the library allocates, synchronises and clears nothing itself), then
replayed several times with eager work and synchronisations between the replays.  Every
replay must reproduce the eager step bit for bit."""
import numpy as np
import pytest

import workloads as W

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("key", ["1", "4a"])
def test_step_replays_match_eager(key):
    import torch
    import bench
    from paper_2408_03865_amd import _lib
    from gpu_common import note
    note(f"graph capture of the step, config {key}")
    cfg = W.config(key)
    d = W.make_inputs(cfg)
    dev = torch.device("cuda:0")
    tens = {k: torch.from_numpy(d[k]).to(torch.bfloat16).to(dev) for k in ("x", "delta", "z", "B", "C", "dout")}
    tens.update({k: torch.from_numpy(np.ascontiguousarray(d[k], dtype=np.float32)).to(dev)
                 for k in ("A", "D", "delta_bias", "w", "bias")})
    tens["pos"] = torch.from_numpy(d["pos"]).to(dev)
    lib = _lib.load()
    side = torch.cuda.Stream(dev)
    with torch.cuda.stream(side):
        stream = torch.cuda.current_stream(dev)
        chain = bench.Chain(lib, tens, _lib.BF16, cfg.width, stream)
        ops = [f for _, f in chain.ops()]
        outs = ("u", "out", "du", "ddl", "dz", "dx", "dA", "dB", "dC", "dD", "ddb", "dw", "dcb")
        for f in ops:                                   # eager reference
            f()
        torch.cuda.synchronize()
        ref = {k: getattr(chain, k).clone() for k in outs}
        graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(graph, stream=side):
            for f in ops:
                f()
    torch.cuda.synchronize()
    for rep in range(3):
        for k in outs:                                  # eager work between the replays
            getattr(chain, k).fill_(float("nan"))
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        for k in outs:
            got, want = getattr(chain, k), ref[k]
            assert torch.equal(got.view(torch.int16) if got.dtype == torch.bfloat16 else got.view(torch.int32),
                               want.view(torch.int16) if want.dtype == torch.bfloat16 else want.view(torch.int32)), (rep, k)
