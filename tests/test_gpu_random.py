"""Seeded random shapes and options against the oracle: batch, channel count (not
multiples of the 16-channel blocks), row length (ragged against the 8-token
vectors, the 128/256-token chunks and the 512-token conv steps, long enough to be
split into segments or not), conv width, dtype, length law (from all-length-1 rows
to one sequence per row) and A recipe.  Every output and gradient of both operators
is compared element by element."""
import numpy as np
import pytest

import workloads as W
from gpu_common import (PER_B, PER_CHANNEL, PER_TOKEN, TOL, check_bf16_rounding, compare, gpu_inputs, note,
                        oracle_run, run_gpu)

pytestmark = pytest.mark.gpu

ALL = PER_TOKEN + PER_CHANNEL + PER_B


def _case(i):
    rng = np.random.default_rng(9100 + i)
    batch = int(rng.integers(1, 5))
    dim = int(rng.integers(1, 71))
    seqlen = int(rng.choice([1, 7, 64, 129, 255, 513, 1000, 2049, 3001]))
    width = int(rng.integers(2, 5))
    dtype = ["f32", "bf16"][i % 2]
    law = [("lognormal", 2.0, 1.5, 1, seqlen), ("lognormal", 6.0, 1.0, 1, seqlen),
           ("lognormal", 0.0, 0.1, 1, 1), ("edges", 1, 64), ("arange",)][int(rng.integers(0, 5))]
    variant = ["paper", "general"][int(rng.integers(0, 2))]
    return batch, dim, seqlen, width, dtype, law, variant


@pytest.mark.parametrize("i", range(12))
def test_random_case(i):
    batch, dim, seqlen, width, dtype, law, variant = _case(i)
    note(f"random case {i}: batch {batch} dim {dim} seqlen {seqlen} width {width} {dtype} {law} {variant}")
    cfg = W.Config("random", "random", batch, seqlen, dim, 16, width, dtype, law, 9200 + i)
    d = W.make_inputs(cfg, variant=variant)
    g = gpu_inputs(d, dtype)
    r = run_gpu(g, out_f32=(dtype == "bf16"))
    compare(r, oracle_run(d), TOL[dtype], ALL, label=f"random {i} ")
    if dtype == "bf16":
        check_bf16_rounding(run_gpu(g, out_f32=False), r, f"random {i} bf16-out ")


def _sweep_case(i):
    rng = np.random.default_rng(50000 + i)
    batch = int(rng.integers(1, 4))
    dim = int(rng.integers(1, 97))
    seqlen = int(rng.choice([1, 2, 3, 8, 9, 127, 128, 129, 256, 257, 511, 512, 1023, 1536, 2048, 2500, 4096, 5000]))
    width = int(rng.integers(2, 5))
    dtype = ["f32", "bf16"][int(rng.integers(0, 2))]
    law = [("lognormal", 2.0, 1.5, 1, seqlen), ("lognormal", 6.0, 1.0, 1, seqlen), ("lognormal", 4.0, 2.0, 1, seqlen),
           ("lognormal", 0.0, 0.1, 1, 1), ("edges", 1, 64), ("edges", 1, 300), ("arange",)][int(rng.integers(0, 7))]
    variant = ["paper", "general"][int(rng.integers(0, 2))]
    return batch, dim, seqlen, width, dtype, law, variant


def test_random_sweep():
    """300 more seeded cases from a wider generator (row lengths on and around every
    chunk and vector edge up to 5000 tokens, up to 96 channels, so that short batches
    split their rows into segments), one after the other; the first mismatch fails
    and names its case."""
    for i in range(300):
        batch, dim, seqlen, width, dtype, law, variant = _sweep_case(i)
        note(f"sweep case {i}: batch {batch} dim {dim} seqlen {seqlen} width {width} {dtype} {law} {variant}")
        cfg = W.Config("sweep", "sweep", batch, seqlen, dim, 16, width, dtype, law, 60000 + i)
        d = W.make_inputs(cfg, variant=variant)
        g = gpu_inputs(d, dtype)
        r = run_gpu(g, out_f32=(dtype == "bf16"))
        compare(r, oracle_run(d), TOL[dtype], ALL, label=f"sweep {i} ")
        if dtype == "bf16":
            check_bf16_rounding(run_gpu(g, out_f32=False), r, f"sweep {i} bf16-out ")
