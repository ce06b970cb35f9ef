"""The seeded generator: packing, position indices, bf16 storage (CPU only)."""
import numpy as np
import pytest

import oracle
import workloads as W


@pytest.mark.parametrize("key", list(W.CONFIGS))
def test_positions_valid(key):
    cfg = W.config(key)
    rng = np.random.Generator(np.random.PCG64(cfg.seed))
    rows = W.draw_row_lengths(cfg.lengths, rng, cfg.batch, cfg.seqlen)
    pos = W.positions_from_lengths(rows, cfg.seqlen)
    assert pos.shape == (cfg.batch, cfg.seqlen) and pos.dtype == np.int32
    assert oracle.check_positions(pos) == -1
    assert int((pos == 0).sum()) == sum(len(r) for r in rows)


def test_edge_rows_hit_tile_edges():
    cfg = W.config("4a")
    rows = W.draw_row_lengths(cfg.lengths, np.random.default_rng(0), cfg.batch, cfg.seqlen)
    pos = W.positions_from_lengths(rows, cfg.seqlen)
    for e in (64, 192, 255, 256, 257, 1024, 4096, cfg.seqlen - 1):
        assert np.all(pos[:, e] == 0), e
    assert np.all(pos[:, 5000:5007] == 0)      # a run of length-1 sequences
    assert np.any(pos[:, 128] != 0)            # some even multiples of 64 carry state


def test_tiny_config_lengths():
    cfg = W.config("0")
    rows = W.draw_row_lengths(cfg.lengths, np.random.default_rng(3), 1, 256)
    assert len(rows[0]) == 5 and all(16 <= n <= 96 for n in rows[0][:4]) and 1 <= rows[0][4] <= 96


def test_bf16_rounding_matches_torch():
    import torch
    a = (np.random.default_rng(1).standard_normal(1 << 16) * 100).astype(np.float32)
    a[:4] = [1 + 2 ** -8, 1 + 3 * 2 ** -8, -(1 + 2 ** -8), 0.0]      # ties to even
    ref = torch.from_numpy(a).to(torch.bfloat16).float().numpy()
    assert np.array_equal(W.bf16_round(a), ref)


def test_inputs_deterministic_and_rounded():
    cfg = W.config("1", dim=64, seqlen=512)
    a, b = W.make_inputs(cfg), W.make_inputs(cfg)
    for k in a:
        assert np.array_equal(a[k], b[k]), k
    for k in W.ACTIVATIONS:
        assert np.array_equal(a[k], W.bf16_round(a[k])), k
    assert np.all(a["A"] == -(np.arange(16) + 1)[None, :])
    g = W.make_inputs(cfg, variant="general")
    assert np.all(g["A"] < 0) and not np.all(g["D"] == 1)


def test_pack_unpack_roundtrip():
    rng = np.random.default_rng(2)
    seqs = [rng.standard_normal((3, n)) for n in (5, 1, 9)]
    packed, pos = W.pack(seqs)
    assert packed.shape == (1, 3, 15)
    assert list(pos[0]) == list(range(5)) + [0] + list(range(9))
    for s, t in zip(seqs, W.unpack(packed, [5, 1, 9])):
        assert np.array_equal(s, t)
