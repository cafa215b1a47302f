"""GPU parity of ubt_topk (softmax statistics and candidate sets) against the oracle."""
from __future__ import annotations

import numpy as np
import pytest

import oracle
import parity
import synth

pytestmark = pytest.mark.gpu


def _run(x: np.ndarray, K: int, view=None):
    import torch

    import paper_2609_39972_amd as ubt
    from gpu_util import dev_values, to_np

    t = dev_values(x)
    if view is not None:
        t = view(t)
    out = ubt.topk(t, K)
    torch.cuda.synchronize()
    return to_np(out)


def _rows(x: np.ndarray) -> np.ndarray:
    return x.reshape(-1, x.shape[-1])


def _check(x: np.ndarray, K: int):
    from gpu_util import say

    say(f"topk shape={x.shape} dtype={x.dtype} K={K}")
    g = _run(x, K)
    parity.check_topk(g, oracle.topk(x, K))
    return g


def _bf16(v: np.ndarray) -> np.ndarray:
    return synth.round_bf16_bits(v)


@pytest.mark.parametrize("V,K", [(1, 1), (8, 8), (33, 8), (100, 64), (1000, 1), (4095, 16), (4096, 4), (8191, 16),
                                 (8192, 8), (8193, 16), (20000, 64), (151937, 16)])
@pytest.mark.parametrize("dt", ["f32", "bf16"])
def test_shapes_and_ragged_tails(V, K, dt):
    rng = np.random.default_rng(V + K)
    x = synth.store(rng.normal(0, 2.5, (2, 3, V)), dt)
    _check(x, K)


@pytest.mark.parametrize("K", list(range(1, 65)))
def test_every_k(K):
    rng = np.random.default_rng(100 + K)
    _check(synth.store(rng.normal(0, 1.5, (1, 2, 12345)), "bf16"), K)


@pytest.mark.parametrize("dt", ["f32", "bf16"])
def test_all_equal_rows_take_lowest_ids(dt):
    x = synth.store(np.full((1, 3, 30000), 0.75), dt)
    g = _check(x, 64)
    assert (g["cand_ids"] == np.arange(64)).all()


@pytest.mark.parametrize("dt", ["f32", "bf16"])
def test_heavy_duplicates(dt):
    rng = np.random.default_rng(7)
    x = synth.store(np.round(rng.normal(0, 1, (2, 4, 50000)) * 2) / 2, dt)
    _check(x, 32)


def test_signed_zero_and_neg_inf():
    x = np.full((1, 2, 9000), -np.inf, np.float32)
    x[0, 0, [17, 4000, 8999]] = [-0.0, 0.0, -0.0]
    x[0, 1, 5] = 3.0
    x[0, 1, 8191] = -2.0
    g = _check(x, 6)
    assert g["cand_ids"][0, 0, :3].tolist() == [17, 4000, 8999]
    xb = synth.round_bf16_bits(x.astype(np.float64))
    _check(xb, 6)


def test_zipf_rows_full_vocab():
    w = synth.WORKLOADS[3]
    x = synth.logits(w, 0, rows=np.arange(40)).reshape(4, 10, w.V)
    _check(x, 8)
    _check(x, 16)


@pytest.mark.parametrize("K", [64, 48, 17])
def test_zipf_rows_large_k(K):
    """The paper's configuration (K = 64) and other large K on permuted-zipf rows."""
    w = synth.WORKLOADS[6]
    x = synth.logits(w, 0, rows=np.arange(24)).reshape(2, 12, w.V)
    _check(x, K)


@pytest.mark.parametrize("dt", ["f32", "bf16"])
def test_rising_rows_fill_every_buffer(dt):
    """Values that rise along the row: the first tiles hold the smallest values, so every
    later group passes the first threshold and each wave's buffer fills and merges again
    and again; with descending rows nothing after the first tiles passes."""
    V = 151936
    up = np.linspace(-4.0, 4.0, V)
    x = synth.store(np.stack([up, up[::-1], np.round(up * 8) / 8]).reshape(1, 3, V), dt)
    _check(x, 64)
    _check(x, 33)


@pytest.mark.parametrize("dt", ["f32", "bf16"])
def test_heavy_duplicates_k64(dt):
    """Long runs of equal values around the K-th: the selection descends into the ids."""
    rng = np.random.default_rng(8)
    x = synth.store(np.round(rng.normal(0, 1, (2, 4, 50000)) * 2) / 2, dt)
    _check(x, 64)


def test_high_entropy_rows():
    w = synth.WORKLOADS[4]
    x = synth.logits(w, 0, rows=np.arange(30)).reshape(2, 15, w.V)
    _check(x, 16)


def test_strided_block_view_and_padding():
    """Rows taken from a [B, L, V] block (skip the anchor row) and rows with padded strides."""
    import torch

    rng = np.random.default_rng(3)
    V = 10007
    block = synth.store(rng.normal(0, 2, (3, 6, V)), "bf16")
    g = _run(block, 8, view=lambda t: t[:, 1:, :])
    parity.check_topk(g, oracle.topk(np.ascontiguousarray(block[:, 1:, :]), 8))
    # padded rows: aligned (bf16 pad of 9 -> row stride 10016 elements = 20032 B) and unaligned (f32 pad of 3)
    for dt, pad in (("bf16", 9), ("f32", 3)):
        big = synth.store(rng.normal(0, 2, (2, 3, V + pad)), dt)
        g = _run(big, 12, view=lambda t: t[:, :, :V])
        parity.check_topk(g, oracle.topk(np.ascontiguousarray(big[:, :, :V]), 12))
    del torch


def test_repeat_is_bitwise_identical():
    import torch

    import paper_2609_39972_amd as ubt
    from gpu_util import dev_values, to_np

    rng = np.random.default_rng(11)
    xa = synth.store(rng.normal(0, 2, (2, 5, 40000)), "bf16")
    ta = dev_values(xa)
    outs = [to_np(ubt.topk(ta, 16)) for _ in range(3)]
    torch.cuda.synchronize()
    parity.check_topk(outs[0], oracle.topk(xa, 16))
    for o in outs[1:]:
        for k in o:
            assert np.array_equal(o[k], outs[0][k]), f"{k} not bitwise reproducible"


@pytest.mark.parametrize("cfg", [1, 2, 3, 4, 5, 6])
def test_workload_full_size(cfg):
    """Every row of the workload at its full size (all buffers of one pool entry)."""
    from gpu_util import say

    w = synth.WORKLOADS[cfg]
    say(f"topk workload {cfg}: {w.describe()}")
    x = synth.logits(w, 0)
    g = _run(x, w.K)
    parity.check_topk(g, oracle.topk(x, w.K))


def test_many_launches_alternating_inputs_are_identical():
    """Two inputs alternating over many back-to-back launches into the same outputs:
    every result must equal that input's first one (no state carried between launches)."""
    import torch

    import paper_2609_39972_amd as ubt
    from gpu_util import dev_values, to_np

    w = synth.WORKLOADS[3]
    xs = [synth.logits(w, b, rows=np.arange(b * 64, b * 64 + 64)).reshape(4, 16, w.V) for b in range(2)]
    ts = [dev_values(x) for x in xs]
    outs = [to_np(ubt.topk(ts[j % 2], 8)) for j in range(200)]
    torch.cuda.synchronize()
    for j in range(2):
        parity.check_topk(outs[j], oracle.topk(xs[j], 8))
    for j in range(2, 200):
        for k in outs[j]:
            assert np.array_equal(outs[j][k], outs[j % 2][k]), f"launch {j}: {k} differs"


@pytest.mark.parametrize("B,gamma", [(1, 1), (4, 63), (64, 4), (5, 60)])
def test_row_counts_around_the_wave_switch(B, gamma):
    """Fewer and more rows than compute units use different workgroup sizes."""
    rng = np.random.default_rng(B * gamma)
    _check(synth.store(rng.normal(0, 2, (B, gamma, 9000)), "bf16"), 8)
