"""The seeded input generator: determinism, shapes, bf16 rounding, recipe structure."""
import numpy as np
import torch

from paper_2602_01219_amd import synth


def test_bf16_rounding_matches_torch():
    x = np.random.default_rng(0).standard_normal(10000).astype(np.float32) * 3
    x[:5] = [0.0, -0.0, 1e-40, 65504.0, -2.5]
    ours = synth.f32_to_bf16_bits(x)
    ref = torch.from_numpy(x).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert (ours == ref).all()
    back = synth.bf16_bits_to_f32(ours)
    assert (back == torch.from_numpy(x).to(torch.bfloat16).float().numpy()).all()


def test_deterministic_and_shaped():
    wl = synth.WORKLOADS["vits_bf16"].with_(B=2, H=3)
    a, b = synth.generate(wl), synth.generate(wl)
    for x, y in zip((a.q, a.k, a.v), (b.q, b.k, b.v)):
        assert x.shape == (2, 3, 196, 64) and x.dtype == np.uint16
        assert (x == y).all()
    assert not (a.q == a.k).all()


def test_workload_table():
    W = synth.WORKLOADS
    assert (W["tiny_f32"].N, W["tiny_f32"].M, W["tiny_f32"].k) == (196, 16, 32)
    assert (W["dense_pred_bf16"].lm_h, W["dense_pred_bf16"].lm_w) == (8, 16)
    for w in W.values():
        assert w.lm_h <= w.grid_h and w.lm_w <= w.grid_w and 1 <= w.k <= w.N


def test_voronoi_map_is_piecewise_and_outliers_scaled():
    wl = synth.WORKLOADS["dense_pred_bf16"].with_(B=1, H=1, grid_h=32, grid_w=32, clusters=8)
    inp = synth.generate(wl)
    q = synth.bf16_bits_to_f32(inp.q)[0, 0]
    norms = np.linalg.norm(q, axis=1)
    n_out = int(round(0.05 * 1024))
    # outliers have 4x the norm: the largest norms are separated from the bulk
    top = np.sort(norms)[::-1]
    assert top[n_out - 1] > 1.8 * np.median(norms)
