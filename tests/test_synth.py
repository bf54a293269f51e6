"""Seeded input generators: shapes, determinism and the stated distributions."""
import numpy as np
import torch

from synth import WORKLOADS, gen_module_inputs, round_half_even_count, workload


def test_workload_sizes():
    assert WORKLOADS["linear256"].n_tiles == 1024
    assert WORKLOADS["down3b"].n_tiles == 352256
    assert WORKLOADS["block3b"].n_weights == 77070336 and WORKLOADS["block3b"].n_tiles == 1204224
    assert WORKLOADS["layer32b"].n_weights == 487587840 and WORKLOADS["layer32b"].n_tiles == 3809280
    assert WORKLOADS["stack3b"].n_weights == 2774532096 and WORKLOADS["stack3b"].n_tiles == 43352064
    assert WORKLOADS["down3b"].candidates == 352256 * 256


def test_outlier_counts():
    assert round_half_even_count(0.01, 11008) == 110
    assert round_half_even_count(0.005, 5120) == 26
    assert round_half_even_count(0.005, 27648) == 138


def test_generators_deterministic_and_shaped():
    wl = workload("block3b")
    m = wl.modules[1]  # k_proj 256 x 2048
    a = gen_module_inputs(wl, m)
    b = gen_module_inputs(wl, m)
    assert a["W"].dtype == torch.bfloat16 and a["W"].shape == (256, 2048)
    assert torch.equal(a["W"], b["W"]) and torch.equal(a["d"], b["d"])
    assert a["d"].shape == (256, 2048) and torch.all(a["d"] > 0)
    # q/k/v share one activation vector: d - 0.5 F is the same across q and k rows
    F = a["d"].double().numpy()
    assert np.isfinite(F).all()


def test_outlier_columns_scaled():
    wl = workload("down3b", modules=(workload("down3b").modules[0].__class__("x", 64, 11008, 0, 0, 0),))
    W = gen_module_inputs(wl, wl.modules[0])["W32"]
    colmax = W.abs().amax(dim=0)
    assert (colmax > 0.2).sum().item() >= 100  # about 110 channels carry 8x the scale


def test_fisher_proxy_moments():
    wl = workload("block3b")
    from synth.workloads import gen_fisher
    f = gen_fisher(wl, wl.modules[1]).double()
    # mean of 64 squared N(0,1): mean 1, variance 2/64
    assert abs(f.mean().item() - 1.0) < 0.01 and abs(f.var().item() - 2 / 64) < 0.003
