"""Seeded synthetic workloads: determinism, shapes and realised densities."""
import hashlib
import json
import os

import numpy as np
import pytest
import torch

import workloads as wl

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _sha(t):
    return hashlib.sha256(t.contiguous().view(torch.uint8).numpy().tobytes()).hexdigest()


def _within(frac, d, n, sig=4.0):
    return abs(frac - d) <= sig * np.sqrt(d * (1 - d) / n) + 1e-12


def test_determinism_and_golden_hashes():
    ref = json.load(open(os.path.join(GOLDEN, "workload_hashes.json")))
    for key, spec in _hash_specs().items():
        a = wl.draw(spec)
        b = wl.draw(spec)
        for name in ("x", "w", "dy"):
            assert torch.equal(a[name].view(torch.uint8) if a[name].dtype == torch.bfloat16 else a[name],
                               b[name].view(torch.uint8) if b[name].dtype == torch.bfloat16 else b[name])
            assert _sha(a[name]) == ref[key][name], (key, name)


def _hash_specs():
    return {
        "config1": wl.config1()[0],
        "config2_N1_H14": wl.config2(N=1, H=14)[0],
        "config3_l2_N1_H8": wl.config3(N=1, H=8)[1],
        "config4_clustered_d0.3_N1": wl.config4(0.3, "clustered", N=1)[0],
    }


def test_config1_recipe():
    s = wl.config1()[0]
    t = wl.draw(s)
    assert t["x"].dtype == torch.float32 and t["x"].shape == (2, 16, 16, 16)
    assert t["w"].shape == (16, 3, 3, 16) and t["dy"].shape == (2, 16, 16, 16)
    x = t["x"].numpy()
    assert np.all(x >= 0)
    assert _within(np.mean(x > 0), 0.5, x.size)
    assert _within(np.mean(t["dy"].numpy() != 0), 0.5, x.size)
    std = np.std(t["w"].numpy())
    assert abs(std - np.sqrt(2 / (9 * 16))) < 0.1 * np.sqrt(2 / (9 * 16))


def test_config2_recipe_small_batch():
    s = wl.config2(N=2)[0]
    t = wl.draw(s)
    assert t["x"].dtype == torch.bfloat16 and t["x"].shape == (2, 56, 56, 256)
    x = t["x"].float().numpy()
    assert _within(np.mean(x > 0), 0.40129, x.size)
    assert _within(np.mean(t["dy"].float().numpy() != 0), 0.4, x.size)


def test_config3_dy_is_next_layer_footprint():
    specs = wl.config3(N=2, H=8)
    assert [(s.C, s.K, s.R) for s in specs] == [(256, 64, 1), (64, 64, 3), (64, 256, 1)]
    t0 = wl.draw(specs[0])
    t1 = wl.draw(specs[1], want=("x",))
    assert torch.equal(t0["dy"] != 0, t1["x"] > 0)
    for s, d in zip(specs, (0.6, 0.45, 0.3)):
        x = wl.draw(s, want=("x",))["x"].float().numpy()
        assert _within(np.mean(x > 0), d, x.size)


@pytest.mark.parametrize("kind", ["bernoulli", "clustered", "channel_shared"])
@pytest.mark.parametrize("d", [0.1, 0.5, 0.9])
def test_config4_densities(kind, d):
    s = wl.config4(d, kind, N=2)[0]
    t = wl.draw(s)
    x = t["x"].float().numpy()
    frac = np.mean(x > 0)
    if kind == "bernoulli":
        assert _within(frac, d, x.size)
    else:
        assert abs(frac - d) < 0.02  # exact quantile threshold on a continuous field
    if kind == "channel_shared":
        live = x > 0
        assert np.all(live == live[..., :1])


def test_config4_clustered_is_spatially_correlated():
    s = wl.config4(0.3, "clustered", N=2)[0]
    live = wl.draw(s, want=("x",))["x"].float().numpy() > 0
    same = np.mean(live[:, 1:, :, :] == live[:, :-1, :, :])
    iid = 0.3 ** 2 + 0.7 ** 2
    assert same > iid + 0.1


def test_config5_layers():
    specs = wl.config5(N=1, scale=8)
    assert len(specs) == 13
    assert [s.masked for s in specs] == [False, True, False, True, False, True, True, False, True, True,
                                         False, True, True]
    assert not specs[0].need_dx
    t = wl.draw(specs[1])
    # maxpool-routed gradient: at most one live position per 2x2 window
    live = t["dy"].float().numpy() != 0
    n, h, w, c = live.shape
    per_win = live.reshape(n, h // 2, 2, w // 2, 2, c).sum(axis=(2, 4))
    assert per_win.max() <= 1
    assert wl.vgg_density(1) == 0.5 and abs(wl.vgg_density(13) - 0.15) < 1e-12


def test_config5_pooled_inputs():
    """The inputs after a max-pool are pooled ReLU outputs: density
    1 - (1 - d)^4 of the layer before (i.i.d. footprint), every value the
    maximum of a 2x2 window; with pooled_mask the four post-pool layers are
    masked (by pooled > 0), the others unchanged."""
    specs = wl.config5(N=2, scale=4)
    pooled = wl.config5(N=2, scale=4, pooled_mask=True)
    after = {3, 5, 8, 11}
    assert [s.masked for s in pooled] == [s.masked or s.layer_id in after for s in specs]
    for s in specs:
        assert (s.x_kind == "pooled_gauss") == (s.layer_id in after)
    for l in (3, 11):
        s = specs[l - 1]
        x = wl.draw(s, want=("x",))["x"].float().numpy()
        assert x.shape == (s.N, s.H, s.W, s.C) and np.all(x >= 0)
        d = 1 - (1 - wl.vgg_density(l - 1)) ** 4
        assert _within(np.mean(x > 0), d, x.size)
        assert torch.equal(wl.draw(pooled[l - 1], want=("x",))["x"].view(torch.uint8),
                           wl.draw(s, want=("x",))["x"].view(torch.uint8))


def test_dense_flops_config2():
    s = wl.config2()[0]
    assert s.dense_flops() == 2 * 32 * 256 * 56 * 56 * 256 * 9


def test_draw_on_device_vgg_recipes_on_the_host():
    """The device-side generator (used for the VGG-16 stack inside the
    benchmark) follows the recipes: post-pool inputs are 2x2 maxima of a
    ReLU output of density d (density 1 - (1 - d)^4), max-pool-routed dY has
    at most one live position per 2x2 window, and the image's padded
    channels are exactly zero.  Run with the CPU generator at reduced size."""
    specs = wl.config5(N=2, scale=8)
    d = wl.draw_on_device(specs[2], device="cpu")          # conv2_1: pooled input
    dens_in = wl.vgg_density(2)
    x_live = (d["x"].float() > 0).float().mean().item()
    assert abs(x_live - (1 - (1 - dens_in) ** 4)) < 0.02
    d = wl.draw_on_device(specs[1], device="cpu")          # conv1_2: followed by a pool
    live = d["dy"].float() != 0
    n, p, q, k = live.shape
    per_win = live.view(n, p // 2, 2, q // 2, 2, k).sum(dim=(2, 4))
    assert per_win.max().item() <= 1
    d_l = wl.vgg_density(2)
    assert abs(per_win.float().mean().item() - (1 - (1 - d_l) ** 4)) < 0.02
    d = wl.draw_on_device(specs[0], device="cpu")          # conv1_1: 3 channels stored as 8
    assert d["x"].shape[-1] == 8 and not d["x"][..., 3:].any() and not d["w"][..., 3:].any()
    assert d["x"][..., :3].any()
    assert d["dy"].dtype == torch.bfloat16
