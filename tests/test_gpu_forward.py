"""GPU parity of the forward convolution with the fused ReLU and footprint
emission (conv_fwd_relu_mask) against the fp64 oracle.

Values are compared with the normwise and per-element bounds of the other
parity tests.  The footprint is an integer decided by floating point, so it
is checked in the precision that decides it: the emitted bits must equal,
word for word, the bitmap of the stored output as cbw_relu_mask_pack computes
it; against the oracle, the bit must match the sign of the fp64 sum wherever
that sum is farther from zero than its error bound.  Every output must be
non-negative with +0.0 zeros, and the output must not depend on whether the
footprint is requested.
"""
import numpy as np
import pytest
import torch

import oracle
import paper_2109_07710_amd as cb
from parity import U_ACC, check_values, tol_for

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    cb.lib()


# name, N, C, H, W, K, R, S, pad, dtype, w_layout
CASES = [
    ("f32_3x3", 2, 16, 16, 16, 16, 3, 3, 1, "f32", "krsc"),          # configuration 1's shape
    ("bf16_3x3_K96", 2, 64, 10, 12, 96, 3, 3, 1, "bf16", "krsc"),    # whole footprint words
    ("bf16_3x3_K40", 2, 32, 9, 11, 40, 3, 3, 1, "bf16", "krsc"),     # words shared by two pixels
    ("bf16_1x1", 2, 256, 7, 9, 64, 1, 1, 0, "bf16", "krsc"),
    ("bf16_5x5_kcrs", 1, 48, 13, 10, 32, 5, 5, 2, "bf16", "kcrs"),
    ("bf16_3x3_pad0", 3, 64, 12, 12, 64, 3, 3, 0, "bf16", "krsc"),
    ("bf16_multi_tile", 4, 256, 28, 28, 288, 3, 3, 1, "bf16", "krsc"),  # 2 channel tiles, 13 pixel tiles
    ("f32_K20", 2, 12, 8, 8, 20, 3, 3, 1, "f32", "krsc"),
    ("bf16_unsplit_K72", 10, 64, 56, 56, 72, 3, 3, 1, "bf16", "krsc"),   # >128 tiles: no split, shared words
    ("bf16_unsplit_K64", 10, 64, 56, 56, 64, 3, 3, 1, "bf16", "krsc"),   # >128 tiles: no split, whole words
]


def _inputs(N, C, H, W, K, R, S, dtype, seed):
    """X = relu(N(0,1) - 0.25) (about 40% non-zero, as after a ReLU), W He-init,
    both rounded to the element type before either side sees them."""
    rng = np.random.default_rng(seed)
    x = np.maximum(rng.standard_normal((N, H, W, C), dtype=np.float32) - 0.25, 0)
    w = rng.standard_normal((K, R, S, C), dtype=np.float32) * np.float32(np.sqrt(2.0 / (C * R * S)))
    tdt = torch.bfloat16 if dtype == "bf16" else torch.float32
    return torch.from_numpy(x).to(tdt), torch.from_numpy(w).to(tdt)


def _run(desc, x, w, want_mask=True):
    N, P, Q, K = desc.N, desc.P, desc.Q, desc.K
    Y = torch.empty((N, P, Q, K), dtype=x.dtype, device="cuda")
    words = max(cb.cbw_dy_mask_words(desc), 1)
    ym = torch.full(((words + 3) // 4 * 4,), -1, dtype=torch.int32, device="cuda") if want_mask else None
    ws = cb.workspace(desc, cb.CBW_OP_FWD)
    cb.conv_fwd_relu_mask(desc, x, w, Y, ym, ws)
    torch.cuda.synchronize()
    return Y, ym


def _reference_bits(Y):
    """cbw_relu_mask_pack of the stored output (Y read as the next layer's X)."""
    N, P, Q, K = Y.shape
    nd = cb.ConvDesc.make(N, K, P, Q, 8, 1, 1, 1, 0, dtype="bf16" if Y.dtype == torch.bfloat16 else "f32")
    bits = torch.zeros(max(cb.cbw_mask_words(nd), 1), dtype=torch.int32, device="cuda")
    cb.cbw_relu_mask_pack(nd, Y, bits)
    torch.cuda.synchronize()
    return bits


def _check(name, N, C, H, W, K, R, S, pad, dtype, w_layout, seed=1):
    print("\n[case] forward %s N=%d C=%d K=%d %dx%d R=%d S=%d pad=%d %s %s" %
          (name, N, C, K, H, W, R, S, pad, dtype, w_layout), flush=True)
    x, w = _inputs(N, C, H, W, K, R, S, dtype, seed)
    desc = cb.ConvDesc.make(N, C, H, W, K, R, S, 1, pad, dtype=dtype, w_layout=w_layout)
    wdev = w.permute(0, 3, 1, 2).contiguous() if w_layout == "kcrs" else w
    Y, ym = _run(desc, x.cuda(), wdev.cuda())

    x64 = oracle.nhwc_to_nchw(x.double().numpy())
    w64 = oracle.krsc_to_kcrs(w.double().numpy())
    z, y, a, n = oracle.conv_fwd_relu(x64, w64, (1, 1), (pad, pad))
    g = oracle.nhwc_to_nchw(Y.float().cpu().double().numpy())
    e = check_values(g, y, a, n, tol_for(dtype), dtype == "bf16", name + " Y")

    # non-negative, and every zero is +0.0
    raw = Y.view(torch.int16 if dtype == "bf16" else torch.int32).cpu().numpy()
    assert not (raw < 0).any(), "negative or -0.0 output"

    # the emitted footprint is the bitmap of the stored output, word for word
    words = cb.cbw_dy_mask_words(desc)
    ref = _reference_bits(Y)
    assert torch.equal(ym[:words].cpu(), ref[:words].cpu()), "emitted footprint differs from the output's bitmap"

    # against the oracle: the bit follows the sign of the fp64 sum where it is unambiguous
    bits = oracle.unpack_bits(ym[:words].cpu().numpy().view(np.uint32), N * K * desc.P * desc.Q)
    live = oracle.nhwc_to_nchw(bits.reshape(N, desc.P, desc.Q, K))
    sure = np.abs(z) > 2.0 * n * U_ACC * a * 1.01 + (2.0 ** -8 if dtype == "bf16" else 0) * np.abs(z)
    assert np.array_equal(live[sure], z[sure] > 0), "footprint bit against the oracle's sign"

    # the output does not depend on whether the footprint is requested
    Y2, _ = _run(desc, x.cuda(), wdev.cuda(), want_mask=False)
    assert torch.equal(Y.view(torch.int16 if dtype == "bf16" else torch.int32),
                       Y2.view(torch.int16 if dtype == "bf16" else torch.int32))
    print("  normwise %.3e, live fraction %.3f" % (e, live.mean()), flush=True)


@pytest.mark.parametrize("case", CASES, ids=[c[0] for c in CASES])
def test_forward_parity(case):
    _check(*case)


def test_forward_reference_chain():
    """The emitted footprint drives the next layer's masked data gradient
    exactly as the packed bitmap of the stored output does."""
    N, C, H, W, K = 2, 64, 10, 12, 64
    x, w = _inputs(N, C, H, W, K, 3, 3, "bf16", 5)
    desc = cb.ConvDesc.make(N, C, H, W, K, 3, 3, 1, 1, dtype="bf16")
    Y, ym = _run(desc, x.cuda(), w.cuda())
    nxt = cb.ConvDesc.make(N, K, desc.P, desc.Q, 32, 3, 3, 1, 1, dtype="bf16")
    rng = np.random.default_rng(9)
    w2 = torch.from_numpy(rng.standard_normal((32, 3, 3, K), dtype=np.float32) * 0.1).to(torch.bfloat16).cuda()
    dy = torch.from_numpy(rng.standard_normal((N, nxt.P, nxt.Q, 32), dtype=np.float32)).to(torch.bfloat16).cuda()
    outs = []
    for mask in (ym, _reference_bits(Y)):
        dx = torch.empty_like(Y)
        cb.conv_bwd_data_masked(nxt, dy, w2, mask, dx, cb.workspace(nxt, cb.CBW_OP_BWD_DATA_MASKED))
        outs.append(dx.view(torch.int16).clone())
    torch.cuda.synchronize()
    assert torch.equal(outs[0], outs[1])


def test_forward_full_size_sampled():
    """The benchmark layer (N=32, C=K=256, 56x56, bf16) in full: the footprint
    against the stored output's bitmap over the whole tensor, values at
    sampled outputs (random ones plus every image border) against the
    oracle evaluated one by one."""
    import workloads as wl
    spec = wl.config2()[0]
    print("\n[case] forward full size N=%d C=%d K=%d %dx%d" % (spec.N, spec.C, spec.K, spec.H, spec.W), flush=True)
    t = wl.draw(spec)
    x, w = t["x"], t["w"]
    desc = cb.ConvDesc.make(spec.N, spec.C, spec.H, spec.W, spec.K, spec.R, spec.S, 1, spec.pad, dtype="bf16")
    Y, ym = _run(desc, x.cuda(), w.cuda())
    words = cb.cbw_dy_mask_words(desc)
    assert torch.equal(ym[:words].cpu(), _reference_bits(Y)[:words].cpu())
    assert not (Y.view(torch.int16) < 0).any().item()
    rng = np.random.default_rng(2109)
    m = 3000
    co = np.stack([rng.integers(0, spec.N, m), rng.integers(0, spec.K, m), rng.integers(0, desc.P, m),
                   rng.integers(0, desc.Q, m)], 1)
    border = [[spec.N - 1, k, p, q] for k in (0, spec.K - 1) for p in range(desc.P) for q in (0, desc.Q - 1)]
    border += [[0, spec.K // 2, p, q] for q in range(desc.Q) for p in (0, desc.P - 1)]
    co = np.concatenate([co, np.array(border)]).astype(np.int32)
    x64 = oracle.nhwc_to_nchw(x.double().numpy())
    w64 = oracle.krsc_to_kcrs(w.double().numpy())
    z, a, n = oracle.conv_fwd_at(x64, w64, co, (1, 1), (spec.pad, spec.pad))
    g = Y.float().cpu().numpy()[co[:, 0], co[:, 2], co[:, 3], co[:, 1]].astype(np.float64)
    e = check_values(g, oracle.relu(z), a, n, tol_for("bf16"), True, "forward full size (sampled)")
    print("  sampled normwise %.3e" % e, flush=True)
