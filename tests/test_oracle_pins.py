"""Pins of the oracle against what the mathematics and the paper fix.

Each test checks the oracle against something other than itself: an exact
identity (adjointness), an independent loop order (brute force), a textbook or
library special case (matrix product, identity filter, one-hot gradient,
torch CPU fp64 convolution gradients), the paper's worked MAC counts
(Sec. III-B, Fig. "Compaction") and the paper's closed-form compute model
(Sec. II-A).  The mutation tests at the end plant plausible mistakes into the
oracle's operands and show that the pins catch them.
"""
import itertools
import json
import os

import numpy as np
import pytest
import torch

import oracle
from oracle import brute

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _rand(rng, shape, density=1.0):
    a = rng.standard_normal(shape)
    if density < 1.0:
        a *= rng.random(shape) < density
    return a


def _shapes():
    """Small shapes sweeping filter size, stride and pad (all outputs non-empty)."""
    out = []
    for (R, S), st, pad in itertools.product([(1, 1), (2, 3), (3, 3), (5, 5)], [1, 2, 3], [0, 1, 2]):
        for H, W in [(5, 6), (7, 4)]:
            if (H + 2 * pad - R) // st + 1 <= 0 or (W + 2 * pad - S) // st + 1 <= 0:
                continue
            out.append(dict(N=2, C=3, K=2, H=H, W=W, R=R, S=S, stride=(st, st), pad=(pad, pad)))
    return out


SHAPES = _shapes()


def _rel(a, b):
    return np.max(np.abs(np.asarray(a) - np.asarray(b))) / max(np.max(np.abs(b)), 1e-300)


# ------------------------------------------------------------- brute force

@pytest.mark.parametrize("sh", SHAPES[::3])
def test_brute_force_agrees(sh):
    rng = np.random.default_rng(7)
    x = _rand(rng, (sh["N"], sh["C"], sh["H"], sh["W"]))
    w = _rand(rng, (sh["K"], sh["C"], sh["R"], sh["S"]))
    y = oracle.conv_fwd(x, w, sh["stride"], sh["pad"])
    assert _rel(y, np.array(brute.conv_fwd(x, w, sh["stride"], sh["pad"]))) < 1e-12
    dy = _rand(rng, y.shape, 0.6)
    dx = oracle.conv_bwd_data(dy, w, (sh["H"], sh["W"]), sh["stride"], sh["pad"])
    bdx = np.array(brute.conv_bwd_data(dy, w, (sh["H"], sh["W"]), sh["stride"], sh["pad"]))
    assert _rel(dx, bdx) < 1e-12
    dw = oracle.conv_bwd_weight(x, dy, (sh["R"], sh["S"]), sh["stride"], sh["pad"])
    bdw = np.array(brute.conv_bwd_weight(x, dy, (sh["R"], sh["S"]), sh["stride"], sh["pad"]))
    assert _rel(dw, bdw) < 1e-12


# ------------------------------------------------------ adjoint identities

@pytest.mark.parametrize("sh", SHAPES)
def test_adjoint_identities(sh):
    """<dY, conv(X,W)> = <bwd_data(dY,W), X> = <bwd_weight(X,dY), W> exactly
    (up to fp64 rounding): the two gradients are the adjoints of the forward
    map in X and in W (Sec. IV-B: the backward pass is the forward operation
    with M and C interchanged)."""
    rng = np.random.default_rng(11)
    x = _rand(rng, (sh["N"], sh["C"], sh["H"], sh["W"]))
    w = _rand(rng, (sh["K"], sh["C"], sh["R"], sh["S"]))
    y = oracle.conv_fwd(x, w, sh["stride"], sh["pad"])
    dy = _rand(rng, y.shape)
    lhs = np.sum(dy * y)
    dx = oracle.conv_bwd_data(dy, w, (sh["H"], sh["W"]), sh["stride"], sh["pad"])
    dw = oracle.conv_bwd_weight(x, dy, (sh["R"], sh["S"]), sh["stride"], sh["pad"])
    scale = np.sum(np.abs(dy) * np.abs(oracle.conv_fwd(np.abs(x), np.abs(w), sh["stride"], sh["pad"])))
    assert abs(lhs - np.sum(dx * x)) <= 1e-12 * scale
    assert abs(lhs - np.sum(dw * w)) <= 1e-12 * scale


def test_finite_differences():
    """L(X) = <dY, conv(X,W)> is linear in X and in W, so a central difference
    along a random direction equals the directional derivative <grad, E> up to
    rounding; the gradients are dX and dW."""
    rng = np.random.default_rng(3)
    N, C, K, H, W, R, S = 2, 3, 4, 6, 5, 3, 3
    st, pad = (2, 1), (1, 0)
    x = _rand(rng, (N, C, H, W))
    w = _rand(rng, (K, C, R, S))
    y = oracle.conv_fwd(x, w, st, pad)
    dy = _rand(rng, y.shape)
    L = lambda xx, ww: np.sum(dy * oracle.conv_fwd(xx, ww, st, pad))
    eps = 1e-3
    ex = _rand(rng, x.shape)
    ew = _rand(rng, w.shape)
    fdx = (L(x + eps * ex, w) - L(x - eps * ex, w)) / (2 * eps)
    fdw = (L(x, w + eps * ew) - L(x, w - eps * ew)) / (2 * eps)
    dx = oracle.conv_bwd_data(dy, w, (H, W), st, pad)
    dw = oracle.conv_bwd_weight(x, dy, (R, S), st, pad)
    assert abs(fdx - np.sum(dx * ex)) < 1e-8 * max(1.0, abs(fdx))
    assert abs(fdw - np.sum(dw * ew)) < 1e-8 * max(1.0, abs(fdw))


# ------------------------------------------------ special cases / library

def test_one_by_one_is_matrix_product():
    """A 1x1, stride-1, pad-0 convolution is a matrix product per pixel:
    dX[n,:,h,w] = W^T dY[n,:,h,w] and dW = sum over pixels dY X^T."""
    rng = np.random.default_rng(5)
    N, C, K, H, W = 3, 5, 7, 4, 6
    w = _rand(rng, (K, C, 1, 1))
    dy = _rand(rng, (N, K, H, W), 0.5)
    x = _rand(rng, (N, C, H, W))
    dx = oracle.conv_bwd_data(dy, w, (H, W))
    ref = np.matmul(w[:, :, 0, 0].T, dy.transpose(0, 2, 3, 1)[..., None])[..., 0].transpose(0, 3, 1, 2)
    assert _rel(dx, ref) < 1e-13
    dw = oracle.conv_bwd_weight(x, dy, (1, 1))
    refw = np.matmul(dy.transpose(1, 0, 2, 3).reshape(K, -1), x.transpose(1, 0, 2, 3).reshape(C, -1).T)
    assert _rel(dw[:, :, 0, 0], refw) < 1e-13


@pytest.mark.parametrize("R", [1, 3, 5])
def test_identity_filter_passes_gradient_through(R):
    """W[k,c,R//2,R//2] = [k == c] with 'same' padding: dX = dY exactly."""
    rng = np.random.default_rng(R)
    N, C, H, W = 2, 4, 7, 5
    w = np.zeros((C, C, R, R))
    for c in range(C):
        w[c, c, R // 2, R // 2] = 1.0
    dy = _rand(rng, (N, C, H, W), 0.5)
    dx = oracle.conv_bwd_data(dy, w, (H, W), pad=(R // 2, R // 2))
    assert np.array_equal(dx, dy)


@pytest.mark.parametrize("stride,pad", [((1, 1), (1, 1)), ((2, 2), (1, 1)), ((2, 3), (0, 2))])
def test_one_hot_gradient_places_the_filter(stride, pad):
    """A one-hot dY at (n0,k0,p0,q0) yields dX[n0,c,p0*sh-ph+r,q0*sw-pw+s] =
    W[k0,c,r,s] for in-range positions and 0 everywhere else."""
    rng = np.random.default_rng(9)
    N, C, K, H, W, R, S = 2, 3, 4, 8, 9, 3, 4
    w = _rand(rng, (K, C, R, S))
    P = (H + 2 * pad[0] - R) // stride[0] + 1
    Q = (W + 2 * pad[1] - S) // stride[1] + 1
    for (n0, k0, p0, q0) in [(0, 0, 0, 0), (1, 3, P - 1, Q - 1), (1, 2, P // 2, 1)]:
        dy = np.zeros((N, K, P, Q))
        dy[n0, k0, p0, q0] = 1.0
        dx = oracle.conv_bwd_data(dy, w, (H, W), stride, pad)
        ref = np.zeros((N, C, H, W))
        for r in range(R):
            for s in range(S):
                h, ww = p0 * stride[0] - pad[0] + r, q0 * stride[1] - pad[1] + s
                if 0 <= h < H and 0 <= ww < W:
                    ref[n0, :, h, ww] = w[k0, :, r, s]
        assert np.array_equal(dx, ref)


@pytest.mark.parametrize("sh", SHAPES[1::4])
def test_matches_torch_cpu_fp64_gradients(sh):
    """An independent library routine: torch CPU fp64 conv2d and its
    gradient functions (used only here, never in the oracle)."""
    rng = np.random.default_rng(13)
    x = _rand(rng, (sh["N"], sh["C"], sh["H"], sh["W"]))
    w = _rand(rng, (sh["K"], sh["C"], sh["R"], sh["S"]))
    tx, tw = torch.from_numpy(x), torch.from_numpy(w)
    y = torch.nn.functional.conv2d(tx, tw, stride=sh["stride"], padding=sh["pad"]).numpy()
    assert _rel(oracle.conv_fwd(x, w, sh["stride"], sh["pad"]), y) < 1e-12
    dy = _rand(rng, y.shape, 0.5)
    tdy = torch.from_numpy(dy)
    tdx = torch.nn.grad.conv2d_input(tx.shape, tw, tdy, stride=sh["stride"], padding=sh["pad"]).numpy()
    tdw = torch.nn.grad.conv2d_weight(tx, tw.shape, tdy, stride=sh["stride"], padding=sh["pad"]).numpy()
    assert _rel(oracle.conv_bwd_data(dy, w, (sh["H"], sh["W"]), sh["stride"], sh["pad"]), tdx) < 1e-12
    assert _rel(oracle.conv_bwd_weight(x, dy, (sh["R"], sh["S"]), sh["stride"], sh["pad"]), tdw) < 1e-12


# ------------------------------------------------------- masked semantics

def test_masked_equals_dense_times_mask_with_positive_zeros():
    """Output sparsity (Sec. III-B): the masked gradient is the dense gradient
    at live outputs and exactly +0.0 at killed outputs."""
    rng = np.random.default_rng(17)
    N, C, K, H, W = 2, 5, 3, 6, 7
    w = _rand(rng, (K, C, 3, 3))
    dy = _rand(rng, (N, K, H, W), 0.5)
    x = np.maximum(_rand(rng, (N, C, H, W)), 0.0)
    mask = oracle.relu_mask(x)
    dense = oracle.conv_bwd_data(dy, w, (H, W), pad=(1, 1))
    masked = oracle.conv_bwd_data(dy, w, (H, W), pad=(1, 1), mask=mask)
    assert np.array_equal(masked[mask], dense[mask])
    assert np.all(masked[~mask].view(np.uint64) == 0)  # +0.0 bit pattern
    all_live = oracle.conv_bwd_data(dy, w, (H, W), pad=(1, 1), mask=np.ones_like(mask))
    assert np.array_equal(all_live, dense)


def test_maxpool_matches_torch_cpu():
    """The 2x2 max-pool and its backward against torch's CPU fp64 max_pool2d
    and its autograd (continuous values, so the maximum is unique)."""
    rng = np.random.default_rng(23)
    a = rng.standard_normal((2, 3, 6, 8))
    pooled, arg = oracle.maxpool2x2(a)
    ta = torch.from_numpy(a).requires_grad_(True)
    tp = torch.nn.functional.max_pool2d(ta, 2, 2)
    assert np.array_equal(pooled, tp.detach().numpy())
    g = rng.standard_normal(pooled.shape)
    tp.backward(torch.from_numpy(g))
    assert np.array_equal(oracle.maxpool2x2_backward(g, arg), ta.grad.numpy())


def test_maxpool_ties_route_to_first_position():
    """A window of equal values (e.g. four ReLU zeros) routes to its first position."""
    pooled, arg = oracle.maxpool2x2(np.zeros((1, 1, 2, 4)))
    assert pooled.shape == (1, 1, 1, 2) and np.all(pooled == 0) and np.all(arg == 0)
    back = oracle.maxpool2x2_backward(np.array([[[[5.0, -2.0]]]]), arg)
    assert back.tolist() == [[[[5.0, 0.0, -2.0, 0.0], [0.0, 0.0, 0.0, 0.0]]]]


def test_pooled_footprint_mask_is_exact():
    """MaxPool -> CONV boundary (the layers after a pool in Sec. VI, where the
    paper applies no output sparsity): masking the conv's data gradient by
    pooled > 0 leaves the gradient that reaches the pre-pool ReLU unchanged,
    bit for bit.  A pooled value of 0 means every ReLU output of its window
    is 0, so the ReLU derivative (mask = output > 0) kills whatever max-pool
    backward routes there."""
    rng = np.random.default_rng(29)
    N, C, K, H, W = 2, 4, 3, 4, 6          # pooled size; the pre-pool map is 2H x 2W
    z = rng.standard_normal((N, C, 2 * H, 2 * W)) - 0.8   # pre-activation: most windows all dead
    a = oracle.relu(z)
    x, arg = oracle.maxpool2x2(a)
    w = _rand(rng, (K, C, 3, 3))
    dy = _rand(rng, (N, K, H, W), 0.6)
    dense = oracle.conv_bwd_data(dy, w, (H, W), pad=(1, 1))
    masked = oracle.conv_bwd_data(dy, w, (H, W), pad=(1, 1), mask=oracle.relu_mask(x))
    assert np.any((dense != 0) & ~(x > 0)), "the mask must remove something"
    relu_deriv = oracle.relu_mask(a)
    g_dense = np.where(relu_deriv, oracle.maxpool2x2_backward(dense, arg), 0.0)
    g_masked = np.where(relu_deriv, oracle.maxpool2x2_backward(masked, arg), 0.0)
    assert np.array_equal(g_dense, g_masked)
    # and the masked gradient is the dense one with the pooled-dead outputs at zero
    assert np.array_equal(np.where(x > 0, dense, 0.0), masked)


def test_relu_mask_reading_at_zero():
    """mask = (ReLU output > 0): exact zeros of either sign are killed."""
    x = np.array([-1.0, -0.0, 0.0, 1e-300, 2.0])
    assert oracle.relu_mask(x).tolist() == [False, False, False, True, True]


def test_paper_compaction_example_mac_counts():
    """Sec. III-B, Fig. "Compaction": a live output whose gradient column has
    two zeros of four needs 2 MACs, not 4; an output killed by the ReLU
    derivative needs none.  The example is posed as a 1x1 convolution."""
    g = json.load(open(os.path.join(GOLDEN, "compaction_example.json")))
    W2 = np.array(g["W2"])            # [c][k]
    d3 = np.array(g["delta3"])        # [k][j]
    a1 = np.array(g["a1_prime"])      # [c][j]
    C, K = W2.shape
    J = d3.shape[1]
    w = W2.T.reshape(K, C, 1, 1)
    dy = d3.reshape(1, K, 1, J)
    mask = a1.reshape(1, C, 1, J)
    total, per = oracle.bwd_data_macs(dy, (1, J), (1, 1), C, mask=mask, per_output=True)
    assert per.reshape(C, J).tolist() == g["expected_macs"]
    assert per[0, 0, 0, 0] == 2 and per[0, 1, 0, 0] == 0
    assert total == int(np.sum(g["expected_macs"]))
    _, dense_per = oracle.bwd_data_macs(np.ones_like(dy), (1, J), (1, 1), C, per_output=True)
    assert np.all(dense_per == g["dense_macs_per_output"])
    dx = oracle.conv_bwd_data(dy, w, (1, J), mask=mask).reshape(C, J)
    assert dx.tolist() == g["expected_delta1"]
    assert np.signbit(dx[1, 0]) == False  # killed output is +0.0


def test_compute_model_closed_forms():
    """Sec. II-A: a layer costs M*U*V*C*R*S MACs (here K*P*Q*C*R*S per
    image); with pad 0 and stride 1 every forward term has exactly one
    backward term, so the dense backward-data count is that number, and with
    a sparse dY it is nnz(dY)*C*R*S (the input-sparsity factor)."""
    rng = np.random.default_rng(19)
    N, C, K, H, W, R, S = 2, 3, 4, 7, 6, 3, 2
    P, Q = H - R + 1, W - S + 1
    dense = oracle.bwd_data_macs(np.ones((N, K, P, Q)), (H, W), (R, S), C)
    assert dense == N * K * P * Q * C * R * S
    dy = _rand(rng, (N, K, P, Q), 0.4)
    assert oracle.bwd_data_macs(dy, (H, W), (R, S), C) == np.count_nonzero(dy) * C * R * S


def test_mac_counter_brute_force():
    rng = np.random.default_rng(23)
    N, C, K, H, W, R, S = 2, 3, 2, 5, 4, 3, 3
    st, pad = (2, 1), (1, 2)
    P, Q = (H + 2 * pad[0] - R) // st[0] + 1, (W + 2 * pad[1] - S) // st[1] + 1
    dy = _rand(rng, (N, K, P, Q), 0.5)
    mask = rng.random((N, C, H, W)) < 0.5
    _, per = oracle.bwd_data_macs(dy, (H, W), (R, S), C, st, pad, mask=mask, per_output=True)
    ref = np.zeros((N, C, H, W), np.int64)
    for n, k, p, q in itertools.product(range(N), range(K), range(P), range(Q)):
        if dy[n, k, p, q] == 0:
            continue
        for c, r, s in itertools.product(range(C), range(R), range(S)):
            h, w = p * st[0] - pad[0] + r, q * st[1] - pad[1] + s
            if 0 <= h < H and 0 <= w < W and mask[n, c, h, w]:
                ref[n, c, h, w] += 1
    assert np.array_equal(per, ref)


def test_error_bound_terms_brute_force():
    """The per-output conditioning sum(|a*b|) and term counts."""
    rng = np.random.default_rng(29)
    N, C, K, H, W = 1, 2, 3, 4, 5
    w = _rand(rng, (K, C, 3, 3))
    dy = _rand(rng, (N, K, H, W))
    x = _rand(rng, (N, C, H, W))
    _, absd, nt = oracle.conv_bwd_data(dy, w, (H, W), pad=(1, 1), with_bound=True)
    ref = oracle.conv_bwd_data(np.abs(dy), np.abs(w), (H, W), pad=(1, 1))
    assert _rel(absd, ref) < 1e-13
    cnt = oracle.conv_bwd_data(np.ones_like(dy), np.ones_like(w), (H, W), pad=(1, 1))
    assert np.array_equal(nt, cnt.astype(np.int64))
    _, absw, ntw = oracle.conv_bwd_weight(x, dy, (3, 3), pad=(1, 1), with_bound=True)
    assert _rel(absw, oracle.conv_bwd_weight(np.abs(x), np.abs(dy), (3, 3), pad=(1, 1))) < 1e-13
    assert np.array_equal(ntw, oracle.conv_bwd_weight(np.ones_like(x), np.ones_like(dy), (3, 3),
                                                      pad=(1, 1)).astype(np.int64))


def test_sampled_entry_points_match_full():
    rng = np.random.default_rng(31)
    N, C, K, H, W, R, S = 2, 4, 3, 6, 5, 3, 3
    st, pad = (1, 2), (1, 1)
    x = _rand(rng, (N, C, H, W))
    w = _rand(rng, (K, C, R, S))
    P, Q = (H + 2 - R) // 1 + 1, (W + 2 - S) // 2 + 1
    dy = _rand(rng, (N, K, P, Q))
    dx, absd, nt = oracle.conv_bwd_data(dy, w, (H, W), st, pad, with_bound=True)
    dw, absw, ntw = oracle.conv_bwd_weight(x, dy, (R, S), st, pad, with_bound=True)
    cx = np.stack(np.meshgrid(range(N), range(C), range(H), range(W), indexing="ij"), -1).reshape(-1, 4)
    v, a, t = oracle.conv_bwd_data_at(dy, w, (H, W), cx, st, pad)
    assert np.array_equal(v, dx.reshape(-1)) and np.array_equal(a, absd.reshape(-1))
    assert np.array_equal(t, nt.reshape(-1))
    cw = np.stack(np.meshgrid(range(K), range(C), range(R), range(S), indexing="ij"), -1).reshape(-1, 4)
    v, a, t = oracle.conv_bwd_weight_at(x, dy, (R, S), cw, st, pad)
    assert np.array_equal(v, dw.reshape(-1)) and np.array_equal(a, absw.reshape(-1))
    assert np.array_equal(t, ntw.reshape(-1))


# --------------------------------------------- forward with the ReLU fused

def _brute_fwd_terms(x, w, stride, pad):
    """Pure-Python loops: per output (sum x*w, sum |x*w|, number of terms)."""
    N, C, H, W = x.shape
    K, _, R, S = w.shape
    P = (H + 2 * pad[0] - R) // stride[0] + 1
    Q = (W + 2 * pad[1] - S) // stride[1] + 1
    z, a, n = np.zeros((N, K, P, Q)), np.zeros((N, K, P, Q)), np.zeros((N, K, P, Q), np.int64)
    for nn, k, p, q in itertools.product(range(N), range(K), range(P), range(Q)):
        for c, r, t in itertools.product(range(C), range(R), range(S)):
            h, ww = p * stride[0] - pad[0] + r, q * stride[1] - pad[1] + t
            if 0 <= h < H and 0 <= ww < W:
                z[nn, k, p, q] += x[nn, c, h, ww] * w[k, c, r, t]
                a[nn, k, p, q] += abs(x[nn, c, h, ww] * w[k, c, r, t])
                n[nn, k, p, q] += 1
    return z, a, n


@pytest.mark.parametrize("sh", SHAPES[::5])
def test_forward_relu_brute_force(sh):
    rng = np.random.default_rng(17)
    x = _rand(rng, (sh["N"], sh["C"], sh["H"], sh["W"]), 0.6)
    w = _rand(rng, (sh["K"], sh["C"], sh["R"], sh["S"]))
    z, y, a, n = oracle.conv_fwd_relu(x, w, sh["stride"], sh["pad"])
    zb, ab, nb = _brute_fwd_terms(x, w, sh["stride"], sh["pad"])
    assert _rel(z, zb) < 1e-12 and _rel(a, ab) < 1e-12
    assert np.array_equal(n, nb)
    assert np.array_equal(y > 0, zb > 0)                      # the footprint is the sign of the sum
    assert np.all(y[zb <= 0] == 0) and _rel(y[zb > 0], zb[zb > 0]) < 1e-12
    # the emitted footprint is the bitmap of the stored output
    assert np.array_equal(oracle.relu_mask(y), y > 0)


def test_relu_reading_of_zero_and_nan():
    y = oracle.relu(np.array([-0.0, 0.0, -1.0, 2.0, np.nan, 1e-300, -1e-300]))
    assert np.array_equal(np.signbit(y[:3]), [False, False, False])    # every zero is +0.0
    assert y[3] == 2.0 and y[4] == 0.0 and y[5] == 1e-300 and y[6] == 0.0


def test_sampled_forward_matches_full():
    rng = np.random.default_rng(37)
    N, C, K, H, W, R, S = 2, 3, 4, 6, 5, 3, 2
    for st, pad in [((1, 1), (1, 1)), ((2, 1), (0, 1))]:
        x = _rand(rng, (N, C, H, W), 0.5)
        w = _rand(rng, (K, C, R, S))
        z, _, a, n = oracle.conv_fwd_relu(x, w, st, pad)
        P, Q = z.shape[2:]
        co = np.stack(np.meshgrid(range(N), range(K), range(P), range(Q), indexing="ij"), -1).reshape(-1, 4)
        v, av, nv = oracle.conv_fwd_at(x, w, co, st, pad)
        assert _rel(v, z.reshape(-1)) < 1e-12 and _rel(av, a.reshape(-1)) < 1e-12
        assert np.array_equal(nv, n.reshape(-1))


# ---------------------------------------------------- bitmaps and indexing

@pytest.mark.parametrize("stride,pad,tpg,chunk,ktile,ctile", [((1, 1), (1, 1), 1, 8, 4, 4), ((2, 1), (0, 2), 4, 5, 3, 8),
                                                               ((1, 2), (1, 0), 9, 16, 8, 2)])
def test_weight_block_liveness_brute_force(stride, pad, tpg, chunk, ktile, ctile):
    """The weight-gradient block liveness against nested loops over every
    operand element of every block: live iff both the block's dY operand and
    its (tap-shifted) X operand hold a non-zero; and every product of a dead
    block vanishes, so skipping it changes no sum."""
    rng = np.random.default_rng(31)
    N, C, H, W, K, R, S = 2, 8, 6, 7, 6, 3, 3
    x = _rand(rng, (N, C, H, W), 0.3)
    x[:, :, 1:4] = 0
    dy_shape = (N, K, oracle.out_size(H, R, stride[0], pad[0]), oracle.out_size(W, S, stride[1], pad[1]))
    dy = _rand(rng, dy_shape, 0.2)
    dy[0] = 0
    P, Q = dy_shape[2:]
    live = oracle.weight_block_liveness(x != 0, dy != 0, (R, S), stride, pad, chunk, ktile, ctile, tpg)
    nch = -(-N * P * Q // chunk)
    assert live.shape == (-(-R * S // tpg), -(-C // ctile), -(-K // ktile), nch)
    for g, ct, kt, b in itertools.product(*map(range, live.shape)):
        dy_nz = x_nz = prod_nz = False
        for pix in range(b * chunk, min((b + 1) * chunk, N * P * Q)):
            n, rem = divmod(pix, P * Q)
            p, q = divmod(rem, Q)
            for k in range(kt * ktile, min((kt + 1) * ktile, K)):
                dy_nz |= dy[n, k, p, q] != 0
            for tap in range(g * tpg, min((g + 1) * tpg, R * S)):
                r, s = divmod(tap, S)
                h, w = p * stride[0] - pad[0] + r, q * stride[1] - pad[1] + s
                if not (0 <= h < H and 0 <= w < W):
                    continue
                for c in range(ct * ctile, min((ct + 1) * ctile, C)):
                    x_nz |= x[n, c, h, w] != 0
                    for k in range(kt * ktile, min((kt + 1) * ktile, K)):
                        prod_nz |= dy[n, k, p, q] * x[n, c, h, w] != 0
        assert live[g, ct, kt, b] == (dy_nz and x_nz), (g, ct, kt, b)
        assert live[g, ct, kt, b] or not prod_nz
    assert live.any() and not live.all()


def test_pack_bits_brute_force():
    rng = np.random.default_rng(37)
    for n in [1, 31, 32, 33, 100, 257]:
        live = rng.random(n) < 0.5
        words = oracle.pack_bits(live)
        assert len(words) == (n + 31) // 32
        for i in range(len(words) * 32):
            bit = (int(words[i // 32]) >> (i % 32)) & 1
            assert bit == (1 if i < n and live[i] else 0)
        assert np.array_equal(oracle.unpack_bits(words, n), live)


def test_live_pixel_lists_brute_force():
    rng = np.random.default_rng(41)
    npix, C = 37, 48
    live = rng.random((npix, C)) < 0.03
    live[5] = True
    bits = oracle.pack_bits(live.reshape(-1))
    for G in (16, 32, 48):
        lists = oracle.live_pixel_lists(bits, npix, C, G)
        assert len(lists) == (C + G - 1) // G
        for g, lst in enumerate(lists):
            ref = [p for p in range(npix) if any(live[p, c] for c in range(g * G, min(C, (g + 1) * G)))]
            assert lst.tolist() == ref


def test_block_occupancy_brute_force():
    rng = np.random.default_rng(43)
    npix, K = 50, 24
    d = _rand(rng, (npix, K), 0.05)
    d[7, 3] = -0.0
    occ = oracle.block_occupancy(d, 8, 8)
    for j in range(occ.shape[0]):
        for g in range(occ.shape[1]):
            ref = any(d[p, k] != 0 for p in range(j * 8, min(npix, j * 8 + 8)) for k in range(g * 8, g * 8 + 8))
            assert occ[j, g] == ref


# ----------------------------------------------------------- mutation tests

def _adjoint_gap(dx_fn, sh):
    rng = np.random.default_rng(47)
    x = _rand(rng, (sh["N"], sh["C"], sh["H"], sh["W"]))
    w = _rand(rng, (sh["K"], sh["C"], sh["R"], sh["S"]))
    y = oracle.conv_fwd(x, w, sh["stride"], sh["pad"])
    dy = _rand(rng, y.shape)
    return abs(np.sum(dy * y) - np.sum(dx_fn(dy, w) * x)) / np.sum(np.abs(dy * y))


@pytest.mark.parametrize("mutation", ["flipped_filter", "transposed_channels", "dropped_tap", "wrong_pad", "sign"])
def test_pins_catch_planted_mistakes(mutation):
    """Plant a plausible mistake in the oracle's data gradient (through its
    operands) and show that the adjoint pin fails for it."""
    sh = dict(N=2, C=3, K=3, H=6, W=7, R=3, S=3, stride=(2, 1), pad=(1, 1))
    hw = (sh["H"], sh["W"])

    def good(dy, w):
        return oracle.conv_bwd_data(dy, w, hw, sh["stride"], sh["pad"])

    def bad(dy, w):
        if mutation == "flipped_filter":
            return oracle.conv_bwd_data(dy, w[:, :, ::-1, ::-1], hw, sh["stride"], sh["pad"])
        if mutation == "transposed_channels":
            return oracle.conv_bwd_data(dy, w.transpose(1, 0, 2, 3), hw, sh["stride"], sh["pad"])
        if mutation == "dropped_tap":
            w2 = w.copy()
            w2[:, :, 0, 0] = 0
            return oracle.conv_bwd_data(dy, w2, hw, sh["stride"], sh["pad"])
        if mutation == "wrong_pad":
            return oracle.conv_bwd_data(dy[:, :, :, 1:-1], w, hw, sh["stride"], (1, 0))
        if mutation == "sign":
            return -good(dy, w)
        raise AssertionError

    assert _adjoint_gap(good, sh) < 1e-13
    try:
        gap = _adjoint_gap(bad, sh)
    except (AssertionError, ValueError):
        return  # the mistake does not even produce a well-formed gradient
    assert gap > 1e-3
