"""Seeded synthetic layer workloads for the masked convolution backward pass.

This module only draws inputs.  It holds none of the method's arithmetic (no
mask packing, no compaction, no convolution); both the HIP library's tests and
the oracle's tests draw their inputs here.

The paper measures on layer-wise activation and gradient traces recorded while
training VGGNet, ResNet, GoogLeNet, DenseNet and MobileNet on ImageNet
(Sec. V-A).  Neither the dataset, the trained models nor the traces are
available, so seeded synthetic layers stand in for them: the layer shapes of
the benchmark networks and the activation densities of the paper's observed
sparsity range (about 30% to 70% zeros, Sec. II-A).

Every tensor is drawn with numpy's PCG64 seeded by
``SeedSequence([210907710, config_id, layer_id, tensor_id])`` in float32, in
the storage order NHWC (activations and gradients) or KRSC (filters), and then
rounded to bfloat16 with round-to-nearest-even (torch CPU ``.to``) unless the
layer is float32.  Tensors come back as CPU torch tensors.

Configurations
--------------
1. 3x3 conv, stride 1, pad 1, fp32, N=2, C=K=16, 16x16.  X = relu(N(0,1));
   W ~ N(0, 2/(9C)); dY = N(0,1) * Bernoulli(0.5).
2. VGG-style 3x3 conv, N=32, C=K=256, 56x56, bf16.  X = relu(N(0,1) - 0.25)
   (density 1 - Phi(0.25) = 0.401); dY = N(0,1) * Bernoulli(0.4); He-init W.
3. ResNet-50 bottleneck at 56x56, N=64, bf16: 1x1 256->64, 3x3 64->64 (pad 1),
   1x1 64->256.  Layer inputs X_i = relu(N(0,1) - t_i) with densities
   0.6 / 0.45 / 0.3; dY_i = N(0,1) * [X_{i+1} > 0] (the next layer's ReLU
   footprint: no batch norm between), with a fresh density-0.6 footprint
   after the last layer.
4. Sparsity sweep, 3x3 conv N=128, C=K=512, 14x14, bf16, density
   d in {0.1,...,0.9}; footprint either i.i.d. Bernoulli(d) per element or
   spatially clustered (per (n,c) plane, N(0,1) noise box-blurred 5x5 with
   wrap-around, thresholded at its empirical (1-d) quantile); X = footprint *
   |N(0,1)|; dY = N(0,1) * an independent footprint of the same kind and d.
   A diagnostic kind "channel_shared" draws one clustered field per image
   and shares it across channels.
5. VGG-16 conv stack at 224x224, N=32, bf16: 13 3x3 stride-1 pad-1 layers,
   2x2 max pool after conv1_2, 2_2, 3_3, 4_3, 5_3.  The ReLU output after
   conv_l has density d_l = 0.5 - 0.35 (l-1)/12; conv_l's input has density
   d_{l-1}; layers right after a pool (conv2_1, 3_1, 4_1, 5_1) get a dense
   (unmasked) data gradient and conv1_1 (input = image) only a weight
   gradient.  dY_l = N(0,1) * Bernoulli(d_l), and at a layer followed by a
   pool dY is routed as max-pool backward would route it: per 2x2 window at
   most one position (uniform) keeps the value if any position is live.
"""
from dataclasses import dataclass, field
from math import erf, sqrt
from typing import Optional

import numpy as np
import torch

ROOT_SEED = 210907710


@dataclass
class LayerSpec:
    """Shape and sparsity recipe of one convolution layer (paper notation
    [C,H,W] --[K,C,R,S]--> [K,P,Q], Sec. II-A)."""
    name: str
    config_id: int
    layer_id: int
    N: int
    C: int
    H: int
    W: int
    K: int
    R: int
    S: int
    stride: int = 1
    pad: int = 1
    dtype: str = "bf16"           # "bf16" or "f32" for X, W, dY (and dX)
    masked: bool = True           # data gradient restricted by X's ReLU footprint
    need_dx: bool = True          # False for a network's first layer
    x_kind: str = "shifted_gauss"  # how X is drawn, see draw()
    x_param: float = 0.0
    dy_kind: str = "bernoulli"    # how dY's footprint is drawn
    dy_param: float = 0.5
    extra: dict = field(default_factory=dict)

    @property
    def P(self):
        return (self.H + 2 * self.pad - self.R) // self.stride + 1

    @property
    def Q(self):
        return (self.W + 2 * self.pad - self.S) // self.stride + 1

    def dense_flops(self):
        """Conventional FLOP count of one gradient GEMM, 2*N*K*P*Q*C*R*S, with
        the layer's true channel count when its input is stored padded."""
        c = self.extra.get("true_c", self.C)
        return 2 * self.N * self.K * self.P * self.Q * c * self.R * self.S


def _rng(cfg, layer, tensor):
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence([ROOT_SEED, cfg, layer, tensor])))


def _phi(x):
    return 0.5 * (1.0 + erf(x / sqrt(2.0)))


def threshold_for_density(d):
    """t such that P(N(0,1) - t > 0) = d, by bisection on the normal CDF."""
    lo, hi = -10.0, 10.0
    for _ in range(200):
        mid = 0.5 * (lo + hi)
        if 1.0 - _phi(mid) > d:
            lo = mid
        else:
            hi = mid
    return 0.5 * (lo + hi)


def _to_torch(a, dtype):
    t = torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32))
    return t.to(torch.bfloat16) if dtype == "bf16" else t


def _clustered_footprint(rng, n, c, h, w, d, shared=False):
    """Spatially clustered footprint of density d in NHWC order."""
    planes = n if shared else n * c
    g = rng.standard_normal((planes, h, w), dtype=np.float32)
    acc = np.zeros_like(g)
    for dy in range(-2, 3):
        for dx in range(-2, 3):
            acc += np.roll(np.roll(g, dy, axis=1), dx, axis=2)
    acc /= 25.0
    thr = np.quantile(acc, 1.0 - d)
    fp = acc > thr
    if shared:
        fp = np.broadcast_to(fp[:, None], (n, c, h, w))
    else:
        fp = fp.reshape(n, c, h, w)
    return np.ascontiguousarray(fp.transpose(0, 2, 3, 1))


def _footprint(rng, kind, n, c, h, w, d):
    if kind == "bernoulli":
        return rng.random((n, h, w, c), dtype=np.float32) < d
    if kind == "clustered":
        return _clustered_footprint(rng, n, c, h, w, d)
    if kind == "channel_shared":
        return _clustered_footprint(rng, n, c, h, w, d, shared=True)
    raise ValueError(kind)


def _maxpool_route(rng, live):
    """At most one live position per 2x2 window: where the window has a live
    position, one position chosen uniformly carries the gradient."""
    n, h, w, c = live.shape
    win = live.reshape(n, h // 2, 2, w // 2, 2, c).any(axis=(2, 4))
    pick = rng.integers(0, 4, size=win.shape)
    out = np.zeros((n, h // 2, 2, w // 2, 2, c), dtype=bool)
    for i in range(4):
        sel = win & (pick == i)
        out[:, :, i // 2, :, i % 2, :] = sel
    return out.reshape(n, h, w, c)


def draw(spec: LayerSpec, want=("x", "w", "dy")):
    """Draw the layer's tensors.  Returns a dict of CPU torch tensors:
    x [N,H,W,C], w [K,R,S,C], dy [N,P,Q,K] in spec.dtype."""
    n, c, h, w_, k = spec.N, spec.C, spec.H, spec.W, spec.K
    # an input stored with zero-padded channels (the 3-channel image as 8
    # channels): the tensors are drawn at the true width and padded after
    c_store, c = c, spec.extra.get("true_c", c)
    out = {}
    cid, lid = spec.config_id, spec.layer_id
    if "x" in want:
        rng = _rng(cid, lid, 0)
        if spec.x_kind == "shifted_gauss":
            x = rng.standard_normal((n, h, w_, c), dtype=np.float32)
            x -= np.float32(spec.x_param)
            np.maximum(x, np.float32(0.0), out=x)
        elif spec.x_kind == "pooled_gauss":
            # the input of a layer that follows a 2x2 max-pool: the previous
            # layer's ReLU output, drawn at twice the size, then pooled
            z = rng.standard_normal((n, 2 * h, 2 * w_, c), dtype=np.float32)
            z -= np.float32(spec.x_param)
            np.maximum(z, np.float32(0.0), out=z)
            x = z.reshape(n, h, 2, w_, 2, c).max(axis=(2, 4))
            del z
        elif spec.x_kind in ("bernoulli", "clustered", "channel_shared"):
            fp = _footprint(rng, spec.x_kind, n, c, h, w_, spec.x_param)
            x = rng.standard_normal((n, h, w_, c), dtype=np.float32)
            np.abs(x, out=x)
            x *= fp
        else:
            raise ValueError(spec.x_kind)
        if c_store != c:
            x = np.concatenate([x, np.zeros((n, h, w_, c_store - c), np.float32)], axis=3)
        out["x"] = _to_torch(x, spec.dtype)
    if "w" in want:
        rng = _rng(cid, lid, 1)
        std = sqrt(2.0 / (c * spec.R * spec.S))
        wt = rng.standard_normal((k, spec.R, spec.S, c), dtype=np.float32)
        wt *= np.float32(std)
        if c_store != c:
            wt = np.concatenate([wt, np.zeros((k, spec.R, spec.S, c_store - c), np.float32)], axis=3)
        out["w"] = _to_torch(wt, spec.dtype)
    if "dy" in want:
        p, q = spec.P, spec.Q
        rng = _rng(cid, lid, 2)
        vals = rng.standard_normal((n, p, q, k), dtype=np.float32)
        rngm = _rng(cid, lid, 3)
        if spec.dy_kind == "next_layer_x":
            # footprint of the next layer's ReLU output, drawn by that layer's spec
            nxt = spec.extra["next_spec"]
            live = draw(nxt, want=("x",))["x"].float().numpy() > 0
        elif spec.dy_kind == "fresh_shifted_gauss":
            g = rngm.standard_normal((n, p, q, k), dtype=np.float32)
            live = (g - np.float32(spec.dy_param)) > 0
        else:
            live = _footprint(rngm, spec.dy_kind, n, k, p, q, spec.dy_param)
        if spec.extra.get("maxpool_route"):
            live = _maxpool_route(rngm, live)
        np.putmask(vals, ~live, np.float32(0.0))  # +0.0 where dead
        out["dy"] = _to_torch(vals, spec.dtype)
    return out


def draw_on_device(spec: LayerSpec, device="cuda"):
    """The layer's tensors drawn directly in device memory with torch's
    seeded device generator: for sizes whose host-side generation would take
    minutes (the largest tensors a buffer descriptor can address, the VGG-16
    stack inside the benchmark).  Same recipe as draw() for "shifted_gauss"
    and "pooled_gauss" X, "bernoulli" dY (with the max-pool routing of
    spec.extra["maxpool_route"]) and zero-padded image channels; the values
    differ from draw() (another generator).  bf16 only."""
    assert spec.dtype == "bf16" and spec.x_kind in ("shifted_gauss", "pooled_gauss") and spec.dy_kind == "bernoulli"
    g = torch.Generator(device=device)
    g.manual_seed(ROOT_SEED * 1000 + spec.config_id * 100 + spec.layer_id)
    n, c, h, w_, k = spec.N, spec.C, spec.H, spec.W, spec.K
    c_store, c = c, spec.extra.get("true_c", c)
    if spec.x_kind == "shifted_gauss":
        x = torch.randn((n, h, w_, c), generator=g, device=device, dtype=torch.float32)
        x.sub_(spec.x_param).clamp_(min=0.0)
    else:
        # the previous layer's ReLU output at twice the size, max-pooled 2x2
        z = torch.randn((n, 2 * h, 2 * w_, c), generator=g, device=device, dtype=torch.float32)
        z.sub_(spec.x_param).clamp_(min=0.0)
        x = z.view(n, h, 2, w_, 2, c).amax(dim=(2, 4))
        del z
    wt = torch.randn((k, spec.R, spec.S, c), generator=g, device=device, dtype=torch.float32)
    wt.mul_(sqrt(2.0 / (c * spec.R * spec.S)))
    if c_store != c:
        x = torch.nn.functional.pad(x, (0, c_store - c))
        wt = torch.nn.functional.pad(wt, (0, c_store - c))
    x = x.to(torch.bfloat16)
    wt = wt.to(torch.bfloat16)
    p, q = spec.P, spec.Q
    dy = torch.randn((n, p, q, k), generator=g, device=device, dtype=torch.float32)
    live = torch.rand((n, p, q, k), generator=g, device=device) < spec.dy_param
    if spec.extra.get("maxpool_route"):
        # at most one live position per 2x2 window, chosen uniformly
        win = live.view(n, p // 2, 2, q // 2, 2, k).any(dim=4).any(dim=2)
        pick = torch.randint(0, 4, win.shape, generator=g, device=device)
        routed = torch.zeros((n, p // 2, 2, q // 2, 2, k), dtype=torch.bool, device=device)
        for i in range(4):
            routed[:, :, i // 2, :, i % 2, :] = win & (pick == i)
        live = routed.view(n, p, q, k)
        del win, pick, routed
    dy.masked_fill_(~live, 0.0)          # +0.0 where dead
    dy = dy.to(torch.bfloat16)
    return {"x": x, "w": wt, "dy": dy}


# ------------------------------------------------------------ configurations

def config1():
    return [LayerSpec("conv3x3_c16_16x16_f32", 1, 0, N=2, C=16, H=16, W=16, K=16, R=3, S=3,
                      dtype="f32", x_kind="shifted_gauss", x_param=0.0,
                      dy_kind="bernoulli", dy_param=0.5)]


def config2(N=32, H=56):
    return [LayerSpec("vgg_conv3x3_c256_56x56", 2, 0, N=N, C=256, H=H, W=H, K=256, R=3, S=3,
                      x_kind="shifted_gauss", x_param=0.25,
                      dy_kind="bernoulli", dy_param=0.4)]


def config3(N=64, H=56):
    dens = (0.6, 0.45, 0.3)
    ts = [threshold_for_density(d) for d in dens]
    shapes = [(256, 64, 1, 0), (64, 64, 3, 1), (64, 256, 1, 0)]
    specs = []
    for i, ((c, k, r, pad), t) in enumerate(zip(shapes, ts)):
        specs.append(LayerSpec(f"resnet50_bottleneck_l{i + 1}_{r}x{r}_{c}to{k}", 3, i,
                               N=N, C=c, H=H, W=H, K=k, R=r, S=r, pad=pad,
                               x_kind="shifted_gauss", x_param=t))
    for i in range(3):
        if i + 1 < 3:
            specs[i].dy_kind = "next_layer_x"
            specs[i].extra["next_spec"] = specs[i + 1]
        else:
            specs[i].dy_kind = "fresh_shifted_gauss"
            specs[i].dy_param = threshold_for_density(0.6)
    return specs


SWEEP_DENSITIES = tuple(round(0.1 * i, 1) for i in range(1, 10))


def config4(d, kind="bernoulli", N=128, H=14):
    """kind: "bernoulli" (i.i.d.), "clustered", or the diagnostic "channel_shared"."""
    kid = {"bernoulli": 0, "clustered": 1, "channel_shared": 2}[kind]
    lid = kid * 100 + int(round(d * 10))
    return [LayerSpec(f"sweep_conv3x3_c512_14x14_{kind}_d{d:.1f}", 4, lid, N=N, C=512, H=H, W=H,
                      K=512, R=3, S=3, x_kind=kind, x_param=d, dy_kind=kind, dy_param=d,
                      extra={"density": d, "kind": kind})]


VGG16 = [  # (name, C, K, spatial, followed_by_pool)
    ("conv1_1", 3, 64, 224, False), ("conv1_2", 64, 64, 224, True),
    ("conv2_1", 64, 128, 112, False), ("conv2_2", 128, 128, 112, True),
    ("conv3_1", 128, 256, 56, False), ("conv3_2", 256, 256, 56, False),
    ("conv3_3", 256, 256, 56, True),
    ("conv4_1", 256, 512, 28, False), ("conv4_2", 512, 512, 28, False),
    ("conv4_3", 512, 512, 28, True),
    ("conv5_1", 512, 512, 14, False), ("conv5_2", 512, 512, 14, False),
    ("conv5_3", 512, 512, 14, True),
]


def vgg_density(l):
    """Density of the ReLU output after conv_l, l = 1..13."""
    return 0.5 - 0.35 * (l - 1) / 12.0


def config5(N=32, scale=1, pooled_mask=False):
    """VGG-16 conv stack; scale > 1 divides every spatial size (test sizes).

    The inputs of the four layers after a max-pool are the pooled ReLU output
    of the layer before (density 1 - (1 - d)^4 for i.i.d. footprints).  Their
    data gradient is dense (the paper applies no output sparsity there) unless
    pooled_mask is set, in which case it is masked by pooled > 0."""
    specs = []
    for i, (name, c, k, hw, pool) in enumerate(VGG16):
        l = i + 1
        hw_s = max(2, hw // scale)
        after_pool = l in (3, 5, 8, 11)
        d_in = vgg_density(l - 1) if l > 1 else 1.0
        extra = {"maxpool_route": pool}
        if c % 8:
            # the image: stored with its channels zero-padded to a multiple of 8
            # (the 16-byte vector of 8 bf16), which leaves the weight gradient of
            # the real channels unchanged and gives exact zeros for the padding
            extra["true_c"] = c
            c = (c + 7) // 8 * 8
        spec = LayerSpec(f"vgg16_{name}", 5, l, N=N, C=c, H=hw_s, W=hw_s, K=k, R=3, S=3,
                         masked=(l > 1 and (pooled_mask or not after_pool)), need_dx=(l > 1),
                         x_kind="pooled_gauss" if after_pool else "shifted_gauss",
                         x_param=threshold_for_density(d_in) if l > 1 else -10.0,
                         dy_kind="bernoulli", dy_param=vgg_density(l),
                         extra=extra)
        specs.append(spec)
    return specs


def all_configs():
    return {1: config1, 2: config2, 3: config3, 4: config4, 5: config5}
