"""The five synthetic workloads and the lattice pipelines run on them.

A workload is a seeded cloud plus a list of lattice operations (a small
pipeline description).  The GPU runner and the oracle runner each interpret
that list on their own; this module only describes inputs and the order of
operations, it computes nothing of the method.

Operations (fields in brackets):
  create        [level=0]                 lattice of the cloud at scale sigma
  coarsen       [level]                   lattice of the cloud at scale 2^level * sigma
  splat         [dst, normalize]          point features -> level-0 vertex values
  conv          [level, src, dst, w, relu]        1-hop convolution on one level
  conv_down     [level, src, dst, w, relu]        strided convolution level-1 -> level
  refine        [level, src, dst, w, relu]        transposed convolution level+1 -> level
  slice         [level, src, out]                 vertex values -> points
  deform_slice  [level, src, wv, beta, out]       DeformSlice to points
  distribute    [level, dst, layers, norm]        Distribute + PointNet of the point
                                                  positions and features (layers: names
                                                  of (W [out][in], b) pairs in `mlp`;
                                                  norm: the GroupNorm parameters in `norms`)
`src`/`dst` are (buffer, first column, channels); buffers are row-major
(vertices of their level) x (total channels), so several ops can write
disjoint column ranges of one buffer (concatenation without a copy).
"""
from __future__ import annotations

from dataclasses import dataclass, field

import numpy as np

from . import generators as gen

TAPS = 9  # 2(d+1)+1 vertices of the 1-hop neighbourhood for d = 3


@dataclass
class Workload:
    cfg: int
    name: str
    seed: int
    positions: np.ndarray            # m x 3 float32
    sigma: np.ndarray                # 3 float32
    dtype: str                       # "f32" or "bf16"
    features: np.ndarray             # m x C float32 (already bf16-representable when dtype == bf16)
    weights: dict = field(default_factory=dict)    # name -> float32 array
    vectors: dict = field(default_factory=dict)    # DeformSlice weight vectors
    mlp: dict = field(default_factory=dict)        # name -> (W [out][in], b) of 1x1 layers
    grads: dict = field(default_factory=dict)      # point output -> dL/d(output), m x C float32
    norms: dict = field(default_factory=dict)      # name -> (gamma, beta) of a GroupNorm pre-activation
    classifiers: dict = field(default_factory=dict)  # name -> (W [class][channel], b)
    buffers: dict = field(default_factory=dict)    # name -> (level, channels)
    ops: list = field(default_factory=list)
    levels: int = 1

    @property
    def m(self) -> int:
        return int(self.positions.shape[0])


def _round_bf16(x: np.ndarray) -> np.ndarray:
    return gen.bf16_bits_to_f32(gen.to_bf16_bits(x))


def _finish(wl: Workload) -> Workload:
    if wl.dtype == "bf16":
        wl.features = _round_bf16(wl.features)
        wl.weights = {k: _round_bf16(v) for k, v in wl.weights.items()}
    wl.levels = 1 + max([op["level"] for op in wl.ops if op["op"] == "coarsen"] + [0])
    return wl


def _conv(wl, kind, level, src, dst, relu, seed, std=None):
    name = f"{kind}{level}_{src[0]}_{dst[0]}_{dst[1]}"
    wl.weights[name] = gen.conv_weights(seed, name, TAPS, src[2], dst[2], std)
    wl.ops.append(dict(op=kind, level=level, src=src, dst=dst, w=name, relu=relu))


def config1(seed: int = 0, m: int = 4096) -> Workload:
    """4,096 points uniform in the unit cube, sigma 0.1, 8 features N(0,1);
    splat -> conv 8->16 (weights N(0, 0.1^2)) -> slice, fp32."""
    pos = gen.uniform_cube(seed, m)
    F = gen.normal_matrix(seed, "F", m, 8, 1.0)
    wl = Workload(1, "uniform-cube", seed, pos, np.full(3, 0.1, np.float32), "f32", F)
    wl.buffers = {"s0": (0, 8), "c0": (0, 16)}
    wl.ops = [dict(op="create", level=0), dict(op="splat", dst=("s0", 0, 8), normalize=1)]
    _conv(wl, "conv", 0, ("s0", 0, 8), ("c0", 0, 16), False, seed, std=0.1)
    wl.ops.append(dict(op="slice", level=0, src=("c0", 0, 16), out="slice"))
    return _finish(wl)


def config2(seed: int = 1, m: int = 2048) -> Workload:
    """ShapeNet-sized object (2,048 surface points), sigma 0.05, 32 features;
    splat -> conv 32->64 -> coarsen (strided conv 64->64) -> conv 64->64 ->
    slice at the coarse level, fp32."""
    pos = gen.object_surfaces(seed, m)
    F = gen.normal_matrix(seed, "F", m, 32, 1.0)
    wl = Workload(2, "object", seed, pos, np.full(3, 0.05, np.float32), "f32", F)
    wl.buffers = {"s0": (0, 32), "c0": (0, 64), "d1": (1, 64), "c1": (1, 64)}
    wl.ops = [dict(op="create", level=0), dict(op="splat", dst=("s0", 0, 32), normalize=1)]
    _conv(wl, "conv", 0, ("s0", 0, 32), ("c0", 0, 64), True, seed)
    wl.ops.append(dict(op="coarsen", level=1))
    _conv(wl, "conv_down", 1, ("c0", 0, 64), ("d1", 0, 64), True, seed)
    _conv(wl, "conv", 1, ("d1", 0, 64), ("c1", 0, 64), False, seed)
    wl.ops.append(dict(op="slice", level=1, src=("c1", 0, 64), out="slice"))
    return _finish(wl)


def _room_features(seed, pos, channels, st_name="rgb"):
    st = gen.Stream(seed, st_name)
    rgb = st.uniform(3 * pos.shape[0]).reshape(-1, 3)
    raw = np.concatenate([pos.astype(np.float64), rgb], axis=1)
    return gen.lifted_features(seed, raw, channels)


def _deform_vector(wl, seed, C, name="deform"):
    wl.vectors[name] = (gen.normal_matrix(seed, "wv:" + name, 1, C, 1.0 / np.sqrt(C))[0], 0.1)


def config3(seed: int = 2, m: int = 200_000) -> Workload:
    """ScanNet-sized room (200k points, 8x8x3 m, 20 boxes, 1 cm noise),
    xyz+RGB lifted to 64 channels, sigma 0.05 m; splat -> conv 64->64 ->
    slice and DeformSlice, fp32."""
    pos = gen.room(seed, m, (8.0, 8.0, 3.0), 20, 0.01)
    F = _room_features(seed, pos, 64)
    wl = Workload(3, "indoor-room", seed, pos, np.full(3, 0.05, np.float32), "f32", F)
    wl.buffers = {"s0": (0, 64), "c0": (0, 64)}
    wl.ops = [dict(op="create", level=0), dict(op="splat", dst=("s0", 0, 64), normalize=1)]
    _conv(wl, "conv", 0, ("s0", 0, 64), ("c0", 0, 64), False, seed)
    _deform_vector(wl, seed, 64)
    wl.ops.append(dict(op="slice", level=0, src=("c0", 0, 64), out="slice"))
    wl.ops.append(dict(op="deform_slice", level=0, src=("c0", 0, 64), wv="deform", out="deform"))
    return _finish(wl)


def config4(seed: int = 3, m: int = 120_000) -> Workload:
    """SemanticKITTI-sized LiDAR scan (120k points), intensity lifted to 64
    channels, sigma 0.3 m, three lattice levels, fp32:
      L0 conv 64->64, coarsen 64->128, L1 conv 128->128, coarsen 128->128,
      L2 conv 128->128, refine 128->128 to L1, refine 128->64 to L0,
      then slice and DeformSlice of the L0 result."""
    pos = gen.lidar_scan(seed, m)
    st = gen.Stream(seed, "intensity")
    F = gen.lifted_features(seed, st.uniform(m).reshape(m, 1), 64)
    wl = Workload(4, "lidar-scan", seed, pos, np.full(3, 0.3, np.float32), "f32", F)
    wl.buffers = {"s0": (0, 64), "e0": (0, 64), "d1": (1, 128), "e1": (1, 128),
                  "d2": (2, 128), "e2": (2, 128), "u1": (1, 128), "u0": (0, 64)}
    wl.ops = [dict(op="create", level=0), dict(op="splat", dst=("s0", 0, 64), normalize=1)]
    _conv(wl, "conv", 0, ("s0", 0, 64), ("e0", 0, 64), True, seed)
    wl.ops.append(dict(op="coarsen", level=1))
    _conv(wl, "conv_down", 1, ("e0", 0, 64), ("d1", 0, 128), True, seed)
    _conv(wl, "conv", 1, ("d1", 0, 128), ("e1", 0, 128), True, seed)
    wl.ops.append(dict(op="coarsen", level=2))
    _conv(wl, "conv_down", 2, ("e1", 0, 128), ("d2", 0, 128), True, seed)
    _conv(wl, "conv", 2, ("d2", 0, 128), ("e2", 0, 128), True, seed)
    _conv(wl, "refine", 1, ("e2", 0, 128), ("u1", 0, 128), True, seed)
    _conv(wl, "refine", 0, ("u1", 0, 128), ("u0", 0, 64), False, seed)
    _deform_vector(wl, seed, 64)
    wl.ops.append(dict(op="slice", level=0, src=("u0", 0, 64), out="slice"))
    wl.ops.append(dict(op="deform_slice", level=0, src=("u0", 0, 64), wv="deform", out="deform"))
    return _finish(wl)


def config5(seed: int = 4, m: int = 1_000_000, size=(20.0, 20.0, 3.0), nboxes: int = 125) -> Workload:
    """Large indoor stack (1M points, 20x20x3 m room, 125 boxes), 64 lifted
    channels, sigma 0.05 m, a 4-level U-Net of lattice convolutions at
    64/128/192/256 channels with concatenated skips, bf16 storage and MFMA
    inputs with fp32 accumulation, DeformSlice to the points."""
    pos = gen.room(seed, m, size, nboxes, 0.01)
    F = _room_features(seed, pos, 64)
    wl = Workload(5, "large-indoor-unet", seed, pos, np.full(3, 0.05, np.float32), "bf16", F)
    wl.buffers = {"s0": (0, 64), "cat0": (0, 128), "d1": (1, 128), "cat1": (1, 256),
                  "d2": (2, 192), "cat2": (2, 384), "d3": (3, 256), "e3": (3, 256),
                  "u2": (2, 192), "u1": (1, 128), "out0": (0, 64)}
    wl.ops = [dict(op="create", level=0), dict(op="splat", dst=("s0", 0, 64), normalize=1)]
    _conv(wl, "conv", 0, ("s0", 0, 64), ("cat0", 64, 64), True, seed)
    wl.ops.append(dict(op="coarsen", level=1))
    _conv(wl, "conv_down", 1, ("cat0", 64, 64), ("d1", 0, 128), True, seed)
    _conv(wl, "conv", 1, ("d1", 0, 128), ("cat1", 128, 128), True, seed)
    wl.ops.append(dict(op="coarsen", level=2))
    _conv(wl, "conv_down", 2, ("cat1", 128, 128), ("d2", 0, 192), True, seed)
    _conv(wl, "conv", 2, ("d2", 0, 192), ("cat2", 192, 192), True, seed)
    wl.ops.append(dict(op="coarsen", level=3))
    _conv(wl, "conv_down", 3, ("cat2", 192, 192), ("d3", 0, 256), True, seed)
    _conv(wl, "conv", 3, ("d3", 0, 256), ("e3", 0, 256), True, seed)
    _conv(wl, "refine", 2, ("e3", 0, 256), ("cat2", 0, 192), True, seed)
    _conv(wl, "conv", 2, ("cat2", 0, 384), ("u2", 0, 192), True, seed)
    _conv(wl, "refine", 1, ("u2", 0, 192), ("cat1", 0, 128), True, seed)
    _conv(wl, "conv", 1, ("cat1", 0, 256), ("u1", 0, 128), True, seed)
    _conv(wl, "refine", 0, ("u1", 0, 128), ("cat0", 0, 64), True, seed)
    _conv(wl, "conv", 0, ("cat0", 0, 128), ("out0", 0, 64), False, seed)
    _deform_vector(wl, seed, 64)
    wl.ops.append(dict(op="deform_slice", level=0, src=("out0", 0, 64), wv="deform", out="deform"))
    return _finish(wl)


def config6(seed: int = 3, m: int = 120_000) -> Workload:
    """The LiDAR scan of config 4 entering the network the paper's way:
    Distribute + PointNet of the positions and 4 raw point features
    (intensity U[0,1] and a random unit vector) through 1x1 layers
    16/32/64, then a 1-hop convolution 64->64 and slice, fp32."""
    pos = gen.lidar_scan(seed, m)
    st = gen.Stream(seed, "raw-features")
    inten = st.uniform(m).reshape(m, 1)
    u = st.normal(3 * m).reshape(m, 3)
    u /= np.linalg.norm(u, axis=1, keepdims=True)
    F = np.concatenate([inten, u], axis=1).astype(np.float32)
    wl = Workload(6, "lidar-distribute", seed, pos, np.full(3, 0.3, np.float32), "f32", F)
    wl.buffers = {"p0": (0, 64), "e0": (0, 64)}
    names = _pointnet(wl, seed, (16, 32, 64))
    wl.ops = [dict(op="create", level=0),
              dict(op="distribute", level=0, dst=("p0", 0, 64), layers=names, norm="pointnet")]
    _conv(wl, "conv", 0, ("p0", 0, 64), ("e0", 0, 64), True, seed)
    wl.ops.append(dict(op="slice", level=0, src=("e0", 0, 64), out="slice"))
    return _finish(wl)


def _pointnet(wl, seed, widths):
    """The PointNet block's three 1x1 layers (W ~ N(0, 1/fan_in), biases
    N(0, 0.1^2)) and its three GroupNorms (gamma ~ 1 + N(0, 0.1^2), beta ~
    N(0, 0.1^2), concatenated over the layer inputs); returns the layer names."""
    k = 3 + wl.features.shape[1]
    names, fan_ins = [], []
    for i, c in enumerate(widths):
        W = gen.normal_matrix(seed, f"pointnet{i}", c, k, 1.0 / np.sqrt(k))
        b = gen.normal_matrix(seed, f"pointnet{i}:bias", 1, c, 0.1)[0]
        wl.mlp[f"pointnet{i}"] = (W, b)
        names.append(f"pointnet{i}")
        fan_ins.append(k)
        k = c
    tot = sum(fan_ins)
    gam = 1.0 + gen.normal_matrix(seed, "gn-gamma:pointnet", 1, tot, 0.1)[0]
    bet = gen.normal_matrix(seed, "gn-beta:pointnet", 1, tot, 0.1)[0]
    wl.norms["pointnet"] = (gam.astype(np.float32), bet.astype(np.float32))
    return names


def _preact(wl, kind, level, src, dst, seed, res=None, groups=32):
    """A pre-activated convolution conv(relu(GN(src))) (+ res)."""
    name = f"{kind}{level}_{src[0]}{src[1]}_{dst[0]}{dst[1]}_{len(wl.ops)}"
    wl.weights[name] = gen.conv_weights(seed, name, TAPS, src[2], dst[2])
    gam = 1.0 + gen.normal_matrix(seed, "gn-gamma:" + name, 1, src[2], 0.1)[0]
    bet = gen.normal_matrix(seed, "gn-beta:" + name, 1, src[2], 0.1)[0]
    wl.norms[name] = (gam.astype(np.float32), bet.astype(np.float32))
    op = dict(op=kind, level=level, src=src, dst=dst, w=name, relu=False, pre=dict(norm=name, groups=groups))
    if res is not None:
        op["res"] = res
    wl.ops.append(op)


def _resnet(wl, level, x, tmp, out, seed):
    """ResNet block of the architecture figure: out = x + [GN, ReLU, conv]^2 (x)."""
    _preact(wl, "conv", level, x, tmp, seed)
    _preact(wl, "conv", level, tmp, out, seed, res=x)


def _latticenet(wl, seed, widths=(64, 128, 256), classes=20):
    """The LatticeNet forward network of the architecture figure on wl's
    points (raw features wl.features): Distribute + PointNet (16/32/64) ->
    ResNet -> Downsample -> ResNet x2 -> Downsample -> ResNet x2 -> Upsample
    -> concatenate the level-1 skip -> ResNet x2 -> Upsample -> concatenate
    the level-0 skip -> ResNet -> DeformSlice fused with the linear
    classifier.  Every convolution is pre-activated by GroupNorm(32) + ReLU;
    levels carry widths[0..2] channels; the concatenations are column ranges
    of one buffer per level (no copies)."""
    c0, c1, c2 = widths
    wl.buffers = {"p0": (0, c0), "h0": (0, c0), "cat0": (0, 2 * c0), "d1": (1, c1), "h1": (1, c1), "r1": (1, c1),
                  "cat1": (1, 2 * c1), "d2": (2, c2), "h2": (2, c2), "r2": (2, c2), "b2": (2, c2),
                  "hu1": (1, 2 * c1), "ru1": (1, 2 * c1), "u1": (1, 2 * c1), "hu0": (0, 2 * c0), "u0": (0, 2 * c0)}
    wl.ops = [dict(op="create", level=0), dict(op="coarsen", level=1), dict(op="coarsen", level=2)]
    names = _pointnet(wl, seed, (16, 32, c0))
    wl.ops.append(dict(op="distribute", level=0, dst=("p0", 0, c0), layers=names, norm="pointnet"))
    _resnet(wl, 0, ("p0", 0, c0), ("h0", 0, c0), ("cat0", c0, c0), seed)           # skip of level 0
    _preact(wl, "conv_down", 1, ("cat0", c0, c0), ("d1", 0, c1), seed)
    _resnet(wl, 1, ("d1", 0, c1), ("h1", 0, c1), ("r1", 0, c1), seed)
    _resnet(wl, 1, ("r1", 0, c1), ("h1", 0, c1), ("cat1", c1, c1), seed)          # skip of level 1
    _preact(wl, "conv_down", 2, ("cat1", c1, c1), ("d2", 0, c2), seed)
    _resnet(wl, 2, ("d2", 0, c2), ("h2", 0, c2), ("r2", 0, c2), seed)
    _resnet(wl, 2, ("r2", 0, c2), ("h2", 0, c2), ("b2", 0, c2), seed)
    _preact(wl, "refine", 1, ("b2", 0, c2), ("cat1", 0, c1), seed)
    _resnet(wl, 1, ("cat1", 0, 2 * c1), ("hu1", 0, 2 * c1), ("ru1", 0, 2 * c1), seed)
    _resnet(wl, 1, ("ru1", 0, 2 * c1), ("hu1", 0, 2 * c1), ("u1", 0, 2 * c1), seed)
    _preact(wl, "refine", 0, ("u1", 0, 2 * c1), ("cat0", 0, c0), seed)
    _resnet(wl, 0, ("cat0", 0, 2 * c0), ("hu0", 0, 2 * c0), ("u0", 0, 2 * c0), seed)
    _deform_vector(wl, seed, 2 * c0)
    wl.classifiers["classifier"] = (gen.normal_matrix(seed, "classifier", classes, 2 * c0, 1.0 / np.sqrt(2 * c0)),
                                    gen.normal_matrix(seed, "classifier:bias", 1, classes, 0.1)[0])
    wl.ops.append(dict(op="deform_classify", level=0, src=("u0", 0, 2 * c0), wv="deform", cls="classifier",
                       out="logits"))


def config8(seed: int = 3, m: int = 120_000) -> Workload:
    """LatticeNet forward on the SemanticKITTI-sized LiDAR scan of config 4:
    raw feature = intensity, sigma 0.3 m, widths 64/128/256, 20 classes,
    fp32."""
    pos = gen.lidar_scan(seed, m)
    inten = gen.Stream(seed, "intensity").uniform(m).reshape(m, 1).astype(np.float32)
    wl = Workload(8, "latticenet-lidar", seed, pos, np.full(3, 0.3, np.float32), "f32", inten)
    _latticenet(wl, seed)
    return _finish(wl)


def config9(seed: int = 2, m: int = 200_000, size=(8.0, 8.0, 3.0), nboxes: int = 20) -> Workload:
    """LatticeNet forward on the ScanNet-sized room of config 3: raw
    features = RGB, sigma 0.05 m, widths 64/128/256, 20 classes, fp32."""
    pos = gen.room(seed, m, size, nboxes, 0.01)
    rgb = gen.Stream(seed, "rgb").uniform(3 * m).reshape(m, 3).astype(np.float32)
    wl = Workload(9, "latticenet-room", seed, pos, np.full(3, 0.05, np.float32), "f32", rgb)
    _latticenet(wl, seed)
    return _finish(wl)


def _backward(wl, loss_out):
    """Append the backward pass of wl's forward ops for a loss whose gradient
    with respect to the point output `loss_out` is wl.grads[loss_out]: the
    ops in reverse order, each turning the gradient of its output buffer
    into that of its input buffer ("g" + name) and of its parameters."""
    fwd = list(wl.ops)
    for name, (lv, total) in list(wl.buffers.items()):
        wl.buffers["g" + name] = (lv, total)
    for op in reversed(fwd):
        kind = op["op"]
        if kind == "deform_slice" and op["out"] == loss_out:
            name, c0, cc = op["src"]
            wl.ops.append(dict(op="deform_slice_bwd", level=op["level"], x=op["src"], wv=op["wv"], grad=loss_out,
                               dst=("g" + name, c0, cc), out="dwv:" + op["wv"]))
        elif kind in ("conv", "conv_down", "refine"):
            (sn, s0, sc), (dn, d0, dc) = op["src"], op["dst"]
            wl.ops.append(dict(op="conv_bwd", kind=kind, level=op["level"], x=op["src"], y=op["dst"], w=op["w"],
                               relu=op["relu"], src=("g" + dn, d0, dc), dst=("g" + sn, s0, sc), out="dW:" + op["w"]))
        elif kind == "splat":
            name, c0, cc = op["dst"]
            wl.ops.append(dict(op="splat_bwd", normalize=op["normalize"], src=("g" + name, c0, cc), out="dfeat"))
        elif kind in ("create", "coarsen"):
            continue
        else:
            raise ValueError(f"no backward for {kind}")


def config7(seed: int = 3, m: int = 120_000) -> Workload:
    """A training step on the LiDAR scan of config 4: its forward network
    ending in DeformSlice (no plain slice), then the backward pass of every
    operator for a loss gradient dL/d(DeformSlice output) ~ N(0, 1): dL/dx
    through DeformSlice, the two Upsamples, the three convolutions and the
    two strided convolutions down to the splat, dL/dW and dL/dbias of every
    convolution, dL/dwv and dL/dbeta of DeformSlice and dL/dfeatures."""
    wl = config4(seed, m)
    wl.cfg, wl.name = 7, "lidar-train-step"
    wl.ops = [op for op in wl.ops if op["op"] != "slice"]
    wl.grads["deform"] = gen.Stream(seed, "loss-grad").normal(wl.m * 64).reshape(wl.m, 64).astype(np.float32)
    _backward(wl, "deform")
    return wl


def config10(seed: int = 4, m: int = 1_000_000, size=(20.0, 20.0, 3.0), nboxes: int = 125) -> Workload:
    """LatticeNet forward on the large indoor stack of config 5 (1M points,
    20x20x3 m room, 125 boxes): raw features = RGB, sigma 0.05 m, widths
    64/128/256, 20 classes, bf16 storage of every lattice activation and
    bf16 MFMA inputs with fp32 accumulation (Distribute + PointNet in fp32,
    its output rounded to bf16; the classifier in fp32 from the bf16
    values)."""
    pos = gen.room(seed, m, size, nboxes, 0.01)
    rgb = gen.Stream(seed, "rgb").uniform(3 * m).reshape(m, 3).astype(np.float32)
    wl = Workload(10, "latticenet-large-indoor", seed, pos, np.full(3, 0.05, np.float32), "bf16", rgb)
    _latticenet(wl, seed)
    return _finish(wl)


CONFIGS = {1: config1, 2: config2, 3: config3, 4: config4, 5: config5, 6: config6, 7: config7, 8: config8,
           9: config9, 10: config10}


def make(cfg: int, seed: int | None = None, **kw) -> Workload:
    fn = CONFIGS[cfg]
    return fn(**kw) if seed is None else fn(seed=seed, **kw)
