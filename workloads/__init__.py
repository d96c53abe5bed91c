"""Seeded synthetic workloads shared by the HIP path's tests/bench and by the oracle.

This module only *draws* inputs: shapes, value distributions and seeds of the
five training / contraction workloads of the MagmaDNN-style SGD step.  It holds
none of the method's arithmetic (no GEMM, convolution, loss, update or storage
rounding of intermediate results); the only conversions here turn an fp64 draw
into the bits of the storage type the workload names, which *defines* the
input.

Seeding: workload ``i`` uses base seed ``1188 + i``; every tensor comes from its
own child stream ``numpy.random.default_rng(SeedSequence([base, tensor_id]))``
so that drawing one tensor never shifts another.

Storage dtypes are returned as numpy arrays:
  * ``"f32"``  -> float32
  * ``"f16"``  -> float16
  * ``"bf16"`` -> uint16 bit patterns (numpy has no bfloat16); the fp32 value is
    rounded to nearest-even by torch's CPU conversion.
"""
from __future__ import annotations

import dataclasses
import math
from typing import List, Optional, Sequence, Tuple

import numpy as np

DTYPES = ("f32", "f16", "bf16")

# Layer kinds of the fixed training chains (paper section 2.1: a compute graph
# of tensor ops trained by backpropagation; here the graph is a fixed chain).
FC, CONV, MAXPOOL2 = 0, 1, 2
ACT_NONE, ACT_RELU = 0, 1
LOSS_XENT, LOSS_MSE = 0, 1


def rng(base_seed: int, tensor_id: int) -> np.random.Generator:
    return np.random.default_rng(np.random.SeedSequence([base_seed, tensor_id]))


def to_storage(x: np.ndarray, dtype: str) -> np.ndarray:
    """Round an fp64 draw to the storage type that defines the input."""
    x = np.asarray(x, dtype=np.float64)
    if dtype == "f32":
        return x.astype(np.float32)
    if dtype == "f16":
        return x.astype(np.float16)
    if dtype == "bf16":
        import torch

        t = torch.from_numpy(x.astype(np.float32)).to(torch.bfloat16)
        return t.view(torch.int16).numpy().view(np.uint16).copy()
    raise ValueError(f"unknown dtype {dtype!r}")


def bf16_bits_to_f32(bits: np.ndarray) -> np.ndarray:
    """Widen bf16 bit patterns to float32 (exact: bf16 is the top half of fp32)."""
    b = np.asarray(bits, dtype=np.uint16).astype(np.uint32) << 16
    return b.view(np.float32)


def storage_to_f64(a: np.ndarray, dtype: str) -> np.ndarray:
    """Exact widening of stored input bits to fp64."""
    if dtype == "bf16":
        return bf16_bits_to_f32(a).astype(np.float64)
    return np.asarray(a).astype(np.float64)


# ---------------------------------------------------------------------------
# Layer chains
# ---------------------------------------------------------------------------

@dataclasses.dataclass(frozen=True)
class Layer:
    kind: int
    c_in: int            # FC: in_features; CONV/POOL: channels in
    h: int = 1           # spatial input height (CONV/POOL)
    w: int = 1           # spatial input width  (CONV/POOL)
    c_out: int = 0       # FC: out_features; CONV: filters; POOL: = c_in
    r: int = 0
    s: int = 0
    pad: int = 0
    act: int = ACT_NONE

    @property
    def n_weight(self) -> int:
        if self.kind == FC:
            return self.c_in * self.c_out
        if self.kind == CONV:
            return self.c_out * self.r * self.s * self.c_in
        return 0

    @property
    def n_bias(self) -> int:
        return self.c_out if self.kind in (FC, CONV) else 0

    @property
    def fan_in(self) -> int:
        if self.kind == FC:
            return self.c_in
        return self.c_in * self.r * self.s

    def out_features(self) -> int:
        if self.kind == FC:
            return self.c_out
        if self.kind == CONV:
            return self.h * self.w * self.c_out  # stride 1, "same" padding
        return (self.h // 2) * (self.w // 2) * self.c_in


@dataclasses.dataclass(frozen=True)
class TrainConfig:
    name: str
    base_seed: int
    layers: Tuple[Layer, ...]
    batch: int
    in_features: int
    dtype: str            # storage type of activations / working weights
    loss: int
    lr: float
    momentum: float = 0.0
    loss_scaling: bool = False
    init_scale: float = 1.0
    n_classes: int = 10   # cross-entropy only
    steps: int = 10
    x_dist: str = "uniform"  # "uniform" U[0,1) or "normal" N(0,1)

    @property
    def n_params(self) -> int:
        return sum(l.n_weight + l.n_bias for l in self.layers)

    def param_offsets(self) -> List[Tuple[int, int]]:
        """(weight offset, bias offset) of each layer in the flat parameter buffer.

        Packing order: per layer in chain order, weights then bias.  FC weights
        are [in, out] row-major, conv filters are [Cout][R][S][Cin]."""
        out, off = [], 0
        for l in self.layers:
            wo = off
            off += l.n_weight
            bo = off
            off += l.n_bias
            out.append((wo, bo))
        return out

    def flops_per_step(self) -> int:
        """Algorithmic FLOPs of one step: 2*M*N*K per contraction (fwd, bwd-data
        except for the first layer, bwd-weight); element-wise work not counted."""
        total = 0
        for i, l in enumerate(self.layers):
            if l.kind == FC:
                mnk = 2 * self.batch * l.c_in * l.c_out
            elif l.kind == CONV:
                mnk = 2 * self.batch * l.h * l.w * l.c_out * l.r * l.s * l.c_in
            else:
                continue
            total += mnk * (3 if i > 0 else 2)
        return total


def mlp784_fp32() -> TrainConfig:
    """MLP 784->128(ReLU)->10, softmax cross-entropy, batch 64, fp32, SGD lr 0.05."""
    return TrainConfig(
        name="mlp784_fp32_b64", base_seed=1188 + 1,
        layers=(Layer(FC, 784, c_out=128, act=ACT_RELU), Layer(FC, 128, c_out=10)),
        batch=64, in_features=784, dtype="f32", loss=LOSS_XENT, lr=0.05)


def lenet_bf16() -> TrainConfig:
    """LeNet-style CNN, batch 256, bf16 storage, fp32 accumulate/master, lr 0.01."""
    return TrainConfig(
        name="lenet_bf16_b256", base_seed=1188 + 3,
        layers=(
            Layer(CONV, 1, 28, 28, 32, 5, 5, 2, ACT_RELU),
            Layer(MAXPOOL2, 32, 28, 28, 32),
            Layer(CONV, 32, 14, 14, 64, 5, 5, 2, ACT_RELU),
            Layer(MAXPOOL2, 64, 14, 14, 64),
            Layer(FC, 3136, c_out=1024, act=ACT_RELU),
            Layer(FC, 1024, c_out=10),
        ),
        batch=256, in_features=784, dtype="bf16", loss=LOSS_XENT, lr=0.01)


def wide_mlp_fp16(batch: int = 4096, width: int = 4096, init_scale: float = 2.0 ** 16) -> TrainConfig:
    """Wide regression MLP 1024->4x4096(ReLU)->1, MSE, fp16 storage with dynamic
    loss scaling (initial scale 2^16), fp32 master weights, SGD momentum 0.9.
    The learning rate is not given by the workload; 1e-4 is used: at 1e-3
    (with momentum 0.9 and 4096-wide layers) training diverges within a few
    steps, the fp16 forward pass overflows and the loss scaler then skips
    every update.  ``width`` shrinks the hidden layers for quick multi-step
    checks."""
    layers = [Layer(FC, 1024, c_out=width, act=ACT_RELU)]
    layers += [Layer(FC, width, c_out=width, act=ACT_RELU) for _ in range(3)]
    layers += [Layer(FC, width, c_out=1)]
    suffix = "" if width == 4096 else f"_w{width}"
    return TrainConfig(
        name=f"wide_mlp_fp16_b{batch}{suffix}", base_seed=1188 + 5, layers=tuple(layers),
        batch=batch, in_features=1024, dtype="f16", loss=LOSS_MSE, lr=1e-4,
        momentum=0.9, loss_scaling=True, init_scale=init_scale, x_dist="normal")


TRAIN_CONFIGS = {
    "mlp784_fp32": mlp784_fp32,
    "lenet_bf16": lenet_bf16,
    "wide_mlp_fp16": wide_mlp_fp16,
}


# tensor ids inside a training workload's seed space
_TID_W = 100      # + layer index
_TID_X = 1000     # + step index
_TID_T = 2000     # + step index


def init_params(cfg: TrainConfig) -> np.ndarray:
    """He-normal fp32 master weights (std sqrt(2/fan_in), untruncated), bias 0."""
    p = np.zeros(cfg.n_params, dtype=np.float32)
    for i, (l, (wo, bo)) in enumerate(zip(cfg.layers, cfg.param_offsets())):
        if l.n_weight:
            std = math.sqrt(2.0 / l.fan_in)
            p[wo:wo + l.n_weight] = to_storage(
                rng(cfg.base_seed, _TID_W + i).standard_normal(l.n_weight) * std, "f32")
    return p


def batch_inputs(cfg: TrainConfig, step: int, rows: Optional[int] = None):
    """Input batch ``step`` (fp32 [B, in_features], NHWC-flattened for images) and
    its targets: int32 labels U{0..C-1} for cross-entropy, fp32 [B,1] N(0,1) for MSE.

    ``rows`` draws only the first ``rows`` samples of the batch (same values)."""
    b = cfg.batch
    g = rng(cfg.base_seed, _TID_X + step)
    if cfg.x_dist == "uniform":
        x = g.random((b, cfg.in_features))
    else:
        x = g.standard_normal((b, cfg.in_features))
    gt = rng(cfg.base_seed, _TID_T + step)
    if cfg.loss == LOSS_XENT:
        t = gt.integers(0, cfg.n_classes, size=b).astype(np.int32)
    else:
        t = to_storage(gt.standard_normal((b, 1)), "f32")
    x = to_storage(x, "f32")
    if rows is not None:
        x, t = x[:rows].copy(), t[:rows].copy()
    return x, t


# ---------------------------------------------------------------------------
# Contraction workloads
# ---------------------------------------------------------------------------

GEMM_SIZES = (1024, 4096, 8192)
GEMM_LAYOUTS = ("NN", "NT", "TN")
GEMM_BASE_SEED = 1188 + 2


def gemm_operands(layout: str, m: int, n: int, k: int, dtype: str = "f16",
                  seed: int = GEMM_BASE_SEED, scale: Optional[float] = None):
    """A, B with N(0,1)/sqrt(K) entries, stored per layout (row-major):
    NN: A[M,K], B[K,N];  NT: A[M,K], B[N,K];  TN: A[K,M], B[K,N]."""
    s = 1.0 / math.sqrt(k) if scale is None else scale
    a_shape = (k, m) if layout == "TN" else (m, k)
    b_shape = (n, k) if layout == "NT" else (k, n)
    tid = 10 * GEMM_LAYOUTS.index(layout)
    a = rng(seed, tid + 1).standard_normal(a_shape) * s
    b = rng(seed, tid + 2).standard_normal(b_shape) * s
    return to_storage(a, dtype), to_storage(b, dtype)


@dataclasses.dataclass(frozen=True)
class ConvShape:
    n: int
    h: int
    w: int
    c_in: int
    c_out: int
    r: int = 3
    s: int = 3
    pad: int = 1

    def gemm_mnk(self, op: str) -> Tuple[int, int, int]:
        nhw = self.n * self.h * self.w
        if op == "fwd":
            return nhw, self.c_out, self.r * self.s * self.c_in
        if op == "bwd_data":
            return nhw, self.c_in, self.r * self.s * self.c_out
        return self.c_out, self.r * self.s * self.c_in, nhw

    def flops(self) -> int:
        m, n, k = self.gemm_mnk("fwd")
        return 2 * m * n * k


RESNET_LAYERS = (ConvShape(128, 32, 32, 64, 64), ConvShape(128, 16, 16, 128, 128),
                 ConvShape(128, 8, 8, 256, 256))
CONV_BASE_SEED = 1188 + 4


def conv_operands(shape: ConvShape, dtype: str = "f16", seed: int = CONV_BASE_SEED):
    """x [N,H,W,Cin], w [Cout,R,S,Cin], dy [N,H,W,Cout]; all N(0,1)/sqrt(R*S*Cin)."""
    s = 1.0 / math.sqrt(shape.r * shape.s * shape.c_in)
    tid = 10 * (shape.c_in + 1000 * shape.h)
    x = rng(seed, tid + 1).standard_normal((shape.n, shape.h, shape.w, shape.c_in)) * s
    w = rng(seed, tid + 2).standard_normal((shape.c_out, shape.r, shape.s, shape.c_in)) * s
    dy = rng(seed, tid + 3).standard_normal((shape.n, shape.h, shape.w, shape.c_out)) * s
    return to_storage(x, dtype), to_storage(w, dtype), to_storage(dy, dtype)


def normal(shape: Sequence[int], seed: int, tensor_id: int, dtype: str = "f32",
           scale: float = 1.0) -> np.ndarray:
    return to_storage(rng(seed, tensor_id).standard_normal(tuple(shape)) * scale, dtype)


def uniform(shape: Sequence[int], seed: int, tensor_id: int, dtype: str = "f32",
            lo: float = 0.0, hi: float = 1.0) -> np.ndarray:
    return to_storage(lo + (hi - lo) * rng(seed, tensor_id).random(tuple(shape)), dtype)


def small_ints(shape: Sequence[int], seed: int, tensor_id: int, lo: int = -4, hi: int = 4,
               dtype: str = "f16") -> np.ndarray:
    """Integers in [lo, hi]: every product and partial sum stays exact in fp32."""
    v = rng(seed, tensor_id).integers(lo, hi + 1, size=tuple(shape)).astype(np.float64)
    return to_storage(v, dtype)
