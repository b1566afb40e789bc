"""Seeded synthetic workloads for the LionMuon step.

This module only draws inputs: it holds none of the optimizer's arithmetic and
is shared, as the single input source, by the oracle-based tests, the GPU
parity tests and the benchmark.

The paper trains GPT-2 / LLaMA models on FineWeb, SlimPajama and WikiText-103;
none of those datasets or trained weights are available, so gradients are
drawn from seeded distributions of the same shapes:

* ``single768``  -- one 768x768 matrix, W ~ N(0, 0.02^2), M = 0,
  G ~ N(0, 1e-2^2), four steps with P = 2 (fp32 Newton-Schulz path).
* ``gpt2-124m``  -- 12 layers x {768x2304 qkv, 768x768 attn-proj,
  768x3072 fc, 3072x768 mlp-proj}, G ~ N(0, 1e-3^2).
* ``gpt2-355m``  -- 24 layers, d = 1024, ffn 4096, heavy-tailed gradients
  1e-3 * T_3 / sqrt(3) (Student-t with 3 degrees of freedom has variance 3,
  so the standard deviation is 1e-3).
* ``gpt2-720m``  -- 36 layers, d = 1280, ffn 5120, G ~ N(0, 1e-3^2), plus a
  Lion-only 50257x1280 token embedding and every 1-D bias / norm vector.

CPU draws use ``numpy.random.default_rng([config_id, tensor_index, stream,
step])``; device draws (for the large sets, where CPU generation would
dominate) use a seeded ``torch.Generator`` on the GPU.
"""
from __future__ import annotations

from dataclasses import dataclass, field

import numpy as np

W_STD = 0.02


@dataclass(frozen=True)
class TensorSpec:
    name: str
    rows: int
    cols: int           # 1-D tensors have rows = 1
    lion_only: bool = False

    @property
    def numel(self) -> int:
        return self.rows * self.cols

    @property
    def shape(self):
        return (self.cols,) if self.rows == 1 else (self.rows, self.cols)


@dataclass(frozen=True)
class Workload:
    name: str
    config_id: int
    tensors: tuple
    grad_dist: str          # "normal" or "student_t3"
    grad_std: float
    P: int = 2
    beta1: float = 0.9
    beta2: float = 0.99
    lr_muon: float = 3e-3
    lr_lion: float = 2e-5
    wd: float = 0.1
    ns_precision: str = "bf16"
    extra: dict = field(default_factory=dict)

    @property
    def numel(self) -> int:
        return sum(t.numel for t in self.tensors)

    @property
    def matrix_numel(self) -> int:
        return sum(t.numel for t in self.tensors if not t.lion_only and t.rows > 1)


def _block(prefix, layers, d, ffn, qkv_cols):
    out = []
    for i in range(layers):
        out += [TensorSpec(f"{prefix}{i}.attn.qkv", d, qkv_cols),
                TensorSpec(f"{prefix}{i}.attn.proj", d, d),
                TensorSpec(f"{prefix}{i}.mlp.fc", d, ffn),
                TensorSpec(f"{prefix}{i}.mlp.proj", ffn, d)]
    return out


def _gpt2_vectors(layers, d, ffn):
    out = []
    for i in range(layers):
        out += [TensorSpec(f"h{i}.ln1.w", 1, d, True),
                TensorSpec(f"h{i}.ln1.b", 1, d, True),
                TensorSpec(f"h{i}.attn.qkv.b", 1, 3 * d, True),
                TensorSpec(f"h{i}.attn.proj.b", 1, d, True),
                TensorSpec(f"h{i}.ln2.w", 1, d, True),
                TensorSpec(f"h{i}.ln2.b", 1, d, True),
                TensorSpec(f"h{i}.mlp.fc.b", 1, ffn, True),
                TensorSpec(f"h{i}.mlp.proj.b", 1, d, True)]
    out += [TensorSpec("ln_f.w", 1, d, True), TensorSpec("ln_f.b", 1, d, True)]
    return out


def single768() -> Workload:
    return Workload("single768", 0, (TensorSpec("w", 768, 768),), "normal",
                    1e-2, P=2, lr_muon=0.02, lr_lion=0.02, wd=0.1,
                    ns_precision="fp32", extra={"steps": (1, 2, 3, 4)})


def gpt2_124m() -> Workload:
    return Workload("gpt2-124m", 1, tuple(_block("h", 12, 768, 3072, 2304)),
                    "normal", 1e-3)


def gpt2_355m() -> Workload:
    return Workload("gpt2-355m", 2, tuple(_block("h", 24, 1024, 4096, 3072)),
                    "student_t3", 1e-3)


def gpt2_720m() -> Workload:
    mats = _block("h", 36, 1280, 5120, 3840)
    emb = [TensorSpec("wte", 50257, 1280, True)]
    return Workload("gpt2-720m", 3, tuple(mats + emb + _gpt2_vectors(36, 1280, 5120)),
                    "normal", 1e-3)


WORKLOADS = {"single768": single768, "gpt2-124m": gpt2_124m,
             "gpt2-355m": gpt2_355m, "gpt2-720m": gpt2_720m}


def get(name: str) -> Workload:
    return WORKLOADS[name]()


# ----------------------------------------------------------------------------
# CPU draws (numpy, float64 -> float32)
# ----------------------------------------------------------------------------
STREAM_W, STREAM_M, STREAM_G = 0, 1, 2


def _rng(config_id, index, stream, step):
    return np.random.default_rng([int(config_id), int(index), int(stream), int(step)])


def draw(dist: str, std: float, shape, rng) -> np.ndarray:
    """fp32 sample of a zero-mean distribution with standard deviation std."""
    if dist == "normal":
        x = rng.standard_normal(shape) * std
    elif dist == "student_t3":
        x = rng.standard_t(3, size=shape) * (std / np.sqrt(3.0))
    else:
        raise ValueError(dist)
    return x.astype(np.float32)


def initial_weight(wl: Workload, index: int) -> np.ndarray:
    spec = wl.tensors[index]
    return draw("normal", W_STD, spec.shape, _rng(wl.config_id, index, STREAM_W, 0))


def initial_momentum(wl: Workload, index: int, warm: bool = False) -> np.ndarray:
    """M = 0 (Algorithm 1's M_{-1}); ``warm`` gives a seeded non-zero buffer of
    the gradient scale, as a mid-training state for single-step tests."""
    spec = wl.tensors[index]
    if not warm:
        return np.zeros(spec.shape, dtype=np.float32)
    return draw(wl.grad_dist, wl.grad_std, spec.shape,
                _rng(wl.config_id, index, STREAM_M, 0))


def gradient(wl: Workload, index: int, step: int) -> np.ndarray:
    spec = wl.tensors[index]
    return draw(wl.grad_dist, wl.grad_std, spec.shape,
                _rng(wl.config_id, index, STREAM_G, step))


def random_matrix(seed, rows, cols, std=1.0, dist="normal") -> np.ndarray:
    """Free-standing seeded fp32 matrix for edge-case tests."""
    return draw(dist, std, (rows, cols), np.random.default_rng(seed))


# ----------------------------------------------------------------------------
# Device draws (torch, for the full-size sets)
# ----------------------------------------------------------------------------
def device_draw(torch, dist, std, numel, gen, device):
    """Seeded fp32 draw of ``numel`` values on ``device`` via ``gen``."""
    if dist == "normal":
        x = torch.randn(numel, generator=gen, device=device, dtype=torch.float32)
        return x.mul_(std)
    if dist == "student_t3":
        # T_3 = Z / sqrt(V/3), V ~ chi^2_3 = sum of three squared normals.
        z = torch.randn(numel, generator=gen, device=device, dtype=torch.float32)
        v = torch.randn(3, numel, generator=gen, device=device,
                        dtype=torch.float32).square_().sum(0)
        return z.mul_(torch.rsqrt(v.div_(3.0))).mul_(std / np.sqrt(3.0))
    raise ValueError(dist)


def device_state(torch, wl: Workload, device, seed=1234, warm=True, n_grad=2):
    """Allocate W, M and ``n_grad`` gradient sets for every tensor on device.

    Returns (params, moms, grad_sets) as lists of contiguous fp32 tensors.
    """
    gen = torch.Generator(device=device)
    gen.manual_seed(seed * 1000 + wl.config_id)
    params, moms = [], []
    grad_sets = [[] for _ in range(n_grad)]
    for spec in wl.tensors:
        params.append(device_draw(torch, "normal", W_STD, spec.numel, gen,
                                  device).view(spec.shape))
        if warm:
            moms.append(device_draw(torch, wl.grad_dist, wl.grad_std, spec.numel,
                                    gen, device).view(spec.shape))
        else:
            moms.append(torch.zeros(spec.shape, device=device, dtype=torch.float32))
        for g in grad_sets:
            g.append(device_draw(torch, wl.grad_dist, wl.grad_std, spec.numel,
                                 gen, device).view(spec.shape))
    return params, moms, grad_sets
