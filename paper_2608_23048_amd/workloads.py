"""Seeded synthetic workloads (shapes and value distributions only).

This module holds none of the sampler's arithmetic: it lays out the weight
stacks of the Qwen2.5-shaped workloads and fills them with seeded random
values.  It is the one module that both the HIP path and the CPU oracle's
callers (the tests, the benchmark's CPU baseline) draw inputs from.

Distributions: W ~ N(0, 0.02^2) rounded to bf16, logits ~ N(0, 1) in fp32,
upstream gradient dL/dW_masked ~ N(0, (1e-3)^2) rounded to bf16.  The real
checkpoints and calibration data are not used; only their shapes are.

A stack is laid out back to back in one slab per operand (layer-major, and
within a layer q, k, v, o, gate, up, down); tensor t starts at the global
element offset equal to the sizes of the tensors before it, which is also the
offset of its noise stream.
"""
from __future__ import annotations

from dataclasses import dataclass, field

W_STD = 0.02
LOGIT_STD = 1.0
GRAD_STD = 1e-3


@dataclass(frozen=True)
class Tensor:
    name: str
    rows: int
    cols: int
    offset: int  # global element offset in the slab

    @property
    def numel(self) -> int:
        return self.rows * self.cols


@dataclass(frozen=True)
class Workload:
    name: str
    tensors: tuple[Tensor, ...]
    n: int
    m: int
    tau: float
    description: str = ""
    tau_schedule: tuple[float, float, int] | None = None  # (init, end, T_anneal) over steps
    extra_patterns: tuple[tuple[int, int], ...] = field(default_factory=tuple)

    @property
    def numel(self) -> int:
        return sum(t.numel for t in self.tensors)


def _stack(layer_shapes, layers):
    out, off = [], 0
    for layer in range(layers):
        for name, (r, c) in layer_shapes:
            out.append(Tensor(f"layers.{layer}.{name}", r, c, off))
            off += r * c
    return tuple(out)


def qwen_layer(hidden: int, kv: int, inter: int):
    return [("q_proj", (hidden, hidden)), ("k_proj", (kv, hidden)), ("v_proj", (kv, hidden)),
            ("o_proj", (hidden, hidden)), ("gate_proj", (inter, hidden)),
            ("up_proj", (inter, hidden)), ("down_proj", (hidden, inter))]


QWEN_05B = qwen_layer(896, 128, 4864)
QWEN_15B = qwen_layer(1536, 256, 8960)
QWEN_7B = qwen_layer(3584, 512, 18944)

WORKLOADS = {
    "single-896x896-2:4": Workload(
        "single-896x896-2:4", (Tensor("linear", 896, 896, 0),), 2, 4, 1.0,
        "one 896x896 linear layer, 2:4, tau=1"),
    "qwen2.5-0.5b-stack-2:4": Workload(
        "qwen2.5-0.5b-stack-2:4", _stack(QWEN_05B, 24), 2, 4, 1.0,
        "0.5B-class decoder stack, 24 layers x 7 linears (168 tensors), 2:4, tau=1"),
    "qwen2.5-7b-layer-2:4": Workload(
        "qwen2.5-7b-layer-2:4", _stack(QWEN_7B, 1), 2, 4, 0.5,
        "7B-class single decoder layer (7 tensors), 2:4, tau=0.5"),
    "qwen2.5-7b-layer-4:8": Workload(
        "qwen2.5-7b-layer-4:8", _stack(QWEN_7B, 1), 4, 8, 0.5,
        "7B-class single decoder layer (7 tensors), 4:8, tau=0.5"),
    "qwen2.5-7b-stack-2:4": Workload(
        "qwen2.5-7b-stack-2:4", _stack(QWEN_7B, 28), 2, 4, 1.0,
        "7B-class full stack, 28 layers x 7 linears (196 tensors, 6.53e9 masked weights), 2:4, "
        "tau annealed 1.0 -> 0.1 over 10 steps", tau_schedule=(1.0, 0.1, 9)),
    "qwen2.5-1.5b-stack-8:16": Workload(
        "qwen2.5-1.5b-stack-8:16", _stack(QWEN_15B, 28), 8, 16, 1.0,
        "1.5B-class stack, 28 layers x 7 linears (196 tensors), 8:16, tau=1"),
    "qwen2.5-1.5b-stack-16:32": Workload(
        "qwen2.5-1.5b-stack-16:32", _stack(QWEN_15B, 28), 16, 32, 1.0,
        "1.5B-class stack, 28 layers x 7 linears (196 tensors), 16:32, tau=1"),
}


def tensor_seeds(t_index: int, step: int = 0) -> tuple[int, int, int]:
    """Seeds of W, logits and the upstream gradient of tensor t at a step."""
    return 1_000_000 + t_index, 2_000_000 + t_index, 3_000_000 + 1000 * step + t_index


def _bf16_normal(n, std, gen, device):
    import torch
    x = torch.empty(n, dtype=torch.float32, device=device)
    x.normal_(0.0, std, generator=gen)
    return x.to(torch.bfloat16)


def fill_slab(workload: Workload, device, step: int = 0, W=None, logits=None, grad=None,
              tensors=None):
    """Fill (or allocate) flat slabs W (bf16), logits (fp32), grad (bf16) for a
    workload, tensor by tensor with per-tensor seeds.  `tensors` restricts the
    fill to a subset of tensor indices (the others are left as they are)."""
    import torch
    total = workload.numel
    if W is None:
        W = torch.empty(total, dtype=torch.bfloat16, device=device)
    if logits is None:
        logits = torch.empty(total, dtype=torch.float32, device=device)
    if grad is None:
        grad = torch.empty(total, dtype=torch.bfloat16, device=device)
    idxs = range(len(workload.tensors)) if tensors is None else tensors
    for i in idxs:
        t = workload.tensors[i]
        sw, sl, sg = tensor_seeds(i, step)
        sl_ = slice(t.offset, t.offset + t.numel)
        g = torch.Generator(device=device)
        g.manual_seed(sw)
        W[sl_] = _bf16_normal(t.numel, W_STD, g, device)
        g.manual_seed(sl)
        logits[sl_].normal_(0.0, LOGIT_STD, generator=g)
        g.manual_seed(sg)
        grad[sl_] = _bf16_normal(t.numel, GRAD_STD, g, device)
    return W, logits, grad


def small_case(rows: int, cols: int, seed: int, device="cpu", w_std=W_STD, logit_std=LOGIT_STD,
               grad_std=GRAD_STD):
    """One seeded [rows, cols] case (W bf16, logits fp32, grad bf16)."""
    import torch
    g = torch.Generator(device="cpu")
    g.manual_seed(seed)
    W = (torch.randn(rows, cols, generator=g) * w_std).to(torch.bfloat16)
    L = torch.randn(rows, cols, generator=g) * logit_std
    G = (torch.randn(rows, cols, generator=g) * grad_std).to(torch.bfloat16)
    return W.to(device), L.to(device), G.to(device)
