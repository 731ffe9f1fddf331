"""Seeded synthetic optimizer-step inputs (W, G, M_prev) for the benchmark
stacks.  Holds no part of the NormPre arithmetic: it only draws tensors.

The paper trains on OpenWebText / C4 / Pile; those datasets and trained
weights are not used.  These inputs stand in for them with the layer shapes of
the models in the paper's model table (App. A) and gradient spectra of the
kinds listed per workload:

  single_256  one 256 x 256 matrix, G = Z diag(s), Z ~ N(0,1), s_j = 1/j
  gpt2_small  12 layers x {768x2304, 768x768, 768x3072, 3072x768};
              G = A B^T / sqrt(32) + 0.1 N  (rank-32 signal plus noise)
  llama_1b    16 layers x {2048x2048 x2, 2048x512 x2, 2048x5632 x2, 5632x2048};
              G = U diag(i^-0.7) V^T with Haar U, V
  qwen3_1p7b  28 layers x {2048x2048 x2, 2048x1024 x2, 2048x6144 x2, 6144x2048};
              G i.i.d. Student-t with nu = 3
  large_sweep 4096^2, 4096x16384, 8192^2, 8192x28672 with the power-law spectrum

W ~ N(0, 0.02^2) (GPT-2 / LLaMA initialisation scale); M_prev is an
independent draw from the distribution of G so the momentum read is not
trivial.  Every tensor has its own generator seed
seed_base + 1000 * workload_index + 10 * matrix_index + kind.
"""
from __future__ import annotations

import math
from dataclasses import dataclass, field

import torch


@dataclass
class Workload:
    name: str
    index: int
    shapes: list            # [(m, n), ...] in caller order
    grad_kind: str          # "decay", "lowrank", "powerlaw", "student_t"
    lr: float
    rank: int
    oversample: int = 8
    power_iters: int = 1
    description: str = ""
    extra: dict = field(default_factory=dict)

    @property
    def elements(self) -> int:
        return sum(m * n for m, n in self.shapes)


def _layers(n_layers, per_layer):
    out = []
    for _ in range(n_layers):
        out.extend(per_layer)
    return out


WORKLOADS = {
    "single_256": Workload("single_256", 0, [(256, 256)], "decay", 6e-4, rank=16,
                           description="one 256x256 matrix, G = Z diag(1/j)"),
    "gpt2_small": Workload("gpt2_small", 1,
                           _layers(12, [(768, 2304), (768, 768), (768, 3072), (3072, 768)]),
                           "lowrank", 6e-4, rank=32,
                           description="GPT-2 Small hidden matrices (48), rank-32 signal + 0.1 noise"),
    "llama_1b": Workload("llama_1b", 2,
                         _layers(16, [(2048, 2048), (2048, 2048), (2048, 512), (2048, 512),
                                      (2048, 5632), (2048, 5632), (5632, 2048)]),
                         "powerlaw", 3e-4, rank=64,
                         description="LLaMA-1B-shaped stack (112), power-law spectrum i^-0.7"),
    "qwen3_1p7b": Workload("qwen3_1p7b", 3,
                           _layers(28, [(2048, 2048), (2048, 2048), (2048, 1024), (2048, 1024),
                                        (2048, 6144), (2048, 6144), (6144, 2048)]),
                           "student_t", 3e-4, rank=32,
                           description="Qwen3-1.7B stack (196), Student-t(3) gradients"),
    "large_sweep": Workload("large_sweep", 4,
                            [(4096, 4096), (4096, 16384), (8192, 8192), (8192, 28672)],
                            "powerlaw", 3e-4, rank=64,
                            description="large single matrices, power-law spectrum",
                            extra={"ranks": [64, 128, 256]}),
}

KIND_W, KIND_G, KIND_M = 0, 1, 2


def _gen(device, seed):
    g = torch.Generator(device=device)
    g.manual_seed(int(seed))
    return g


def _haar(rows, cols, gen, device):
    """rows x cols matrix with orthonormal columns (QR of a Gaussian, signs fixed)."""
    z = torch.randn(rows, cols, generator=gen, device=device, dtype=torch.float32)
    q, r = torch.linalg.qr(z)
    d = torch.sign(torch.diagonal(r))
    d[d == 0] = 1.0
    return q * d


def draw_gradient(kind: str, m: int, n: int, gen, device) -> torch.Tensor:
    f32 = torch.float32
    if kind == "decay":
        z = torch.randn(m, n, generator=gen, device=device, dtype=f32)
        s = 1.0 / torch.arange(1, n + 1, device=device, dtype=f32)
        return z * s[None, :]
    if kind == "lowrank":
        a = torch.randn(m, 32, generator=gen, device=device, dtype=f32)
        b = torch.randn(n, 32, generator=gen, device=device, dtype=f32)
        noise = torch.randn(m, n, generator=gen, device=device, dtype=f32)
        return (a @ b.T) / math.sqrt(32.0) + 0.1 * noise
    if kind == "powerlaw":
        s = min(m, n)
        u = _haar(m, s, gen, device)
        v = _haar(n, s, gen, device)
        sig = torch.arange(1, s + 1, device=device, dtype=f32) ** -0.7
        return (u * sig[None, :]) @ v.T
    if kind == "student_t":
        z0 = torch.randn(m, n, generator=gen, device=device, dtype=f32)
        chi = torch.zeros(m, n, device=device, dtype=f32)
        for _ in range(3):
            zi = torch.randn(m, n, generator=gen, device=device, dtype=f32)
            chi += zi * zi
        return z0 / torch.sqrt(chi / 3.0)
    raise ValueError(f"unknown gradient kind {kind!r}")


def make_matrix(wl: Workload, i: int, device="cpu", seed_base: int = 1337, shape=None):
    """(W, G, M_prev) of matrix i of a workload (shape override for tests)."""
    m, n = shape if shape is not None else wl.shapes[i]
    base = seed_base + 1000 * wl.index + 10 * i
    w = 0.02 * torch.randn(m, n, generator=_gen(device, base + KIND_W), device=device, dtype=torch.float32)
    g = draw_gradient(wl.grad_kind, m, n, _gen(device, base + KIND_G), device)
    mp = draw_gradient(wl.grad_kind, m, n, _gen(device, base + KIND_M), device)
    return w.contiguous(), g.contiguous(), mp.contiguous()


def make_stack(wl: Workload, device="cpu", seed_base: int = 1337, indices=None):
    """Lists W, G, M_prev for the whole stack (or the given matrix indices)."""
    idx = range(len(wl.shapes)) if indices is None else indices
    ws, gs, ms = [], [], []
    for i in idx:
        w, g, mp = make_matrix(wl, i, device, seed_base)
        ws.append(w)
        gs.append(g)
        ms.append(mp)
    return ws, gs, ms
