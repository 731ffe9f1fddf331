"""``torch.optim`` front end of the NormPre library.

The paper applies its matrix optimizers to the hidden two-dimensional
attention and MLP weights and trains every other parameter (token
embeddings, output heads, normalization weights, biases) with AdamW
(App. A.1).  ``NormPreOptimizer`` follows that split: parameter groups marked
``normpre=True`` are stepped together by one ``normpre_step`` call of the C
library (every matrix of the group in one batched step, on the current HIP
stream); all other groups are handed to ``torch.optim.AdamW``.

Momentum buffers and the step counter t (which picks the row/column
orientation, Sec. 3.1, and keys the NormPre-L sketch) live here and are part
of ``state_dict()``.
"""
from __future__ import annotations

import torch

from . import normpre as N


class NormPreOptimizer(torch.optim.Optimizer):
    """Hidden matrices by NormPre (variant "G", "L", "MUON" or "NORM"), the
    rest by AdamW.

    Args:
        params: parameter groups (dicts) or an iterable of parameters; a group
            with ``normpre=True`` holds hidden 2-D fp32 matrices.  Plain
            parameters are split automatically: 2-D tensors go to NormPre
            unless ``matrix_filter`` says otherwise.
        lr: NormPre learning rate (eta of Alg. 1).
        variant: "G" (Newton-Schulz), "L" (sketch), or the reference steps
            "MUON" / "NORM" of the library.
        adamw_lr, adamw_betas, adamw_eps: AdamW for the other parameters
            (App. A.1 uses betas (0.9, 0.95) and the model's learning rate).
        Other keyword arguments are NormPre hyper-parameters (momentum,
        weight_decay, rank, oversample, power_iters, ns_iters, seed, flags...).
    """

    def __init__(self, params, lr: float = 6e-4, variant: str = "G", weight_decay: float = 0.1,
                 adamw_lr: float | None = None, adamw_betas=(0.9, 0.95), adamw_eps: float = 1e-8,
                 matrix_filter=None, **hparams):
        params = list(params)
        if params and not isinstance(params[0], dict):
            keep = matrix_filter or (lambda p: p.dim() == 2)
            mats = [p for p in params if keep(p)]
            rest = [p for p in params if not keep(p)]
            params = []
            if mats:
                params.append({"params": mats, "normpre": True})
            if rest:
                params.append({"params": rest, "normpre": False})
        defaults = dict(lr=lr, weight_decay=weight_decay, normpre=False)
        super().__init__(params, defaults)
        self.variant = variant.upper()
        self.hparams = dict(hparams)
        self.t = int(self.hparams.pop("step", 0))
        adam_groups = []
        for g in self.param_groups:
            if g["normpre"]:
                for p in g["params"]:
                    if p.dim() != 2 or p.dtype != torch.float32 or not p.is_contiguous():
                        raise ValueError("NormPre groups take contiguous 2-D fp32 matrices")
            else:
                adam_groups.append({"params": g["params"], "lr": adamw_lr if adamw_lr is not None else g["lr"],
                                    "weight_decay": g["weight_decay"]})
        self._adamw = (torch.optim.AdamW(adam_groups, betas=adamw_betas, eps=adamw_eps)
                       if adam_groups else None)
        self._ctx = None

    def _context(self, device):
        if self._ctx is None:
            self._ctx = N.normpre_init(device.index if device.index is not None else 0)
        return self._ctx

    @torch.no_grad()
    def step(self, closure=None):
        loss = None
        if closure is not None:
            with torch.enable_grad():
                loss = closure()
        for g in self.param_groups:
            if not g["normpre"]:
                continue
            ps = [p for p in g["params"] if p.grad is not None]
            if not ps:
                continue
            ms = []
            for p in ps:
                st = self.state[p]
                if "momentum" not in st:
                    st["momentum"] = torch.zeros_like(p)
                ms.append(st["momentum"])
            grads = [p.grad if p.grad.is_contiguous() else p.grad.contiguous() for p in ps]
            hp = N.normpre_default_hparams(lr=g["lr"], weight_decay=g["weight_decay"], step=self.t,
                                           **self.hparams)
            N.normpre_step(self._context(ps[0].device), N.VARIANTS[self.variant], ps, grads, ms, hp,
                           stream=torch.cuda.current_stream(ps[0].device))
        if self._adamw is not None:
            self._adamw.step()
        self.t += 1
        return loss

    def zero_grad(self, set_to_none: bool = True):
        super().zero_grad(set_to_none=set_to_none)
        if self._adamw is not None:
            self._adamw.zero_grad(set_to_none=set_to_none)

    def state_dict(self):
        sd = super().state_dict()
        sd["normpre_t"] = self.t
        sd["adamw"] = self._adamw.state_dict() if self._adamw is not None else None
        return sd

    def load_state_dict(self, state_dict):
        state_dict = dict(state_dict)
        self.t = int(state_dict.pop("normpre_t", 0))
        adam = state_dict.pop("adamw", None)
        super().load_state_dict(state_dict)
        if adam is not None and self._adamw is not None:
            self._adamw.load_state_dict(adam)

    def close(self):
        if self._ctx is not None:
            N.normpre_destroy(self._ctx)
            self._ctx = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass
