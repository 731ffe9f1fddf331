"""End-to-end GPT-2 Small training steps on synthetic tokens.

Random-initialized GPT-2 Small (12 layers, width 768; no checkpoint, no
dataset: uniform random token ids), forward + backward + optimizer step.  The
48 hidden attention/MLP matrices are stepped by the NormPre library through
``NormPreOptimizer``; embeddings, layer norms and biases by AdamW (App. A.1).
The optimizer step is timed between device synchronizations, as in the
paper's efficiency tables (Sec. 4.2); the model runs in fp32.

Prints one JSON line: fwd+bwd and optimizer milliseconds per step, the
optimizer's share of the step, tokens/s, and the descent alignment of the
last step (App. A.3: mean over the hidden matrices of the cosine between the
gradient and the update direction, weight decay excluded).

    python -m paper_2609_36692_amd.e2e_gpt2 --optimizer normpre-g --batch 4
"""
from __future__ import annotations

import argparse
import json
import time

import torch

HIDDEN_SUFFIXES = ("attn.c_attn.weight", "attn.c_proj.weight", "mlp.c_fc.weight", "mlp.c_proj.weight")


def build(seq):
    from transformers import GPT2Config, GPT2LMHeadModel
    torch.manual_seed(1337)
    cfg = GPT2Config(n_layer=12, n_embd=768, n_head=12, n_positions=seq, vocab_size=50257)
    return GPT2LMHeadModel(cfg)


def make_optimizer(name, model, lr, wd):
    hidden = [p for n, p in model.named_parameters() if n.endswith(HIDDEN_SUFFIXES)]
    hidden_ids = {id(p) for p in hidden}
    others = [p for p in model.parameters() if id(p) not in hidden_ids]
    if name == "adamw":
        return torch.optim.AdamW(model.parameters(), lr=lr, betas=(0.9, 0.95), weight_decay=wd), hidden
    from .optim import NormPreOptimizer
    variant = {"normpre-g": "G", "normpre-l": "L", "muon": "MUON", "normalize-only": "NORM"}[name]
    groups = [{"params": hidden, "normpre": True, "lr": lr, "weight_decay": wd},
              {"params": others, "normpre": False, "lr": lr, "weight_decay": wd}]
    return NormPreOptimizer(groups, lr=lr, variant=variant, weight_decay=wd), hidden


def main(argv=None):
    ap = argparse.ArgumentParser()
    ap.add_argument("--optimizer", default="normpre-g",
                    choices=["normpre-g", "normpre-l", "muon", "normalize-only", "adamw"])
    ap.add_argument("--batch", type=int, default=4)
    ap.add_argument("--seq", type=int, default=1024)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--lr", type=float, default=6e-4)
    ap.add_argument("--weight-decay", type=float, default=0.1)
    a = ap.parse_args(argv)
    if not torch.cuda.is_available():
        raise SystemExit("needs a GPU")
    dev = torch.device("cuda:0")
    model = build(a.seq).to(dev)
    opt, hidden = make_optimizer(a.optimizer, model, a.lr, a.weight_decay)
    gen = torch.Generator(device=dev)
    gen.manual_seed(1337)
    fb_ms, op_ms = [], []
    align = None
    for it in range(a.warmup + a.steps):
        tokens = torch.randint(0, 50257, (a.batch, a.seq), generator=gen, device=dev)
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        loss = model(tokens, labels=tokens).loss
        loss.backward()
        torch.cuda.synchronize()
        t1 = time.perf_counter()
        last = it == a.warmup + a.steps - 1
        if last:
            before = [(p.detach().clone(), p.grad.detach().clone()) for p in hidden]
        opt.step()
        torch.cuda.synchronize()
        t2 = time.perf_counter()
        if last:
            # App. A descent alignment, computed by the library's kernels.
            from . import normpre as N
            actx = N.normpre_init(dev.index or 0)
            try:
                _, align = N.normpre_descent_alignment(actx, [b[1] for b in before], [b[0] for b in before],
                                                       [p.detach() for p in hidden], a.lr, a.weight_decay)
            finally:
                N.normpre_destroy(actx)
        opt.zero_grad(set_to_none=True)
        if it >= a.warmup:
            fb_ms.append(1e3 * (t1 - t0))
            op_ms.append(1e3 * (t2 - t1))
    fb = sum(fb_ms) / len(fb_ms)
    op = sum(op_ms) / len(op_ms)
    out = {"metric": "GPT-2 Small end-to-end step (synthetic tokens, random init, fp32)",
           "optimizer": a.optimizer, "batch": a.batch, "seq_len": a.seq, "steps": a.steps,
           "fwd_bwd_ms": round(fb, 3), "optimizer_ms": round(op, 3), "step_ms": round(fb + op, 3),
           "optimizer_share": round(op / (fb + op), 4),
           "tokens_per_s": round(a.batch * a.seq / ((fb + op) / 1e3), 1),
           "descent_alignment_last_step": None if align is None else round(align, 4),
           "final_loss": round(float(loss.detach()), 4)}
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
