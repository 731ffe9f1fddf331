"""Descent alignment on the device and two end-to-end GPT-2 Small training
steps.

* normpre_descent_alignment (App. A, training dynamics) against the oracle's
  cosine on synthetic (G, W_before, W_after) made on the host, and on real
  steps of the library against the oracle's update.  The update of a step
  matches the oracle's to the Newton-Schulz tolerance e (2e-2), so the cosine
  with a fixed G moves by at most about e.
* Two optimizer steps of a random-init GPT-2 Small (uniform random token ids,
  batch 1, fp32 model) through the torch.optim front end: sampled hidden
  matrices are compared with the oracle step on the same (W, G, M_prev).
"""
import math
import sys

import numpy as np
import pytest

torch = pytest.importorskip("torch")

from oracle import normpre_oracle as O  # noqa: E402
from paper_2609_36692_amd import normpre as N  # noqa: E402
from paper_2609_36692_amd import workloads as WL  # noqa: E402
from parity_util import check_update, record  # noqa: E402

pytestmark = pytest.mark.gpu

TOL_G = 2e-2
U16 = 2.0 ** -11


def _say(msg):
    print(msg, flush=True)
    sys.stdout.flush()


@pytest.fixture(scope="module")
def ctx():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    c = N.normpre_init(0)
    yield c
    N.normpre_destroy(c)


def test_alignment_kernel_matches_oracle(ctx):
    _say("descent alignment on synthetic inputs")
    rng = np.random.default_rng(8)
    shapes = [(300, 200), (1, 7), (64, 4096), (513, 257)]
    lr, wd = 3e-3, 0.1
    g_h, wb_h, wa_h = [], [], []
    for i, (m, n) in enumerate(shapes):
        g = rng.standard_normal((m, n)).astype(np.float32)
        wb = (0.02 * rng.standard_normal((m, n))).astype(np.float32)
        # an update that is partly aligned with G, partly not
        u = (0.6 * g / np.linalg.norm(g) + rng.standard_normal((m, n)) / math.sqrt(m * n)).astype(np.float64)
        wa = (wb - lr * (u + wd * wb)).astype(np.float32)
        g_h.append(g); wb_h.append(wb); wa_h.append(wa)
    dev = torch.device("cuda:0")
    to = lambda xs: [torch.from_numpy(x).to(dev) for x in xs]  # noqa: E731
    cos, mean = N.normpre_descent_alignment(ctx, to(g_h), to(wb_h), to(wa_h), lr, wd)
    # the oracle on the same fp32 arrays: Phi from the same difference, in fp64
    phi = [(b.astype(np.float64) - a.astype(np.float64)) / np.float64(np.float32(lr))
           - np.float64(np.float32(wd)) * b.astype(np.float64) for b, a in zip(wb_h, wa_h)]
    ref_cos, ref_mean = O.descent_alignment(g_h, phi)
    err = float(np.max(np.abs(cos - np.array(ref_cos))))
    record("descent alignment, synthetic", "max |cos - oracle|", err, 1e-12)
    assert err < 1e-12 and abs(mean - ref_mean) < 1e-12
    assert 0.3 < ref_mean < 0.9


@pytest.mark.parametrize("variant", ["G", "L", "MUON"])
def test_alignment_of_library_steps(ctx, variant):
    _say(f"descent alignment of NormPre-{variant} steps")
    wl = WL.WORKLOADS["gpt2_small"]
    idx = [0, 1, 2, 3]
    dev = torch.device("cuda:0")
    ws, gs, ms = WL.make_stack(wl, dev, indices=idx)
    w0 = [w.clone() for w in ws]
    host = [(w.cpu(), g.cpu(), m.cpu()) for w, g, m in zip(ws, gs, ms)]
    lr, wd = 6e-4, 0.1
    hp = N.normpre_default_hparams(lr=lr, weight_decay=wd, step=1)
    N.normpre_step(ctx, N.VARIANTS[variant], ws, gs, ms, hp)
    cos, mean = N.normpre_descent_alignment(ctx, gs, w0, ws, lr, wd)
    refs = [O.normpre_step(w.numpy(), g.numpy(), m.numpy(), 1, O.HParams(lr=lr, weight_decay=wd), variant,
                           matrix_id=i) for i, (w, g, m) in enumerate(host)]
    ref_cos, ref_mean = O.descent_alignment([h[1].numpy() for h in host], [r["update"] for r in refs])
    err = float(np.max(np.abs(cos - np.array(ref_cos))))
    _say(f"  Align = {mean:.4f} (oracle {ref_mean:.4f}), max cosine error {err:.2e}")
    record(f"descent alignment NormPre-{variant}", "max |cos - oracle|", err, TOL_G)
    assert err < TOL_G and abs(mean - ref_mean) < TOL_G


HIDDEN_SAMPLE = ("transformer.h.0.attn.c_attn.weight", "transformer.h.0.attn.c_proj.weight",
                 "transformer.h.0.mlp.c_fc.weight", "transformer.h.11.mlp.c_proj.weight")


@pytest.mark.parametrize("variant", ["G", "L"])
def test_gpt2_small_two_steps(variant):
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    pytest.importorskip("transformers")
    from paper_2609_36692_amd import e2e_gpt2 as E
    _say(f"GPT-2 Small end to end, NormPre-{variant}, batch 1")
    dev = torch.device("cuda:0")
    seq, lr, wd = 256, 6e-4, 0.1
    model = E.build(seq).to(dev)
    opt, hidden = E.make_optimizer({"G": "normpre-g", "L": "normpre-l"}[variant], model, lr, wd)
    assert len(hidden) == 48
    named = dict(model.named_parameters())
    sample = [named[n] for n in HIDDEN_SAMPLE]
    order = {id(p): i for i, p in enumerate(hidden)}
    gen = torch.Generator(device=dev)
    gen.manual_seed(7)
    for t in range(2):
        tokens = torch.randint(0, 50257, (1, seq), generator=gen, device=dev)
        loss = model(tokens, labels=tokens).loss
        assert torch.isfinite(loss)
        loss.backward()
        before = []
        for p in sample:
            st = opt.state[p]
            mp = st["momentum"].cpu().double().numpy() if "momentum" in st else np.zeros(tuple(p.shape))
            before.append((p.detach().cpu().double().numpy(), p.grad.detach().cpu().double().numpy(), mp))
        opt.step()
        torch.cuda.synchronize()
        assert opt.t == t + 1
        for name, p, (w, g, mp) in zip(HIDDEN_SAMPLE, sample, before):
            ref = O.normpre_step(w, g, mp, t, O.HParams(lr=lr, weight_decay=wd), variant, matrix_id=order[id(p)])
            u = (w - p.detach().cpu().double().numpy()) / lr - wd * w
            if variant == "G":
                tol = TOL_G
            else:
                lam = ref["ritz_values"][ref["ritz_values"] > 1.0][: ref["n_selected"]]
                kappa = math.sqrt(float(np.sum(lam))) / max(np.linalg.norm(ref["t"]), 1e-300)
                tol = max(1e-2, 8.0 * U16 * kappa)
            err = check_update(f"GPT-2 E2E NormPre-{variant} step {t} {name}", u, ref["update"], tol)
            _say(f"  step {t} {name} {tuple(p.shape)}: update err {err:.2e} (tol {tol:.1e})")
        opt.zero_grad(set_to_none=True)
    opt.close()
