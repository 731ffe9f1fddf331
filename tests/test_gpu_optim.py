"""The torch.optim front end on the GPU: one step over a small model matches
the oracle on the hidden matrices (NormPre-G tolerance 2e-2, fp16 Newton-Schulz)
and AdamW on the rest; the step counter drives the orientation."""
import math

import numpy as np
import pytest

torch = pytest.importorskip("torch")

from oracle import normpre_oracle as O  # noqa: E402
from paper_2609_36692_amd.optim import NormPreOptimizer  # noqa: E402

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("variant", ["G", "L"])
def test_optimizer_step_matches_oracle(variant):
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    torch.manual_seed(0)
    dev = torch.device("cuda:0")
    m = torch.nn.Sequential(torch.nn.Linear(96, 192), torch.nn.GELU(), torch.nn.Linear(192, 64)).to(dev)
    ref_bias = torch.nn.Sequential(torch.nn.Linear(96, 192), torch.nn.GELU(), torch.nn.Linear(192, 64)).to(dev)
    ref_bias.load_state_dict(m.state_dict())
    lr, wd = 0.5, 0.0
    opt = NormPreOptimizer(m.parameters(), lr=lr, variant=variant, weight_decay=wd, adamw_lr=1e-3, rank=16)
    ref_adam = torch.optim.AdamW([ref_bias[0].bias, ref_bias[2].bias], lr=1e-3, betas=(0.9, 0.95), weight_decay=wd)
    for t in range(2):
        with torch.no_grad():   # same weights, so the bias gradients agree
            ref_bias[0].weight.copy_(m[0].weight)
            ref_bias[2].weight.copy_(m[2].weight)
        x = torch.randn(32, 96, device=dev)
        for mod in (m, ref_bias):
            mod(x).square().mean().backward()
        mats = [m[0].weight, m[2].weight]
        before = [(p.detach().cpu().double().numpy(), p.grad.detach().cpu().double().numpy(),
                   opt.state[p]["momentum"].cpu().double().numpy() if "momentum" in opt.state[p]
                   else np.zeros(tuple(p.shape))) for p in mats]
        opt.step()
        ref_adam.step()
        torch.cuda.synchronize()
        for i, (p, (w0, g, mp)) in enumerate(zip(mats, before)):
            hp = O.HParams(lr=lr, weight_decay=wd, rank=16)
            ref = O.normpre_step(w0, g, mp, t, hp, variant, matrix_id=i)
            u = (w0 - p.detach().cpu().double().numpy()) / lr
            err = O.relative_fro(u, ref["update"])
            if variant == "G":
                tol = 2e-2
            else:   # fp16 apply: max(1e-2, 8 u16 kappa), as in the parity tests
                lam = ref["ritz_values"][ref["ritz_values"] > 1.0][: ref["n_selected"]]
                kappa = math.sqrt(float(np.sum(lam))) / max(np.linalg.norm(ref["t"]), 1e-300)
                tol = max(1e-2, 8.0 * 2.0 ** -11 * kappa)
            assert err < tol, (t, i, err, tol)
            assert math.isclose(np.linalg.norm(u), 0.2 * math.sqrt(w0.size), rel_tol=2e-3)
        for a, b in ((m[0].bias, ref_bias[0].bias), (m[2].bias, ref_bias[2].bias)):
            torch.testing.assert_close(a, b, rtol=1e-6, atol=1e-7)
        opt.zero_grad()
        ref_adam.zero_grad()
        ref_bias.zero_grad()
    assert opt.t == 2
    opt.close()
