"""Host-side checks of the torch.optim front end (no GPU, no library call):
parameter split between NormPre and AdamW, argument checks, state_dict."""
import pytest

torch = pytest.importorskip("torch")

from paper_2609_36692_amd.optim import NormPreOptimizer  # noqa: E402


def _model():
    return torch.nn.Sequential(torch.nn.Linear(8, 16), torch.nn.GELU(), torch.nn.Linear(16, 4))


def test_plain_parameters_split_by_dimension():
    m = _model()
    opt = NormPreOptimizer(m.parameters(), lr=1e-3)
    groups = {g["normpre"]: g["params"] for g in opt.param_groups}
    assert [tuple(p.shape) for p in groups[True]] == [(16, 8), (4, 16)]
    assert [tuple(p.shape) for p in groups[False]] == [(16,), (4,)]
    assert opt._adamw is not None


def test_explicit_groups_and_checks():
    m = _model()
    with pytest.raises(ValueError):
        NormPreOptimizer([{"params": [m[0].bias], "normpre": True}])
    with pytest.raises(ValueError):
        NormPreOptimizer([{"params": [m[0].weight.double()], "normpre": True}])
    opt = NormPreOptimizer([{"params": [m[0].weight, m[2].weight], "normpre": True, "lr": 2e-3}], variant="l")
    assert opt.variant == "L" and opt._adamw is None


def test_state_dict_keeps_step_counter():
    m = _model()
    opt = NormPreOptimizer(m.parameters(), step=7)
    sd = opt.state_dict()
    assert sd["normpre_t"] == 7
    opt2 = NormPreOptimizer(_model().parameters())
    opt2.load_state_dict(sd)
    assert opt2.t == 7
