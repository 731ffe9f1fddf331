"""normpre_step_noalloc (the entry point that allocates nothing: its
workspace is the library's static device scratch array) against
normpre_step, through the C ABI.  Two calls in a row, the second with a
smaller input, so the second runs over what the first left in the array;
then a stack larger than the array, which runs in several rounds through it.
Where both entry points plan the step identically (everything fits the array
in one round) the results are bitwise equal; the multi-round case pools
fewer matrices per launch, which may change fp16 rounding, and is held to
the Newton-Schulz parity tolerance against normpre_step and the oracle."""
import sys

import numpy as np
import pytest

torch = pytest.importorskip("torch")

from oracle import normpre_oracle as O  # noqa: E402
from paper_2609_36692_amd import normpre as N  # noqa: E402
from paper_2609_36692_amd import workloads as WL  # noqa: E402
from parity_util import check_update  # noqa: E402

pytestmark = pytest.mark.gpu

TOL_G = 2e-2


def _say(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def _mats(shapes, seed):
    wl = WL.Workload("t", 70 + seed, shapes, "lowrank", 1.0, rank=8)
    return [WL.make_matrix(wl, i, "cpu") for i in range(len(shapes))]


def _run(entry, ctx, variant, mats, t, **over):
    dev = torch.device("cuda:0")
    Ws = [m[0].to(dev).clone() for m in mats]
    Gs = [m[1].to(dev).clone() for m in mats]
    Ms = [m[2].to(dev).clone() for m in mats]
    hp = N.normpre_default_hparams(lr=1.0, weight_decay=0.0, step=t, rank=16, **over)
    torch.cuda.synchronize()
    entry(ctx, N.VARIANTS[variant], Ws, Gs, Ms, hp)
    torch.cuda.synchronize()
    return [(w.cpu(), m.cpu()) for w, m in zip(Ws, Ms)]


@pytest.fixture(scope="module")
def ctx():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    c = N.normpre_init(0)
    yield c
    N.normpre_destroy(c)


@pytest.mark.parametrize("variant", ["G", "L"])
def test_noalloc_matches_step_twice_in_a_row(ctx, variant):
    first = _mats([(512, 1024)] * 4 + [(300, 700), (700, 300)], seed=1)
    second = _mats([(256, 256), (130, 400)], seed=2)
    for t, mats in ((0, first), (1, second)):
        _say(f"noalloc {variant} t={t}: {len(mats)} matrices")
        got = _run(N.normpre_step_noalloc, ctx, variant, mats, t)
        want = _run(N.normpre_step, ctx, variant, mats, t)
        for (wg, mg), (ww, mw) in zip(got, want):
            assert torch.equal(mg, mw)
            assert torch.equal(wg, ww)


def test_noalloc_multi_round_stack(ctx):
    # 12 matrices of 2048 x 4096 need about four times the array: several
    # rounds through it, each a fresh use of the same memory.
    shapes = [(2048, 4096)] * 12
    mats = _mats(shapes, seed=3)
    for t in (0, 1):
        _say(f"noalloc multi-round G t={t}")
        got = _run(N.normpre_step_noalloc, ctx, "G", mats, t)
        want = _run(N.normpre_step, ctx, "G", mats, t)
        for i, ((wg, mg), (ww, mw)) in enumerate(zip(got, want)):
            assert torch.equal(mg, mw)
            w0 = mats[i][0].double().numpy()
            u_got = w0 - wg.double().numpy()
            u_want = w0 - ww.double().numpy()
            check_update(f"noalloc multi-round #{i} t={t} vs normpre_step", u_got, u_want, TOL_G)
            if i in (0, 11):
                ref = O.normpre_step(w0, mats[i][1].numpy(), mats[i][2].numpy(), t,
                                     O.HParams(lr=1.0, weight_decay=0.0), "G", matrix_id=i)
                check_update(f"noalloc multi-round #{i} t={t} vs oracle", u_got, ref["update"], TOL_G)


def test_noalloc_rejects_what_it_cannot_do(ctx):
    dev = torch.device("cuda:0")
    w, g, m = (x.to(dev) for x in _mats([(64, 64)], seed=4)[0])
    hp = N.normpre_default_hparams(flags=N.NORMPRE_FLAG_DEBUG)
    with pytest.raises(N.NormPreError) as ei:
        N.normpre_step_noalloc(ctx, N.NORMPRE_VARIANT_G, [w], [g], [m], hp)
    assert ei.value.code == N.NORMPRE_ERR_INVALID_ARG
    # one 8192 x 16384 matrix needs more than the whole array: refused before
    # any launch, so the shapes alone decide (no buffers of that size needed)
    hp = N.normpre_default_hparams()
    base = torch.zeros(8, device=dev).data_ptr()
    ptrs = [base + (i << 30) for i in range(3)]   # disjoint 512 MiB ranges, never dereferenced
    with pytest.raises(N.NormPreError) as ei:
        N.normpre_step_noalloc(ctx, N.NORMPRE_VARIANT_G, [ptrs[0]], [ptrs[1]], [ptrs[2]], hp,
                               shapes=[(8192, 16384)])
    assert ei.value.code == N.NORMPRE_ERR_UNSUPPORTED
