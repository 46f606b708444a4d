"""The allocation-free entry point malt_init_state_scratch, through the C ABI.

A scratch plan uses the library's static per-device array as its workspace.
Two scratch plans in a row (the second over smaller shapes, taking the array
over) must step exactly like plans over caller-allocated workspaces on the
same inputs, and both must meet the oracle's bars; the older scratch plan must
then refuse to step.
"""
import numpy as np
import pytest

from gpu_harness import TOL_NS, TOL_STATE, say, to_dev
from oracle import OracleHparams, oracle_init, oracle_step, rel_fro
from paper_2608_05088_amd import libmalt as lm
from paper_2608_05088_amd import workloads as wl

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    lm.lib()


def _run(shapes, variant, seed, scratch, steps=2):
    import torch
    W0 = [wl.weight(seed, i, s) for i, s in enumerate(shapes)]
    grads = [[wl.grad(seed, t, i, s, "row_loguniform") for i, s in enumerate(shapes)] for t in range(1, steps + 1)]
    plan = lm.Plan(shapes, variant, scratch=scratch)
    hp = lm.make_hparams(lr=5e-3)
    Wd = to_dev(W0)
    dW = []
    for Gs in grads:
        before = [w.clone() for w in Wd]
        plan.step(Wd, to_dev(Gs), hp)
        torch.cuda.synchronize()
        dW.append([(a.double() - b.double()).cpu().numpy() for a, b in zip(Wd, before)])
    state = [tuple(x.clone() if x is not None else None for x in plan.state_views(i)) for i in range(len(shapes))]
    W = [w.cpu().numpy() for w in Wd]
    return plan, W0, grads, W, dW, state


# First call: three matrices (a wide and a tall 1024-class pair, a ragged one);
# second call: one smaller matrix.  Both workspaces fit the 64 MiB array.
CASES = [([(1024, 3072), (3072, 1024), (300, 700)], "malter", 71), ([(256, 512)], "malt", 72)]


def test_scratch_plans_match_workspace_plans_and_oracle():
    plans = []
    for shapes, variant, seed in CASES:
        sb, wb = lm.malt_state_size(shapes, variant)
        assert wb <= lm.MALT_SCRATCH_BYTES
        say(f"[no-alloc] {variant} {shapes}: workspace {wb} bytes, scratch plan vs workspace plan")
        ref = _run(shapes, variant, seed, scratch=False)
        got = _run(shapes, variant, seed, scratch=True)
        ref[0].close()
        plans.append(got[0])
        # Same kernels on the same inputs: the parameters and the state agree bitwise.
        for k in range(len(shapes)):
            assert np.array_equal(got[3][k], ref[3][k]), f"{shapes[k]}: W differs"
            for a, b in zip(got[5][k], ref[5][k]):
                if a is not None:
                    assert bool((a == b).all().item())
        # And both meet the oracle's bars.
        ost = oracle_init(shapes, variant)
        ohp = OracleHparams(variant=variant, lr=5e-3)
        W = [w.astype(np.float64) for w in got[1]]
        for t, Gs in enumerate(got[2]):
            W, inter = oracle_step(W, Gs, ost, ohp)
            for k in range(len(shapes)):
                assert rel_fro(got[4][t][k], inter[k].dW) <= TOL_NS
        for k in range(len(shapes)):
            assert rel_fro(got[5][k][0].double().cpu().numpy(), ost.M[k]) <= TOL_STATE
        say(f"[no-alloc] {shapes}: scratch plan bitwise equal to the workspace plan")
    # The second scratch plan took the array over: the first must refuse to step.
    import torch
    shapes = CASES[0][0]
    Wd = [torch.zeros(s, device="cuda") for s in shapes]
    with pytest.raises(lm.MaltError) as ei:
        plans[0].step(Wd, [torch.zeros_like(w) for w in Wd], lm.make_hparams())
    assert ei.value.status == lm.MALT_ERR_STATE_MISMATCH
    for p in plans:
        p.close()


def test_scratch_rejects_workspaces_beyond_the_array():
    import torch
    shapes = [(4096, 4096)]
    sb, wb = lm.malt_state_size(shapes)
    assert wb > lm.MALT_SCRATCH_BYTES
    with pytest.raises(lm.MaltError) as ei:
        lm.Plan(shapes, "malt", scratch=True)
    assert ei.value.status == lm.MALT_ERR_SCRATCH_SIZE
    torch.cuda.synchronize()
