"""lsgd_lars_step_plan_noalloc (through the C ABI) against lsgd_lars_step_plan
with a caller-owned workspace: the same trust ratios, parameters, momentum and
replicas, bit for bit, on consecutive calls that share the library's scratch
array (the second on a smaller plan, which finds the first call's contents
there), at the ResNet-50 size, and the size limit."""
import numpy as np
import pytest
import torch

import workloads

pytestmark = pytest.mark.gpu

if torch.cuda.device_count() > 0:
    import paper_1906_05936_amd as lsgd
    from paper_1906_05936_amd._lib import NOALLOC_SCRATCH_BYTES
else:  # collected but skipped on machines without a GPU
    lsgd = None

DEV = torch.device("cuda:0")
TRUST_COEF = 1e-3


def make_plan(sizes, G, W, R, gdt, seed):
    gen = torch.Generator(device=DEV)
    gen.manual_seed(seed)
    gt = torch.bfloat16 if gdt == "bf16" else torch.float32
    params = [torch.randn(s, device=DEV, generator=gen) * 0.05 for s in sizes]
    mom = [torch.randn(s, device=DEV, generator=gen) * 0.01 for s in sizes]
    grads = [[(torch.randn(s, device=DEV, generator=gen) * 1e-2).to(gt) for s in sizes] for _ in range(G * W)]
    reps = [[torch.full((s,), float("nan"), device=DEV) for s in sizes] for _ in range(R)]
    gow = workloads.shuffled_groups(G, W, seed)
    plan = lsgd.Plan(params, mom, grads, gow, G, reps)
    return plan, params, mom, grads, reps


def both_ways(plan, params, mom, reps, lr, mu, wd):
    """One LARS step without a workspace, then the same step (same starting
    state) with one; returns both results."""
    p0 = [x.clone() for x in params]
    m0 = [x.clone() for x in mom]
    out = []
    for noalloc in (True, False):
        for t in range(len(params)):
            params[t].copy_(p0[t])
            mom[t].copy_(m0[t])
        for row in reps:
            for x in row:
                x.fill_(float("nan"))
        trust = torch.full((len(params),), -1.0, device=DEV)
        if noalloc:
            plan.lars_step_noalloc(lr, mu, wd, TRUST_COEF, trust_out=trust)
        else:
            plan.lars_step(lr, mu, wd, TRUST_COEF, trust_out=trust)
        torch.cuda.synchronize()
        out.append((trust.clone(), [x.clone() for x in params], [x.clone() for x in mom],
                    [[x.clone() for x in row] for row in reps]))
    return out


def assert_same(a, b, what):
    assert torch.equal(a[0], b[0]), what + ": trust ratios"
    for t in range(len(a[1])):
        assert torch.equal(a[1][t], b[1][t]), "%s: params[%d]" % (what, t)
        assert torch.equal(a[2][t], b[2][t]), "%s: momentum[%d]" % (what, t)
        for r in range(len(a[3])):
            assert torch.equal(a[3][r][t], b[3][r][t]), "%s: replica %d tensor %d" % (what, r, t)


def test_noalloc_matches_workspace_on_two_calls_in_a_row():
    """A larger plan, then a smaller one: the second call reuses the array the
    first one filled, and both equal the workspace form bit for bit."""
    big = [1_000_003, 64, 2_359_296, 9408, 5, 70_001]
    plan, params, mom, grads, reps = make_plan(big, 4, 4, 3, "f32", seed=1)
    a, b = both_ways(plan, params, mom, reps, 0.1, 0.9, 1e-4)
    assert_same(a, b, "first call")
    plan.close()
    small = [4099, 3, 1000]
    plan, params, mom, grads, reps = make_plan(small, 2, 2, 2, "bf16", seed=2)
    a, b = both_ways(plan, params, mom, reps, 0.2, 0.5, 0.0)
    assert_same(a, b, "second call, smaller plan")
    plan.close()


def test_noalloc_at_resnet50_size():
    wl = workloads.WORKLOADS["resnet50_tensors"]
    plan, params, mom, grads, reps = make_plan(list(wl.tensor_sizes), 4, 4, 2, "f32", seed=3)
    assert plan.lars_workspace_size() <= NOALLOC_SCRATCH_BYTES
    a, b = both_ways(plan, params, mom, reps, wl.lr, wl.mu, wl.wd)
    assert_same(a, b, "resnet50")
    plan.close()


def test_noalloc_rejects_plans_beyond_the_array():
    n = NOALLOC_SCRATCH_BYTES // 4 + 1           # the mean-gradient scratch alone exceeds the array
    p = torch.zeros(n, device=DEV)
    m = torch.zeros(n, device=DEV)
    g = [[torch.ones(n, device=DEV)]]
    plan = lsgd.Plan([p], [m], g, [0], 1)
    assert plan.lars_workspace_size() > NOALLOC_SCRATCH_BYTES
    with pytest.raises(lsgd.LsgdError) as e:
        plan.lars_step_noalloc(0.1, 0.9, 1e-4, TRUST_COEF)
    assert e.value.name == "LSGD_ERR_SIZE"
    torch.cuda.synchronize()
    assert torch.count_nonzero(p).item() == 0      # nothing launched
    plan.close()
