"""GPU parity of the LARS plan step (lsgd_lars_step_plan, through the C ABI)
against the CPU oracle (oracle_lars_step, one tensor at a time).

Bar: each tensor's trust ratio within one binary32 ulp of the oracle's (both
evaluate the norms in binary64 and round once; the GPU sums in a blocked
order, the oracle sequentially, so a ratio may differ in its last bit in rare
cases) and within one ulp of the exact ratio (exact sums of squares, 60-digit
square roots and division). Where the trust ratios agree bit for bit,
parameters, momentum and replicas are bit-exact; otherwise the contract
tolerance |gpu - ref| <= 1e-6*|ref| + 1e-6*rms(ref) applies, and that
tensor's GPU state is then reset to the oracle's, so that every step starts
both sides from the oracle's trajectory.
"""
import sys

import numpy as np
import pytest
import torch

import fullsize
import oracle
import workloads

pytestmark = pytest.mark.gpu

if torch.cuda.device_count() > 0:
    import paper_1906_05936_amd as lsgd
else:  # collected but skipped on machines without a GPU
    lsgd = None

DEV = torch.device("cuda:0")
TRUST_COEF = 1e-3   # eta of the LARS paper's experiments


def log(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def to_dev(a):
    if a.dtype == np.uint16:
        return torch.from_numpy(a.view(np.int16).copy()).view(torch.bfloat16).to(DEV)
    return torch.from_numpy(np.ascontiguousarray(a)).to(DEV)


def to_host(t):
    t = t.detach()
    if t.dtype == torch.bfloat16:
        return t.view(torch.int16).cpu().numpy().view(np.uint16)
    return t.cpu().numpy()


def rand_host(rng, n, std, dtype):
    x = (rng.standard_normal(n) * std).astype(np.float32)
    return oracle.f32_to_bf16(x) if dtype == "bf16" else x


def close(gpu, ref, what):
    assert gpu.shape == ref.shape, what
    fin = np.isfinite(ref)
    assert np.array_equal(np.isfinite(gpu), fin), what
    rms = float(np.sqrt(np.mean(ref[fin].astype(np.float64) ** 2))) if fin.any() else 0.0
    err = np.abs(gpu[fin].astype(np.float64) - ref[fin])
    assert np.all(err <= 1e-6 * np.abs(ref[fin]) + 1e-6 * rms), "%s: max err %g" % (what, err.max())


def ulps(a, b):
    return abs(int(np.float32(a).view(np.int32)) - int(np.float32(b).view(np.int32)))


def oracle_gbar(grads_h, gow, G):
    """The oracle's binary32 mean gradient of one tensor (mean of means)."""
    return oracle.global_mean(oracle.group_means(grads_h, gow, G))


def check_exact_trust(t_gpu, p_before, gbar, wd, eta, what):
    """The GPU trust ratio within one binary32 ulp of the exact ratio."""
    exact = fullsize.trust_60_digits(p_before, gbar, wd, eta)
    assert fullsize.within_one_ulp(t_gpu, exact), "%s: trust %r, exact %s" % (what, t_gpu, exact)


def reset_to_oracle(params_t, mom_t, ph_t, mh_t):
    """After a one-ulp trust difference: the GPU tensor continues from the
    oracle's state (the oracle's trajectory is never taken from the GPU)."""
    params_t.copy_(to_dev(ph_t))
    mom_t.copy_(to_dev(mh_t))


# Mixed sizes: ragged ends, single elements, several pieces, an empty tensor;
# tensor ZERO_P starts at p = 0 and tensor ZERO_G gets zero gradients (trust 1).
SIZES = [1, 3, 64, 1000, 8191, 8193, 0, 20_000, 5, 4096, 9408, 16_385, 70_001]
ZERO_P, ZERO_G = 4, 9


class Case:
    def __init__(self, G, W, gdt, R, rdt, seed):
        self.rng = np.random.default_rng(seed)
        self.G, self.W, self.N, self.gdt, self.R, self.rdt = G, W, G * W, gdt, R, rdt
        self.gow = workloads.shuffled_groups(G, W, seed)
        self.ph = [(self.rng.standard_normal(s) * 0.05).astype(np.float32) for s in SIZES]
        self.ph[ZERO_P][:] = 0.0
        self.mh = [np.zeros(s, np.float32) for s in SIZES]
        self.params = [to_dev(x) for x in self.ph]
        self.mom = [to_dev(x) for x in self.mh]
        self.grads = [[torch.empty(s, device=DEV, dtype=torch.bfloat16 if gdt == "bf16" else torch.float32)
                       for s in SIZES] for _ in range(self.N)]
        rtd = torch.bfloat16 if rdt == "bf16" else torch.float32
        self.reps = [[torch.empty(s, device=DEV, dtype=rtd) for s in SIZES] for _ in range(R)]
        self.plan = lsgd.Plan(self.params, self.mom, self.grads, self.gow, G, self.reps)

    def new_grads(self):
        self.gh = [[rand_host(self.rng, s, 1e-2 * self.rng.uniform(0.2, 5), self.gdt) for s in SIZES]
                   for _ in range(self.N)]
        for w in range(self.N):
            self.gh[w][ZERO_G][:] = 0
            for t in range(len(SIZES)):
                self.grads[w][t].copy_(to_dev(self.gh[w][t]))

    def check(self, lr, mu, wd, eta, step):
        trust = torch.full((len(SIZES),), -1.0, device=DEV)
        self.plan.lars_step(lr, mu, wd, eta, trust_out=trust)
        torch.cuda.synchronize()
        tg = to_host(trust)
        exact = 0
        for t, s in enumerate(SIZES):
            rr = [np.zeros(s, np.uint16 if self.rdt == "bf16" else np.float32) for _ in range(self.R)]
            g_t = [self.gh[w][t] for w in range(self.N)]
            if s:
                check_exact_trust(tg[t], self.ph[t], oracle_gbar(g_t, self.gow, self.G), wd, eta,
                                  "tensor %d step %d" % (t, step))
            tr = oracle.lars_step(self.ph[t], self.mh[t], g_t, self.gow, self.G, lr, mu, wd, eta, rr,
                                  oracle.BF16 if self.rdt == "bf16" else oracle.F32)
            assert ulps(tg[t], tr) <= 1, "tensor %d step %d: trust %r vs %r" % (t, step, tg[t], tr)
            if t == ZERO_G or s == 0 or (t == ZERO_P and step == 0):   # p = 0 only before the first update
                assert tg[t] == 1.0, (t, tg[t])
            pg, mg = to_host(self.params[t]), to_host(self.mom[t])
            if np.float32(tg[t]) == np.float32(tr):
                exact += 1
                assert np.array_equal(pg, self.ph[t]), "params[%d] step %d differ in bits" % (t, step)
                assert np.array_equal(mg, self.mh[t]), "momentum[%d] step %d differ in bits" % (t, step)
                for r in range(self.R):
                    assert np.array_equal(to_host(self.reps[r][t]), rr[r]), (t, r, step)
            else:
                close(pg, self.ph[t], "params[%d] step %d" % (t, step))
                close(mg, self.mh[t], "momentum[%d] step %d" % (t, step))
                reset_to_oracle(self.params[t], self.mom[t], self.ph[t], self.mh[t])
        log("  step %d: %d of %d trust ratios bit-equal" % (step, exact, len(SIZES)))


@pytest.mark.parametrize("G,W,gdt,R,rdt", [(4, 4, "f32", 16, "f32"), (2, 2, "f32", 0, "f32"),
                                           (8, 8, "bf16", 3, "bf16"), (3, 5, "f32", 1, "bf16"),
                                           (1, 1, "f32", 1, "f32"), (5, 3, "bf16", 0, "f32"),
                                           (32, 4, "f32", 1, "f32"), (1, 64, "bf16", 0, "f32"),
                                           (12, 8, "f32", 1, "f32"), (20, 3, "bf16", 0, "f32"),
                                           (16, 4, "f32", 2, "f32"), (5, 1, "bf16", 1, "f32"),
                                           (4, 3, "f32", 1, "f32"), (2, 5, "bf16", 0, "f32"),
                                           (6, 2, "f32", 1, "f32"), (12, 4, "bf16", 0, "f32"),
                                           (4, 12, "bf16", 1, "f32"), (3, 32, "f32", 0, "f32")])
def test_lars_plan_matches_oracle(G, W, gdt, R, rdt):
    log("lars plan G=%d W=%d %s R=%d %s" % (G, W, gdt, R, rdt))
    c = Case(G, W, gdt, R, rdt, seed=G * 10 + W)
    for step in range(3):
        c.new_grads()
        c.check(0.1, 0.9, 1e-4, TRUST_COEF, step)
    c.plan.close()


@pytest.mark.parametrize("mode", ["fused", "separate"])
@pytest.mark.parametrize("R,rdt", [(5, "f32"), (6, "bf16")])
def test_lars_copy_out_modes(mode, R, rdt):
    """The replicas written inside the update kernel and by the copy-out pass
    (replica groups that do not divide R) both match the oracle."""
    log("lars copy-out %s R=%d %s" % (mode, R, rdt))
    lsgd.set_copy_out_mode(lsgd.COPY_OUT_FUSED if mode == "fused" else lsgd.COPY_OUT_SEPARATE)
    try:
        c = Case(2, 2, "f32", R, rdt, seed=31 + R)
        for step in range(2):
            c.new_grads()
            c.check(0.1, 0.9, 1e-4, TRUST_COEF, step)
        c.plan.close()
    finally:
        lsgd.set_copy_out_mode(lsgd.COPY_OUT_AUTO)


def test_lars_results_independent_of_launch_shape_for_one_plan():
    """One plan (its pieces, hence the order of its norm sums, fixed at
    creation): the LARS step gives the same trust ratios, parameters, momentum
    and replicas whatever the XCD renumbering and the copy-out grid cap at
    step time."""
    c = Case(4, 4, "f32", 5, "f32", seed=57)
    c.new_grads()
    p0 = [x.clone() for x in c.params]
    m0 = [x.clone() for x in c.mom]
    default = lsgd.get_launch_shape()
    outs = []
    try:
        for sh in [(-1, 0, 1), (0, 0, 1), (4, 0, 1), (2, 3, 1)]:
            lsgd.set_launch_shape(*sh)
            for mode in (lsgd.COPY_OUT_FUSED, lsgd.COPY_OUT_SEPARATE):
                lsgd.set_copy_out_mode(mode)
                for t in range(len(SIZES)):
                    c.params[t].copy_(p0[t])
                    c.mom[t].copy_(m0[t])
                trust = torch.empty(len(SIZES), device=DEV)
                c.plan.lars_step(0.1, 0.9, 1e-4, TRUST_COEF, trust_out=trust)
                torch.cuda.synchronize()
                outs.append(((sh, mode), trust.clone(), [x.clone() for x in c.params],
                             [x.clone() for x in c.mom], [x.clone() for x in c.reps[c.R - 1]]))
    finally:
        lsgd.set_launch_shape(*default)
        lsgd.set_copy_out_mode(lsgd.COPY_OUT_AUTO)
    for key, trust, ps, ms, rs in outs[1:]:
        assert torch.equal(trust, outs[0][1]), key
        for t in range(len(SIZES)):
            assert torch.equal(ps[t], outs[0][2][t]) and torch.equal(ms[t], outs[0][3][t]), (key, t)
            assert torch.equal(rs[t], outs[0][4][t]), (key, t)
    c.plan.close()


def test_lars_special_coefficients():
    """eta = 0 (trust 0: the momentum only decays) and wd = 0, on the same plan."""
    c = Case(4, 4, "f32", 2, "f32", seed=77)
    c.new_grads()
    c.check(0.1, 0.9, 1e-4, 0.0, 0)
    c.new_grads()
    c.check(0.2, 0.5, 0.0, 0.02, 1)
    c.plan.close()


def test_lars_full_size_resnet50_tensors():
    """The 161 ResNet-50 tensors (25,557,032 elements), 4 x 4 workers, two
    steps, every element compared."""
    wl = workloads.WORKLOADS["resnet50_tensors"]
    G, W, N, R = wl.groups, wl.workers_per_group, wl.n_workers, 2
    sizes = list(wl.tensor_sizes)
    offs = np.cumsum([0] + sizes)
    gow = workloads.contiguous_groups(G, W)
    flat_p = workloads.init_params(wl, DEV)
    params = workloads.split_tensors(flat_p, sizes)
    ph = [to_host(x) for x in params]
    del flat_p
    mom = [torch.zeros_like(x) for x in params]
    mh = [np.zeros(s, np.float32) for s in sizes]
    grads = [[torch.empty(s, device=DEV) for s in sizes] for _ in range(N)]
    reps = [[torch.empty(s, device=DEV) for s in sizes] for _ in range(R)]
    plan = lsgd.Plan(params, mom, grads, gow, G, reps)
    tmp = torch.empty(wl.n, device=DEV)
    trust = torch.empty(len(sizes), device=DEV)
    for step in range(2):
        gh = []
        for w in range(N):
            workloads.fill_worker_grad(wl, step, w, tmp)
            for t in range(len(sizes)):
                grads[w][t].copy_(tmp[offs[t]:offs[t + 1]])
            gh.append(to_host(tmp))
        plan.lars_step(wl.lr, wl.mu, wl.wd, TRUST_COEF, trust_out=trust)
        torch.cuda.synchronize()
        tg = to_host(trust)
        exact = 0
        for t, s in enumerate(sizes):
            rr = [np.zeros(s, np.float32) for _ in range(R)]
            g_t = [g[offs[t]:offs[t + 1]] for g in gh]
            check_exact_trust(tg[t], ph[t], oracle_gbar(g_t, gow, G), wl.wd, TRUST_COEF,
                              "tensor %d step %d" % (t, step))
            tr = oracle.lars_step(ph[t], mh[t], g_t, gow, G, wl.lr, wl.mu, wl.wd, TRUST_COEF, rr)
            assert ulps(tg[t], tr) <= 1, (t, step, tg[t], tr)
            pg, mg = to_host(params[t]), to_host(mom[t])
            if np.float32(tg[t]) == np.float32(tr):
                exact += 1
                assert np.array_equal(pg, ph[t]) and np.array_equal(mg, mh[t]), (t, step)
                assert np.array_equal(to_host(reps[R - 1][t]), rr[R - 1]), (t, step)
            else:
                close(pg, ph[t], "params[%d]" % t)
                close(mg, mh[t], "momentum[%d]" % t)
                reset_to_oracle(params[t], mom[t], ph[t], mh[t])
        log("  resnet50 step %d: %d of %d trust ratios bit-equal" % (step, exact, len(sizes)))
    plan.close()


def test_lars_above_the_cache_limit():
    """Two tensors of 2e7 elements (parameters and momentum beyond the cached
    form's 288 MB limit: the update's nontemporal form), 2 x 2 workers, four
    binary32 replicas (a copy-out pass), two steps, every element compared."""
    sizes = [20_000_000, 20_000_004]
    G, W, R = 2, 2, 4
    N = G * W
    gow = workloads.contiguous_groups(G, W)
    rng = np.random.default_rng(12)
    ph = [(rng.standard_normal(s) * 0.05).astype(np.float32) for s in sizes]
    mh = [np.zeros(s, np.float32) for s in sizes]
    params = [to_dev(x) for x in ph]
    mom = [torch.zeros(s, device=DEV) for s in sizes]
    grads = [[torch.empty(s, device=DEV) for s in sizes] for _ in range(N)]
    reps = [[torch.empty(s, device=DEV) for s in sizes] for _ in range(R)]
    plan = lsgd.Plan(params, mom, grads, gow, G, reps)
    trust = torch.empty(len(sizes), device=DEV)
    for step in range(2):
        gh = [[(rng.standard_normal(s) * 1e-2).astype(np.float32) for s in sizes] for _ in range(N)]
        for w in range(N):
            for t in range(len(sizes)):
                grads[w][t].copy_(to_dev(gh[w][t]))
        plan.lars_step(0.1, 0.9, 1e-4, TRUST_COEF, trust_out=trust)
        torch.cuda.synchronize()
        tg = to_host(trust)
        for t, s in enumerate(sizes):
            rr = [np.zeros(s, np.float32) for _ in range(R)]
            g_t = [gh[w][t] for w in range(N)]
            check_exact_trust(tg[t], ph[t], oracle_gbar(g_t, gow, G), 1e-4, TRUST_COEF,
                              "tensor %d step %d" % (t, step))
            tr = oracle.lars_step(ph[t], mh[t], g_t, gow, G, 0.1, 0.9, 1e-4, TRUST_COEF, rr)
            assert ulps(tg[t], tr) <= 1, (t, step, tg[t], tr)
            pg, mg = to_host(params[t]), to_host(mom[t])
            if np.float32(tg[t]) == np.float32(tr):
                assert np.array_equal(pg, ph[t]) and np.array_equal(mg, mh[t]), (t, step)
                for r in range(R):
                    assert np.array_equal(to_host(reps[r][t]), rr[r]), (t, r, step)
            else:
                close(pg, ph[t], "params[%d]" % t)
                close(mg, mh[t], "momentum[%d]" % t)
                reset_to_oracle(params[t], mom[t], ph[t], mh[t])
        log("  step %d ok" % step)
    plan.close()


def test_lars_argument_errors():
    """Workspace too small, misaligned, or overlapping a plan buffer: the call
    raises and launches nothing."""
    n = 10_000
    p = torch.zeros(n, device=DEV)
    m = torch.zeros(n, device=DEV)
    g = [[torch.ones(n, device=DEV)] for _ in range(2)]
    plan = lsgd.Plan([p], [m], g, [0, 1], 2)
    need = plan.lars_workspace_size()
    assert need >= n * 4
    ws = torch.empty(need + 512, dtype=torch.uint8, device=DEV)
    for bad, status in [(ws[:need - 1], "LSGD_ERR_SIZE"), (ws[16:16 + need], "LSGD_ERR_ALIGN")]:
        with pytest.raises(lsgd.LsgdError) as e:
            plan.lars_step(0.1, 0.9, 1e-4, TRUST_COEF, workspace=bad)
        assert e.value.name == status
    big = torch.zeros(need // 4 + 1024, device=DEV)
    plan2 = lsgd.Plan([big[:n]], [m], g, [0, 1], 2)
    with pytest.raises(lsgd.LsgdError) as e:
        plan2.lars_step(0.1, 0.9, 1e-4, TRUST_COEF, workspace=big.view(torch.uint8))
    assert e.value.name == "LSGD_ERR_ALIAS"
    torch.cuda.synchronize()
    assert torch.count_nonzero(p).item() == 0 and torch.count_nonzero(big[:n]).item() == 0
    plan.lars_step(0.1, 0.9, 1e-4, TRUST_COEF, workspace=ws)   # a valid call goes through
    torch.cuda.synchronize()
    assert torch.count_nonzero(p).item() == n
    plan.close()
    plan2.close()


def test_lars_graph_follows_the_device_schedule():
    """A HIP graph holding the device-side learning-rate schedule step and a
    LARS plan step that reads the rate from device memory: every replay equals
    an eager LARS step run with the oracle's rate for that iteration, bit for
    bit (three launches per step, no host work, no allocation in the graph)."""
    rng = np.random.default_rng(12)
    sizes = [1000, 4097, 65_536, 3]
    G, W = 2, 2
    gow = workloads.contiguous_groups(G, W)
    p0 = [(rng.standard_normal(s) * 0.05).astype(np.float32) for s in sizes]
    gh = [[rand_host(rng, s, 1e-2, "f32") for s in sizes] for _ in range(G * W)]

    def make():
        params = [to_dev(x) for x in p0]
        mom = [torch.zeros(s, device=DEV) for s in sizes]
        grads = [[to_dev(x) for x in row] for row in gh]
        reps = [[torch.empty(s, device=DEV) for s in sizes]]
        return params, mom, grads, reps, lsgd.Plan(params, mom, grads, gow, G, reps)

    pg, mg, gg, rg, plan_g = make()
    pe, me, ge, re_, plan_e = make()
    ws = torch.empty(plan_g.lars_workspace_size(), dtype=torch.uint8, device=DEV)
    sched = (0.1, 256.0, 1024.0, 3, 5, 0.5)
    s = lsgd.lr_schedule(*sched)
    it = torch.zeros(1, device=DEV, dtype=torch.int64)
    lr_t = torch.zeros(1, device=DEV)
    stream = torch.cuda.Stream()
    stream.wait_stream(torch.cuda.current_stream())
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.stream(stream):
        with torch.cuda.graph(graph, stream=stream):
            lsgd.lr_schedule_step(s, it, lr_t, stream=stream)
            plan_g.lars_step(0.0, 0.9, 1e-4, TRUST_COEF, workspace=ws, stream=stream, lr_device=lr_t)
    torch.cuda.synchronize()
    for k in range(8):
        graph.replay()
        plan_e.lars_step(float(oracle.lr_at(k, *sched)), 0.9, 1e-4, TRUST_COEF)
        torch.cuda.synchronize()
        for t in range(len(sizes)):
            assert torch.equal(pg[t], pe[t]) and torch.equal(mg[t], me[t]), (k, t)
            assert torch.equal(rg[0][t], re_[0][t]), (k, t)
    assert it.item() == 8
    del graph
    plan_g.close()
    plan_e.close()


def test_lars_excluded_tensors_take_the_plain_step():
    """Tensors flagged with lsgd_plan_set_lars_exclude take trust 1: their step
    is the oracle's plain step bit for bit, the others' the LARS step; clearing
    the flags brings every tensor back to LARS."""
    c = Case(4, 4, "f32", 2, "f32", seed=91)
    excl = [s < 100 or t == 7 for t, s in enumerate(SIZES)]   # the small vectors and one large tensor
    c.plan.set_lars_exclude(excl)
    for step in range(2):
        c.new_grads()
        trust = torch.full((len(SIZES),), -1.0, device=DEV)
        c.plan.lars_step(0.1, 0.9, 1e-4, TRUST_COEF, trust_out=trust)
        torch.cuda.synchronize()
        tg = to_host(trust)
        for t, s in enumerate(SIZES):
            rr = [np.zeros(s, np.float32) for _ in range(c.R)]
            g = [c.gh[w][t] for w in range(c.N)]
            if excl[t]:
                oracle.lsgd_step(c.ph[t], c.mh[t], g, c.gow, c.G, 0.1, 0.9, 1e-4, rr)
                assert tg[t] == 1.0, (t, tg[t])
            else:
                tr = oracle.lars_step(c.ph[t], c.mh[t], g, c.gow, c.G, 0.1, 0.9, 1e-4, TRUST_COEF, rr)
                assert np.float32(tg[t]) == np.float32(tr), (t, tg[t], tr)
            assert np.array_equal(to_host(c.params[t]), c.ph[t]), (t, step)
            assert np.array_equal(to_host(c.mom[t]), c.mh[t]), (t, step)
            for r in range(c.R):
                assert np.array_equal(to_host(c.reps[r][t]), rr[r]), (t, r, step)
    c.plan.set_lars_exclude(None)
    c.new_grads()
    c.check(0.1, 0.9, 1e-4, TRUST_COEF, 2)
    c.plan.close()
