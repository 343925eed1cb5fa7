"""GPU parity: liblsgd (HIP, through its C ABI) against the CPU oracle on the
same seeded inputs.

Bar: parameters, momentum, group means and mean gradient bit-exact (the kernels
and the oracle use the same pairwise order and the same binary32 operations);
the contract tolerance |gpu - ref| <= 1e-6*|ref| + 1e-6*rms(ref) is asserted
as well. Replicas and all indexing are bit-exact.

Sizes: small shapes that span several workgroups and end ragged, shapes large
enough that the kernels renumber their workgroups across the XCDs (every
grid the benchmark's workloads launch is renumbered), and the five workloads at
full size in the launch configuration the benchmark times: every element of
the first steps, and sampled elements over the full step count (every element
is independent of the others).
"""
import os
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


def log(msg):
    print(msg, flush=True)
    sys.stdout.flush()


# ---------------------------------------------------------------- helpers

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


def assert_close(gpu, ref, what):
    """Bitwise equality, and the contract tolerance for binary32 results."""
    assert gpu.shape == ref.shape, what
    if gpu.dtype == np.float32:
        nan = np.isnan(ref)
        assert np.array_equal(np.isnan(gpu), nan), what
        fin = np.isfinite(ref)
        assert np.array_equal(gpu[~fin & ~nan], ref[~fin & ~nan]), what   # infinities
        rms = float(np.sqrt(np.mean(ref[fin].astype(np.float64) ** 2))) if fin.any() else 0.0
        err = np.abs(gpu[fin].astype(np.float64) - ref[fin])
        tol = 1e-6 * np.abs(ref[fin]) + 1e-6 * rms
        assert np.all(err <= tol), "%s: max err %g" % (what, err.max() if err.size else 0)
        mism = np.count_nonzero(gpu[~nan].view(np.uint32) != ref[~nan].view(np.uint32))
        assert mism == 0, "%s: %d of %d elements differ in bits" % (what, mism, ref.size)
    else:
        assert np.array_equal(gpu, ref), what


def groups_for(G, W, layout, seed=0):
    if layout == "contiguous":
        return workloads.contiguous_groups(G, W)
    return workloads.shuffled_groups(G, W, seed)


# ---------------------------------------------------------------- flat fused step

STEP_CASES = [
    # G, W, gdt, n, R, rdt, layout
    (2, 2, "f32", 1_000_003, 4, "f32", "shuffled"),
    (4, 4, "f32", 65_541, 16, "f32", "contiguous"),
    (4, 4, "f32", 3, 1, "f32", "contiguous"),
    (16, 8, "f32", 20_001, 128, "f32", "shuffled"),
    (8, 8, "bf16", 40_007, 64, "bf16", "shuffled"),
    (8, 8, "bf16", 7, 2, "f32", "contiguous"),
    (2, 16, "bf16", 33_333, 3, "bf16", "shuffled"),
    (16, 4, "f32", 12_345, 0, "f32", "shuffled"),
    (1, 16, "f32", 12_289, 0, "f32", "contiguous"),
    (16, 1, "f32", 4_099, 1, "bf16", "contiguous"),
    (1, 1, "f32", 1, 1, "f32", "contiguous"),
    (3, 5, "f32", 10_007, 2, "bf16", "shuffled"),
    (5, 3, "bf16", 9_999, 0, "f32", "shuffled"),
    (7, 1, "f32", 5_000, 1, "f32", "contiguous"),
    (1, 100, "f32", 777, 0, "f32", "contiguous"),
    (128, 1, "bf16", 513, 1, "f32", "shuffled"),
    (6, 7, "bf16", 2_050, 42, "bf16", "shuffled"),
    # XCD-renumbered grids (the chunked, padded launch the workloads take):
    # 4x4 fp32 two-unit tiles cover 2048 elements per workgroup, chunk 64, from
    # 512 workgroups; 8x8 bf16 one-unit tiles 2048, chunk 128, from 1024; 16x8
    # fp32 four-unit tiles 4096, chunk 32, from 256. Ragged ends in each.
    (4, 4, "f32", 2_000_003, 16, "f32", "contiguous"),
    (8, 8, "bf16", 4_000_003, 64, "bf16", "shuffled"),
    (16, 8, "f32", 2_000_003, 128, "f32", "shuffled"),
    (16, 4, "f32", 2_000_003, 8, "f32", "shuffled"),    # 16 groups of 4: two-unit tiles
    # kernels with a wave cap, on the chunked grid: 8 bf16 groups of 3 (cap 2),
    # 2 fp32 groups of 5 and 2 bf16 groups of 2 with cached state (cap 2), one
    # fp32 group of 3 (cap 3)
    (8, 3, "bf16", 4_000_003, 0, "f32", "shuffled"),
    (2, 5, "f32", 2_000_003, 10, "f32", "shuffled"),
    (2, 2, "bf16", 4_000_003, 4, "f32", "contiguous"),
    (1, 3, "f32", 2_000_003, 3, "f32", "contiguous"),
    # compile-time kernels for 32 to 128 groups of few workers, and for groups
    # of 32 to 128 workers (members streamed through an accumulator)
    (32, 4, "f32", 300_007, 8, "f32", "shuffled"),
    (32, 4, "bf16", 70_001, 2, "bf16", "shuffled"),
    (64, 2, "f32", 50_001, 0, "f32", "shuffled"),
    (128, 1, "f32", 9_999, 1, "f32", "shuffled"),
    (4, 32, "f32", 60_003, 3, "f32", "shuffled"),
    (2, 64, "bf16", 40_009, 1, "f32", "shuffled"),
    (1, 128, "f32", 20_011, 2, "bf16", "contiguous"),
    (1, 32, "bf16", 33_335, 1, "bf16", "contiguous"),
    # non-power-of-two group counts with power-of-two groups, and groups of 3,
    # 5 or 6 (the segmented kernel)
    (3, 8, "f32", 100_003, 24, "f32", "shuffled"),
    (6, 4, "bf16", 50_001, 2, "bf16", "shuffled"),
    (12, 8, "f32", 30_007, 1, "f32", "shuffled"),
    (4, 6, "f32", 65_537, 24, "f32", "shuffled"),
    (9, 1, "bf16", 5_555, 0, "f32", "contiguous"),
    (3, 2, "f32", 4_101, 6, "f32", "shuffled"),
    # the segmented kernel's accumulator forms: counts up to 7 take 3 levels
    # (above), up to 15 four, up to 31 five, larger eight (1 x 100 above)
    (1, 9, "f32", 6_007, 3, "f32", "contiguous"),
    (20, 3, "f32", 7_001, 2, "f32", "shuffled"),
    (3, 20, "bf16", 5_003, 1, "bf16", "shuffled"),
    # one worker per group in a non-power-of-two count: run as one group of
    # all N workers in the member order (shuffled: that order is not the
    # workers' ids)
    (12, 1, "f32", 33_333, 3, "f32", "shuffled"),
    (6, 1, "bf16", 20_005, 2, "bf16", "shuffled"),
    (12, 1, "f32", 2_000_003, 12, "f32", "shuffled"),
    # compile-time kernels for groups of 3, 5, 6 or 7 in a power-of-two count
    # (the group mean a true division); 16 and 32 groups of 3 stream their
    # groups in power-of-two batches
    (8, 3, "f32", 100_003, 24, "f32", "shuffled"),
    (16, 3, "f32", 2_000_003, 4, "f32", "shuffled"),
    (32, 3, "f32", 10_007, 2, "f32", "shuffled"),
    (8, 3, "bf16", 50_001, 3, "bf16", "shuffled"),
    (4, 5, "bf16", 40_009, 2, "bf16", "shuffled"),
    (8, 5, "bf16", 9_001, 0, "f32", "shuffled"),
    (2, 7, "f32", 30_011, 14, "f32", "contiguous"),
    (4, 7, "bf16", 7_003, 1, "f32", "contiguous"),
    (16, 6, "f32", 20_003, 1, "f32", "shuffled"),
    # compile-time kernels for 3, 5, 6, 7 or 12 groups (the total a true
    # division; 12 groups stream through the accumulator in batches of a
    # divisor of 12)
    (12, 4, "f32", 2_000_003, 12, "f32", "shuffled"),
    (12, 8, "bf16", 30_001, 2, "bf16", "shuffled"),
    (7, 16, "bf16", 9_999, 1, "f32", "shuffled"),
    (5, 16, "f32", 8_011, 3, "f32", "contiguous"),
    (6, 3, "f32", 60_013, 18, "f32", "shuffled"),
    (12, 1, "bf16", 11_111, 2, "bf16", "shuffled"),
    # groups of 12 workers: compile-time kernels for power-of-two counts and
    # for 3, 5, 6 and 7 groups
    (4, 12, "f32", 100_003, 12, "f32", "shuffled"),
    (8, 12, "bf16", 30_007, 2, "bf16", "shuffled"),
    (3, 12, "f32", 20_011, 3, "f32", "shuffled"),
    (7, 12, "bf16", 9_001, 0, "f32", "shuffled"),
    (1, 12, "f32", 8_191, 1, "f32", "contiguous"),
    # 3 groups of 32: members streamed through the accumulator, G a division
    (3, 32, "f32", 20_011, 2, "f32", "shuffled"),
    (3, 32, "bf16", 9_001, 0, "f32", "contiguous"),
]


@pytest.mark.parametrize("G,W,gdt,n,R,rdt,layout", STEP_CASES)
def test_fused_step_matches_oracle(G, W, gdt, n, R, rdt, layout):
    log("case G=%d W=%d gdt=%s n=%d R=%d rdt=%s %s" % (G, W, gdt, n, R, rdt, layout))
    rng = np.random.default_rng(G * 7919 + W * 31 + n)
    N = G * W
    gow = groups_for(G, W, layout, seed=n)
    p_ref = (rng.standard_normal(n) * 0.05).astype(np.float32)
    m_ref = np.zeros(n, np.float32)
    p, m = to_dev(p_ref), to_dev(m_ref)
    rtd = torch.bfloat16 if rdt == "bf16" else torch.float32
    reps = [torch.full((n,), float("nan"), device=DEV, dtype=rtd) for _ in range(R)]
    for step in range(3):
        host_grads = [rand_host(rng, n, 1e-2, gdt) for _ in range(N)]
        grads = [to_dev(g) for g in host_grads]
        lsgd.step(p, m, grads, gow, G, 0.1, 0.9, 1e-4, reps)
        ref_reps = [np.zeros(n, np.uint16 if rdt == "bf16" else np.float32) for _ in range(R)]
        oracle.lsgd_step(p_ref, m_ref, host_grads, gow, G, 0.1, 0.9, 1e-4, ref_reps,
                         oracle.BF16 if rdt == "bf16" else oracle.F32)
        torch.cuda.synchronize()
        assert_close(to_host(p), p_ref, "params step %d" % step)
        assert_close(to_host(m), m_ref, "momentum step %d" % step)
        for r in range(R):
            assert np.array_equal(to_host(reps[r]), ref_reps[r]), "replica %d step %d" % (r, step)


def test_fused_step_empty_and_errors():
    p = torch.zeros(0, device=DEV)
    lsgd.step(p, torch.zeros(0, device=DEV), [torch.zeros(0, device=DEV)] * 2, [0, 1], 2, 0.1, 0.9, 0.0)
    base = torch.zeros(1025, device=DEV)
    p, m = base[1:], torch.zeros(1024, device=DEV)          # p is 4 bytes off 16-byte alignment
    g = [torch.zeros(1024, device=DEV) for _ in range(2)]
    with pytest.raises(lsgd.LsgdError) as e:
        lsgd.step(p, m, g, [0, 1], 2, 0.1, 0.9, 0.0)
    assert e.value.name == "LSGD_ERR_ALIGN"
    with pytest.raises(lsgd.LsgdError) as e:
        lsgd.step(m, m, g, [0, 1], 2, 0.1, 0.9, 0.0)
    assert e.value.name == "LSGD_ERR_ALIAS"
    with pytest.raises(TypeError):
        lsgd.step(m.clone(), m, [g[0], g[1].bfloat16()], [0, 1], 2, 0.1, 0.9, 0.0)


def test_non_finite_values_propagate_like_the_oracle():
    n = 1024
    g = np.full(n, 1e-3, np.float32)
    g[:6] = [np.nan, np.inf, -np.inf, 3e38, -3e38, 1e-45]
    grads_h = [g, g.copy(), g[::-1].copy(), g.copy()]
    p_ref = np.ones(n, np.float32)
    m_ref = np.zeros(n, np.float32)
    p, m = to_dev(p_ref), to_dev(m_ref)
    lsgd.step(p, m, [to_dev(x) for x in grads_h], [0, 0, 1, 1], 2, 0.1, 0.9, 1e-4)
    oracle.lsgd_step(p_ref, m_ref, grads_h, [0, 0, 1, 1], 2, 0.1, 0.9, 1e-4)
    assert_close(to_host(p), p_ref, "params")
    assert_close(to_host(m), m_ref, "momentum")


def test_fixed_point_on_gpu():
    """Identical worker gradients: the mean is the gradient itself, bitwise."""
    for G, W, gdt in [(4, 4, "f32"), (8, 8, "bf16"), (16, 8, "f32")]:
        rng = np.random.default_rng(G + W)
        gh = rand_host(rng, 50_003, 1e-2, gdt)
        g = to_dev(gh)
        outs = [torch.empty(50_003, device=DEV) for _ in range(G)]
        lsgd.group_mean([g] * (G * W), workloads.contiguous_groups(G, W), G, outs)
        gbar = torch.empty(50_003, device=DEV)
        lsgd.global_mean(outs, gbar)
        want = oracle.bf16_to_f32(gh) if gdt == "bf16" else gh
        assert to_host(gbar).tobytes() == want.tobytes()


# ---------------------------------------------------------------- unfused calls

@pytest.mark.parametrize("G,W,gdt,n,R,rdt", [(4, 4, "f32", 100_003, 2, "f32"),
                                             (8, 8, "bf16", 20_001, 1, "bf16"),
                                             (3, 5, "f32", 7_777, 0, "f32"),
                                             (1, 1, "bf16", 5, 1, "f32"),
                                             (12, 8, "f32", 9_001, 1, "f32"),
                                             (2, 12, "bf16", 3_001, 0, "f32"),
                                             (20, 3, "f32", 4_003, 0, "f32"),
                                             (6, 1, "f32", 4_001, 1, "f32")])
def test_unfused_calls_match_oracle_and_fused(G, W, gdt, n, R, rdt):
    log("unfused G=%d W=%d %s n=%d" % (G, W, gdt, n))
    rng = np.random.default_rng(n)
    N = G * W
    gow = groups_for(G, W, "shuffled", seed=3)
    gh = [rand_host(rng, n, 1e-2, gdt) for _ in range(N)]
    grads = [to_dev(x) for x in gh]
    gm = [torch.empty(n, device=DEV) for _ in range(G)]
    lsgd.group_mean(grads, gow, G, gm)
    gm_ref = oracle.group_means(gh, gow, G)
    for j in range(G):
        assert_close(to_host(gm[j]), gm_ref[j], "group mean %d" % j)
    gbar = torch.empty(n, device=DEV)
    lsgd.global_mean(gm, gbar)
    gbar_ref = oracle.global_mean(gm_ref)
    assert_close(to_host(gbar), gbar_ref, "mean gradient")

    p0 = (rng.standard_normal(n) * 0.05).astype(np.float32)
    m0 = (rng.standard_normal(n) * 0.01).astype(np.float32)
    rtd = torch.bfloat16 if rdt == "bf16" else torch.float32
    p_ref, m_ref = p0.copy(), m0.copy()
    ref_reps = [np.zeros(n, np.uint16 if rdt == "bf16" else np.float32) for _ in range(R)]
    oracle.sgd_step(p_ref, m_ref, gbar_ref, 0.1, 0.9, 1e-4, ref_reps,
                    oracle.BF16 if rdt == "bf16" else oracle.F32)
    try:   # replicas written by the update kernel, then by a copy-out pass of their own
        for mode in (lsgd.COPY_OUT_FUSED, lsgd.COPY_OUT_SEPARATE, lsgd.COPY_OUT_AUTO):
            lsgd.set_copy_out_mode(mode)
            p, m = to_dev(p0), to_dev(m0)
            reps = [torch.empty(n, device=DEV, dtype=rtd) for _ in range(R)]
            lsgd.sgd_step(p, m, gbar, 0.1, 0.9, 1e-4, reps)
            assert_close(to_host(p), p_ref, "params mode %d" % mode)
            assert_close(to_host(m), m_ref, "momentum mode %d" % mode)
            for r in range(R):
                assert np.array_equal(to_host(reps[r]), ref_reps[r]), (mode, r)
    finally:
        lsgd.set_copy_out_mode(lsgd.COPY_OUT_AUTO)

    pf, mf = to_dev(p0), to_dev(m0)
    lsgd.step(pf, mf, grads, gow, G, 0.1, 0.9, 1e-4)
    assert torch.equal(pf, p) and torch.equal(mf, m)   # fused == unfused, bitwise


# ---------------------------------------------------------------- multi-tensor plans

PLAN_SIZES = [1, 3, 64, 1000, 8191, 8192, 8193, 20_000, 5, 64, 4096, 9408, 16_385]


@pytest.mark.parametrize("G,W,gdt,R,rdt", [(4, 4, "f32", 16, "f32"), (2, 2, "f32", 0, "f32"),
                                           (8, 8, "bf16", 3, "bf16"), (3, 5, "f32", 1, "bf16"),
                                           (16, 8, "f32", 2, "f32"), (5, 3, "bf16", 0, "f32"),
                                           (32, 4, "f32", 2, "f32"), (2, 64, "bf16", 1, "bf16"),
                                           (12, 8, "f32", 1, "f32"), (20, 3, "bf16", 0, "f32"),
                                           (16, 4, "f32", 2, "f32"), (6, 1, "f32", 2, "f32"),
                                           (8, 3, "bf16", 1, "f32"), (4, 6, "f32", 2, "f32"),
                                           (2, 12, "f32", 2, "f32"), (3, 32, "bf16", 1, "f32"),
                                           (2, 2, "bf16", 2, "f32"), (32, 3, "bf16", 1, "f32"),
                                           (1, 3, "f32", 3, "f32")])
def test_plan_matches_oracle(G, W, gdt, R, rdt):
    log("plan G=%d W=%d %s R=%d" % (G, W, gdt, R))
    rng = np.random.default_rng(G * 100 + W)
    N = G * W
    gow = groups_for(G, W, "shuffled", seed=G)
    T = len(PLAN_SIZES)
    ph = [(rng.standard_normal(s) * 0.05).astype(np.float32) for s in PLAN_SIZES]
    mh = [np.zeros(s, np.float32) for s in PLAN_SIZES]
    params = [to_dev(x) for x in ph]
    mom = [to_dev(x) for x in mh]
    gh = [[rand_host(rng, s, 1e-2, gdt) for s in PLAN_SIZES] for _ in range(N)]
    grads = [[to_dev(x) for x in row] for row in gh]
    rtd = torch.bfloat16 if rdt == "bf16" else torch.float32
    reps = [[torch.empty(s, device=DEV, dtype=rtd) for s in PLAN_SIZES] for _ in range(R)]
    plan = lsgd.Plan(params, mom, grads, gow, G, reps)
    for step in range(2):
        if step:
            gh = [[rand_host(rng, s, 1e-2, gdt) for s in PLAN_SIZES] for _ in range(N)]
            for w in range(N):
                for t in range(T):
                    grads[w][t].copy_(to_dev(gh[w][t]))
        plan.step(0.1, 0.9, 1e-4)
        torch.cuda.synchronize()
        for t in range(T):
            rr = [np.zeros(PLAN_SIZES[t], np.uint16 if rdt == "bf16" else np.float32) for _ in range(R)]
            oracle.lsgd_step(ph[t], mh[t], [gh[w][t] for w in range(N)], gow, G, 0.1, 0.9, 1e-4, rr,
                             oracle.BF16 if rdt == "bf16" else oracle.F32)
            assert_close(to_host(params[t]), ph[t], "params[%d] step %d" % (t, step))
            assert_close(to_host(mom[t]), mh[t], "momentum[%d] step %d" % (t, step))
            for r in range(R):
                assert np.array_equal(to_host(reps[r][t]), rr[r]), (t, r)
    plan.close()


def test_plan_equals_flat_bitwise():
    """Different launch shapes (plan buckets vs grid-stride flat kernel) give the
    same bits: every element's result depends only on its own inputs."""
    sizes = workloads.resnet50_param_sizes()[:40]
    n = sum(sizes)
    G, W = 4, 4
    gen = torch.Generator(device=DEV)
    gen.manual_seed(5)
    flat_p = torch.randn(n, device=DEV, generator=gen) * 0.05
    flat_g = [torch.randn(n, device=DEV, generator=gen) * 1e-2 for _ in range(G * W)]
    params = workloads.split_tensors(flat_p, sizes)
    mom = [torch.zeros_like(x) for x in params]
    grads = [workloads.split_tensors(g, sizes) for g in flat_g]
    flat_m = torch.zeros(n, device=DEV)
    gow = workloads.contiguous_groups(G, W)
    plan = lsgd.Plan(params, mom, grads, gow, G)
    for _ in range(3):
        plan.step(0.1, 0.9, 1e-4)
        lsgd.step(flat_p, flat_m, flat_g, gow, G, 0.1, 0.9, 1e-4)
    torch.cuda.synchronize()
    assert torch.equal(torch.cat(params), flat_p) and torch.equal(torch.cat(mom), flat_m)
    plan.close()


def test_repeat_runs_are_bit_identical():
    rng = np.random.default_rng(0)
    n = 300_007
    gh = [rand_host(rng, n, 1e-2, "f32") for _ in range(16)]
    p0 = (rng.standard_normal(n) * 0.05).astype(np.float32)
    outs = []
    for _ in range(2):
        p, m = to_dev(p0), torch.zeros(n, device=DEV)
        for _ in range(4):
            lsgd.step(p, m, [to_dev(x) for x in gh], workloads.contiguous_groups(4, 4), 4, 0.1, 0.9, 1e-4)
        outs.append((to_host(p), to_host(m)))
    assert outs[0][0].tobytes() == outs[1][0].tobytes()
    assert outs[0][1].tobytes() == outs[1][1].tobytes()


def test_bf16_gradients_within_2e3_of_fp32_gradients():
    """bf16 gradient storage against fp32 storage of the same fp32 draws: the
    mean gradient agrees within 2e-3 normwise (64 workers, std 1e-3)."""
    n, G, W = 1_000_000, 8, 8
    gen = torch.Generator(device=DEV)
    gen.manual_seed(77)
    g32 = [torch.randn(n, device=DEV, generator=gen) * 1e-3 for _ in range(G * W)]
    g16 = [g.bfloat16() for g in g32]
    gow = workloads.contiguous_groups(G, W)
    res = []
    for gl in (g32, g16):
        gm = [torch.empty(n, device=DEV) for _ in range(G)]
        lsgd.group_mean(gl, gow, G, gm)
        out = torch.empty(n, device=DEV)
        lsgd.global_mean(gm, out)
        res.append(out.double())
    rel = (torch.linalg.vector_norm(res[1] - res[0]) / torch.linalg.vector_norm(res[0])).item()
    log("bf16 vs fp32 gradient storage: normwise relative difference %.3e" % rel)
    assert rel <= 2e-3


# ---------------------------------------------------------------- full-size workloads

@pytest.mark.parametrize("name", workloads.ORDER + ["resnet50_unequal"])
def test_workload_full_size_sampled(name):
    """Each workload at its full size and step count, R = N replicas, in the
    benchmark's launch configuration. Inputs are regenerated every step; the
    oracle follows the sampled elements (all of them for the tiny workload).
    Unequal subgroups take the paper-literal reduction."""
    wl = workloads.WORKLOADS[name]
    N, G, W = wl.n_workers, wl.groups, wl.workers_per_group
    log("workload %s: n=%d G=%d W=%d %s steps=%d" % (name, wl.n, G, W, wl.grad_dtype, wl.steps))
    gow = wl.group_of_worker()
    literal = bool(wl.group_sizes)
    rtd = torch.bfloat16 if wl.replica_dtype == "bf16" else torch.float32
    R = N
    flat_p = workloads.init_params(wl, DEV)
    if wl.tensor_sizes:
        params = workloads.split_tensors(flat_p, wl.tensor_sizes)
        del flat_p
        mom = [torch.zeros_like(x) for x in params]
        grads = [[torch.empty(s, device=DEV, dtype=wl.torch_grad_dtype) for s in wl.tensor_sizes]
                 for _ in range(N)]
        reps = [[torch.empty(s, device=DEV, dtype=rtd) for s in wl.tensor_sizes] for _ in range(R)]
        plan = lsgd.Plan(params, mom, grads, gow, G, reps)
        offs = np.cumsum([0] + list(wl.tensor_sizes))
    else:
        params, mom = [flat_p], [torch.zeros_like(flat_p)]
        grads = [[torch.empty(wl.n, device=DEV, dtype=wl.torch_grad_dtype)] for _ in range(N)]
        reps = [[torch.empty(wl.n, device=DEV, dtype=rtd)] for _ in range(R)]
        plan = None
        offs = np.array([0, wl.n])
    full = wl.n <= 1_000_000
    idx = np.arange(wl.n) if full else workloads.sample_indices(wl.n, 4096, wl.seed)
    if wl.tensor_sizes:   # also each tensor's first and last element
        idx = np.unique(np.concatenate([idx, offs[:-1], offs[1:] - 1]))
    # (tensor, local index) of every sampled element
    tid = np.searchsorted(offs, idx, side="right") - 1
    loc = idx - offs[tid]
    sel = [(t, torch.from_numpy(loc[tid == t]).to(DEV)) for t in np.unique(tid)]

    def gather(tensors):
        return to_host(torch.cat([tensors[t].index_select(0, li) for t, li in sel]))

    p_ref = gather(params)
    m_ref = gather(mom)
    scratch = torch.empty(max(wl.tensor_sizes or (wl.n,)), device=DEV) if wl.grad_dtype == "bf16" else None
    flat_tmp = torch.empty(wl.n, device=DEV, dtype=wl.torch_grad_dtype) if wl.tensor_sizes else None
    for step in range(wl.steps):
        for w in range(N):
            if wl.tensor_sizes:
                workloads.fill_worker_grad(wl, step, w, flat_tmp)
                for t, s in enumerate(wl.tensor_sizes):
                    grads[w][t].copy_(flat_tmp[offs[t]:offs[t + 1]])
            else:
                workloads.fill_worker_grad(wl, step, w, grads[w][0], scratch)
        g_ref = [gather(grads[w]) for w in range(N)]
        if plan is not None:
            plan.step(wl.lr, wl.mu, wl.wd)
        else:
            lsgd.step(params[0], mom[0], [g[0] for g in grads], gow, G, wl.lr, wl.mu, wl.wd,
                      [r[0] for r in reps], reduction="literal" if literal else "mean_of_means")
        rr = [np.zeros(idx.size, np.uint16 if rtd == torch.bfloat16 else np.float32) for _ in range(R)]
        ref_step = oracle.lsgd_step_literal if literal else oracle.lsgd_step
        ref_step(p_ref, m_ref, g_ref, gow, G, wl.lr, wl.mu, wl.wd, rr,
                 oracle.BF16 if rtd == torch.bfloat16 else oracle.F32)
        torch.cuda.synchronize()
        assert_close(gather(params), p_ref, "%s params step %d" % (name, step))
        assert_close(gather(mom), m_ref, "%s momentum step %d" % (name, step))
        for r in range(R):   # every replica: the copy-out pass writes each from its own workgroups
            assert np.array_equal(gather(reps[r]), rr[r]), "%s replica %d step %d" % (name, r, step)
        if step % 10 == 0 or step == wl.steps - 1:
            log("  %s step %d ok (%d sampled elements)" % (name, step, idx.size))
    if plan is not None:
        plan.close()
    del params, mom, grads, reps
    torch.cuda.empty_cache()


# Steps compared element by element at full size (every element of p, m and
# of replicas 0 and R-1; all R replicas against replica 0 on the device).
FULL_COMPARE_STEPS = {"tiny": 10, "resnet50_flat": 3, "resnet50_tensors": 3, "wide": 1, "large": 1,
                      "resnet50_unequal": 3}


@pytest.mark.parametrize("name", workloads.ORDER + ["resnet50_unequal"])
def test_workload_full_size_every_element(name):
    """Each workload at its full size, R = N replicas, in the benchmark's launch
    configuration, against the oracle on every element: the oracle runs block
    by block over the host threads (elements are independent, so the blocks
    give the bits of one call over the whole vector). Inputs are regenerated
    every step. Unequal subgroups take the paper-literal reduction."""
    wl = workloads.WORKLOADS[name]
    steps = FULL_COMPARE_STEPS[name]
    N, G = wl.n_workers, wl.groups
    T = fullsize.host_threads()
    log("workload %s every element: n=%d N=%d %s, %d step(s), %d host threads"
        % (name, wl.n, N, wl.grad_dtype, steps, T))
    gow = wl.group_of_worker()
    literal = bool(wl.group_sizes)
    bf16_rep = wl.replica_dtype == "bf16"
    rtd = torch.bfloat16 if bf16_rep else torch.float32
    R = N
    flat_p = workloads.init_params(wl, DEV)
    if wl.tensor_sizes:
        params = workloads.split_tensors(flat_p, wl.tensor_sizes)
        del flat_p
        mom = [torch.zeros_like(x) for x in params]
        grads = [[torch.empty(s, device=DEV, dtype=wl.torch_grad_dtype) for s in wl.tensor_sizes]
                 for _ in range(N)]
        reps = [[torch.empty(s, device=DEV, dtype=rtd) for s in wl.tensor_sizes] for _ in range(R)]
        plan = lsgd.Plan(params, mom, grads, gow, G, reps)
        offs = np.cumsum([0] + list(wl.tensor_sizes))
        flat_tmp = torch.empty(wl.n, device=DEV, dtype=wl.torch_grad_dtype)
    else:
        params, mom = [flat_p], [torch.zeros_like(flat_p)]
        grads = [[torch.empty(wl.n, device=DEV, dtype=wl.torch_grad_dtype)] for _ in range(N)]
        reps = [[torch.empty(wl.n, device=DEV, dtype=rtd)] for _ in range(R)]
        plan = None
    scratch = torch.empty(max(wl.tensor_sizes or (wl.n,)), device=DEV) if wl.grad_dtype == "bf16" else None
    vp, vm = fullsize.FlatView(params), fullsize.FlatView(mom)
    vg = [fullsize.FlatView(g) for g in grads]
    vr0, vrl = fullsize.FlatView(reps[0]), fullsize.FlatView(reps[R - 1])
    p_ref = vp.range(0, wl.n).copy()
    m_ref = np.zeros(wl.n, np.float32)
    # element blocks of at most about 2 GB of host copies
    per_elem = N * wl.grad_bytes + 16 + 2 * (2 if bf16_rep else 4)
    block = int(min(wl.n, max(1 << 20, (2 << 30) // per_elem)))
    ref_step = oracle.lsgd_step_literal if literal else oracle.lsgd_step
    rdt = oracle.BF16 if bf16_rep else oracle.F32
    for step in range(steps):
        for w in range(N):
            if wl.tensor_sizes:
                workloads.fill_worker_grad(wl, step, w, flat_tmp)
                for t in range(len(wl.tensor_sizes)):
                    grads[w][t].copy_(flat_tmp[offs[t]:offs[t + 1]])
            else:
                workloads.fill_worker_grad(wl, step, w, grads[w][0], scratch)
        if plan is not None:
            plan.step(wl.lr, wl.mu, wl.wd)
        else:
            lsgd.step(params[0], mom[0], [g[0] for g in grads], gow, G, wl.lr, wl.mu, wl.wd,
                      [r[0] for r in reps], reduction="literal" if literal else "mean_of_means")
        torch.cuda.synchronize()
        for r in range(1, R):          # every replica equals replica 0, bit for bit
            for t in range(len(reps[0])):
                assert torch.equal(reps[r][t], reps[0][t]), "%s replica %d tensor %d step %d" % (name, r, t, step)
        for lo in range(0, wl.n, block):
            hi = min(wl.n, lo + block)
            g_h = [v.range(lo, hi) for v in vg]
            rr = np.zeros(hi - lo, np.uint16 if bf16_rep else np.float32)
            pb, mb = p_ref[lo:hi], m_ref[lo:hi]

            def run(a, b):
                ref_step(pb[a:b], mb[a:b], [x[a:b] for x in g_h], gow, G, wl.lr, wl.mu, wl.wd, [rr[a:b]], rdt)
            fullsize.run_blocks(run, hi - lo, T)
            where = "%s step %d elements [%d, %d)" % (name, step, lo, hi)
            assert_close(vp.range(lo, hi), pb, "params " + where)
            assert_close(vm.range(lo, hi), mb, "momentum " + where)
            assert np.array_equal(vr0.range(lo, hi), rr), "replica 0 " + where
            assert np.array_equal(vrl.range(lo, hi), rr), "replica %d %s" % (R - 1, where)
            del g_h
        log("  %s step %d: all %d elements equal the oracle" % (name, step, wl.n))
    if plan is not None:
        plan.close()
    del params, mom, grads, reps
    torch.cuda.empty_cache()


def test_long_vectors_in_ranges_match_oracle():
    """Vectors above 2^26 elements whose copy-out runs as a pass of its own, or
    which have no replicas, are processed range by range (the step kernel, then
    its copy passes, over ranges of about 2^24 elements): lsgd_step with the
    literal reduction and the gradient broadcast, lsgd_step without replicas,
    and lsgd_sgd_step with and without replicas, against the oracle on every
    element, on a length that leaves seven ranges and a ragged end."""
    n = (1 << 26) + (1 << 25) + 12_345
    G, W, R = 2, 2, 2
    T = fullsize.host_threads()
    log("ranges: n=%d G=%d W=%d R=%d" % (n, G, W, R))
    gen = torch.Generator(device=DEV)
    gen.manual_seed(77)
    grads = [torch.randn(n, device=DEV, generator=gen) * 1e-2 for _ in range(G * W)]
    p = torch.randn(n, device=DEV, generator=gen) * 0.05
    m = torch.randn(n, device=DEV, generator=gen) * 0.01
    gh = [to_host(g).copy() for g in grads]
    p0, m0 = to_host(p).copy(), to_host(m).copy()
    gow = workloads.contiguous_groups(G, W)
    reps = [torch.empty(n, device=DEV) for _ in range(R)]
    lsgd.set_copy_out_mode(lsgd.COPY_OUT_SEPARATE)
    try:
        lsgd.step(p, m, grads, gow, G, 0.1, 0.9, 1e-4, reps, reduction="literal", broadcast_grad=True)
        torch.cuda.synchronize()
        p_ref, m_ref, rr = p0.copy(), m0.copy(), np.zeros(n, np.float32)
        fullsize.run_blocks(lambda a, b: oracle.lsgd_step_literal(
            p_ref[a:b], m_ref[a:b], [x[a:b] for x in gh], gow, G, 0.1, 0.9, 1e-4, [rr[a:b]],
            broadcast_grad=True), n, T)
        assert_close(to_host(p), p_ref, "params")
        assert_close(to_host(m), m_ref, "momentum")
        for r in range(R):
            assert np.array_equal(to_host(reps[r]), rr), "replica %d" % r
        for w in range(G * W):
            assert np.array_equal(to_host(grads[w]), gh[w]), "broadcast to worker %d" % w
        gbar = grads[0]                       # now holds the mean gradient
        p2, m2 = torch.from_numpy(p0).to(DEV), torch.from_numpy(m0).to(DEV)
        lsgd.sgd_step(p2, m2, gbar, 0.1, 0.9, 1e-4, reps)
        torch.cuda.synchronize()
        p_ref2, m_ref2, rr2 = p0.copy(), m0.copy(), np.zeros(n, np.float32)
        fullsize.run_blocks(lambda a, b: oracle.sgd_step(p_ref2[a:b], m_ref2[a:b], gh[0][a:b], 0.1, 0.9, 1e-4,
                                                         [rr2[a:b]]), n, T)
        assert_close(to_host(p2), p_ref2, "sgd params")
        assert_close(to_host(m2), m_ref2, "sgd momentum")
        for r in range(R):
            assert np.array_equal(to_host(reps[r]), rr2), "sgd replica %d" % r
        # no replicas: the step kernel alone, range by range (automatic mode)
        lsgd.set_copy_out_mode(lsgd.COPY_OUT_AUTO)
        p3, m3 = torch.from_numpy(p0).to(DEV), torch.from_numpy(m0).to(DEV)
        lsgd.step(p3, m3, grads, gow, G, 0.1, 0.9, 1e-4, [])
        lsgd.sgd_step(p2, m2, gbar, 0.1, 0.9, 1e-4, [])
        torch.cuda.synchronize()
        p_ref3, m_ref3 = p0.copy(), m0.copy()        # gh: the broadcast gradients, as on the device
        fullsize.run_blocks(lambda a, b: oracle.lsgd_step(p_ref3[a:b], m_ref3[a:b], [x[a:b] for x in gh], gow, G,
                                                          0.1, 0.9, 1e-4, []), n, T)
        assert_close(to_host(p3), p_ref3, "params (no replicas)")
        assert_close(to_host(m3), m_ref3, "momentum (no replicas)")
        fullsize.run_blocks(lambda a, b: oracle.sgd_step(p_ref2[a:b], m_ref2[a:b], gh[0][a:b], 0.1, 0.9, 1e-4, []),
                            n, T)
        assert_close(to_host(p2), p_ref2, "sgd params (no replicas)")
        assert_close(to_host(m2), m_ref2, "sgd momentum (no replicas)")
    finally:
        lsgd.set_copy_out_mode(lsgd.COPY_OUT_AUTO)
    del grads, reps, p, m, p2, m2, p3, m3
    torch.cuda.empty_cache()


def test_results_independent_of_launch_shape():
    """Every launch shape (XCD chunking, grid-stride caps, units per lane) gives
    the same bits: each element is computed by one lane from its own inputs."""
    shapes = [(-1, 0, 1), (0, 0, 1), (256, 0, 1), (0, 8, 1), (16, 0, 4), (4, 2, 8), (0, 1, 1),
              (1, 0, 3), (64, 0, 1)]
    default = lsgd.get_launch_shape()
    try:
        for gdt, G, W, n in [("f32", 4, 4, 1_000_003), ("bf16", 8, 8, 400_009), ("f32", 3, 5, 77_777)]:
            log("launch shapes %s G=%d W=%d n=%d" % (gdt, G, W, n))
            rng = np.random.default_rng(n)
            gh = [rand_host(rng, n, 1e-2, gdt) for _ in range(G * W)]
            grads = [to_dev(x) for x in gh]
            p0 = to_dev((rng.standard_normal(n) * 0.05).astype(np.float32))
            gow = groups_for(G, W, "shuffled", seed=1)
            outs = []
            for sh in shapes:
                lsgd.set_launch_shape(*sh)
                for mode in (lsgd.COPY_OUT_FUSED, lsgd.COPY_OUT_SEPARATE):   # the copy-out grid strides too
                    lsgd.set_copy_out_mode(mode)
                    p, m = p0.clone(), torch.zeros(n, device=DEV)
                    reps = [torch.empty(n, device=DEV) for _ in range(3)]
                    for _ in range(2):
                        lsgd.step(p, m, grads, gow, G, 0.1, 0.9, 1e-4, reps)
                    gm = [torch.empty(n, device=DEV) for _ in range(G)]
                    lsgd.group_mean(grads, gow, G, gm)
                    gbar = torch.empty(n, device=DEV)
                    lsgd.global_mean(gm, gbar)
                    outs.append((sh, mode, (p, m, reps[0], reps[2], gbar)))
            for sh, mode, o in outs[1:]:
                for a, b in zip(outs[0][2], o):
                    assert torch.equal(a, b), (sh, mode)
    finally:
        lsgd.set_launch_shape(*default)
        lsgd.set_copy_out_mode(lsgd.COPY_OUT_AUTO)


@pytest.mark.parametrize("nbytes", [16, 48, 4096 + 16, 1 << 20, (1 << 27) + 16 * 333])
def test_stream_copy_is_exact(nbytes):
    src = torch.randint(-2 ** 31, 2 ** 31 - 1, (nbytes // 4,), device=DEV, dtype=torch.int32)
    dst = torch.zeros_like(src)
    lsgd.stream_copy(dst, src)
    torch.cuda.synchronize()
    assert torch.equal(dst, src)


def test_resume_from_host_copy_is_bit_exact():
    """The optimizer state is (params, momentum): copying it to host memory and
    back into fresh buffers mid-run continues bit for bit."""
    rng = np.random.default_rng(21)
    n, G, W = 200_003, 4, 4
    gow = groups_for(G, W, "shuffled", seed=2)
    steps = [[to_dev(rand_host(rng, n, 1e-2, "f32")) for _ in range(G * W)] for _ in range(6)]
    p0 = to_dev((rng.standard_normal(n) * 0.05).astype(np.float32))
    p, m = p0.clone(), torch.zeros(n, device=DEV)
    for g in steps:
        lsgd.step(p, m, g, gow, G, 0.1, 0.9, 1e-4)
    q, v = p0.clone(), torch.zeros(n, device=DEV)
    for g in steps[:3]:
        lsgd.step(q, v, g, gow, G, 0.1, 0.9, 1e-4)
    host_p, host_m = to_host(q).copy(), to_host(v).copy()
    del q, v
    q, v = to_dev(host_p), to_dev(host_m)
    for g in steps[3:]:
        lsgd.step(q, v, g, gow, G, 0.1, 0.9, 1e-4)
    assert torch.equal(p, q) and torch.equal(m, v)


def test_graph_capture_replays_match_eager():
    """lsgd_step and lsgd_step_plan captured in a HIP graph: every replay (with
    eager work and synchronizations in between) gives the eager bits."""
    rng = np.random.default_rng(22)
    n, G, W = 100_003, 2, 4
    gow = groups_for(G, W, "shuffled", seed=3)
    grads = [to_dev(rand_host(rng, n, 1e-2, "f32")) for _ in range(G * W)]
    p0 = to_dev((rng.standard_normal(n) * 0.05).astype(np.float32))
    sizes = [1000, 4096, 3, 70_000]
    pt0 = [to_dev((rng.standard_normal(s) * 0.05).astype(np.float32)) for s in sizes]
    gt = [[to_dev(rand_host(rng, s, 1e-2, "f32")) for s in sizes] for _ in range(G * W)]

    # eager reference: three steps
    pe, me = p0.clone(), torch.zeros(n, device=DEV)
    re = [torch.empty(n, device=DEV) for _ in range(2)]
    pte, mte = [x.clone() for x in pt0], [torch.zeros_like(x) for x in pt0]
    plan_e = lsgd.Plan(pte, mte, gt, gow, G)
    eager = []
    for _ in range(3):
        lsgd.step(pe, me, grads, gow, G, 0.1, 0.9, 1e-4, re)
        plan_e.step(0.1, 0.9, 1e-4)
        torch.cuda.synchronize()
        eager.append((pe.clone(), me.clone(), re[1].clone(), [x.clone() for x in pte]))
    plan_e.close()

    pg, mg = p0.clone(), torch.zeros(n, device=DEV)
    rg = [torch.empty(n, device=DEV) for _ in range(2)]
    ptg, mtg = [x.clone() for x in pt0], [torch.zeros_like(x) for x in pt0]
    plan_g = lsgd.Plan(ptg, mtg, gt, gow, G)
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.stream(s):
        with torch.cuda.graph(graph, stream=s):
            lsgd.step(pg, mg, grads, gow, G, 0.1, 0.9, 1e-4, rg, stream=s)
            plan_g.step(0.1, 0.9, 1e-4, stream=s)
    torch.cuda.synchronize()
    # capture does not execute: state is still the initial one
    assert torch.equal(pg, p0)
    for k in range(3):
        graph.replay()
        torch.cuda.synchronize()
        _ = (torch.ones(1000, device=DEV) * 2).sum().item()   # eager work between replays
        assert torch.equal(pg, eager[k][0]) and torch.equal(mg, eager[k][1]), k
        assert torch.equal(rg[1], eager[k][2]), k
        for a, b in zip(ptg, eager[k][3]):
            assert torch.equal(a, b), k
    del graph
    plan_g.close()


# ---------------------------------------------------------------- step variants (lsgd_step_ex)

LITERAL_CASES = [
    # group_of_worker, G, gdt, n, R, broadcast
    ([0, 1, 1, 1], 2, "f32", 100_003, 2, False),
    ([2, 0, 1, 1, 2, 0, 0, 0, 1], 3, "bf16", 50_001, 1, False),
    ("shuffled4x4", 4, "f32", 65_541, 0, True),
    ([0] * 5 + [1], 2, "f32", 7, 1, True),
    (list(range(7)), 7, "f32", 3_001, 0, False),
    ([3, 0, 6, 1, 5, 2, 4], 7, "f32", 3_001, 1, False),   # one worker per group, shuffled: divides per group
    ([0, 0, 0, 1, 1, 2] * 20, 3, "f32", 4_099, 3, True),
    # equal power-of-two groups: the compile-time kernels, on XCD-renumbered
    # grids, with the replicas and the broadcast in copy passes of their own
    ("shuffled4x4", 4, "f32", 2_000_003, 16, False),
    ("shuffled4x4", 4, "f32", 2_000_003, 16, True),
    ("shuffled4x4", 4, "f32", 33_333, 2, True),
    ("contiguous8x8", 8, "bf16", 100_003, 2, False),
    ("contiguous2x2", 2, "f32", 1_000_001, 1, True),
    # equal groups of 3 in a power-of-two count: the compile-time kernel, each
    # group's sum divided by N = 24
    (workloads.shuffled_groups(8, 3, 5), 8, "f32", 40_003, 3, True),
]


@pytest.mark.parametrize("gow,G,gdt,n,R,bcast", LITERAL_CASES)
def test_literal_reduction_matches_oracle(gow, G, gdt, n, R, bcast):
    if gow == "shuffled4x4":
        gow = workloads.shuffled_groups(4, 4, seed=9)
    elif isinstance(gow, str) and gow.startswith("contiguous"):
        g, w = (int(x) for x in gow[len("contiguous"):].split("x"))
        gow = workloads.contiguous_groups(g, w)
    log("literal G=%d N=%d %s n=%d R=%d bcast=%s" % (G, len(gow), gdt, n, R, bcast))
    rng = np.random.default_rng(n + G)
    gh = [rand_host(rng, n, 1e-2, gdt) for _ in range(len(gow))]
    grads = [to_dev(x) for x in gh]
    p_ref = (rng.standard_normal(n) * 0.05).astype(np.float32)
    m_ref = (rng.standard_normal(n) * 0.01).astype(np.float32)
    p, m = to_dev(p_ref), to_dev(m_ref)
    reps = [torch.empty(n, device=DEV) for _ in range(R)]
    lsgd.step(p, m, grads, gow, G, 0.1, 0.9, 1e-4, reps, reduction="literal", broadcast_grad=bcast)
    rr = [np.zeros(n, np.float32) for _ in range(R)]
    gw = [x.copy() for x in gh]
    oracle.lsgd_step_literal(p_ref, m_ref, gw, gow, G, 0.1, 0.9, 1e-4, rr, broadcast_grad=bcast)
    torch.cuda.synchronize()
    assert_close(to_host(p), p_ref, "params")
    assert_close(to_host(m), m_ref, "momentum")
    for r in range(R):
        assert np.array_equal(to_host(reps[r]), rr[r])
    for w in range(len(gow)):
        assert np.array_equal(to_host(grads[w]), gw[w]), w   # broadcast target (or untouched)


def extreme_grads(rng, n, N, gdt):
    """Gradients at the ends of the binary32 range, one regime per element for
    all workers: small integer multiples of the smallest subnormal (where a
    group's sum / N and the mean of means round differently), values near the
    overflow threshold (where some sums overflow), and ordinary values."""
    out = []
    kind = rng.integers(0, 3, n)
    for _ in range(N):
        sub = (rng.integers(-6, 7, n).astype(np.float64) * 2.0 ** -149).astype(np.float32)
        big = (rng.choice([-1.0, 1.0], n) * rng.uniform(0.6e38, 1.7e38, n)).astype(np.float32)
        mid = (rng.standard_normal(n) * 1e-2).astype(np.float32)
        x = np.where(kind == 0, sub, np.where(kind == 1, big, mid)).astype(np.float32)
        out.append(oracle.f32_to_bf16(x) if gdt == "bf16" else x)
    return out


@pytest.mark.parametrize("gdt", ["f32", "bf16"])
def test_literal_power_of_two_groups_at_range_extremes(gdt):
    """The paper-literal reduction on equal power-of-two groups (the
    compile-time kernels, flat and plan) with subnormal and near-overflow
    gradients: bit-exact against the oracle's literal step. With binary32
    gradients that step differs from the mean of means on some of these
    elements (division by N against division by W then G, where the quotient
    is subnormal); bfloat16 subnormals are multiples of 2^-133, whose
    quotients by 16 are exact in binary32, so there the two agree."""
    G, W, n = 4, 4, 65_541
    N = G * W
    rng = np.random.default_rng(2024 + len(gdt))
    gow = workloads.shuffled_groups(G, W, seed=11)
    gh = extreme_grads(rng, n, N, gdt)
    p0 = (rng.standard_normal(n) * 0.05).astype(np.float32)
    lit = oracle.lsgd_step_literal
    p_lit, m_lit = p0.copy(), np.zeros(n, np.float32)
    rr = [np.zeros(n, np.float32)]
    lit(p_lit, m_lit, [x.copy() for x in gh], gow, G, 0.5, 0.0, 0.0, rr)
    p_mom, m_mom = p0.copy(), np.zeros(n, np.float32)
    oracle.lsgd_step(p_mom, m_mom, gh, gow, G, 0.5, 0.0, 0.0)
    differ = np.count_nonzero(m_lit.view(np.uint32) != m_mom.view(np.uint32))
    log("literal vs mean of means (%s): %d of %d mean gradients differ" % (gdt, differ, n))
    assert differ > 0 or gdt == "bf16"
    grads = [to_dev(x) for x in gh]
    p, m = to_dev(p0), torch.zeros(n, device=DEV)
    reps = [torch.empty(n, device=DEV)]
    lsgd.step(p, m, grads, gow, G, 0.5, 0.0, 0.0, reps, reduction="literal")
    torch.cuda.synchronize()
    assert_close(to_host(p), p_lit, "params")
    assert_close(to_host(m), m_lit, "momentum")
    assert_close(to_host(reps[0]), rr[0], "replica")   # NaN where inf - inf: compared as NaN
    # the same elements as two plan tensors
    cut = 40_000
    pt = [to_dev(p0[:cut]), to_dev(p0[cut:])]
    mt = [torch.zeros(cut, device=DEV), torch.zeros(n - cut, device=DEV)]
    gt = [[to_dev(x[:cut]), to_dev(x[cut:])] for x in gh]
    plan = lsgd.Plan(pt, mt, gt, gow, G)
    plan.step(0.5, 0.0, 0.0, reduction="literal")
    torch.cuda.synchronize()
    assert_close(np.concatenate([to_host(x) for x in pt]), p_lit, "plan params")
    assert_close(np.concatenate([to_host(x) for x in mt]), m_lit, "plan momentum")
    plan.close()


@pytest.mark.parametrize("G,W", [(4, 4), (3, 5), (2, 16)])
def test_gradient_broadcast_with_mean_of_means(G, W):
    """broadcast_grad with the default reduction: every worker buffer receives
    the global mean of the group means; params and momentum as lsgd_step."""
    n = 70_001
    rng = np.random.default_rng(G * W)
    gow = groups_for(G, W, "shuffled", seed=4)
    gh = [rand_host(rng, n, 1e-2, "f32") for _ in range(G * W)]
    grads = [to_dev(x) for x in gh]
    p_ref = (rng.standard_normal(n) * 0.05).astype(np.float32)
    m_ref = np.zeros(n, np.float32)
    p, m = to_dev(p_ref), to_dev(m_ref)
    lsgd.step(p, m, grads, gow, G, 0.1, 0.9, 1e-4, broadcast_grad=True)
    want = oracle.global_mean(oracle.group_means(gh, gow, G))
    oracle.lsgd_step(p_ref, m_ref, gh, gow, G, 0.1, 0.9, 1e-4)
    torch.cuda.synchronize()
    assert_close(to_host(p), p_ref, "params")
    assert_close(to_host(m), m_ref, "momentum")
    for g in grads:
        assert to_host(g).tobytes() == want.tobytes()


def test_learning_rate_from_device_memory():
    n, G, W = 50_003, 2, 4
    rng = np.random.default_rng(5)
    gow = groups_for(G, W, "contiguous")
    gh = [rand_host(rng, n, 1e-2, "f32") for _ in range(G * W)]
    grads = [to_dev(x) for x in gh]
    lr_t = torch.tensor([0.37], device=DEV)
    p_ref = (rng.standard_normal(n) * 0.05).astype(np.float32)
    m_ref = np.zeros(n, np.float32)
    p, m = to_dev(p_ref), to_dev(m_ref)
    lsgd.step(p, m, grads, gow, G, 123.0, 0.9, 1e-4, lr_device=lr_t)   # the lr argument is ignored
    oracle.lsgd_step(p_ref, m_ref, gh, gow, G, np.float32(0.37), 0.9, 1e-4)
    sizes = [1000, 3, 4097]
    ph = [(rng.standard_normal(s) * 0.05).astype(np.float32) for s in sizes]
    gth = [[rand_host(rng, s, 1e-2, "f32") for s in sizes] for _ in range(G * W)]
    pt = [to_dev(x) for x in ph]
    mt = [torch.zeros(s, device=DEV) for s in sizes]
    plan = lsgd.Plan(pt, mt, [[to_dev(x) for x in row] for row in gth], gow, G)
    plan.step(-1.0, 0.9, 1e-4, lr_device=lr_t)
    torch.cuda.synchronize()
    assert_close(to_host(p), p_ref, "params")
    assert_close(to_host(m), m_ref, "momentum")
    for t, s in enumerate(sizes):
        mm = np.zeros(s, np.float32)
        oracle.lsgd_step(ph[t], mm, [gth[w][t] for w in range(G * W)], gow, G, np.float32(0.37), 0.9, 1e-4)
        assert_close(to_host(pt[t]), ph[t], "plan params %d" % t)
    plan.close()


def test_device_schedule_matches_oracle():
    sched = (0.1, 256.0, 16384.0, 390, 2340, 0.1)
    s = lsgd.lr_schedule(*sched)
    it = torch.tensor([2300], device=DEV, dtype=torch.int64)
    lr_out = torch.empty(1, device=DEV)
    hist = torch.empty(100, device=DEV)
    for k in range(100):
        lsgd.lr_schedule_step(s, it, lr_out)
        hist[k:k + 1].copy_(lr_out)
    torch.cuda.synchronize()
    assert it.item() == 2400
    want = np.array([oracle.lr_at(2300 + k, *sched) for k in range(100)], np.float32)
    assert to_host(hist).tobytes() == want.tobytes()


def test_graph_captured_whole_step_follows_the_schedule():
    """A HIP graph holding (schedule step, fused step reading the rate from
    device memory): each replay advances the schedule, bitwise equal to eager
    steps run with the oracle's rates."""
    n, G, W = 40_009, 2, 2
    rng = np.random.default_rng(6)
    gow = groups_for(G, W, "contiguous")
    grads = [to_dev(rand_host(rng, n, 1e-2, "f32")) for _ in range(G * W)]
    p0 = to_dev((rng.standard_normal(n) * 0.05).astype(np.float32))
    sched = (0.1, 256.0, 1024.0, 4, 7, 0.5)
    s = lsgd.lr_schedule(*sched)
    it = torch.zeros(1, device=DEV, dtype=torch.int64)
    lr_t = torch.zeros(1, device=DEV)
    p, m = p0.clone(), torch.zeros(n, device=DEV)
    stream = torch.cuda.Stream()
    stream.wait_stream(torch.cuda.current_stream())
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.stream(stream):
        with torch.cuda.graph(graph, stream=stream):
            lsgd.lr_schedule_step(s, it, lr_t, stream=stream)
            lsgd.step(p, m, grads, gow, G, 0.0, 0.9, 1e-4, lr_device=lr_t, stream=stream)
    torch.cuda.synchronize()
    pe, me = p0.clone(), torch.zeros(n, device=DEV)
    for k in range(12):
        graph.replay()
        lr_k = float(oracle.lr_at(k, *sched))
        lsgd.step(pe, me, grads, gow, G, lr_k, 0.9, 1e-4)
        torch.cuda.synchronize()
        assert abs(lr_t.item() - lr_k) == 0.0, k
        assert torch.equal(p, pe) and torch.equal(m, me), k
    assert it.item() == 12
    del graph


# ---------------------------------------------------------------- copy-out pass

@pytest.mark.parametrize("G,W,gdt,R,rdt,n", [(4, 4, "f32", 33, "f32", 100_003), (2, 2, "bf16", 9, "bf16", 77_777),
                                             (8, 8, "f32", 3, "f32", 65_539), (3, 5, "f32", 20, "bf16", 4_099),
                                             (2, 2, "f32", 5, "f32", 4_500_007), (2, 1, "bf16", 7, "bf16", 4_500_011)])
def test_copy_out_pass_matches_oracle_in_every_mode(G, W, gdt, R, rdt, n):
    """The replicas written in the step kernel, in a copy-out pass of their own
    (with the step kernel writing none, some or all of them first), and by the
    automatic choice: all bitwise equal to the oracle, flat and through a plan
    (ragged sizes; the last two cases span three 8 MB windows of the copy-out
    pass, the last one partial, and replica counts that the
    replicas-per-workgroup grouping does not divide)."""
    log("copy-out modes G=%d W=%d %s R=%d %s n=%d" % (G, W, gdt, R, rdt, n))
    rng = np.random.default_rng(n)
    N = G * W
    gow = groups_for(G, W, "shuffled", seed=3)
    gh = [rand_host(rng, n, 1e-2, gdt) for _ in range(N)]
    grads = [to_dev(x) for x in gh]
    p0 = (rng.standard_normal(n) * 0.05).astype(np.float32)
    ph, mh = p0.copy(), np.zeros(n, np.float32)
    rr = [np.zeros(n, np.uint16 if rdt == "bf16" else np.float32) for _ in range(R)]
    oracle.lsgd_step(ph, mh, gh, gow, G, 0.1, 0.9, 1e-4, rr, oracle.BF16 if rdt == "bf16" else oracle.F32)
    rtd = torch.bfloat16 if rdt == "bf16" else torch.float32
    sizes = [n // 3, 1, n - n // 3 - 1]
    default_shape = lsgd.get_launch_shape()
    try:
        # then the separate pass after a step kernel that writes the first 1, 3
        # and R replicas itself; the last pass: the copy-out pass on a grid of
        # one workgroup per CU, striding
        for mode in (lsgd.COPY_OUT_FUSED, lsgd.COPY_OUT_SEPARATE, lsgd.COPY_OUT_AUTO, "k1", "k3", "kR",
                     "strided"):
            lsgd.set_step_replicas(-1)
            if mode == "strided":
                lsgd.set_launch_shape(default_shape[0], 1, default_shape[2])
                mode = lsgd.COPY_OUT_SEPARATE
            elif isinstance(mode, str):
                lsgd.set_step_replicas(R if mode == "kR" else int(mode[1:]))
                mode = lsgd.COPY_OUT_SEPARATE
            lsgd.set_copy_out_mode(mode)
            p, m = to_dev(p0), torch.zeros(n, device=DEV)
            reps = [torch.full((n,), 7, device=DEV, dtype=rtd) for _ in range(R)]
            lsgd.step(p, m, grads, gow, G, 0.1, 0.9, 1e-4, reps)
            torch.cuda.synchronize()
            assert_close(to_host(p), ph, "params mode %d" % mode)
            for r in range(R):
                assert np.array_equal(to_host(reps[r]), rr[r]), (mode, r)
            # the same step through a three-tensor plan
            offs = np.cumsum([0] + sizes)
            pt = [to_dev(p0[offs[t]:offs[t + 1]].copy()) for t in range(3)]
            mt = [torch.zeros(s, device=DEV) for s in sizes]
            gt = [[g[offs[t]:offs[t + 1]].clone() for t in range(3)] for g in grads]
            rt = [[torch.full((s,), 7, device=DEV, dtype=rtd) for s in sizes] for _ in range(R)]
            plan = lsgd.Plan(pt, mt, gt, gow, G, rt)
            plan.step(0.1, 0.9, 1e-4)
            torch.cuda.synchronize()
            for t in range(3):
                assert_close(to_host(pt[t]), ph[offs[t]:offs[t + 1]], "plan params %d mode %d" % (t, mode))
                for r in range(R):
                    assert np.array_equal(to_host(rt[r][t]), rr[r][offs[t]:offs[t + 1]]), (mode, t, r)
            # the plan's copy-out on its own (lsgd_plan_copy_out) rewrites the same replicas
            for rl in rt:
                for x in rl:
                    x.fill_(7)
            plan.copy_out()
            torch.cuda.synchronize()
            for t in range(3):
                for r in range(R):
                    assert np.array_equal(to_host(rt[r][t]), rr[r][offs[t]:offs[t + 1]]), ("copy_out", mode, t, r)
            plan.close()
    finally:
        lsgd.set_copy_out_mode(lsgd.COPY_OUT_AUTO)
        lsgd.set_step_replicas(-1)
        lsgd.set_launch_shape(*default_shape)


@pytest.mark.parametrize("n,R,rdt,strided", [(1, 1, "f32", False), (7, 3, "bf16", False), (4097, 16, "f32", False),
                                              (4097, 5, "bf16", False), (4_500_007, 3, "f32", False),
                                              (4_500_011, 4, "bf16", True), (2_000_001, 9, "f32", True)])
def test_copy_out_entry_matches_oracle(n, R, rdt, strided):
    """lsgd_copy_out on its own: binary32 replicas equal params bit for bit,
    bfloat16 replicas equal the oracle's nearest-even rounding (values include
    NaN, infinities, signed zeros, subnormals and ties); params untouched.
    Ragged sizes, several 8 MB windows, replica counts the replicas-per-workgroup
    grouping does not divide, and a strided grid (one workgroup per CU)."""
    log("copy_out n=%d R=%d %s strided=%s" % (n, R, rdt, strided))
    rng = np.random.default_rng(n + R)
    ph = (rng.standard_normal(n) * 3).astype(np.float32)
    special = np.array([np.nan, np.inf, -np.inf, 0.0, -0.0, 1e-45, -1e-40, 1.0 + 2 ** -8, 1.0 + 3 * 2 ** -8,
                        3.3895314e38, -1.0 - 2 ** -8], np.float32)
    k = min(n, special.size)
    ph[rng.choice(n, k, replace=False)] = special[:k]
    p = to_dev(ph)
    rtd = torch.bfloat16 if rdt == "bf16" else torch.float32
    reps = [torch.full((n,), 3, device=DEV, dtype=rtd) for _ in range(R)]
    default = lsgd.get_launch_shape()
    try:
        if strided:
            lsgd.set_launch_shape(default[0], 1, default[2])
        lsgd.copy_out(p, reps)
        torch.cuda.synchronize()
    finally:
        lsgd.set_launch_shape(*default)
    want = oracle.f32_to_bf16(ph) if rdt == "bf16" else ph
    assert np.array_equal(to_host(p).view(np.uint32), ph.view(np.uint32))
    for r in range(R):
        got = to_host(reps[r])
        assert np.array_equal(got.view(np.uint16 if rdt == "bf16" else np.uint32),
                              want.view(np.uint16 if rdt == "bf16" else np.uint32)), r


def test_graph_with_separate_copy_out_matches_eager():
    """The step kernel and its copy-out pass captured in one graph: every
    replay equals eager steps, bit for bit."""
    n, G, W, R = 50_021, 4, 4, 40
    rng = np.random.default_rng(8)
    gow = groups_for(G, W, "contiguous")
    grads = [to_dev(rand_host(rng, n, 1e-2, "f32")) for _ in range(G * W)]
    p0 = to_dev((rng.standard_normal(n) * 0.05).astype(np.float32))
    p, m = p0.clone(), torch.zeros(n, device=DEV)
    reps = [torch.empty(n, device=DEV) for _ in range(R)]
    pe, me = p0.clone(), torch.zeros(n, device=DEV)
    reps_e = [torch.empty(n, device=DEV) for _ in range(R)]
    try:
        lsgd.set_copy_out_mode(lsgd.COPY_OUT_SEPARATE)
        stream = torch.cuda.Stream()
        stream.wait_stream(torch.cuda.current_stream())
        graph = torch.cuda.CUDAGraph()
        with torch.cuda.stream(stream):
            with torch.cuda.graph(graph, stream=stream):
                lsgd.step(p, m, grads, gow, G, 0.1, 0.9, 1e-4, reps, stream=stream)
        torch.cuda.synchronize()
        for k in range(5):
            graph.replay()
            lsgd.step(pe, me, grads, gow, G, 0.1, 0.9, 1e-4, reps_e)
            torch.cuda.synchronize()
            assert torch.equal(p, pe) and torch.equal(m, me), k
            for r in (0, R // 2, R - 1):
                assert torch.equal(reps[r], reps_e[r]) and torch.equal(reps[r], p), (k, r)
        del graph
    finally:
        lsgd.set_copy_out_mode(lsgd.COPY_OUT_AUTO)


# ---------------------------------------------------------------- plans: literal reduction, broadcast

@pytest.mark.parametrize("gow,G,gdt,R,bcast", [
    ([0, 0, 1, 1, 1, 2, 2, 2, 2, 2, 3, 3, 3, 3, 3, 3], 4, "f32", 3, False),   # node sizes 2, 3, 5, 6
    ([2, 0, 1, 1, 0, 2, 1], 3, "bf16", 2, False),
    ([0, 0, 1, 1, 1, 2, 2, 2, 2, 2, 3, 3, 3, 3, 3, 3], 4, "f32", 1, True),
    (workloads.contiguous_groups(4, 4), 4, "f32", 16, True),
    (workloads.shuffled_groups(4, 4, 6), 4, "f32", 2, True),
    (workloads.shuffled_groups(2, 4, 7), 2, "bf16", 3, False),
])
def test_plan_literal_reduction_and_broadcast_match_oracle(gow, G, gdt, R, bcast):
    """Plans over any partition take the paper-literal reduction, optionally
    broadcasting the mean gradient into every worker's tensors; every tensor
    bit-exact against the oracle's literal step."""
    log("plan literal gow=%s G=%d %s R=%d bcast=%d" % (gow, G, gdt, R, bcast))
    rng = np.random.default_rng(len(gow) * 7 + R)
    N = len(gow)
    T = len(PLAN_SIZES)
    ph = [(rng.standard_normal(s) * 0.05).astype(np.float32) for s in PLAN_SIZES]
    mh = [np.zeros(s, np.float32) for s in PLAN_SIZES]
    params = [to_dev(x) for x in ph]
    mom = [to_dev(x) for x in mh]
    gh = [[rand_host(rng, s, 1e-2, gdt) for s in PLAN_SIZES] for _ in range(N)]
    grads = [[to_dev(x) for x in row] for row in gh]
    reps = [[torch.empty(s, device=DEV) for s in PLAN_SIZES] for _ in range(R)]
    plan = lsgd.Plan(params, mom, grads, gow, G, reps)
    equal = len(set(gow.count(j) for j in range(G))) == 1
    if not equal:
        with pytest.raises(lsgd.LsgdError) as e:
            plan.step(0.1, 0.9, 1e-4)
        assert e.value.name == "LSGD_ERR_GROUPS"
        with pytest.raises(lsgd.LsgdError) as e:
            plan.lars_step(0.1, 0.9, 1e-4, 1e-3)
        assert e.value.name == "LSGD_ERR_GROUPS"
    for step in range(2):
        if step:
            gh = [[rand_host(rng, s, 1e-2, gdt) for s in PLAN_SIZES] for _ in range(N)]
            for w in range(N):
                for t in range(T):
                    grads[w][t].copy_(to_dev(gh[w][t]))
        plan.step(0.1, 0.9, 1e-4, reduction="literal", broadcast_grad=bcast)
        torch.cuda.synchronize()
        for t in range(T):
            rr = [np.zeros(PLAN_SIZES[t], np.float32) for _ in range(R)]
            gt = [gh[w][t].copy() for w in range(N)]
            oracle.lsgd_step_literal(ph[t], mh[t], gt, gow, G, 0.1, 0.9, 1e-4, rr, oracle.F32,
                                     broadcast_grad=bcast)
            assert_close(to_host(params[t]), ph[t], "params[%d] step %d" % (t, step))
            assert_close(to_host(mom[t]), mh[t], "momentum[%d] step %d" % (t, step))
            for r in range(R):
                assert np.array_equal(to_host(reps[r][t]), rr[r]), (t, r)
            for w in range(N):   # the broadcast's targets, or untouched
                assert np.array_equal(to_host(grads[w][t]), gt[w]), (t, w)
    plan.close()


def test_plan_broadcast_rejects_shared_gradient_tensors():
    """With the broadcast every gradient tensor is written: two workers
    sharing one tensor are rejected (LSGD_ERR_ALIAS), bf16 gradients too
    (LSGD_ERR_DTYPE); the plain step on the same plan still runs."""
    n = 4096
    p, m = torch.zeros(n, device=DEV), torch.zeros(n, device=DEV)
    g = torch.ones(n, device=DEV)
    plan = lsgd.Plan([p], [m], [[g], [g]], [0, 1], 2)
    with pytest.raises(lsgd.LsgdError) as e:
        plan.step(0.1, 0.9, 1e-4, broadcast_grad=True)
    assert e.value.name == "LSGD_ERR_ALIAS"
    plan.step(0.1, 0.9, 1e-4)
    torch.cuda.synchronize()
    assert torch.count_nonzero(p).item() == n
    gb = [torch.ones(n, device=DEV, dtype=torch.bfloat16) for _ in range(2)]
    plan2 = lsgd.Plan([p], [m], [[gb[0]], [gb[1]]], [0, 1], 2)
    with pytest.raises(lsgd.LsgdError) as e:
        plan2.step(0.1, 0.9, 1e-4, broadcast_grad=True)
    assert e.value.name == "LSGD_ERR_DTYPE"
    plan.close()
    plan2.close()


def test_vector_longer_than_2_to_31_elements():
    """n = 2^31 + 13 (8.6 GB per fp32 buffer, five buffers): the 64-bit
    element offsets of the fused step, the copy-out pass and the ragged tail,
    checked on sampled elements (including the last 64) against the oracle."""
    n = (1 << 31) + 13
    G, W, R = 1, 2, 1
    log("n = %d (%.1f GB per buffer)" % (n, n * 4 / 1e9))
    gen = torch.Generator(device=DEV)
    gen.manual_seed(2 ** 31)
    p = torch.randn(n, generator=gen, device=DEV).mul_(0.05)
    m = torch.zeros(n, device=DEV)
    grads = [torch.randn(n, generator=gen, device=DEV).mul_(0.01) for _ in range(G * W)]
    rep = torch.empty(n, device=DEV)
    idx = workloads.sample_indices(n, 4096, seed=31)
    ti = torch.from_numpy(idx).to(DEV)
    ph, mh = to_host(p.index_select(0, ti)), np.zeros(idx.size, np.float32)
    gh = [to_host(g.index_select(0, ti)) for g in grads]
    try:
        for mode in (lsgd.COPY_OUT_FUSED, lsgd.COPY_OUT_SEPARATE):
            lsgd.set_copy_out_mode(mode)
            lsgd.step(p, m, grads, [0, 0], G, 0.1, 0.9, 1e-4, [rep])
            rr = [np.zeros(idx.size, np.float32)]
            oracle.lsgd_step(ph, mh, gh, [0, 0], G, 0.1, 0.9, 1e-4, rr)
            torch.cuda.synchronize()
            assert_close(to_host(p.index_select(0, ti)), ph, "params mode %d" % mode)
            assert_close(to_host(m.index_select(0, ti)), mh, "momentum mode %d" % mode)
            assert np.array_equal(to_host(rep.index_select(0, ti)), rr[0]), mode
        # the update alone on the same vector (its nontemporal form: p and m exceed the caches)
        lsgd.sgd_step(p, m, grads[0], 0.1, 0.9, 1e-4, [rep])
        rr = [np.zeros(idx.size, np.float32)]
        oracle.sgd_step(ph, mh, gh[0], 0.1, 0.9, 1e-4, rr)
        torch.cuda.synchronize()
        assert_close(to_host(p.index_select(0, ti)), ph, "params after sgd_step")
        assert_close(to_host(m.index_select(0, ti)), mh, "momentum after sgd_step")
        assert np.array_equal(to_host(rep.index_select(0, ti)), rr[0])
    finally:
        lsgd.set_copy_out_mode(lsgd.COPY_OUT_AUTO)
    del p, m, grads, rep
    torch.cuda.empty_cache()


@pytest.mark.parametrize("G,W,gdt,R,rdt,plan", [(4, 4, "f32", 16, "f32", False), (3, 5, "f32", 5, "bf16", False),
                                                (2, 2, "bf16", 2, "bf16", False), (4, 4, "f32", 16, "f32", True)])
def test_nontemporal_forms_above_the_cache_limit(G, W, gdt, R, rdt, plan):
    """Vectors whose parameters and momentum exceed the cached form's limit
    (8n > 288 MB) take the nontemporal kernels even with 16 or fewer workers:
    two steps on sampled elements against the oracle, flat (compile-time and
    segmented) and through a three-tensor plan."""
    n = 40_000_003
    log("n = %d above the cache limit: G=%d W=%d %s R=%d %s plan=%s" % (n, G, W, gdt, R, rdt, plan))
    N = G * W
    gow = groups_for(G, W, "shuffled", seed=9)
    gen = torch.Generator(device=DEV)
    gen.manual_seed(40)
    gt = torch.bfloat16 if gdt == "bf16" else torch.float32
    rt = torch.bfloat16 if rdt == "bf16" else torch.float32
    p = torch.randn(n, generator=gen, device=DEV).mul_(0.05)
    m = torch.zeros(n, device=DEV)
    grads = [torch.randn(n, generator=gen, device=DEV).mul_(0.01).to(gt) for _ in range(N)]
    reps = [torch.empty(n, device=DEV, dtype=rt) for _ in range(R)]
    idx = workloads.sample_indices(n, 4096, seed=41)
    sizes = [13_333_336, 8, n - 13_333_344]   # views at 16-byte-aligned offsets
    idx = np.unique(np.concatenate([idx, np.cumsum([0] + sizes)[1:-1], np.cumsum(sizes)[:-1] - 1]))
    ti = torch.from_numpy(idx).to(DEV)
    ph, mh = to_host(p.index_select(0, ti)), np.zeros(idx.size, np.float32)
    gh = [to_host(g.index_select(0, ti)) for g in grads]
    pl = None
    if plan:
        v = lambda t: workloads.view_tensors(t, sizes)
        pl = lsgd.Plan(v(p), v(m), [v(g) for g in grads], gow, G, [v(r) for r in reps])
    for step in range(2):
        if pl is not None:
            pl.step(0.1, 0.9, 1e-4)
        else:
            lsgd.step(p, m, grads, gow, G, 0.1, 0.9, 1e-4, reps)
        rr = [np.zeros(idx.size, np.uint16 if rdt == "bf16" else np.float32) for _ in range(R)]
        oracle.lsgd_step(ph, mh, gh, gow, G, 0.1, 0.9, 1e-4, rr, oracle.BF16 if rdt == "bf16" else oracle.F32)
        torch.cuda.synchronize()
        assert_close(to_host(p.index_select(0, ti)), ph, "params step %d" % step)
        assert_close(to_host(m.index_select(0, ti)), mh, "momentum step %d" % step)
        for r in range(R):
            assert np.array_equal(to_host(reps[r].index_select(0, ti)), rr[r]), (step, r)
    if pl is not None:
        pl.close()
    del p, m, grads, reps
    torch.cuda.empty_cache()


# ---------------------------------------------------------------- tail sizes

TAIL_SIZES = list(range(1, 68)) + [2 ** k + d for k in (7, 10, 11, 12, 13, 17) for d in (-1, 1)]


@pytest.mark.parametrize("gdt,G,W,R,rdt", [("f32", 2, 2, 1, "f32"), ("bf16", 4, 4, 2, "bf16"), ("f32", 3, 5, 1, "f32"),
                                           ("f32", 8, 4, 2, "f32")])
def test_every_tail_size_flat(gdt, G, W, R, rdt):
    """n = 1..67 and 2^k +- 1: every ragged end of the 4- and 8-element units,
    flat step bit-exact against the oracle."""
    rng = np.random.default_rng(67)
    gow = groups_for(G, W, "shuffled", seed=2)
    rtd = torch.bfloat16 if rdt == "bf16" else torch.float32
    for n in TAIL_SIZES:
        gh = [rand_host(rng, n, 1e-2, gdt) for _ in range(G * W)]
        p0 = (rng.standard_normal(n) * 0.05).astype(np.float32)
        ph, mh = p0.copy(), np.zeros(n, np.float32)
        rr = [np.zeros(n, np.uint16 if rdt == "bf16" else np.float32) for _ in range(R)]
        oracle.lsgd_step(ph, mh, gh, gow, G, 0.1, 0.9, 1e-4, rr, oracle.BF16 if rdt == "bf16" else oracle.F32)
        p, m = to_dev(p0), torch.zeros(n, device=DEV)
        reps = [torch.empty(n, device=DEV, dtype=rtd) for _ in range(R)]
        lsgd.step(p, m, [to_dev(g) for g in gh], gow, G, 0.1, 0.9, 1e-4, reps)
        torch.cuda.synchronize()
        assert_close(to_host(p), ph, "params n=%d" % n)
        assert_close(to_host(m), mh, "momentum n=%d" % n)
        for r in range(R):
            assert np.array_equal(to_host(reps[r]), rr[r]), (n, r)


@pytest.mark.parametrize("gdt,G,W", [("f32", 2, 4), ("bf16", 2, 4), ("f32", 8, 4)])
def test_every_tail_size_as_plan_tensors(gdt, G, W):
    """The same sizes as the tensors of one plan (many small tensors share a
    bucket): plain step, then a LARS step, each tensor bit-exact against the
    oracle (8x4 binary32: four-unit tiles and 4096-element pieces)."""
    rng = np.random.default_rng(68)
    N = G * W
    gow = groups_for(G, W, "shuffled", seed=4)
    sizes = TAIL_SIZES
    ph = [(rng.standard_normal(s) * 0.05).astype(np.float32) for s in sizes]
    mh = [np.zeros(s, np.float32) for s in sizes]
    params = [to_dev(x) for x in ph]
    mom = [to_dev(x) for x in mh]
    gh = [[rand_host(rng, s, 1e-2, gdt) for s in sizes] for _ in range(N)]
    grads = [[to_dev(x) for x in row] for row in gh]
    reps = [[torch.empty(s, device=DEV) for s in sizes]]
    plan = lsgd.Plan(params, mom, grads, gow, G, reps)
    plan.step(0.1, 0.9, 1e-4)
    torch.cuda.synchronize()
    for t, s in enumerate(sizes):
        rr = [np.zeros(s, np.float32)]
        oracle.lsgd_step(ph[t], mh[t], [gh[w][t] for w in range(N)], gow, G, 0.1, 0.9, 1e-4, rr)
        assert_close(to_host(params[t]), ph[t], "plan params size %d" % s)
        assert np.array_equal(to_host(reps[0][t]), rr[0]), s
    trust = torch.empty(len(sizes), device=DEV)
    plan.lars_step(0.1, 0.9, 1e-4, 1e-3, trust_out=trust)
    torch.cuda.synchronize()
    tg = to_host(trust)
    for t, s in enumerate(sizes):
        tr = oracle.lars_step(ph[t], mh[t], [gh[w][t] for w in range(N)], gow, G, 0.1, 0.9, 1e-4, 1e-3)
        assert np.float32(tg[t]) == np.float32(tr), (s, tg[t], tr)
        assert_close(to_host(params[t]), ph[t], "LARS params size %d" % s)
        assert_close(to_host(mom[t]), mh[t], "LARS momentum size %d" % s)
    # the plan's copy-out pass on its own over every tail size (shared buckets too)
    for x in reps[0]:
        x.fill_(3)
    plan.copy_out()
    torch.cuda.synchronize()
    for t, s in enumerate(sizes):
        assert torch.equal(reps[0][t], params[t]), ("copy_out", s)
    plan.close()
