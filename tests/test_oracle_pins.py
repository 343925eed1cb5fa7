"""Pins of the CPU oracle against what the paper and mathematics fix.

Yu et al., arXiv 1906.05936. The paper prints no worked example, so each part
of the oracle is pinned by something other than itself:
  - the two-level mean equals the flat mean (Sec. 4.2: Algorithms 2 and 3 give
    the same parameters; Sec. 3: equal-size partition), bit for bit for
    power-of-two counts with the pairwise order;
  - identical worker gradients are a fixed point of the aggregation;
  - a two-step example worked by hand in dyadic arithmetic (tests/golden/);
  - the momentum recurrence against its closed form over many steps;
  - special cases that reduce to textbook routines (Alg. 1, Alg. 2, plain copy,
    torch's bfloat16 rounding);
  - brute force in exact rational arithmetic on tiny inputs, within the
    forward error bound of the binary32 operations;
  - the summation order (largest-power-of-two split) written out by hand.
"""
import json
import math
import os
from fractions import Fraction

import numpy as np
import pytest
import torch

import oracle
import workloads

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")
U = 2.0 ** -24  # unit roundoff of binary32


def f32(x):
    return np.float32(x)


def rand_grads(rng, n_workers, n, std=1e-2):
    return [(rng.standard_normal(n) * std).astype(np.float32) for _ in range(n_workers)]


def run_step(p, m, grads, gow, G, lr, mu, wd, replicas=(), rdt=oracle.F32):
    p, m = p.copy(), m.copy()
    oracle.lsgd_step(p, m, grads, gow, G, lr, mu, wd, replicas, rdt)
    return p, m


# ---------------------------------------------------------------- summation order

def test_pairwise_split_written_out():
    """PW splits at the largest power of two below k (the fixed order of the
    oracle). Terms are chosen so that every other association of these sums
    rounds differently in binary32."""
    x = np.array([1e8, 3.0, -1e8, 5.0, 7.0, -3.0, 1e-3, 2.5, 11.0], dtype=np.float32)
    a = [f32(v) for v in x]
    expect = {
        1: a[0],
        2: a[0] + a[1],
        3: (a[0] + a[1]) + a[2],
        4: (a[0] + a[1]) + (a[2] + a[3]),
        5: ((a[0] + a[1]) + (a[2] + a[3])) + a[4],
        6: ((a[0] + a[1]) + (a[2] + a[3])) + (a[4] + a[5]),
        7: ((a[0] + a[1]) + (a[2] + a[3])) + ((a[4] + a[5]) + a[6]),
        8: ((a[0] + a[1]) + (a[2] + a[3])) + ((a[4] + a[5]) + (a[6] + a[7])),
        9: (((a[0] + a[1]) + (a[2] + a[3])) + ((a[4] + a[5]) + (a[6] + a[7]))) + a[8],
    }
    for k, e in expect.items():
        got = np.float32(oracle.pairwise(x[:k]))
        assert got.tobytes() == np.float32(e).tobytes(), k
    # a half split (k // 2) would differ at k = 6: (a0+a1+a2) + (a3+a4+a5)
    half = ((a[0] + a[1]) + a[2]) + ((a[3] + a[4]) + a[5])
    assert np.float32(half) != np.float32(expect[6])


def test_group_sums_follow_ascending_worker_id():
    """Each group is summed in ascending worker id with the pairwise split
    (members of a non-power-of-two group written out), then divided by W;
    groups are combined in ascending group id."""
    f = np.float32
    # row = worker, column = element; in column 0 group 0 holds (1, 1e8, -1e8): ascending
    # order gives (1 + 1e8) - 1e8 = 0, the reverse order (-1e8 + 1e8) + 1 = 1
    vals = np.array([[2.0, 1e8], [1.0, -3.0], [3.0, -1e8], [1e8, 7.0], [4.0, 2.5], [-1e8, 1e-3]],
                    dtype=np.float32)
    grads = [vals[w].copy() for w in range(6)]
    gow = [1, 0, 1, 0, 1, 0]                      # group 0 = {1, 3, 5}, group 1 = {0, 2, 4}
    gm = oracle.group_means(grads, gow, 2)
    for i in range(2):
        g = vals[:, i]
        m0 = ((g[1] + g[3]) + g[5]) / f(3)
        m1 = ((g[0] + g[2]) + g[4]) / f(3)
        assert gm[0][i].tobytes() == f(m0).tobytes() and gm[1][i].tobytes() == f(m1).tobytes(), i
        reversed_m0 = ((g[5] + g[3]) + g[1]) / f(3)
        assert i != 0 or f(reversed_m0) != f(m0)      # the order is observable here
    gbar = oracle.global_mean(gm)
    assert gbar.tobytes() == ((gm[0] + gm[1]) / f(2)).tobytes()


@pytest.mark.parametrize("k", [1, 2, 3, 5, 8, 13, 64, 100, 128, 255])
def test_pairwise_error_bound(k):
    """|PW(x) - sum(x)| <= gamma_h * sum|x|, h = ceil(log2 k): the pairwise bound
    (Higham, Accuracy and Stability of Numerical Algorithms, Sec. 4.2)."""
    rng = np.random.default_rng(k)
    x = (rng.standard_normal(k) * 10.0 ** rng.uniform(-3, 3, size=k)).astype(np.float32)
    exact = sum(Fraction(float(v)) for v in x)
    h = max(0, math.ceil(math.log2(k)))
    gamma = h * U / (1 - h * U)
    bound = gamma * float(sum(abs(Fraction(float(v))) for v in x))
    assert abs(Fraction(float(oracle.pairwise(x))) - exact) <= Fraction(bound)
    # the binary64 build is within binary64 rounding of the exact sum
    assert abs(Fraction(oracle.pairwise(x.astype(np.float64))) - exact) <= Fraction(bound) * Fraction(2 ** -29)


# ---------------------------------------------------------------- membership

def test_members_contiguous_and_shuffled():
    assert oracle.members([0, 0, 1, 1], 2).tolist() == [[0, 1], [2, 3]]
    assert oracle.members([1, 0, 1, 0, 2, 2], 3).tolist() == [[1, 3], [0, 2], [4, 5]]
    gow = workloads.shuffled_groups(16, 8, seed=7)
    rows = oracle.members(gow, 16)
    assert rows.shape == (16, 8)
    for j, row in enumerate(rows):
        assert list(row) == sorted(row) and all(gow[i] == j for i in row)
    assert sorted(rows.ravel().tolist()) == list(range(128))


@pytest.mark.parametrize("gow,G", [([0, 0, 1], 2),          # G does not divide N
                                   ([0, 0, 0, 1], 2),       # unequal groups
                                   ([0, 1, 2, 2], 2),       # id out of range
                                   ([0, -1, 0, 1], 2)])     # negative id
def test_members_rejects_invalid_partitions(gow, G):
    with pytest.raises(oracle.OracleError) as e:
        oracle.members(gow, G)
    assert e.value.status == oracle.ERR_GROUPS


def test_members_rejects_bad_counts():
    with pytest.raises(oracle.OracleError) as e:
        oracle.members([0, 0], 0)
    assert e.value.status == oracle.ERR_SIZE


# ---------------------------------------------------------------- P1 two-level == flat

@pytest.mark.parametrize("G,W", [(2, 2), (4, 4), (16, 8), (8, 8), (1, 16), (16, 1), (2, 8),
                                 (32, 4), (4, 32)])
@pytest.mark.parametrize("gdt", ["f32", "bf16"])
def test_two_level_equals_flat_bitwise(G, W, gdt):
    """Alg. 3 (Reduce + divide, then Allreduce over communicators) reaches the
    same parameters as Alg. 2 (Allreduce over all N, divide by N): with power-of-
    two W and G and the pairwise order the two are bit-identical."""
    rng = np.random.default_rng(G * 1000 + W)
    n = 1500
    grads = rand_grads(rng, G * W, n)
    if gdt == "bf16":
        grads = [oracle.f32_to_bf16(g) for g in grads]
    p = (rng.standard_normal(n) * 0.05).astype(np.float32)
    m = (rng.standard_normal(n) * 0.01).astype(np.float32)
    two = run_step(p, m, grads, workloads.contiguous_groups(G, W), G, 0.1, 0.9, 1e-4)
    flat = run_step(p, m, grads, [0] * (G * W), 1, 0.1, 0.9, 1e-4)
    assert two[0].tobytes() == flat[0].tobytes()
    assert two[1].tobytes() == flat[1].tobytes()


@pytest.mark.parametrize("G,W", [(4, 4), (3, 5), (16, 8)])
def test_membership_relabelling_bitwise(G, W):
    """A shuffled worker->group map equals the contiguous map applied to the
    gradient list reordered by the same membership (ascending ids per group)."""
    rng = np.random.default_rng(5)
    n = 700
    grads = rand_grads(rng, G * W, n)
    gow = workloads.shuffled_groups(G, W, seed=11)
    rows = oracle.members(gow, G)
    relabelled = [grads[i] for i in rows.ravel()]
    p = (rng.standard_normal(n) * 0.05).astype(np.float32)
    m = np.zeros(n, np.float32)
    a = run_step(p, m, grads, gow, G, 0.1, 0.9, 1e-4)
    b = run_step(p, m, relabelled, workloads.contiguous_groups(G, W), G, 0.1, 0.9, 1e-4)
    assert a[0].tobytes() == b[0].tobytes() and a[1].tobytes() == b[1].tobytes()


# ---------------------------------------------------------------- P2 fixed point

@pytest.mark.parametrize("G,W", [(2, 2), (4, 4), (16, 8), (8, 8), (1, 1), (1, 128), (128, 1)])
def test_identical_inputs_are_a_fixed_point(G, W):
    """Every worker holding the same gradient g gives mean g exactly (Alg. 2/3:
    the average of equal terms), here for power-of-two counts, subnormals and
    large values included (no partial sum may overflow: 128 * |g| < 3.4e38)."""
    rng = np.random.default_rng(3)
    g = (rng.standard_normal(2048) * 10.0 ** rng.uniform(-40, 30, size=2048)).astype(np.float32)
    g[:4] = [1e-45, -3e-44, 2e36, -0.0]  # 128 * 2e36 stays below the binary32 maximum
    grads = [g] * (G * W)
    gm = oracle.group_means(grads, workloads.contiguous_groups(G, W), G)
    for j in range(G):
        assert gm[j].tobytes() == g.tobytes()
    assert oracle.global_mean(gm).tobytes() == g.tobytes()


# ---------------------------------------------------------------- P3 hand-worked example

def test_dyadic_two_steps_golden():
    with open(os.path.join(GOLDEN, "dyadic_two_steps.json")) as f:
        gold = json.load(f)
    p = np.array(gold["p0"], np.float32)
    m = np.zeros_like(p)
    for st in gold["steps"]:
        grads = [np.array(g, np.float32) for g in st["grads"]]
        gm = oracle.group_means(grads, gold["group_of_worker"], gold["groups"])
        assert oracle.global_mean(gm).tolist() == st["gbar"]
        reps = [np.zeros_like(p), np.zeros_like(p)]
        oracle.lsgd_step(p, m, grads, gold["group_of_worker"], gold["groups"], gold["lr"],
                         gold["momentum"], gold["weight_decay"], reps)
        assert m.tolist() == st["m"]
        assert p.tolist() == st["p"]
        for r in reps:
            assert r.tobytes() == p.tobytes()


# ---------------------------------------------------------------- P4 closed forms

def _closed_form(p0, gbar, lr, mu, wd, k):
    """x_k = A^k x_0 + (A^0 + A^1 + ... + A^(k-1)) b for x = (m, p), m_0 = 0,
    with m' = mu*m + gbar + wd*p and p' = p - lr*m' written as x' = A x + b.
    (I - A is singular when wd = 0, so the geometric sum is taken term by term.)"""
    A = np.array([[mu, wd], [-lr * mu, 1.0 - lr * wd]])
    Ak = np.linalg.matrix_power(A, k)
    S = sum(np.linalg.matrix_power(A, t) for t in range(k))
    m_out = np.empty_like(p0)
    p_out = np.empty_like(p0)
    for i in range(p0.size):
        b = np.array([gbar[i], -lr * gbar[i]])
        x = Ak @ np.array([0.0, p0[i]]) + S @ b
        m_out[i], p_out[i] = x
    return p_out, m_out


@pytest.mark.parametrize("wd", [0.0, 0.01])
def test_momentum_recurrence_closed_form(wd):
    """k steps with a constant mean gradient against the closed form of the
    heavy-ball recurrence with L2 weight decay (Sec. 5.3 settings, reading of
    the update in the design notes). With wd = 0 it is also checked against the
    scalar closed form m_k = g(1-mu^k)/(1-mu),
    p_k = p0 - lr*g*(k/(1-mu) - mu(1-mu^k)/(1-mu)^2)."""
    rng = np.random.default_rng(17)
    n, G, W, k = 64, 2, 2, 60
    lr, mu = 0.1, 0.9
    grads = rand_grads(rng, G * W, n)
    gow = workloads.contiguous_groups(G, W)
    gbar = np.mean(np.stack(grads).astype(np.float64), axis=0)  # exact for these four terms
    p0 = (rng.standard_normal(n) * 0.05).astype(np.float32)
    p, m = p0.astype(np.float64), np.zeros(n)
    p32, m32 = p0.copy(), np.zeros(n, np.float32)
    for _ in range(k):
        oracle.lsgd_step(p, m, grads, gow, G, lr, mu, wd)
        oracle.lsgd_step(p32, m32, grads, gow, G, lr, mu, wd)
    pc, mc = _closed_form(p0.astype(np.float64), gbar, lr, mu, wd, k)
    scale = np.max(np.abs(pc))
    assert np.max(np.abs(p - pc)) <= 1e-12 * scale
    assert np.max(np.abs(m - mc)) <= 1e-12 * np.max(np.abs(mc))
    # binary32 build: k steps of a handful of roundings, amplified at most 1/(1-mu)
    assert np.max(np.abs(p32 - pc)) <= k * 10 * 8 * U * scale
    assert np.max(np.abs(m32 - mc)) <= k * 10 * 8 * U * np.max(np.abs(mc))
    if wd == 0.0:
        mk = gbar * (1 - mu ** k) / (1 - mu)
        pk = p0 - lr * gbar * (k / (1 - mu) - mu * (1 - mu ** k) / (1 - mu) ** 2)
        assert np.max(np.abs(m - mk)) <= 1e-12 * np.max(np.abs(mk))
        assert np.max(np.abs(p - pk)) <= 1e-12 * scale


# ---------------------------------------------------------------- P5 special cases

def test_plain_sgd_special_case():
    """N = 1, mu = wd = 0 is Alg. 1: w <- w - eps * dw, each operation a binary32
    operation (numpy float32 as the independent IEEE implementation)."""
    rng = np.random.default_rng(1)
    n = 5000
    g = rand_grads(rng, 1, n, std=1.0)[0]
    p = (rng.standard_normal(n)).astype(np.float32)
    p1, m1 = run_step(p, np.zeros(n, np.float32), [g], [0], 1, 0.1, 0.0, 0.0)
    assert m1.tobytes() == (np.float32(0.0) * np.zeros(n, np.float32) + g).tobytes()
    assert p1.tobytes() == (p - np.float32(0.1) * g).tobytes()


def test_momentum_sgd_single_worker_each_operation_rounded():
    """N = 1 with momentum and weight decay: each of the five operations is one
    binary32 operation with no contraction or excess precision."""
    rng = np.random.default_rng(2)
    n = 5000
    g = rand_grads(rng, 1, n)[0]
    p = (rng.standard_normal(n) * 0.05).astype(np.float32)
    m = (rng.standard_normal(n) * 0.01).astype(np.float32)
    lr, mu, wd = f32(0.1), f32(0.9), f32(1e-4)
    p1, m1 = run_step(p, m, [g], [0], 1, lr, mu, wd)
    d = g + wd * p
    m_ref = mu * m + d
    p_ref = p - lr * m_ref
    assert m1.tobytes() == m_ref.tobytes() and p1.tobytes() == p_ref.tobytes()


def test_csgd_two_workers_is_halved_sum():
    """G = 1 is Alg. 2: Allreduce over the N workers, divide by N (N = 2)."""
    rng = np.random.default_rng(4)
    g0, g1 = rand_grads(rng, 2, 3000)
    gm = oracle.group_means([g0, g1], [0, 0], 1)
    assert gm[0].tobytes() == ((g0 + g1) / np.float32(2)).tobytes()


def test_replica_copy_out():
    """Broadcast to the workers: binary32 replicas are bitwise copies; bf16
    replicas are torch's nearest-even rounding of the updated parameters."""
    rng = np.random.default_rng(6)
    n = 4000
    grads = rand_grads(rng, 4, n)
    p = (rng.standard_normal(n) * 0.05).astype(np.float32)
    reps = [np.full(n, np.nan, np.float32) for _ in range(3)]
    p1, _ = run_step(p, np.zeros(n, np.float32), grads, [0, 0, 1, 1], 2, 0.1, 0.9, 1e-4, reps)
    for r in reps:
        assert r.tobytes() == p1.tobytes()
    breps = [np.zeros(n, np.uint16) for _ in range(2)]
    p2, _ = run_step(p, np.zeros(n, np.float32), grads, [0, 0, 1, 1], 2, 0.1, 0.9, 1e-4, breps,
                     oracle.BF16)
    ref = torch.from_numpy(p2).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    for r in breps:
        assert np.array_equal(r, ref)


def test_bf16_widening_exhaustive():
    bits = np.arange(65536, dtype=np.uint32).astype(np.uint16)
    ours = oracle.bf16_to_f32(bits)
    ref = torch.from_numpy(bits.view(np.int16)).view(torch.bfloat16).float().numpy()
    nan = np.isnan(ref)
    assert np.array_equal(np.isnan(ours), nan)
    assert ours[~nan].tobytes() == ref[~nan].tobytes()


def test_bf16_rounding_matches_torch():
    """Nearest-even binary32 -> bfloat16 against torch's conversion: random bit
    patterns, exact ties (odd and even kept bits), overflow to infinity,
    subnormals, signed zeros and infinities. NaN maps to a NaN."""
    rng = np.random.default_rng(8)
    bits = rng.integers(0, 2 ** 32, size=1_000_000, dtype=np.uint64).astype(np.uint32)
    special = np.array([0x00000000, 0x80000000, 0x7F800000, 0xFF800000, 0x7F7FFFFF, 0x7F7F8000,
                        0x7F7F7FFF, 0x3F808000, 0x3F818000, 0x3F80FFFF, 0x00008000, 0x00018000,
                        0x00000001, 0x807FFFFF, 0x7FC00000, 0xFFC00001, 0x7F800001, 0x4049000F],
                       dtype=np.uint32)
    bits = np.concatenate([special, bits])
    x = bits.view(np.float32)
    ours = oracle.f32_to_bf16(x)
    ref = torch.from_numpy(x.copy()).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    xnan = np.isnan(x)
    assert np.array_equal(ours[~xnan], ref[~xnan])
    assert np.all(np.isnan(oracle.bf16_to_f32(ours[xnan])))


# ---------------------------------------------------------------- P6 brute force

def _exact(v):
    return Fraction(float(v))


def _bounded_op(val, err):
    """Rounding of one binary32 operation whose exact-operand result is `val`
    and whose operands carry absolute error `err` in total."""
    return err + U * (abs(float(val)) + err)


def _brute_force_check(grads, gow, G, p, m, lr, mu, wd, p_out, m_out):
    """Exact rational evaluation of one step from the same binary32 inputs, and a
    running forward error bound for the binary32 evaluation."""
    N = len(grads)
    W = N // G
    rows = [[i for i in range(N) if gow[i] == j] for j in range(G)]
    lr_e, mu_e, wd_e = _exact(f32(lr)), _exact(f32(mu)), _exact(f32(wd))
    hw = math.ceil(math.log2(W)) if W > 1 else 0
    hg = math.ceil(math.log2(G)) if G > 1 else 0
    gw = hw * U / (1 - hw * U)
    gg = hg * U / (1 - hg * U)
    for i in range(p.size):
        means, merrs = [], []
        for row in rows:
            xs = [_exact(grads[w][i]) for w in row]
            s = sum(xs)
            serr = gw * float(sum(abs(x) for x in xs))
            mean = s / W
            means.append(mean)
            merrs.append(_bounded_op(mean, serr / W))
        tot = sum(means)
        terr = sum(merrs) + gg * float(sum(abs(x) + e for x, e in zip(means, merrs)))
        gbar = tot / G
        gerr = _bounded_op(gbar, terr / G)
        pe, me = _exact(p[i]), _exact(m[i])
        wdp = wd_e * pe
        d = gbar + wdp
        derr = _bounded_op(d, gerr + U * abs(float(wdp)))
        mum = mu_e * me
        m_new = mum + d
        m_err = _bounded_op(m_new, derr + U * abs(float(mum)))
        lrm = lr_e * m_new
        p_new = pe - lrm
        p_err = _bounded_op(p_new, float(lr_e) * m_err + U * (abs(float(lrm)) + float(lr_e) * m_err))
        slack = 1.0 + 16 * U
        assert abs(_exact(m_out[i]) - m_new) <= Fraction(m_err * slack), (i, "m")
        assert abs(_exact(p_out[i]) - p_new) <= Fraction(p_err * slack), (i, "p")


@pytest.mark.parametrize("G,W", [(1, 1), (1, 3), (3, 1), (2, 3), (3, 5), (4, 4), (5, 3), (2, 8)])
def test_brute_force_exact_rationals(G, W):
    rng = np.random.default_rng(100 + G * 17 + W)
    n = 8
    grads = rand_grads(rng, G * W, n)
    gow = workloads.shuffled_groups(G, W, seed=G * 31 + W)
    p = (rng.standard_normal(n) * 0.05).astype(np.float32)
    m = (rng.standard_normal(n) * 0.01).astype(np.float32)
    lr, mu, wd = 0.1, 0.9, 1e-4
    p_out, m_out = run_step(p, m, grads, gow, G, lr, mu, wd)
    _brute_force_check(grads, gow, G, p, m, lr, mu, wd, p_out, m_out)


def test_brute_force_detects_a_dropped_weight_decay_term():
    """The bound is tight enough to see the weight-decay term: a step computed
    without it fails the exact check."""
    rng = np.random.default_rng(9)
    n = 8
    grads = rand_grads(rng, 4, n)
    p = (rng.standard_normal(n) * 0.05).astype(np.float32)
    m = np.zeros(n, np.float32)
    p_out, m_out = run_step(p, m, grads, [0, 0, 1, 1], 2, 0.1, 0.9, 0.0)
    with pytest.raises(AssertionError):
        _brute_force_check(grads, [0, 0, 1, 1], 2, p, m, 0.1, 0.9, 1e-4, p_out, m_out)


# ---------------------------------------------------------------- composition

@pytest.mark.parametrize("G,W,gdt", [(2, 2, "f32"), (3, 5, "f32"), (8, 8, "bf16")])
def test_unfused_composition_matches_fused(G, W, gdt):
    """group_means, then global_mean, then sgd_step is the fused step, bitwise."""
    rng = np.random.default_rng(12)
    n = 999
    grads = rand_grads(rng, G * W, n)
    if gdt == "bf16":
        grads = [oracle.f32_to_bf16(g) for g in grads]
    gow = workloads.shuffled_groups(G, W, seed=3)
    p = (rng.standard_normal(n) * 0.05).astype(np.float32)
    m = (rng.standard_normal(n) * 0.01).astype(np.float32)
    pf, mf = run_step(p, m, grads, gow, G, 0.1, 0.9, 1e-4)
    gbar = oracle.global_mean(oracle.group_means(grads, gow, G))
    pu, mu_ = p.copy(), m.copy()
    oracle.sgd_step(pu, mu_, gbar, 0.1, 0.9, 1e-4)
    assert pu.tobytes() == pf.tobytes() and mu_.tobytes() == mf.tobytes()


def test_non_finite_values_propagate():
    g = np.array([np.nan, np.inf, -np.inf, 1.0], np.float32)
    p = np.ones(4, np.float32)
    p1, m1 = run_step(p, np.zeros(4, np.float32), [g, g], [0, 1], 2, 0.1, 0.9, 1e-4)
    assert np.isnan(p1[0]) and np.isnan(m1[0])
    assert p1[1] == -np.inf and p1[2] == np.inf and np.isfinite(p1[3])


def test_workload_shapes():
    sizes = workloads.resnet50_param_sizes()
    assert len(sizes) == 161 and sum(sizes) == workloads.RESNET50_NUMEL
    vec = workloads.resnet50_vector_params()
    assert len(vec) == 161 and sum(vec) == 107                     # 53 BN pairs + the classifier bias
    assert all(s in (64, 128, 256, 512, 1024, 2048, 1000) for s, v in zip(sizes, vec) if v)
    for wl in workloads.WORKLOADS.values():
        if wl.tensor_sizes:
            assert sum(wl.tensor_sizes) == wl.n
    uneq = workloads.WORKLOADS["resnet50_unequal"]
    gow = uneq.group_of_worker()
    assert uneq.n_workers == 16 and len(gow) == 16 and sorted(set(gow)) == [0, 1, 2, 3]
    assert [gow.count(j) for j in range(4)] == [2, 3, 5, 6]
    big = workloads.WORKLOADS["large"]
    assert big.n_workers == 64 and big.algorithmic_bytes(0) == big.n * (64 * 2 + 16)


# ---------------------------------------------------------------- paper-literal reduction

@pytest.mark.parametrize("G,W,gdt", [(2, 2, "f32"), (4, 4, "f32"), (16, 8, "f32"), (8, 8, "bf16"),
                                     (1, 16, "f32")])
def test_literal_reduction_equals_mean_of_means_for_powers_of_two(G, W, gdt):
    """Alg. 3 as printed (each communicator divides its sum by N, the allreduce
    sums) and the mean of subgroup means agree bit for bit when W and G are
    powers of two: dividing by 2^k commutes with rounding."""
    rng = np.random.default_rng(300 + G * W)
    n = 1200
    grads = rand_grads(rng, G * W, n)
    if gdt == "bf16":
        grads = [oracle.f32_to_bf16(g) for g in grads]
    gow = workloads.shuffled_groups(G, W, seed=G + W)
    p = (rng.standard_normal(n) * 0.05).astype(np.float32)
    m = (rng.standard_normal(n) * 0.01).astype(np.float32)
    a = run_step(p, m, grads, gow, G, 0.1, 0.9, 1e-4)
    pl, ml = p.copy(), m.copy()
    oracle.lsgd_step_literal(pl, ml, grads, gow, G, 0.1, 0.9, 1e-4)
    assert pl.tobytes() == a[0].tobytes() and ml.tobytes() == a[1].tobytes()


def _literal_bound_check(grads, gow, G, gbar_out):
    """The literal reduction of any partition has the flat mean sum(g)/N as its
    exact value (sum_j (S_j / N) = S / N): check the binary32 result against it
    within the forward error bound of the per-group pairwise sums, the
    divisions and the pairwise sum over groups."""
    N = len(grads)
    members, start = oracle.partition(gow, G)
    for i in range(gbar_out.size):
        exact = sum(_exact(g[i]) for g in grads) / N
        err = 0.0
        parts_abs = 0.0
        for j in range(G):
            xs = [_exact(grads[w][i]) for w in members[start[j]:start[j + 1]]]
            k = len(xs)
            h = math.ceil(math.log2(k)) if k > 1 else 0
            s_err = h * U / (1 - h * U) * float(sum(abs(x) for x in xs))
            c = sum(xs) / N
            c_err = _bounded_op(c, s_err / N)
            err += c_err
            parts_abs += abs(float(c)) + c_err
        hg = math.ceil(math.log2(G)) if G > 1 else 0
        err += hg * U / (1 - hg * U) * parts_abs
        assert abs(_exact(gbar_out[i]) - exact) <= Fraction(err * (1 + 16 * U)), i


@pytest.mark.parametrize("gow,G", [([0, 1, 1, 1], 2), ([0, 0, 1, 2, 2, 2, 2], 3),
                                   ([2, 0, 1, 1, 2, 0, 0, 0, 1], 3), ([0] * 5 + [1], 2),
                                   (list(range(5)), 5)])
def test_literal_reduction_of_unequal_groups_is_the_flat_mean(gow, G):
    """Any partition, even with unequal subgroups, reaches the conventional
    mean of Alg. 2 (Sec. 4.2: Algorithms 1-3 compute the same SGD)."""
    rng = np.random.default_rng(len(gow) * 7 + G)
    n = 8
    grads = rand_grads(rng, len(gow), n)
    work = [g.copy() for g in grads]
    p = (rng.standard_normal(n) * 0.05).astype(np.float32)
    m = np.zeros(n, np.float32)
    oracle.lsgd_step_literal(p, m, work, gow, G, 0.1, 0.9, 1e-4, broadcast_grad=True)
    for w in work[1:]:
        assert w.tobytes() == work[0].tobytes()        # every worker received the same mean
    _literal_bound_check(grads, gow, G, work[0])


def test_literal_reduction_single_group_is_alg2():
    """G = 1: the communicator sums all N and divides by N, exactly the
    mean-of-means oracle with one group."""
    rng = np.random.default_rng(41)
    grads = rand_grads(rng, 6, 500)
    p = (rng.standard_normal(500) * 0.05).astype(np.float32)
    a = run_step(p, np.zeros(500, np.float32), grads, [0] * 6, 1, 0.1, 0.9, 1e-4)
    pl, ml = p.copy(), np.zeros(500, np.float32)
    oracle.lsgd_step_literal(pl, ml, grads, [0] * 6, 1, 0.1, 0.9, 1e-4)
    assert pl.tobytes() == a[0].tobytes() and ml.tobytes() == a[1].tobytes()


def test_gradient_broadcast_delivers_the_global_mean():
    """Broadcast of the gathered gradient (Sec. 4.1, item 3): afterwards every
    worker's buffer holds the mean gradient, bitwise equal to the global mean of
    the group means for power-of-two groups."""
    rng = np.random.default_rng(42)
    G, W, n = 4, 4, 3000
    grads = rand_grads(rng, G * W, n)
    gow = workloads.contiguous_groups(G, W)
    want = oracle.global_mean(oracle.group_means(grads, gow, G))
    work = [g.copy() for g in grads]
    p = np.zeros(n, np.float32)
    oracle.lsgd_step_literal(p, np.zeros(n, np.float32), work, gow, G, 0.1, 0.9, 1e-4,
                             broadcast_grad=True)
    for w in work:
        assert w.tobytes() == want.tobytes()


@pytest.mark.parametrize("gow,G", [([0, 0, 2, 2], 3), ([0, 1, 3], 3), ([-1, 0], 1)])
def test_partition_rejects_empty_groups_and_bad_ids(gow, G):
    with pytest.raises(oracle.OracleError) as e:
        oracle.partition(gow, G)
    assert e.value.status == oracle.ERR_GROUPS


# ---------------------------------------------------------------- learning-rate schedule

def test_lr_schedule_matches_the_paper():
    with open(os.path.join(GOLDEN, "lr_schedule.json")) as f:
        gold = json.load(f)
    ipe = gold["iters_per_epoch"]
    args = (gold["base_lr"], gold["base_batch"], gold["global_batch"], gold["warmup_epochs"] * ipe,
            gold["decay_epochs"] * ipe, gold["decay_factor"])
    for pt in gold["points"]:
        t = pt["epoch_iter"][0] * ipe + pt["epoch_iter"][1]
        got = oracle.lr_at(t, *args)
        assert abs(got - pt["lr"]) <= 2e-7 * pt["lr"] + 1e-12, (t, got, pt["lr"])


def test_lr_schedule_shape():
    """Linear warmup (equal per-iteration increments), constant plateau, then
    a tenfold drop at every decay boundary."""
    a = (0.1, 256.0, 16384.0, 390, 2340, 0.1)
    w = np.array([oracle.lr_at(t, *a) for t in range(391)], np.float64)
    inc = np.diff(w[:390])
    assert np.allclose(inc, (6.4 - 0.1) / 390, rtol=1e-4)
    assert all(oracle.lr_at(t, *a) == np.float32(6.4) for t in (390, 1000, 2339))
    assert oracle.lr_at(2340, *a) == np.float32(0.64)
    assert oracle.lr_at(4680, *a) == np.float32(6.4 * 0.1 * 0.1)
    # no warmup, no decay: the linearly scaled rate
    assert oracle.lr_at(10 ** 9, 0.1, 256.0, 1024.0, 0, 0, 0.1) == np.float32(0.4)


# ---------------------------------------------------------------- LARS (Sec. 2, Sec. 6)
# The paper names LARS without defining it; the oracle follows You, Gitman and
# Ginsburg (arXiv 1708.03888, eq. 6, Alg. 1). Pins: a step worked by hand, the
# zero-norm fallback to the plain step, the scale symmetries of the trust
# ratio, and the ratio against a 60-digit evaluation.

def _lars(p, m, grads, gow, G, lr, mu, wd, eta):
    p, m = p.copy(), m.copy()
    t = oracle.lars_step(p, m, grads, gow, G, lr, mu, wd, eta)
    return p, m, t


@pytest.mark.parametrize("dtype", [np.float32, np.float64])
def test_lars_constant_tensor_worked_by_hand(dtype):
    """16 elements, p = 2 (or alternating +-2), all four workers (2 x 2) hold 0.5,
    so gbar = 0.5 (fixed point): ||p|| = 8, ||gbar|| = 2, and with eta = 1/8,
    wd = 1/4 the trust is (1/8 * 8) / (2 + 1/4 * 8) = 1/4. Then
    d = 1/4 * (0.5 + 1/4 * p): 1/4 for p = 2, 0 for p = -2; m = d (m0 = 0);
    p - 0.5 * m = 1.875 or -2. Every value is dyadic, so exact in any order."""
    n, G, W = 16, 2, 2
    grads = [np.full(n, 0.5, np.float32) for _ in range(G * W)]
    gow = workloads.contiguous_groups(G, W)
    p0 = np.full(n, 2.0, dtype)
    p, m, t = _lars(p0, np.zeros(n, dtype), grads, gow, G, 0.5, 0.9, 0.25, 0.125)
    assert t == 0.25
    assert np.all(m == 0.25) and np.all(p == 1.875)
    p0 = np.where(np.arange(n) % 2 == 0, 2.0, -2.0).astype(dtype)
    p, m, t = _lars(p0, np.zeros(n, dtype), grads, gow, G, 0.5, 0.9, 0.25, 0.125)
    assert t == 0.25
    assert np.array_equal(m, np.where(np.arange(n) % 2 == 0, 0.25, 0.0).astype(dtype))
    assert np.array_equal(p, np.where(np.arange(n) % 2 == 0, 1.875, -2.0).astype(dtype))


def test_lars_zero_norm_is_the_plain_step():
    """A tensor with ||p|| = 0 or ||gbar|| = 0 takes trust 1, and the LARS
    step is then the plain momentum step bit for bit (zero parameters,
    all-zero gradients, and two workers whose gradients cancel exactly)."""
    rng = np.random.default_rng(41)
    n, G, W = 1000, 2, 2
    gow = workloads.contiguous_groups(G, W)
    m0 = (rng.standard_normal(n) * 1e-3).astype(np.float32)
    g = rand_grads(rng, G * W, n)
    cases = [
        (np.zeros(n, np.float32), g, gow, G),
        ((rng.standard_normal(n) * 0.05).astype(np.float32), [np.zeros(n, np.float32)] * 4, gow, G),
        ((rng.standard_normal(n) * 0.05).astype(np.float32), [g[0], -g[0]], [0, 0], 1),
    ]
    for p0, grads, gw, GG in cases:
        pl, ml, t = _lars(p0, m0, grads, gw, GG, 0.1, 0.9, 1e-4, 1e-3)
        pp, mp = run_step(p0, m0, grads, gw, GG, 0.1, 0.9, 1e-4)
        assert t == 1.0
        assert np.array_equal(pl, pp) and np.array_equal(ml, mp)


@pytest.mark.parametrize("k", [5, -7])
def test_lars_gradient_scale_invariance(k):
    """With wd = 0 the LARS step does not depend on the gradient scale:
    scaling every worker gradient by 2^k scales gbar and ||gbar|| by 2^k
    exactly, the trust by 2^-k exactly, and leaves d = trust * gbar, hence m
    and p, unchanged bit for bit."""
    rng = np.random.default_rng(42)
    n, G, W = 777, 4, 4
    gow = workloads.contiguous_groups(G, W)
    p0 = (rng.standard_normal(n) * 0.05).astype(np.float32)
    m0 = (rng.standard_normal(n) * 1e-3).astype(np.float32)
    g = rand_grads(rng, G * W, n)
    s = np.float32(2.0 ** k)
    pa, ma, ta = _lars(p0, m0, g, gow, G, 0.1, 0.9, 0.0, 1e-3)
    pb, mb, tb = _lars(p0, m0, [x * s for x in g], gow, G, 0.1, 0.9, 0.0, 1e-3)
    assert np.float32(tb) * s == np.float32(ta)
    assert np.array_equal(pa, pb) and np.array_equal(ma, mb)


@pytest.mark.parametrize("k", [3, -4])
def test_lars_parameter_scale_equivariance(k):
    """With wd = 0 and m0 = 0, scaling p by 2^k scales ||p||, the trust, d, m
    and the new p by 2^k exactly."""
    rng = np.random.default_rng(43)
    n, G, W = 513, 2, 4
    gow = workloads.contiguous_groups(G, W)
    p0 = (rng.standard_normal(n) * 0.05).astype(np.float32)
    g = rand_grads(rng, G * W, n)
    s = np.float32(2.0 ** k)
    z = np.zeros(n, np.float32)
    pa, ma, ta = _lars(p0, z, g, gow, G, 0.1, 0.9, 0.0, 1e-3)
    pb, mb, tb = _lars(p0 * s, z, g, gow, G, 0.1, 0.9, 0.0, 1e-3)
    assert np.float32(ta) * s == np.float32(tb)
    assert np.array_equal(pa * s, pb) and np.array_equal(ma * s, mb)


def _trust_60_digits(p, gbar, wd, eta):
    import decimal
    ctx = decimal.Context(prec=60)
    sp = sum(Fraction(float(x)) ** 2 for x in p)
    sg = sum(Fraction(float(x)) ** 2 for x in gbar)
    D = lambda fr: ctx.divide(decimal.Decimal(fr.numerator), decimal.Decimal(fr.denominator))
    wn, gn = ctx.sqrt(D(sp)), ctx.sqrt(D(sg))
    e, w = decimal.Decimal(float(np.float32(eta))), decimal.Decimal(float(np.float32(wd)))
    return ctx.divide(ctx.multiply(e, wn), ctx.add(gn, ctx.multiply(w, wn)))


@pytest.mark.parametrize("n,wd", [(257, 0.0), (1000, 1e-4), (4096, 5e-2)])
def test_lars_trust_against_60_digit_evaluation(n, wd):
    """The binary32 trust ratio is within half an ulp (plus the 1e-15 relative
    slack of its binary64 evaluation) of the ratio evaluated with exact sums of
    squares and 60-digit square roots and division."""
    import decimal
    rng = np.random.default_rng(n)
    p = (rng.standard_normal(n) * 0.05).astype(np.float32)
    gbar = (rng.standard_normal(n) * 1e-2 * rng.uniform(0.1, 10)).astype(np.float32)
    t = np.float32(oracle.lars_trust(p, gbar, wd, 1e-3))
    exact = _trust_60_digits(p, gbar, wd, 1e-3)
    ulp = np.spacing(t)
    err = abs(decimal.Decimal(float(t)) - exact)
    assert err <= decimal.Decimal(float(ulp)) / 2 + exact * decimal.Decimal("1e-15"), (t, exact)


def test_lars_zero_trust_coefficient_keeps_only_momentum():
    """eta = 0 gives trust 0, so d = 0 and the step decays the momentum:
    m = mu*m, p = p - lr*m (two binary32 operations per element)."""
    rng = np.random.default_rng(44)
    n, G, W = 300, 2, 2
    gow = workloads.contiguous_groups(G, W)
    p0 = (rng.standard_normal(n) * 0.05).astype(np.float32)
    m0 = (rng.standard_normal(n) * 1e-3).astype(np.float32)
    p, m, t = _lars(p0, m0, rand_grads(rng, G * W, n), gow, G, 0.1, 0.9, 1e-4, 0.0)
    assert t == 0.0
    m1 = (np.float32(0.9) * m0).astype(np.float32)
    assert np.array_equal(m, m1)
    assert np.array_equal(p, (p0 - np.float32(0.1) * m1).astype(np.float32))
