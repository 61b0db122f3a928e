"""Pins for the oracle's water-filling allocation (Sec. 3.2 Eq. (5), Algorithm 1, integer
ranks) and the coded budget (Sec. 3.1 Eq. (3))."""
import itertools
from fractions import Fraction

import numpy as np
import pytest

from golden_io import fracs, ints, read_blocks


# ---------------------------------------------------------------------------------------
# Independent references (no code shared with the C oracle)

def alg1_exact(u, B, r_min, R):
    """Algorithm 1's water-filling loop run literally with exact rationals, weights = u."""
    N = len(u)
    r = [Fraction(r_min)] * N
    U = set(range(N))
    while True:
        delta = Fraction(B) - sum(r)
        tot = sum(Fraction(u[t]) for t in U)
        for t in U:
            r[t] += delta * u[t] / tot
        S = {t for t in U if r[t] > R}
        for t in S:
            r[t] = Fraction(R)
        U -= S
        if not S:
            return r


def alg1_float(u, B, r_min, R):
    """The same loop in plain fp64 (as the paper's implementation would run it)."""
    N = len(u)
    r = np.full(N, float(r_min))
    U = np.ones(N, bool)
    while True:
        delta = B - r.sum()
        tot = u[U].astype(np.float64).sum()
        r[U] += delta * u[U] / tot
        S = U & (r > R)
        r[S] = R
        U &= ~S
        if not S.any():
            return r


def hamilton(q, u):
    """Largest remainder rounding of exact fractions q with the stated tie rule."""
    fl = [x.numerator // x.denominator for x in q]
    rho = int(sum(q) - sum(fl))
    order = sorted(range(len(q)), key=lambda t: (-(q[t] - fl[t]), -u[t], t))
    out = list(fl)
    for t in order[:rho]:
        out[t] += 1
    return out


def continuous_from_oracle(al, u, r_min, R):
    capped = set(np.argsort(-u.astype(np.int64), kind="stable")[: al.k].tolist())
    return [Fraction(R) if t in capped else Fraction(r_min) + Fraction(int(u[t]) * al.M, al.Q)
            for t in range(len(u))]


# ---------------------------------------------------------------------------------------

@pytest.mark.parametrize("blk", read_blocks("waterfill_handworked.txt"), ids=lambda b: b["name"][0])
def test_waterfill_handworked(oracle_lib, blk):
    N, R, r_min, B = (int(blk[k][0]) for k in ("N", "R", "r_min", "B"))
    u = np.array(ints(blk["u"]), np.uint32)
    if "sbar" in blk:
        sb = np.array([float(x) for x in blk["sbar"]], np.float32)
        assert list(oracle_lib.weights(sb)) == list(u)
    al = oracle_lib.allocate(u, B, r_min, R)
    assert list(al.rank) == ints(blk["rank"])
    assert al.k == int(blk["capped"][0])
    assert continuous_from_oracle(al, u, r_min, R) == fracs(blk["q"])


@pytest.mark.parametrize("seed", range(12))
def test_waterfill_matches_exact_algorithm1(oracle_lib, seed):
    rng = np.random.default_rng(seed)
    N = int(rng.integers(1, 40))
    R = int(rng.integers(2, 20))
    r_min = int(rng.integers(0, R))
    B = int(rng.integers(N * r_min, N * R + 1))
    mode = seed % 3
    if mode == 0:
        u = rng.integers(1, 1 << 25, N)
    elif mode == 1:                       # heavy ties
        u = rng.integers(1, 4, N) * 1000
    else:                                 # spiky: few large weights
        u = np.ones(N, np.int64)
        u[rng.choice(N, size=max(1, N // 8), replace=False)] = rng.integers(1 << 20, 1 << 24)
    u = u.astype(np.uint32)
    al = oracle_lib.allocate(u, B, r_min, R)
    q = alg1_exact(u.tolist(), B, r_min, R)
    assert continuous_from_oracle(al, u, r_min, R) == q
    assert list(al.rank) == hamilton(q, u.tolist())


@pytest.mark.parametrize("seed", range(6))
def test_waterfill_matches_float_algorithm1(oracle_lib, seed):
    """The fp64 loop reaches the same clip set and levels up to rounding (rel 1e-12)."""
    from workloads import CONFIGS, make_layer
    rng = np.random.default_rng(100 + seed)
    N = 3000
    u = (1 + np.floor(rng.random(N) ** 8 * (1 << 24))).astype(np.uint32)
    B = N * 16 + int(rng.integers(0, N * 60))
    al = oracle_lib.allocate(u, B, 16, 128)
    qf = alg1_float(u, B, 16, 128)
    qo = np.array([float(x) for x in continuous_from_oracle(al, u, 16, 128)])
    np.testing.assert_allclose(qf, qo, rtol=1e-12)
    assert int((qf >= 128).sum()) >= al.k


def test_brute_force_rounding_is_least_squares(oracle_lib):
    """Enumerate every integer vector with the bounds and sum B: the oracle's ranks
    minimise sum (r_t - q_t)^2, and among minimisers follow the tie rule."""
    rng = np.random.default_rng(7)
    for trial in range(40):
        N = int(rng.integers(1, 6))
        R = int(rng.integers(2, 8))
        r_min = int(rng.integers(0, R))
        B = int(rng.integers(N * r_min, N * R + 1))
        u = rng.integers(1, 6, N).astype(np.uint32)
        al = oracle_lib.allocate(u, B, r_min, R)
        q = alg1_exact(u.tolist(), B, r_min, R)
        best, argbest = None, []
        for r in itertools.product(range(r_min, R + 1), repeat=N):
            if sum(r) != B:
                continue
            cost = sum((Fraction(x) - y) ** 2 for x, y in zip(r, q))
            if best is None or cost < best:
                best, argbest = cost, [r]
            elif cost == best:
                argbest.append(r)
        assert tuple(al.rank.tolist()) in argbest
        if len(argbest) == 1:
            assert tuple(al.rank.tolist()) == argbest[0]


@pytest.mark.parametrize("seed", range(5))
def test_waterfill_invariants_large(oracle_lib, seed):
    rng = np.random.default_rng(200 + seed)
    N = int(rng.integers(1000, 40000))
    r_min, R = 16, 128
    B = int(rng.integers(N * r_min, N * R + 1))
    u = (1 + np.floor(rng.random(N) ** 6 * (1 << 24))).astype(np.uint32)
    al = oracle_lib.allocate(u, B, r_min, R)
    r = al.rank.astype(np.int64)
    assert r.sum() == B
    assert r.min() >= r_min and r.max() <= R
    # monotone in the weight (equal weights: the lower index may hold the extra unit)
    order = np.lexsort((-np.arange(N), u))
    assert np.all(np.diff(r[order]) >= 0)
    # within one unit of the continuous solution
    qo = np.array([float(x) for x in continuous_from_oracle(al, u, r_min, R)])
    assert np.all(np.abs(r - qo) < 1.0 + 1e-9)


def test_uniform_signal_gives_uniform_codec(oracle_lib):
    """Constant salience collapses Eq. (5) to r_t = B / N (the uniform-rank codec): the
    B - N floor(B/N) extra units go to the lowest indices."""
    N, B = 1001, 1001 * 25 + 417
    al = oracle_lib.allocate(np.full(N, 12345, np.uint32), B, 16, 128)
    want = np.full(N, 25)
    want[:417] = 26
    np.testing.assert_array_equal(al.rank, want)


def test_budget_extremes(oracle_lib):
    u = np.random.default_rng(8).integers(1, 1 << 24, 333).astype(np.uint32)
    np.testing.assert_array_equal(oracle_lib.allocate(u, 333 * 16, 16, 128).rank, 16)
    np.testing.assert_array_equal(oracle_lib.allocate(u, 333 * 128, 16, 128).rank, 128)
    with pytest.raises(oracle_lib.BudgetError):
        oracle_lib.allocate(u, 333 * 16 - 1, 16, 128)
    with pytest.raises(oracle_lib.BudgetError):
        oracle_lib.allocate(u, 333 * 128 + 1, 16, 128)


def test_one_hot_salience(oracle_lib):
    """One salient token: it takes min(R, r_min + E) and the rest of the excess spreads
    uniformly over the others (their epsilon weights are all 1)."""
    N, r_min, R = 200, 16, 128
    u = np.ones(N, np.uint32)
    u[37] = (1 << 24) + 1
    E = 100                               # E * N < 2^24: the epsilon weights stay below one unit
    al = oracle_lib.allocate(u, N * r_min + E, r_min, R)
    # continuous: hot token gets r_min + E (2^24+1)/(2^24+N) < R, the others r_min + tiny
    assert al.rank[37] == r_min + E
    assert np.all(np.delete(al.rank, 37) == r_min)
    E = 5000                              # now the hot token caps at R
    al = oracle_lib.allocate(u, N * r_min + E, r_min, R)
    assert al.rank[37] == R
    rest = np.delete(al.rank, 37)
    left = E - (R - r_min)
    assert rest.sum() == (N - 1) * r_min + left
    assert rest.max() - rest.min() <= 1


def test_zero_floor_allowed(oracle_lib):
    u = np.array([1, 1, 1, 16777217], np.uint32)
    al = oracle_lib.allocate(u, 10, 0, 8)
    assert al.rank.sum() == 10 and al.rank[3] == 8 and al.rank.min() >= 0


# ---------------------------------------------------------------------------------------
# Eq. (3) coded budget

def test_budget_config_values(oracle_lib):
    """B = floor(kappa n d / 100) - w d for the workload shapes (per-head units)."""
    assert oracle_lib.budget(512, 128, 32, 20) == 9011
    assert oracle_lib.budget(32768, 128, 32, 20) == 834764
    assert oracle_lib.budget(16384, 128, 32, 20) == 415334
    assert oracle_lib.budget(131072, 128, 32, 20) == 3351347
    assert oracle_lib.budget(32768, 128, 32, 10) == 415334
    assert oracle_lib.budget(32768, 128, 32, 40) == 1673625


@pytest.mark.parametrize("n,w,kappa", [(512, 32, 20), (1000, 17, 33), (77, 5, 90), (4096, 64, 5)])
def test_budget_matches_storage_fraction(oracle_lib, n, w, kappa):
    """Total storage (exact window + coded coefficients) is the largest integer count not
    above kappa of the full cache, as Eq. (3) requires."""
    d = 128
    B = oracle_lib.budget(n, d, w, kappa)
    total = B + w * d
    assert Fraction(total, n * d) <= Fraction(kappa, 100) < Fraction(total + 1, n * d)


# ---------------------------------------------------------------------------------------
# Reading of the all-zero division in Algorithm 1's loop: the oracle water-fills the integer
# weights u_t = 1 + floor(2^24 s_hat_t) instead of s_hat itself.  As weights w = u / 2^24 =
# s_hat + delta with 0 < delta_t <= 2^-24, and the water level lambda falls as weights grow,
# every token's continuous rank moves by at most (N + 1) lambda_w 2^-24, where lambda_w 2^-24
# = M / Q is the oracle's level per unit of u:
#   q^s_t - clip(r_min + lambda_w s_hat_t) lies in [0, g(lambda_s) - g(lambda_w)] <= lambda_w N 2^-24,
#   |q^w_t - clip(r_min + lambda_w s_hat_t)| <= lambda_w delta_t <= lambda_w 2^-24,
# with g(lambda) = sum_t clip(r_min + lambda s_hat_t), which the budget fixes on both sides.
def _shat_cases():
    rng = np.random.default_rng(4242)
    for i in range(14):
        N = int(rng.integers(2, 36))
        R = int(rng.integers(4, 40))
        r_min = int(rng.integers(0, R // 2 + 1))
        B = int(rng.integers(N * r_min, N * R + 1))
        kind = i % 4
        if kind == 0:
            s = rng.random(N)
        elif kind == 1:                     # spiky: one or two hot tokens, the rest near zero
            s = rng.random(N) ** 16
        elif kind == 2:                     # exact zeros besides the minimum (Q7's 0/0 risk)
            s = np.where(rng.random(N) < 0.6, 0.0, rng.random(N))
        else:                               # heavy ties
            s = rng.integers(0, 3, N) / 2.0
        yield N, R, r_min, B, s.astype(np.float32)


@pytest.mark.parametrize("case", list(_shat_cases()), ids=lambda c: f"N{c[0]}R{c[1]}m{c[2]}B{c[3]}")
def test_epsilon_weights_stay_within_bound_of_algorithm1_on_shat(oracle_lib, case):
    N, R, r_min, B, sbar = case
    if sbar.max() == sbar.min():
        pytest.skip("constant signal: both readings give the uniform codec")
    u = oracle_lib.weights(sbar)
    lo, hi = float(sbar.min()), float(sbar.max())
    shat = [Fraction((float(x) - lo)) / Fraction(hi - lo) for x in sbar]
    if sum(shat) == 0:
        pytest.skip("all-zero s_hat: Algorithm 1 itself divides 0 / 0")
    q_s, stalled = alg1_exact_weights(shat, B, r_min, R)
    al = oracle_lib.allocate(u, B, r_min, R)
    q_w = continuous_from_oracle(al, u, r_min, R)
    assert int(al.rank.sum()) == B
    if stalled:
        # Algorithm 1 reached 0/0: every remaining token has s_hat = 0 while budget is left.
        # Under the reading, tokens with s_hat < 2^-24 weigh u = 1 like the zeros: the loop's
        # capped tokens above that resolution stay capped, and the remainder is spread evenly
        # over the u = 1 tokens.
        assert all(q_w[t] == R for t in range(N) if q_s[t] == R and u[t] > 1)
        ones = [t for t in range(N) if u[t] == 1]
        assert ones and len({q_w[t] for t in ones}) == 1
        assert sum(q_w) == B
        return
    lam = Fraction(al.M, al.Q) if al.Q else Fraction(0)
    bound = (N + 1) * lam
    gap = max(abs(a - b) for a, b in zip(q_w, q_s))
    assert gap <= bound, (float(gap), float(bound))
    # the integer ranks stay within one unit (plus the bound) of Algorithm 1 on s_hat
    assert all(abs(r - q) < 1 + bound for r, q in zip(al.rank.tolist(), q_s))


def alg1_exact_weights(w, B, r_min, R):
    """Algorithm 1's loop in exact rationals with arbitrary non-negative weights w."""
    N = len(w)
    r = [Fraction(r_min)] * N
    U = set(range(N))
    while True:
        delta = Fraction(B) - sum(r)
        tot = sum(w[t] for t in U)
        if tot == 0:
            return r, delta > 0
        for t in U:
            r[t] += delta * w[t] / tot
        S = {t for t in U if r[t] > R}
        for t in S:
            r[t] = Fraction(R)
        U -= S
        if not S:
            return r, False
