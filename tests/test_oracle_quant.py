"""Pins for the oracle's group-wise b-bit coefficient quantiser (Sec. 3.3 "Composability":
the coefficients are quantised group-wise, the allocation is unchanged)."""
import numpy as np
import pytest


def test_half_round_matches_numpy_binary16(oracle_lib):
    """The binary16 rounding (ties to even, subnormals, overflow) against numpy's float16
    conversion, an independent library implementation of the same IEEE definition."""
    rng = np.random.default_rng(3)
    vals = np.concatenate([
        rng.standard_normal(4000) * 10.0 ** rng.uniform(-9, 5, 4000),
        np.array([0.0, 65504.0, 65519.0, 65520.0, 2.0 ** -24, 2.0 ** -25, 3 * 2.0 ** -26, 2.0 ** -14,
                  1.0 + 2.0 ** -11, 1.0 + 3 * 2.0 ** -11, -(1.0 + 2.0 ** -11), 2049.0, 2051.0]),
    ]).astype(np.float32)
    with np.errstate(over="ignore"):
        want = vals.astype(np.float16).astype(np.float32)
    got = np.array([oracle_lib.half_round(v) for v in vals], np.float32)
    np.testing.assert_array_equal(got, want)


def _nearest_code(x, sc, qmax):
    """Brute force over every code: the nearest multiple of sc in [-qmax, qmax], ties to
    the even code."""
    best = None
    for k in range(-qmax, qmax + 1):
        e = abs(np.float64(x) - k * np.float64(sc))
        key = (e, k % 2)
        if best is None or key < best[0]:
            best = (key, k)
    return best[1]


@pytest.mark.parametrize("bits", [3, 4, 8])
def test_codes_are_nearest_grid_points(oracle_lib, bits):
    rng = np.random.default_rng(bits)
    n, G, d = 24, 2, 128
    coef = (rng.standard_normal((n, G, d)) * rng.uniform(0.01, 30, (n, G, 1))).astype(np.float32)
    rank = rng.integers(1, 129, n).astype(np.int32)
    for t in range(n):
        coef[t, :, rank[t]:] = 0.0
    qz = oracle_lib.quantize(coef, rank, bits)
    qmax = 2 ** (bits - 1) - 1
    for t in range(n):
        for g in range(G):
            for s in range(4):
                lo, hi = 32 * s, min(32 * s + 32, int(rank[t]))
                sc = float(qz.scales[t, g, s])
                if lo >= hi:
                    assert sc == 0.0
                    continue
                amax = np.abs(coef[t, g, lo:hi]).max()
                # the scale is binary16(amax / qmax)
                assert sc == oracle_lib.half_round(np.float32(amax) / np.float32(qmax))
                assert abs(sc - amax / qmax) <= 2.0 ** -11 * amax / qmax + 2.0 ** -25
                for j in range(lo, hi):
                    if sc == 0.0:
                        assert qz.codes[t, g, j] == 0
                        continue
                    assert qz.codes[t, g, j] == _nearest_code(coef[t, g, j], sc, qmax), (t, g, j)
                    assert qz.deq[t, g, j] == np.float32(qz.codes[t, g, j]) * np.float32(sc)
                    # half a step of error (plus the last step's clamp, far smaller)
                    assert abs(coef[t, g, j] - qz.deq[t, g, j]) <= 0.5 * sc * (1 + 1e-6) + 2.0 ** -10 * amax
            assert np.all(qz.codes[t, g, rank[t]:] == 0) and np.all(qz.deq[t, g, rank[t]:] == 0)


@pytest.mark.parametrize("bits", [3, 4, 8])
def test_values_on_the_grid_are_kept_exactly(oracle_lib, bits):
    """Groups whose values are integer multiples k * sc of a binary16 step, with max |k| =
    qmax, come back exactly (the scale is found exactly and every x / sc is an integer)."""
    rng = np.random.default_rng(40 + bits)
    qmax = 2 ** (bits - 1) - 1
    n, G, d = 10, 3, 128
    coef = np.zeros((n, G, d), np.float32)
    want_codes = np.zeros((n, G, d), np.int8)
    rank = np.full(n, 128, np.int32)
    for t in range(n):
        for g in range(G):
            for s in range(4):
                sc = np.float32(np.float16(2.0 ** rng.integers(-6, 6) * (1 + rng.integers(0, 1024) / 1024)))
                k = rng.integers(-qmax, qmax + 1, 32)
                k[rng.integers(0, 32)] = qmax * rng.choice([-1, 1])
                coef[t, g, 32 * s:32 * s + 32] = k * sc
                want_codes[t, g, 32 * s:32 * s + 32] = k
    qz = oracle_lib.quantize(coef, rank, bits)
    np.testing.assert_array_equal(qz.codes, want_codes)
    np.testing.assert_array_equal(qz.deq, coef)


def test_error_shrinks_with_bits_and_zero_groups(oracle_lib):
    rng = np.random.default_rng(9)
    coef = rng.standard_normal((50, 2, 128)).astype(np.float32)
    rank = rng.integers(16, 129, 50).astype(np.int32)
    for t in range(50):
        coef[t, :, rank[t]:] = 0
    coef[3, 1, :] = 0.0                      # an all-zero token row: scale 0, codes 0
    errs = {}
    for b in (3, 4, 8):
        qz = oracle_lib.quantize(coef, rank, b)
        errs[b] = np.abs(qz.deq - coef).max(axis=-1)
        assert np.all(qz.scales[3, 1] == 0) and np.all(qz.codes[3, 1] == 0)
    assert np.all(errs[8] <= errs[4] + 1e-7) and np.all(errs[4] <= errs[3] + 1e-7)
    assert errs[8].max() < errs[4].max() < errs[3].max()


def test_quantised_cache_decode_is_decode_of_dequantised_values(oracle_lib):
    """Decode over a quantised cache is the reconstruct-in-place decode of the dequantised
    coefficients; at 8 bits it stays within the quantisation error of the unquantised one,
    and the error grows as the bits fall (tiny workload, fp32 storage)."""
    from workloads import CONFIGS, make_layer
    cfg = CONFIGS["tiny"]
    li = make_layer(cfg, n_queries=1)
    oc = oracle_lib.compress(li.K, li.V, li.Qw, li.PK, li.PV, cfg["H"], cfg["kappa"], cfg["r_min"], "f32")
    base = oracle_lib.decode(oc.coefK, oc.coefV, oc.alloc.rank, oc.Kx, oc.Vx, li.PK, li.PV, li.q[0], cfg["H"])
    prev = 0.0
    for b in (8, 4, 3):
        qk = oracle_lib.quantize(oc.coefK, oc.alloc.rank, b)
        qv = oracle_lib.quantize(oc.coefV, oc.alloc.rank, b)
        o = oracle_lib.decode(qk.deq, qv.deq, oc.alloc.rank, oc.Kx, oc.Vx, li.PK, li.PV, li.q[0], cfg["H"])
        e = np.abs(o - base).max() / np.abs(base).max()
        assert e >= prev * 0.5
        prev = e
        if b == 8:
            assert e < 2e-2
