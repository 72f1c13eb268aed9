"""DN selection (Eq. 11): the oracle pinned by hand-worked tables and by
properties of the constrained minimum, then the C ABI's elasto_select_mode
against the oracle on random tables (host only, no GPU)."""
import math

import numpy as np
import pytest

import oracle
from paper_2609_10018_amd import ffi

# A hand-worked table: five nested DNs, FLOPs falling with the index.
FLOPS = [35.1, 26.4, 17.7, 9.0, 5.7]
LAT = [13.0, 10.5, 8.0, 5.5, 4.4]
MEM = [900.0, 700.0, 500.0, 300.0, 250.0]
ACC = [0.81, 0.80, 0.77, 0.70, 0.62]
POW = [600.0, 520.0, 430.0, 330.0, 300.0]


@pytest.mark.parametrize("bounds,expected", [
    ({}, 4),                                            # nothing binds: cheapest DN
    ({"A_min": 0.75}, 2),                               # accuracy rules out 3 and 4
    ({"A_min": 0.75, "L_d": 7.9}, None),                # fast enough ones are too inaccurate
    ({"A_min": 0.80, "L_d": 12.0}, 1),
    ({"M_d": 260.0}, 4),
    ({"M_d": 240.0}, None),                             # nothing fits in memory
    ({"L_d": 4.4}, 4),                                  # bounds are inclusive
    ({"A_min": 0.81}, 0),                               # only the full model
    ({"P_d": 400.0, "A_min": 0.7}, 3),
    ({"P_d": 299.0}, None),
])
def test_oracle_hand_worked(bounds, expected):
    assert oracle.select_dn(FLOPS, LAT, MEM, ACC, POW, **bounds) == expected


def test_oracle_ties_and_missing_columns():
    # equal cost: the lower index wins; a missing column constrains nothing
    assert oracle.select_dn([2, 1, 1], [1, 1, 1], [1, 1, 1]) == 1
    assert oracle.select_dn([2, 1, 1], [1, 1, 1], [1, 1, 1], A_min=0.99) == 1
    assert oracle.select_dn([5], [1], [1], [0.5], A_min=0.6) is None


def test_oracle_properties_on_random_tables():
    rng = np.random.default_rng(7)
    for _ in range(300):
        n = int(rng.integers(1, 8))
        f, lat, mem, acc, pw = (rng.uniform(0, 10, n).round(1) for _ in range(5))
        b = dict(L_d=rng.uniform(0, 10), M_d=rng.uniform(0, 10), A_min=rng.uniform(0, 10),
                 P_d=rng.uniform(0, 10))
        k = oracle.select_dn(f, lat, mem, acc, pw, **b)
        feas = [(lat[i] <= b["L_d"] and mem[i] <= b["M_d"] and acc[i] >= b["A_min"]
                 and pw[i] <= b["P_d"]) for i in range(n)]
        if k is None:
            assert not any(feas)
            continue
        assert feas[k]                                   # the answer is feasible
        assert all(f[k] <= f[i] for i in range(n) if feas[i])    # and no cheaper one is
        assert all(f[i] > f[k] for i in range(k) if feas[i])     # ties go to the lower index
        # relaxing a bound never makes the choice more expensive
        loose = dict(b, L_d=math.inf)
        k2 = oracle.select_dn(f, lat, mem, acc, pw, **loose)
        assert k2 is not None and f[k2] <= f[k]


def test_c_abi_matches_oracle():
    rng = np.random.default_rng(11)
    for trial in range(500):
        n = int(rng.integers(1, 9))
        f, lat, mem, acc, pw = (rng.integers(0, 6, n).astype(float) for _ in range(5))
        use_acc, use_pw = bool(rng.integers(0, 2)), bool(rng.integers(0, 2))
        b = dict(L_d=float(rng.integers(0, 7)), M_d=float(rng.integers(0, 7)),
                 A_min=float(rng.integers(0, 7)) if use_acc else -math.inf,
                 P_d=float(rng.integers(0, 7)))
        if trial % 5 == 0:
            b["L_d"] = math.inf
        want = oracle.select_dn(f, lat, mem, acc if use_acc else None, pw if use_pw else None,
                                **b)
        got = ffi.select_mode(f, lat, mem, acc if use_acc else None, pw if use_pw else None,
                              max_latency_ms=b["L_d"], max_memory_bytes=b["M_d"],
                              min_accuracy=b["A_min"], max_power_w=b["P_d"])
        assert got == want, (trial, f, lat, mem, acc, pw, b)


def test_c_abi_rejects_bad_tables():
    with pytest.raises(ffi.ElastoError):
        ffi.select_mode([1.0, float("nan")], [1, 1], [1, 1])
    with pytest.raises(ffi.ElastoError):
        ffi.select_mode([1.0], [1.0], [1.0], max_latency_ms=float("nan"))
    with pytest.raises(ffi.ElastoError):            # accuracy bound without accuracy data
        ffi.select_mode([1.0], [1.0], [1.0], min_accuracy=0.5)
    with pytest.raises(ffi.ElastoError):
        ffi.select_mode([], [], [])
    assert ffi.select_mode(FLOPS, LAT, MEM, ACC, POW, min_accuracy=0.75) == 2
