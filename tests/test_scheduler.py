"""Bandwidth allocation under a shared cap (Section 3.6, eqs. (4)-(7)): the
oracle's allocators against the paper's per-request allocation table, brute
force and the optimality conditions; then the library's allocator against
the oracle (host code, no GPU)."""
import ctypes
import math
import random
from itertools import groupby

import numpy as np
import pytest

import paper_2605_22850_amd as oc
from oracle import model
from tests.conftest import golden_rows

GBPS = 1e9 / 8          # bytes/s per Gbps
B_PER_TOKEN = 4096      # Llama 3.1 8B: 2 * 8 KV heads * 128 * 2 B per layer


def paper_workloads():
    """(name, cap, s, c, expected rows) for Workloads A, B, C."""
    cells = {(int(r[0]), float(r[1])): (int(r[2]), float(r[4])) for r in golden_rows("canonical_cells.txt")}
    out = []
    for wl, grp in groupby(golden_rows("per_method_allocations.txt"), key=lambda r: r[0]):
        grp = list(grp)
        s = [cells[(int(r[2]), float(r[3]))][0] * B_PER_TOKEN for r in grp]
        c = [cells[(int(r[2]), float(r[3]))][1] / 1e3 for r in grp]
        want = np.array([[float(x) for x in r[4:9]] for r in grp])
        out.append((wl, float(grp[0][1]) * GBPS, s, c, want))
    return out


def oracle_all(B, s, c, delta=5 * GBPS):
    return np.array([model.alloc_equal(B, len(s)), model.alloc_kv_prop(B, s), model.alloc_bw_prop(B, s, c),
                     model.alloc_stall_opt(B, s, c), model.alloc_cal_stall_opt(B, s, c, delta)]).T


@pytest.mark.parametrize("wl", ["A", "B", "C"])
def test_oracle_reproduces_the_paper_allocation_table(wl):
    name, B, s, c, want = next(w for w in paper_workloads() if w[0] == wl)
    got = oracle_all(B, s, c) / GBPS
    # the table prints 2 decimals from per-layer times printed with 2 decimals
    np.testing.assert_allclose(got, want, atol=0.011)


def _objective(s, r):
    return sum(a / x for a, x in zip(s, r))


def test_stall_opt_two_requests_matches_1d_minimisation():
    rng = random.Random(5)
    for _ in range(50):
        s = [rng.uniform(1, 100), rng.uniform(1, 100)]
        caps = [rng.uniform(0.5, 20), rng.uniform(0.5, 20)]
        B = rng.uniform(0.3, 0.95) * sum(caps)
        got = model.stall_opt(B, s, caps)
        # r1 ranges over [max(eps, B - cap2), min(cap1, B)]; the objective is convex
        lo, hi = max(1e-12, B - caps[1]), min(caps[0], B - 1e-12)
        f = lambda r1: s[0] / r1 + s[1] / (B - r1)
        for _ in range(300):       # golden-section search
            m1, m2 = lo + (hi - lo) * 0.382, lo + (hi - lo) * 0.618
            if f(m1) < f(m2):
                hi = m2
            else:
                lo = m1
        assert got[0] == pytest.approx((lo + hi) / 2, rel=1e-7, abs=1e-9)
        assert sum(got) == pytest.approx(B, rel=1e-12)


def test_stall_opt_three_requests_beats_every_grid_point():
    rng = random.Random(11)
    for _ in range(10):
        s = [rng.uniform(1, 50) for _ in range(3)]
        caps = [rng.uniform(1, 10) for _ in range(3)]
        B = rng.uniform(0.4, 0.9) * sum(caps)
        got = model.stall_opt(B, s, caps)
        best = math.inf
        n = 300
        for i in range(1, n + 1):          # caps included: optima often sit on them
            r0 = caps[0] * i / n
            for j in range(1, n + 1):
                r1 = caps[1] * j / n
                r2 = B - r0 - r1
                if 0 < r2 <= caps[2]:
                    best = min(best, _objective(s, (r0, r1, r2)))
        assert _objective(s, got) <= best * (1 + 1e-12)
        assert _objective(s, got) >= best * (1 - 2e-3)      # and the grid gets close to it


def test_stall_opt_optimality_conditions():
    rng = random.Random(3)
    for _ in range(200):
        n = rng.randint(1, 9)
        s = [rng.uniform(0.1, 1000) for _ in range(n)]
        caps = [rng.uniform(0.1, 100) for _ in range(n)]
        B = rng.uniform(0.05, 1.5) * sum(caps)
        r = model.stall_opt(B, s, caps)
        assert all(0 < x <= cp * (1 + 1e-12) for x, cp in zip(r, caps))
        if sum(caps) <= B:
            assert r == caps
            continue
        assert sum(r) == pytest.approx(B, rel=1e-10)
        free = [a / x ** 2 for a, x, cp in zip(s, r, caps) if x < cp * (1 - 1e-9)]
        if free:
            lam = free[0]
            assert all(v == pytest.approx(lam, rel=1e-6) for v in free)
            # a capped request would take more if it could: its marginal value is higher
            assert all(a / x ** 2 >= lam * (1 - 1e-6) for a, x, cp in zip(s, r, caps) if x >= cp * (1 - 1e-9))


def test_zero_stall_rates_fit_means_no_stall():
    s, c = [10.0, 20.0], [1.0, 4.0]
    r = model.alloc_stall_opt(100.0, s, c)
    assert r == [10.0, 5.0] and model.total_stall(s, c, r) == 0.0
    assert model.per_layer_stall(10.0, 5.0, 1.0) == pytest.approx(1.0)


# ---------------------------------------------------------------------------
# the library's allocator (host code) against the oracle
# ---------------------------------------------------------------------------

POLICIES = ["equal", "kv_prop", "bw_prop", "stall_opt", "cal_stall_opt"]


def lib_alloc(policy, B, s, c, delta):
    import paper_2605_22850_amd as oc
    return np.array(oc.oc_bandwidth_allocate(policy, s, c, B, delta))


def test_library_reproduces_the_paper_allocation_table():
    for name, B, s, c, want in paper_workloads():
        got = np.array([lib_alloc(p, B, s, c, 5 * GBPS) for p in POLICIES]).T / GBPS
        np.testing.assert_allclose(got, want, atol=0.011, err_msg=f"workload {name}")


def test_library_matches_oracle_on_random_sets():
    rng = random.Random(17)
    for _ in range(300):
        n = rng.randint(1, 16)
        s = [rng.uniform(1e5, 5e8) for _ in range(n)]
        c = [rng.uniform(1e-4, 0.3) for _ in range(n)]
        rstar = [a / b for a, b in zip(s, c)]
        B = rng.uniform(0.05, 1.5) * sum(rstar)
        delta = rng.choice([0.0, 5 * GBPS, 0.1 * B])
        want = oracle_all(B, s, c, delta)
        got = np.array([lib_alloc(p, B, s, c, delta) for p in POLICIES]).T
        np.testing.assert_allclose(got, want, rtol=1e-9, atol=1e-6 * B)


def test_library_allocator_rejects_bad_input():
    import paper_2605_22850_amd as oc
    from paper_2605_22850_amd import _lib as L
    with pytest.raises(oc.OcError) as e:
        oc.oc_bandwidth_allocate("stall_opt", [1.0, 2.0], [0.0, 1.0], 1.0, 0.0)
    assert e.value.status == L.OC_EINVAL
    with pytest.raises(oc.OcError):
        oc.oc_bandwidth_allocate("stall_opt", [1.0], [1.0], -1.0, 0.0)
    with pytest.raises(oc.OcError):
        oc.oc_bandwidth_allocate("no_such_policy", [1.0], [1.0], 1.0, 0.0)
    out = (ctypes.c_double * 1)()
    assert oc.lib().oc_bandwidth_allocate(0, 0, None, None, 1.0, 0.0, out) == L.OC_EINVAL


# ---------------------------------------------------------------------------
# scheduling epochs
# ---------------------------------------------------------------------------

def _epoch_cases():
    cases = {}
    for row in golden_rows("epoch_schedule.txt"):
        if row[0] == "case":
            cases[row[1]] = {"policy": row[2], "B": float(row[3]), "L": int(row[4]), "epoch": float(row[5]),
                             "reqs": []}
        else:
            cases[row[1]]["reqs"].append([float(x) for x in row[2:7]])
    return cases


@pytest.mark.parametrize("name", ["periodic", "event", "kvprop", "leftover"])
def test_epoch_schedule_hand_worked_cases(name):
    cs = _epoch_cases()[name]
    s, c, a, want_r, want_t = (list(col) for col in zip(*cs["reqs"]))
    rates, admit = model.epoch_schedule(cs["policy"], s, c, cs["L"], a, cs["B"], epoch=cs["epoch"])
    assert rates == pytest.approx(want_r, rel=1e-12) and admit == pytest.approx(want_t, abs=1e-12)
    rates, admit = oc.oc_epoch_schedule(cs["policy"], s, c, cs["L"], a, cs["B"], epoch_s=cs["epoch"])
    assert rates == pytest.approx(want_r, rel=1e-12) and admit == pytest.approx(want_t, abs=1e-12)


def _check_epoch_rule(policy, s, c, L, a, B, epoch, rates, admit):
    """The rule, checked on a finished schedule: admissions at or after
    arrival and on a boundary; at every boundary the rates of the requests
    still loading fit the budget; a request waits past a boundary only if
    nobody was admitted there and no budget was free."""
    n = len(s)
    end = [admit[i] + L * s[i] / rates[i] for i in range(n)]
    assert all(rates[i] > 0 and admit[i] >= a[i] - 1e-12 for i in range(n))
    if epoch > 0:
        assert all(abs(t / epoch - round(t / epoch)) < 1e-9 for t in admit)
    for t in set(admit):
        loading = sum(rates[j] for j in range(n) if admit[j] <= t + 1e-12 and end[j] > t + 1e-12)
        assert loading <= B * (1 + 1e-9)
    # boundaries a request waited through
    events = sorted(set(a) | set(end) | set(admit))
    bounds = set()
    for e in events:
        bounds.add(e if epoch == 0 else math.ceil(e / epoch - 1e-12) * epoch)
    for i in range(n):
        for b in bounds:
            if a[i] <= b < admit[i] - 1e-12:
                assert not any(abs(admit[j] - b) < 1e-12 for j in range(n)), (i, b)
                held = sum(rates[j] for j in range(n) if admit[j] < b - 1e-12 and end[j] > b + 1e-12)
                assert B - held <= 1e-9 * B * 10 + 1e-12, (i, b, B - held)


@pytest.mark.parametrize("policy", ["equal", "kv_prop", "bw_prop", "stall_opt", "cal_stall_opt"])
def test_epoch_schedule_library_matches_oracle_and_rule(policy):
    rng = np.random.default_rng(11)
    for trial in range(60):
        n = int(rng.integers(1, 9))
        L = int(rng.integers(1, 40))
        s = list(rng.uniform(1e6, 5e8, n))
        c = list(rng.uniform(1e-3, 0.2, n))
        a = [0.0 if rng.random() < 0.3 else float(rng.uniform(0, 3.0)) for _ in range(n)]
        B = float(rng.uniform(1e9, 2e10))
        epoch = 0.0 if trial % 2 else float(rng.choice([0.01, 0.1, 0.5]))
        delta = 0.625e9
        r_o, t_o = model.epoch_schedule(policy, s, c, L, a, B, delta=delta, epoch=epoch)
        r_l, t_l = oc.oc_epoch_schedule(policy, s, c, L, a, B, delta, epoch)
        assert r_l == pytest.approx(r_o, rel=1e-9), (trial, r_l, r_o)
        assert t_l == pytest.approx(t_o, abs=1e-9), (trial, t_l, t_o)
        _check_epoch_rule(policy, s, c, L, a, B, epoch, r_l, t_l)


def test_epoch_schedule_with_every_arrival_at_start_is_one_allocation():
    rng = np.random.default_rng(12)
    for policy in ("equal", "kv_prop", "bw_prop", "stall_opt", "cal_stall_opt"):
        n = 6
        s = list(rng.uniform(1e6, 5e8, n))
        c = list(rng.uniform(1e-3, 0.2, n))
        one = oc.oc_bandwidth_allocate(policy, s, c, 1e10, 0.625e9)
        for epoch in (0.0, 0.25):
            rates, admit = oc.oc_epoch_schedule(policy, s, c, 32, [0.0] * n, 1e10, 0.625e9, epoch)
            assert rates == pytest.approx(one, rel=1e-12) and admit == [0.0] * n


def test_epoch_schedule_rejects_bad_input():
    with pytest.raises(oc.OcError):
        oc.oc_epoch_schedule("equal", [1.0], None, 0, [0.0], 1.0)
    with pytest.raises(oc.OcError):
        oc.oc_epoch_schedule("equal", [1.0], None, 1, [-1.0], 1.0)
    with pytest.raises(oc.OcError):
        oc.oc_epoch_schedule("equal", [1.0], None, 1, [0.0], 1.0, 0.0, -0.5)
    with pytest.raises(oc.OcError):
        oc.oc_epoch_schedule("stall_opt", [1.0], None, 1, [0.0], 1.0)
    with pytest.raises(oc.OcError):
        oc.oc_epoch_schedule("fifo", [1.0], None, 1, [0.0], 1.0)
