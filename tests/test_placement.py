"""CPU: the placement layer (decoder provisioning, prefill latency curve, admission, binding;
Section 4 of the paper). The oracle (oracle/placement.py) is pinned to the paper's worked
provisioning example and to hand-derived cases; the library (include/conserve_sched.h) must then
take exactly the oracle's decisions on seeded random inputs."""
import math
import os

import numpy as np
import pytest

from oracle import placement as op

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _golden(name):
    vals = {}
    for line in open(os.path.join(ROOT, "tests", "golden", name)):
        line = line.strip()
        if line and not line.startswith("#"):
            k, v = line.split()
            vals[k] = float(v)
    return vals


# ---- oracle pins ---------------------------------------------------------------------------
def test_oracle_provisioning_matches_paper_worked_example():
    g = _golden("provisioning_worked_example.txt")
    r, n_thr, n_mem, n = op.provision(g["prefill_tokens_per_s"], g["mean_turn1_tokens"],
                                      g["decoder_tokens_per_s"], g["mean_decoder_tokens"],
                                      convs_per_decoder=1e9, mean_lifetime_s=1.0)
    assert r == pytest.approx(g["saturation_rate"], rel=1e-15)
    assert round(n_thr, 2) == g["n_throughput_printed"]
    assert n == 2                      # smallest integer above 1.67 (the memory bound is tiny)


def test_oracle_provisioning_memory_bound_and_integer_rule():
    # R* = 2/s; throughput bound 2 * 500 / 1000 = 1; memory bound 2 * 60 / 40 = 3 -> N = 4
    r, n_thr, n_mem, n = op.provision(20000, 10000, 1000, 500, 40, 60)
    assert (r, n_thr, n_mem, n) == (2.0, 1.0, 3.0, 4)
    # a non-integer bound rounds up: 2.5 -> 3
    assert op.provision(5000, 1000, 1000, 500, 1e9, 1)[3] == 3


def test_oracle_curve_fit_recovers_exact_quadratic():
    coef = (0.0123, 4.5e-6, 7.25e-11)
    L = [512, 1024, 4096, 16384, 65536, 131072]
    t = [coef[0] + x * coef[1] + x * x * coef[2] for x in L]
    fit, r2 = op.prefill_curve_fit(L, t)
    assert fit == pytest.approx(coef, rel=1e-7)
    assert r2 == pytest.approx(1.0, abs=1e-12)
    # three points: the quadratic through them (Lagrange interpolation) is the fit
    fit3, r23 = op.prefill_curve_fit([1, 2, 3], [1.0, 4.0, 9.0])
    assert fit3 == pytest.approx((0.0, 0.0, 1.0), abs=1e-10) and r23 == pytest.approx(1.0)
    # noise lowers R^2 below 1
    _, r2n = op.prefill_curve_fit(L, [x * (1 + (-1) ** i * 0.05) for i, x in enumerate(t)])
    assert r2n < 1.0


def test_oracle_binding_hand_cases():
    # equal capacities: lowest used wins
    assert op.bind([30, 10, 20], [70, 90, 80], 5) == 1
    # fraction, not absolute pages: 30/300 = 0.10 < 20/100 = 0.20
    assert op.bind([20, 30], [80, 270], 5) == 1
    # ties go to the lower index
    assert op.bind([10, 10, 10], [90, 90, 90], 1) == 0
    # only decoders with room are candidates; none -> -1
    assert op.bind([0, 50], [4, 50], 5) == 1
    assert op.bind([0, 50], [4, 3], 5) == -1


def test_oracle_curve_eval_hand_values():
    """t(L) = c0 + c1 L + c2 L^2, each term checked by hand."""
    assert op.curve_eval((1.0, 2.0, 3.0), 10) == 321.0           # 1 + 20 + 300
    assert op.curve_eval((0.5, 0.0, 0.0), 12345) == 0.5
    assert op.curve_eval((0.0, 0.25, 0.0), 8) == 2.0
    assert op.curve_eval((0.0, 0.0, 0.125), 4) == 2.0
    assert op.curve_eval((3.0, -1.0, 0.5), 0) == 3.0
    assert op.curve_eval((3.0, -1.0, 0.5), 6) == 15.0             # 3 - 6 + 18


def test_oracle_admission_quadratic_timeline():
    # t(L) = 0.5 + 0.25 L + 0.125 L^2 s: L = 2 -> 1.5 s, L = 4 -> 3.5 s
    a = op.Admission((0.5, 0.25, 0.125), max_wait_s=2.0)
    assert a.admit(2, 0.0) == (0.0, 1.5)
    assert a.admit(4, 1.0) == (1.5, 5.0)                           # waits 0.5 s
    assert a.admit(2, 2.0) is None                                 # would wait 3 s
    assert a.admit(2, 3.0) == (5.0, 6.5)                           # waits exactly 2 s


def test_oracle_admission_hand_timeline():
    a = op.Admission((1.0, 0.0, 0.0), max_wait_s=1.5)     # every prefill takes 1 s
    assert a.admit(100, 0.0) == (0.0, 1.0)
    assert a.admit(100, 0.2) == (1.0, 2.0)                 # waits 0.8 s
    assert a.admit(100, 0.4) is None and a.busy_until == 2.0   # would wait 1.6 s > 1.5: refused
    assert a.admit(100, 0.6) == (2.0, 3.0)                 # wait exactly 1.4 s
    assert a.admit(100, 5.0) == (5.0, 6.0)                 # idle prefiller: starts on arrival
    b = op.Admission((1.0, 0.0, 0.0), max_wait_s=1.0)
    assert b.admit(10, 0.0) == (0.0, 1.0) and b.admit(10, 0.0) == (1.0, 2.0)   # wait == bound: admitted


# ---- library vs oracle ------------------------------------------------------------------------
def test_library_provisioning_matches_oracle_exactly():
    import paper_2606_01839_amd as m
    g = _golden("provisioning_worked_example.txt")
    got = m.provision_decoders(g["prefill_tokens_per_s"], g["mean_turn1_tokens"],
                               g["decoder_tokens_per_s"], g["mean_decoder_tokens"], 1e9, 1.0)
    assert round(got["n_throughput"], 2) == g["n_throughput_printed"] and got["n_decoders"] == 2
    rng = np.random.default_rng(11)
    for _ in range(200):
        x = [float(v) for v in rng.uniform(0.5, 5e4, size=6)]
        r, a, b, n = op.provision(*x)
        got = m.provision_decoders(*x)
        assert (got["saturation_rate"], got["n_throughput"], got["n_memory"], got["n_decoders"]) == (r, a, b, n)


def test_library_provisioning_rejects_bad_inputs():
    import paper_2606_01839_amd as m
    from paper_2606_01839_amd import ConserveError, CS_EINVAL
    for bad in [(0, 1, 1, 1, 1, 1), (1, -1, 1, 1, 1, 1), (1, 1, 1, 1, float("inf"), 1),
                (1, 1, 1, 1, 1, float("nan")), (1e300, 1e-300, 1, 1, 1, 1)]:
        with pytest.raises(ConserveError) as e:
            m.provision_decoders(*bad)
        assert e.value.code == CS_EINVAL


def test_library_curve_fit_matches_oracle():
    import paper_2606_01839_amd as m
    rng = np.random.default_rng(12)
    for trial in range(50):
        n = int(rng.integers(3, 20))
        L = np.unique(rng.integers(1, 200000, size=n))
        if L.size < 3:
            continue
        coef = (rng.uniform(1e-4, 1e-2), rng.uniform(1e-7, 1e-5), rng.uniform(1e-12, 1e-10))
        t = np.array([op.curve_eval(coef, int(x)) for x in L]) * rng.uniform(0.97, 1.03, size=L.size)
        want, r2w = op.prefill_curve_fit(L, t)
        got, r2g = m.prefill_curve_fit(L, t)
        for x in L:     # compare the fitted curves where they are used
            assert m.prefill_curve_eval(got, int(x)) == pytest.approx(op.curve_eval(want, int(x)), rel=1e-9)
        assert r2g == pytest.approx(r2w, abs=1e-9)
        for x in (1, 1000, int(L.max())):
            assert m.prefill_curve_eval(got, x) == op.curve_eval(got, x)   # same evaluation order


def test_library_curve_fit_rejects_degenerate_samples():
    import paper_2606_01839_amd as m
    from paper_2606_01839_amd import ConserveError, CS_EINVAL
    for L, t in [([1, 2], [1.0, 2.0]), ([5, 5, 7, 7], [1, 1, 2, 2]), ([1, 2, 3], [1.0, float("nan"), 2.0])]:
        with pytest.raises(ConserveError) as e:
            m.prefill_curve_fit(L, t)
        assert e.value.code == CS_EINVAL


def test_library_binding_matches_oracle_exactly():
    import paper_2606_01839_amd as m
    rng = np.random.default_rng(13)
    for _ in range(500):
        n = int(rng.integers(1, 9))
        cap = rng.integers(1, 5000, size=n)
        used = np.array([int(rng.integers(0, c + 1)) for c in cap])
        free = cap - used
        need = int(rng.integers(0, 800))
        assert m.place_least_occupied(used, free, need) == op.bind(list(map(int, used)), list(map(int, free)), need)
    # huge capacities: the exact comparison must not overflow
    big = 2 ** 40
    assert m.place_least_occupied([big - 1, big - 2], [big + 1, big + 2], 1) == op.bind([big - 1, big - 2], [big + 1, big + 2], 1)


def test_library_admission_matches_oracle_exactly():
    import paper_2606_01839_amd as m
    from paper_2606_01839_amd import KVPool
    pools = [KVPool(1, 4, 2, 64, n_pages=64, max_convs=4, max_pages_per_conv=64, placement_seed=i,
                    device="cpu") for i in range(2)]
    rng = np.random.default_rng(14)
    coef = (0.002, 3e-6, 2e-11)
    for max_wait in (0.0, 0.05, 0.5):
        s = m.Scheduler(coef, max_wait, pools)
        o = op.Admission(coef, max_wait)
        now = 0.0
        for _ in range(300):
            now += float(rng.exponential(0.03))
            L = int(rng.integers(1, 60000))
            assert s.admit(L, now) == o.admit(L, now)
        s.close()
    for p in pools:
        p.close()


def test_scheduler_binds_by_capacity_and_validates():
    import paper_2606_01839_amd as m
    from paper_2606_01839_amd import KVPool, ConserveError, CS_EINVAL
    small = KVPool(1, 4, 2, 64, n_pages=10, max_convs=4, max_pages_per_conv=64, placement_seed=1, device="cpu")
    large = KVPool(1, 4, 2, 64, n_pages=100, max_convs=4, max_pages_per_conv=64, placement_seed=2, device="cpu")
    s = m.Scheduler((0.0, 1e-6, 0.0), 1.0, [small, large])
    assert s.bind(16) == 0                 # both empty: tie -> lower index
    assert s.bind(161) == 1                # 11 pages: only the large pool has room
    assert s.bind(1600) == 1 and s.bind(1601) == -1   # 100 pages fit, 101 do not
    for bad in (lambda: s.bind(0), lambda: s.admit(0, 0.0), lambda: s.admit(5, float("nan"))):
        with pytest.raises(ConserveError) as e:
            bad()
        assert e.value.code == CS_EINVAL
    with pytest.raises(ConserveError) as e:
        m.Scheduler((0, 0, 0), -1.0, [small])
    assert e.value.code == CS_EINVAL
    s.close()
    small.close()
    large.close()


def test_admission_only_scheduler():
    """n_decoders = 0: admission works (the same decisions as the oracle), bind is refused."""
    import paper_2606_01839_amd as m
    from paper_2606_01839_amd import ConserveError, CS_EINVAL
    coef = (0.002, 3e-6, 2e-11)
    s = m.Scheduler(coef, 0.05)
    o = op.Admission(coef, 0.05)
    rng = np.random.default_rng(15)
    now = 0.0
    for _ in range(200):
        now += float(rng.exponential(0.02))
        L = int(rng.integers(1, 40000))
        assert s.admit(L, now) == o.admit(L, now)
    with pytest.raises(ConserveError) as e:
        s.bind(16)
    assert e.value.code == CS_EINVAL
    s.close()
