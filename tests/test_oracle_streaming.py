"""Pins of the weight-streaming oracle (oracle/streaming.py) against a
hand-derived timeline and the closed forms of the paper's streaming model
(Sec. 4, weight-streaming paragraph): lambda >= 1 hides every copy, lambda < 1
makes the copy engine the bottleneck, the overhead never exceeds
Delta = (N - K) W / M, and the device memory of a fully streamed plan is
T_min = 2 W_max + A_max."""
import numpy as np
import pytest

from oracle import streaming as S


def test_hand_derived_timeline():
    # two streamed layers, W = 100 and 200 bytes at 100 B/s (copies 1 s and
    # 2 s), compute 3 s and 1 s, two buffers:
    #   step 1: copy0 [0,1], compute0 [1,4]; copy1 [1,3], compute1 [4,5]
    #   step 2: copy0 waits for buffer 0 (compute0 ends at 4) [4,5],
    #           compute0 [5,8]; copy1 waits for buffer 1 (5) [5,7], compute1 [8,9]
    last, ends = S.simulate([100.0, 200.0], [3.0, 1.0], [0, 0], 2, 100.0, steps=2)
    assert ends == [5.0, 9.0]
    assert last == 4.0                        # steady state: the compute alone
    # one buffer: every copy waits for the previous layer's compute
    #   copy0 [0,1] c0 [1,4]; copy1 [4,6] c1 [6,7]; copy0 [7,8] c0 [8,11]; copy1 [11,13] c1 [13,14]
    last1, ends1 = S.simulate([100.0, 200.0], [3.0, 1.0], [0, 0], 1, 100.0, steps=2)
    assert ends1 == [7.0, 14.0] and last1 == 7.0
    # layer 1 resident: only layer 0 is copied, into alternating buffers
    #   copy0 [0,1] c0 [1,4] c1 [4,5]; copy0' (buffer 1 free) [1,2] c0 [5,8] c1 [8,9]
    last2, ends2 = S.simulate([100.0, 200.0], [3.0, 1.0], [0, 1], 2, 100.0, steps=2)
    assert ends2 == [5.0, 9.0] and last2 == 4.0


@pytest.mark.parametrize("n", [1, 2, 5, 12])
@pytest.mark.parametrize("lam", [1.0, 1.5, 4.0])
def test_lambda_at_least_one_hides_every_copy(n, lam):
    w, rate = 64e6, 50e9
    L = lam * w / rate
    assert S.reservoir_lambda(L, rate, w) == pytest.approx(lam)
    last, _ = S.simulate([w] * n, [L] * n, [0] * n, 2, rate, steps=4)
    assert last == pytest.approx(n * L, rel=1e-12)


@pytest.mark.parametrize("n", [1, 3, 8])
@pytest.mark.parametrize("lam", [0.05, 0.5, 0.9])
def test_lambda_below_one_is_copy_bound(n, lam):
    w, rate = 28e6, 55e9
    tau = w / rate
    L = lam * tau
    last, _ = S.simulate([w] * n, [L] * n, [0] * n, 2, rate, steps=4)
    assert last == pytest.approx(n * tau, rel=1e-12)           # the reservoir drains
    assert last - n * L == pytest.approx(n * (tau - L), rel=1e-9)
    # the paper's overhead with no overlapped layer bounds the exposed time
    assert last - n * L <= S.delta_overhead(n, 0, w, rate) * (1 + 1e-12)


@pytest.mark.parametrize("resident", [[0] * 6, [1, 0, 0, 1, 0, 0], [1, 1, 1, 0, 1, 1]])
def test_delta_is_attained_when_compute_vanishes(resident):
    # with (almost) no compute to hide behind, every streamed copy is exposed:
    # the step is the copies alone, Delta = (N - K) W / M with K resident layers
    n, w, rate, L = len(resident), 12e6, 50e9, 1e-12
    last, _ = S.simulate([w] * n, [L] * n, resident, 2, rate, steps=4)
    k = sum(resident)
    # (the vanishing compute hides in the gaps between copies)
    assert last == pytest.approx(S.delta_overhead(n, k, w, rate), rel=1e-9)


def test_single_buffer_serialises_copy_and_compute():
    w, rate, n = 10e6, 40e9, 6
    tau, L = w / rate, 3e-4
    last, _ = S.simulate([w] * n, [L] * n, [0] * n, 1, rate, steps=3)
    assert last == pytest.approx(n * (tau + L), rel=1e-12)


def test_all_resident_is_the_compute():
    rng = np.random.default_rng(0)
    w = list(rng.uniform(1e6, 1e8, 9))
    c = list(rng.uniform(1e-5, 1e-3, 9))
    last, _ = S.simulate(w, c, [1] * 9, 2, 50e9, steps=3)
    assert last == pytest.approx(sum(c), rel=1e-12)


def test_overhead_bounded_by_delta_and_monotone_in_residency():
    rng = np.random.default_rng(1)
    for _ in range(200):
        n = int(rng.integers(1, 9))
        w = float(rng.uniform(1e6, 5e7))
        rate = 50e9
        L = float(rng.uniform(0.05, 2.0)) * w / rate
        res = [int(b) for b in rng.integers(0, 2, n)]
        last, _ = S.simulate([w] * n, [L] * n, res, 2, rate, steps=4)
        k = sum(res)
        assert n * L * (1 - 1e-12) <= last <= (n * L + S.delta_overhead(n, k, w, rate)) * (1 + 1e-12)
        # any streamed layer made resident: never slower (non-uniform layers too)
        ws = list(rng.uniform(1e6, 5e7, n))
        cs = list(rng.uniform(1e-5, 1e-3, n))
        base, _ = S.simulate(ws, cs, res, 2, rate, steps=4)
        for i in range(n):
            if not res[i]:
                more = list(res)
                more[i] = 1
                t2, _ = S.simulate(ws, cs, more, 2, rate, steps=4)
                assert t2 <= base * (1 + 1e-12)


def test_device_bytes_and_tmin():
    w = [30.0, 50.0, 20.0]
    assert S.device_bytes(w, [0, 0, 0], 7.0) == S.t_min(50.0, 7.0) == 107.0
    assert S.device_bytes(w, [0, 1, 0], 7.0) == 50.0 + 2 * 30.0 + 7.0
    assert S.device_bytes(w, [1, 1, 1], 7.0) == 107.0
    assert S.t_min(50.0, 7.0, slots=3) == 157.0


def test_bruteforce_plan_respects_budget():
    rng = np.random.default_rng(2)
    w = list(rng.uniform(1e6, 4e7, 6))
    c = list(rng.uniform(1e-4, 8e-4, 6))
    a = 5e6
    tmin = S.t_min(max(w), a)
    for budget in (tmin, tmin + 3e7, sum(w) + a):
        (key, bits) = S.best_plan_bruteforce(w, c, 2, 50e9, budget, a)
        assert S.device_bytes(w, bits, a) <= budget
        assert key[0] >= sum(c) - 1e-12
    (key, bits) = S.best_plan_bruteforce(w, c, 2, 50e9, sum(w) + a, a)
    assert key[0] == pytest.approx(sum(c), rel=1e-9)
