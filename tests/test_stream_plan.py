"""The library's weight-streaming model and planner (host code, no GPU)
against the oracle's discrete-event model (oracle/streaming.py), and the
host-side checks of qg_run_layers (every call here fails validation before
any HIP call, so no GPU is touched)."""
import ctypes

import numpy as np
import pytest

import paper_2609_21849_amd as q
from oracle import streaming as S

OK, INVALID, UNSUP, SHAPE, SMALL = 0, 1, 2, 3, 4


def _case(rng, n):
    return (list(rng.uniform(1e6, 5e7, n)), list(rng.uniform(1e-5, 1.5e-3, n)))


def test_simulate_matches_oracle():
    rng = np.random.default_rng(11)
    for _ in range(300):
        n = int(rng.integers(0, 12))
        slots = int(rng.integers(1, 4))
        w, c = _case(rng, n)
        res = [int(b) for b in rng.integers(0, 2, n)]
        steps = int(rng.integers(1, 5))
        st, t = q.qg_stream_simulate(w, c, res, slots, 50e9, steps)
        assert st == OK
        if n == 0:
            assert t == 0.0
            continue
        ref, _ = S.simulate(w, c, res, slots, 50e9, steps)
        assert t == pytest.approx(ref, rel=1e-12, abs=1e-18)


@pytest.mark.parametrize("seed", range(4))
def test_plan_is_optimal_for_small_models(seed):
    rng = np.random.default_rng(100 + seed)
    for _ in range(60):
        n = int(rng.integers(1, 9))
        slots = int(rng.integers(1, 4))
        w, c = _case(rng, n)
        a = float(rng.uniform(0, 2e7))
        lo = min(S.t_min(max(w), a, slots), sum(w) + a)
        budget = float(rng.uniform(0.9 * lo, sum(w) + a + 1e7))
        st, res, t, dev = q.qg_stream_plan(w, c, slots, 50e9, budget, a, check=False)
        best = S.best_plan_bruteforce(w, c, slots, 50e9, budget, a)
        if best is None:
            assert st == SMALL
            continue
        assert st == OK
        assert dev <= budget and dev == pytest.approx(S.device_bytes(w, res, a, slots), rel=1e-12)
        ref, _ = S.simulate(w, c, res, slots, 50e9, 3)
        assert t == pytest.approx(ref, rel=1e-12)
        assert t == pytest.approx(best[0][0], rel=1e-6)          # the best step time


def test_plan_for_a_large_model_is_valid_and_no_worse_than_trivial_plans():
    rng = np.random.default_rng(7)
    n = 40
    w, c = _case(rng, n)
    a = 1e7
    for frac in (0.0, 0.2, 0.5, 0.8, 1.0):
        budget = S.t_min(max(w), a) + frac * sum(w)
        st, res, t, dev = q.qg_stream_plan(w, c, 2, 50e9, budget, a)
        assert st == OK and dev <= budget
        ref, _ = S.simulate(w, c, res, 2, 50e9, 3)
        assert t == pytest.approx(ref, rel=1e-12)
        streamed_all, _ = S.simulate(w, c, [0] * n, 2, 50e9, 3)
        assert t <= streamed_all * (1 + 1e-12)
        assert t >= sum(c) * (1 - 1e-12)
    # everything fits: no exposed copy time
    st, res, t, dev = q.qg_stream_plan(w, c, 2, 50e9, sum(w) + a, a)
    assert t == pytest.approx(sum(c), rel=1e-12)


def test_uniform_layers_reproduce_the_closed_forms():
    # lambda >= 1: a fully streamed model runs at the compute time; lambda < 1:
    # the reservoir drains and the plan keeps layers resident to cut the exposed time
    n, w, rate = 8, 28e6, 55e9
    tau = w / rate
    st, t = q.qg_stream_simulate([w] * n, [1.2 * tau] * n, [0] * n, 2, rate, 4)
    assert t == pytest.approx(n * 1.2 * tau, rel=1e-12)
    st, t = q.qg_stream_simulate([w] * n, [0.3 * tau] * n, [0] * n, 2, rate, 4)
    assert t == pytest.approx(n * tau, rel=1e-12)
    # T_min: below two slots of the largest weight plus activations nothing fits
    a = 5e6
    st, *_ = q.qg_stream_plan([w] * n, [0.3 * tau] * n, 2, rate, S.t_min(w, a) - 1.0, a, check=False)
    assert st == SMALL
    st, res, t, dev = q.qg_stream_plan([w] * n, [0.3 * tau] * n, 2, rate, S.t_min(w, a), a)
    assert st == OK and sum(res) == 0 and dev == S.t_min(w, a)


def test_simulate_and_plan_validation():
    assert q.qg_stream_simulate([1.0], [1.0], [0], 0, 1e9, check=False)[0] == INVALID   # streamed, no slot
    assert q.qg_stream_simulate([1.0], [1.0], [1], 0, 1e9, check=False)[0] == OK        # nothing streamed
    assert q.qg_stream_simulate([1.0], [1.0], [0], 2, 0.0, check=False)[0] == INVALID
    assert q.qg_stream_simulate([-1.0], [1.0], [0], 2, 1e9, check=False)[0] == INVALID
    assert q.qg_stream_simulate([1.0], [float("nan")], [0], 2, 1e9, check=False)[0] == INVALID
    assert q.qg_stream_simulate([1.0], [1.0], [0], 2, 1e9, steps=0, check=False)[0] == INVALID
    assert q.qg_stream_plan([1.0], [1.0], 0, 1e9, 10.0, 0.0, check=False)[0] == INVALID
    assert q.qg_stream_plan([1.0], [1.0], 2, 1e9, -1.0, 0.0, check=False)[0] == INVALID
    assert q.qg_stream_plan([], [], 2, 1e9, 0.0, 0.0, check=False)[0] == OK


# ---------------------------------------------------------------- qg_run_layers host checks
P = 0x100000   # fake, aligned pointers that validation never dereferences


def _layer(**kw):
    d = dict(x=P, a_fmt=q.QG_FMT_FP8_E4M3, a_codes=P, a_block_scales=None, a_tensor_scale=P,
             w_fmt=q.QG_FMT_FP8_E4M3, w_packed=P, w_packed_bytes=1 << 20, resident=0,
             m=64, n=256, k=256, y=P, y_dtype=q.QG_OUT_BF16)
    d.update(kw)
    return q.StreamLayer(**d)


def _run(layers, n_slots=2, slot_bytes=1 << 20, slots=None, cursor=0, events=True):
    slots = [P + 0x10000 * i for i in range(n_slots)] if slots is None else slots
    ev = [0x1000 + i for i in range(n_slots)] if events else [0] * n_slots
    cur = ctypes.c_int32(cursor)
    return q.qg_run_layers(layers, slots, slot_bytes, ev, ev, cur, compute_stream=0, copy_stream=0, check=False)


def test_run_layers_validation():
    assert _run([_layer()], n_slots=0) == INVALID                         # streamed, no slots
    assert _run([_layer()], slots=[P + 16, P]) == INVALID                   # slot alignment
    assert _run([_layer()], cursor=2) == INVALID                            # cursor out of range
    assert _run([_layer()], events=False) == INVALID                        # missing events
    assert _run([_layer()], slot_bytes=4096) == SMALL                       # weight larger than a slot
    assert _run([_layer(w_packed=None)]) == INVALID
    assert _run([_layer(n=40)]) == SHAPE                                    # the GEMM's own checks
    assert _run([_layer(a_fmt=q.QG_FMT_NVFP4, w_fmt=q.QG_FMT_FP8_E4M3)]) == INVALID  # NVFP4 quantize needs scales
    assert _run([_layer(a_fmt=q.QG_FMT_NVFP4, a_block_scales=P, w_fmt=q.QG_FMT_FP8_E4M3)]) == UNSUP
    assert _run([_layer(a_tensor_scale=None)]) == INVALID                   # FP8 quantize needs a scale
    assert _run([_layer(resident=1, w_packed=P + 64)], n_slots=0) == INVALID  # resident weight alignment
    # one bad layer anywhere rejects the whole call (nothing is enqueued)
    assert _run([_layer(resident=1), _layer(k=200)]) == SHAPE
