"""Oracle of the weight-streaming model (test infrastructure only).

The paper's second memory tool (Sec. 4, weight-streaming paragraph) keeps a
resident subset of the layer weights in device memory and copies the others
from pinned host memory ahead of their matrix multiply, so that the copies
overlap the compute. Its quantities, written out here by their definitions:

* reservoir decay factor  lambda = L * M / W   (L: compute time between
  successive matrix multiplies, M: host-to-device rate, W: layer weight size);
  lambda >= 1 hides every copy behind compute;
* overhead when lambda < 1: Delta = (N - K) * W / M  (N layers, K of them
  fully overlapped), the cost of the copies that are waited for;
* minimum device memory  T_min = 2 * W_max + A_max  (the layer being computed
  and the next one both need a buffer, plus the peak activation).

`simulate` is a plain discrete-event model of the same schedule the library
enqueues: layers run in order, step after step; every streamed occurrence
takes the next of `slots` device buffers in turn; one copy engine serves the
copies first come first served; a copy may start once its buffer's previous
occupant has finished computing; a layer computes once the layer before it
has finished and its weights are in place. Only the tests use this module.
"""
from __future__ import annotations

import itertools


def reservoir_lambda(compute_s: float, rate_bps: float, w_bytes: float) -> float:
    """lambda = L * M / W."""
    return compute_s * rate_bps / w_bytes


def delta_overhead(n_layers: int, k_overlapped: int, w_bytes: float, rate_bps: float) -> float:
    """Delta = (N - K) * W / M."""
    return (n_layers - k_overlapped) * w_bytes / rate_bps


def t_min(w_max: float, a_max: float, slots: int = 2) -> float:
    """Minimum device memory with `slots` streaming buffers (2 in the paper)."""
    return slots * w_max + a_max


def device_bytes(w_bytes, resident, a_max: float, slots: int = 2) -> float:
    """Device memory of a plan: resident weights, the streaming buffers (each
    as large as the largest streamed layer) and the peak activation."""
    streamed = [w for w, r in zip(w_bytes, resident) if not r]
    return sum(w for w, r in zip(w_bytes, resident) if r) + (slots * max(streamed) if streamed else 0.0) + a_max


def simulate(w_bytes, compute_s, resident, slots: int, rate_bps: float, steps: int = 3):
    """Return (per-step time of the last step, finish time of every step)."""
    n = len(w_bytes)
    compute_end = []          # per streamed occurrence: finish time of its compute
    copy_free = 0.0           # when the copy engine is idle again
    t = 0.0                   # finish time of the previous layer's compute
    step_end = []
    occ = 0                   # streamed occurrences so far
    for _ in range(steps):
        for i in range(n):
            ready = 0.0
            if not resident[i]:
                # buffer (occ % slots) is free once occurrence occ - slots has computed
                buf_free = compute_end[occ - slots] if occ >= slots else 0.0
                start = max(copy_free, buf_free)
                copy_free = start + w_bytes[i] / rate_bps
                ready = copy_free
            t = max(t, ready) + compute_s[i]
            if not resident[i]:
                compute_end.append(t)
                occ += 1
        step_end.append(t)
    last = step_end[-1] - (step_end[-2] if steps > 1 else 0.0)
    return last, step_end


def best_plan_bruteforce(w_bytes, compute_s, slots: int, rate_bps: float, budget: float, a_max: float,
                         steps: int = 3):
    """Smallest steady-state step time over every resident subset that fits
    the budget (ties: fewer device bytes). Exponential: small cases only."""
    n = len(w_bytes)
    best = None
    for bits in itertools.product((0, 1), repeat=n):
        dev = device_bytes(w_bytes, bits, a_max, slots)
        if dev > budget:
            continue
        tstep, _ = simulate(w_bytes, compute_s, bits, slots, rate_bps, steps)
        key = (round(tstep, 12), dev)
        if best is None or key < best[0]:
            best = (key, bits)
    return best
