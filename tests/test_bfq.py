"""Batch-aware fair queueing (BFQ): the oracle against what the paper and
the mathematics fix, and the library's scheduler (C ABI, host only) against
the oracle, decision by decision.  CPU only."""
import json
import math
import os
import time
from fractions import Fraction

import numpy as np
import pytest

from oracle import bfq_oracle as BO
from paper_2606_09643_amd import binding as B

INF = float("inf")


# --------------------------------------------------------------------------
# oracle pins
# --------------------------------------------------------------------------

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden", "bfq_worked_examples.json")


def _worked_examples():
    with open(GOLDEN) as f:
        return json.load(f)["examples"]


class _OracleView:
    """The oracle's scheduler behind the library binding's query calls."""

    def __init__(self, weights, batch_time, b_max):
        self.q = BO.BFQ(weights, batch_time, b_max)

    def enqueue(self, task, req, arrival):
        self.q.enqueue(task, req, arrival, INF)

    def next_batch(self, now):
        return self.q.next_batch(now)

    def charge(self, task, service):
        self.q.charge(task, service)

    def queued(self, task):
        return self.q.queued(task)

    def tags(self, task, k):
        r = self.q.queues[task][k]
        return r.S, r.F

    def v(self):
        return self.q.v()


@pytest.mark.parametrize("impl", ["oracle", "library"])
@pytest.mark.parametrize("ex", _worked_examples(), ids=lambda e: e["name"])
def test_worked_examples_by_hand(ex, impl):
    """The hand-worked tag sequences of tests/golden/bfq_worked_examples.json
    (Eq. 1-2 tags, the Eq. 3 re-tagging after a batch, token-level charging;
    Section 4.2), replayed step by step on the oracle and on the library.
    The global tag v is checked on the oracle (the library shows it through
    the tags of later arrivals)."""
    fr = lambda x: float(Fraction(x))
    w = [fr(x) for x in ex["weights"]]
    t = [fr(x) for x in ex["batch_time"]]
    q = _OracleView(w, t, ex["b_max"]) if impl == "oracle" else B.BFQ(w, t, ex["b_max"])
    for i, st in enumerate(ex["steps"]):
        op, where = st[0], f"{ex['name']} step {i}: {st}"
        if op == "enqueue":
            q.enqueue(st[1], st[2], fr(st[3]))
        elif op == "batch":
            assert q.next_batch(fr(st[1])) == [tuple(x) for x in st[2]], where
        elif op == "charge":
            q.charge(st[1], fr(st[2]))
        elif op == "tags":
            assert q.queued(st[1]) == len(st[2]), where
            for k, (s_, f_) in enumerate(st[2]):
                s, f = q.tags(st[1], k)
                assert math.isclose(s, fr(s_), abs_tol=1e-12) and math.isclose(f, fr(f_), abs_tol=1e-12), where
        elif op == "v":
            if impl == "oracle":
                assert math.isclose(q.v(), fr(st[1]), abs_tol=1e-12), where
        else:
            raise AssertionError(f"unknown step {op}")


@pytest.mark.parametrize("weights", [[1.0, 1.0], [1.0, 2.0, 4.0], [0.5, 1.0, 2.0, 4.0], [4.0, 1.0]])
def test_oracle_with_single_request_batches_is_textbook_stfq(weights):
    """b_max = 1 and a constant per-request service time: BFQ's dispatch
    order equals start-time fair queueing's (start tags (k-1) l / w_i for a
    backlogged task; dyadic weights so every tag is exact)."""
    counts = [13, 7, 9, 5][:len(weights)]
    q = BO.BFQ(weights, [0.0, 1.0], 1)
    for t, c in enumerate(counts):
        for k in range(c):
            q.enqueue(t, 100 * t + k, 0.0, INF)
    order = []
    while True:
        b = q.next_batch(0.0)
        if not b:
            break
        assert len(b) == 1
        order.append(b[0][1])
    assert order == BO.stfq_order(counts, weights)


@pytest.mark.parametrize("b_max", [1, 4, 32])
def test_oracle_service_shares_follow_weights_under_backlog(b_max):
    """Every task kept backlogged: the dispatched requests per task are in
    proportion to the weights (within a few batches' worth)."""
    w = [1.0, 2.0, 3.0, 6.0]
    T = [0.0] + [1.0 + 0.2 * b for b in range(1, b_max + 1)]   # sublinear batches
    q = BO.BFQ(w, T, b_max)
    nxt = [0] * len(w)
    for t in range(len(w)):
        for _ in range(2 * b_max + 4):
            q.enqueue(t, nxt[t], 0.0, INF)
            nxt[t] += 1
    served = np.zeros(len(w))
    now = 0.0
    for _ in range(max(4000 // b_max, 200)):
        batch = q.next_batch(now)
        now += T[len(batch)]
        for _, t in batch:
            served[t] += 1
            q.enqueue(t, nxt[t], now, INF)     # keep the task backlogged
            nxt[t] += 1
    share = served / served.sum()
    want = np.array(w) / sum(w)
    assert np.all(np.abs(share - want) <= max(0.01, 3.0 * b_max / served.sum())), (share, want)


def test_oracle_admission_respects_deadlines_and_stops_at_the_first_misfit():
    rng = np.random.default_rng(3)
    T = [0.0] + [1.0 + 0.5 * b for b in range(1, 17)]
    q = BO.BFQ([1.0, 1.0, 2.0], T, 16)
    for k in range(60):
        t = int(rng.integers(3))
        q.enqueue(t, k, 0.0, float(rng.uniform(1.0, 9.0)))
    now = 0.0
    while True:
        cand = sorted((r for qq in q.queues for r in qq), key=lambda r: (r.S, r.task, r.seq))
        dl = {r.req: r.deadline for r in cand}
        batch = q.next_batch(now)
        if not batch:
            break
        b = len(batch)
        assert [r.req for r in cand[:b]] == [req for req, _ in batch]     # a prefix in tag order
        if b > 1:
            assert now + T[b] <= min(dl[req] for req, _ in batch)
        if b < 16 and b < len(cand):                                      # why the scan stopped
            assert now + T[b + 1] > min([dl[req] for req, _ in batch] + [cand[b].deadline])
        now += T[b]


# --------------------------------------------------------------------------
# library (C ABI) against the oracle
# --------------------------------------------------------------------------

def _simulate(sched, trace, T):
    """Drives a scheduler over an arrival trace: the server takes the next
    batch whenever it is idle and queues are non-empty; returns the batch
    sequence and the dispatch times."""
    out = []
    now, i = 0.0, 0
    while True:
        while i < len(trace) and trace[i][0] <= now:
            a, t, req, dl = trace[i]
            sched.enqueue(t, req, a, dl)
            i += 1
        batch = sched.next_batch(now)
        if batch:
            out.append((now, batch))
            now += T[len(batch)]
        elif i < len(trace):
            now = trace[i][0]
        else:
            break
    return out


def _trace(seed, n_tasks, n_req, rate, slo):
    rng = np.random.default_rng(seed)
    lam = rng.uniform(0.2, 1.0, n_tasks)
    lam = rate * lam / lam.sum()
    ev = []
    for t in range(n_tasks):
        at = np.cumsum(rng.exponential(1.0 / lam[t], n_req // n_tasks + 1))
        for a in at:
            ev.append((float(a), t, float(a) + slo[t]))
    ev.sort()
    return [(a, t, k, dl) for k, (a, t, dl) in enumerate(ev[:n_req])]


@pytest.mark.parametrize("seed,n_tasks,b_max,rate", [(1, 1, 1, 0.8), (2, 4, 8, 3.0), (3, 16, 32, 20.0),
                                                     (4, 128, 256, 150.0), (5, 7, 5, 1.5)])
def test_library_matches_oracle_on_poisson_traces(seed, n_tasks, b_max, rate):
    """Same arrivals, weights, batch-time table and deadlines: the library
    forms exactly the oracle's batches (request ids and order) and holds the
    same tags afterwards."""
    rng = np.random.default_rng(100 + seed)
    w = rng.choice([0.5, 1.0, 1.5, 2.0, 3.0], n_tasks)
    T = [0.0] + [1.0 + 0.15 * b ** 0.8 for b in range(1, b_max + 1)]
    slo = rng.uniform(3.0, 30.0, n_tasks)
    trace = _trace(seed, n_tasks, 3000, rate, slo)
    lib = B.BFQ(w, T, b_max, max_queued=4096)
    ref = BO.BFQ(w, T, b_max)
    got = _simulate(lib, trace, T)
    want = _simulate(ref, trace, T)
    assert got == want
    assert sum(len(b) for _, b in got) == len(trace)
    # the tags left in the queues (none here: the trace drains) and a fresh
    # arrival's tags agree exactly
    for t in range(n_tasks):
        lib.enqueue(t, -1, want[-1][0], INF)
        ref.enqueue(t, -1, want[-1][0], INF)
        r = ref.queues[t][-1]
        assert lib.tags(t, lib.queued(t) - 1) == (r.S, r.F)


def test_library_tags_match_oracle_while_backlogged():
    w = [1.0, 2.0, 3.0]
    T = [0.0, 1.0, 1.4, 1.7, 1.9]
    lib, ref = B.BFQ(w, T, 4, max_queued=64), BO.BFQ(w, T, 4)
    for k in range(30):
        t = k % 3
        lib.enqueue(t, k, 0.0, INF)
        ref.enqueue(t, k, 0.0, INF)
    now = 0.0
    for _ in range(5):
        assert lib.next_batch(now) == ref.next_batch(now)
        now += 1.0
        for t in range(3):
            assert lib.queued(t) == ref.queued(t)
            for k, r in enumerate(ref.queues[t]):
                assert lib.tags(t, k) == (r.S, r.F)


def test_library_batches_plan_like_the_oracle():
    """A formed batch goes straight to vfm_plan: segments follow the tasks."""
    from oracle import vfm_oracle as O
    w = [1.0] * 8
    T = [0.0] + [1.0 + 0.1 * b for b in range(1, 65)]
    q = B.BFQ(w, T, 64)
    rng = np.random.default_rng(9)
    lens = {}
    for k in range(200):
        t = int(rng.integers(8))
        lens[k] = int(rng.integers(1, 300))
        q.enqueue(t, k, 0.0, INF)
    batch = q.next_batch(0.0)
    task_id = np.array([t for _, t in batch], np.int32)
    seq_len = np.array([lens[r] for r, _ in batch], np.int32)
    host = B.vfm_plan(task_id, seq_len, 8)
    pl = O.plan(task_id, seq_len, 8)
    n = len(batch)
    p = B.VFM_PLAN_HEADER
    assert np.array_equal(host[p:p + n], pl["order"])


def test_library_rejects_bad_arguments():
    lib = B.lib()
    n = B.C.c_size_t()
    w = np.array([1.0, 0.0])
    T = np.array([0.0, 1.0])
    cfg = B.vfm_bfq_config(2, 1, 4, w.ctypes.data_as(B.C.POINTER(B.C.c_double)),
                           T.ctypes.data_as(B.C.POINTER(B.C.c_double)))
    assert lib.vfm_bfq_state_size(B.C.byref(cfg), B.C.byref(n)) == B.VFM_OK
    buf = np.zeros(n.value // 8 + 1, np.float64)
    assert lib.vfm_bfq_init(B.C.byref(cfg), buf.ctypes.data, buf.nbytes) == B.VFM_ERR_SHAPE   # weight 0
    assert lib.vfm_bfq_init(B.C.byref(cfg), None, buf.nbytes) == B.VFM_ERR_ARG
    bad = B.vfm_bfq_config(0, 1, 4, cfg.weight, cfg.batch_time)
    assert lib.vfm_bfq_state_size(B.C.byref(bad), B.C.byref(n)) == B.VFM_ERR_SHAPE
    q = B.BFQ([1.0, 1.0], [0.0, 1.0, 1.5], 2, max_queued=2)
    with pytest.raises(B.VfmError):
        q.enqueue(2, 0, 0.0)                     # task out of range
    q.enqueue(0, 0, 0.0)
    q.enqueue(0, 1, 0.0)
    with pytest.raises(B.VfmError):
        q.enqueue(0, 2, 0.0)                     # queue full
    req = np.zeros(1, np.int64)
    tsk = np.zeros(1, np.int32)
    cnt = B.C.c_int32()
    assert lib.vfm_bfq_next_batch(q.state.ctypes.data, 0.0, req.ctypes.data, tsk.ctypes.data, 1,
                                  B.C.byref(cnt)) == B.VFM_ERR_SHAPE   # capacity < b_max
    assert q.queued(0) == 2                      # nothing changed
    assert lib.vfm_bfq_enqueue(None, 0, 0, 0.0, 0.0) == B.VFM_ERR_ARG
    assert q.next_batch(0.0) == [(0, 0), (1, 0)]
    assert q.next_batch(1.0) == []


def test_library_decision_time():
    """Host cost of one scheduling decision at the decode workload's scale
    (128 tasks, b_max 256, ~512 queued): printed, and bounded well below the
    paper's measured per-request scheduler overhead (0.35 ms on average)."""
    n_tasks, b_max = 128, 256
    T = [0.0] + [1.0 + 0.01 * b for b in range(1, b_max + 1)]
    q = B.BFQ(np.linspace(0.5, 2.0, n_tasks), T, b_max, max_queued=1024)
    rng = np.random.default_rng(0)
    k = 0
    for _ in range(512):
        q.enqueue(int(rng.integers(n_tasks)), k, 0.0, INF)
        k += 1
    reps, spent = 200, 0.0
    for r in range(reps):
        t0 = time.perf_counter()
        batch = q.next_batch(float(r))
        spent += time.perf_counter() - t0
        assert len(batch) == b_max
        for _, t in batch:                        # refill what left (not timed)
            q.enqueue(t, k, float(r), INF)
            k += 1
    dt = spent / reps
    print(f"BFQ: {dt * 1e6:.1f} us per batch decision ({n_tasks} tasks, b_max {b_max}, 512 queued)")
    assert dt < 1e-3


def test_oracle_charging_every_token_keeps_weighted_shares():
    """Two always-backlogged token-based tasks (weights 1 and 3), b_max 1,
    every dispatched request then charged a variable decode length: the
    service each task receives (its requests' lengths) follows the weights
    to within one request's length."""
    rng = np.random.default_rng(7)
    q = BO.BFQ([1.0, 3.0], [0.0, 1.0], 1)
    lens = {}
    k = 0
    for _ in range(50):
        for t in (0, 1):
            q.enqueue(t, k, 0.0, INF)
            lens[k] = float(rng.integers(1, 20))
            k += 1
    got = [0.0, 0.0]
    for _ in range(60):
        (req, t), = q.next_batch(0.0)
        q.charge(t, lens[req] - 1.0)           # T(1) = 1 already counted at dispatch
        got[t] += lens[req]
    assert abs(got[1] / 3.0 - got[0]) <= 20.0


def test_library_charge_matches_oracle():
    """The library's charge gives bit-identical tags and batches to the
    oracle's on a random mix of arrivals, batches and charges."""
    rng = np.random.default_rng(11)
    w = [1.0, 2.0, 0.5, 3.0]
    T = [0.0] + [1.0 + 0.2 * b for b in range(1, 9)]
    lib, ref = B.BFQ(w, T, 8), BO.BFQ(w, T, 8)
    k = 0
    for step in range(400):
        now = float(step)
        for _ in range(int(rng.integers(0, 4))):
            t = int(rng.integers(0, 4))
            lib.enqueue(t, k, now, INF)
            ref.enqueue(t, k, now, INF)
            k += 1
        if rng.random() < 0.5:
            assert lib.next_batch(now) == ref.next_batch(now)
        t = int(rng.integers(0, 4))
        s = float(rng.uniform(0.0, 5.0))
        lib.charge(t, s)
        ref.charge(t, s)
        for tt in range(4):
            for j in range(ref.queued(tt)):
                r = ref.queues[tt][j]
                assert lib.tags(tt, j) == (r.S, r.F)
    lib_state = lib.state.copy()
    with pytest.raises(B.VfmError):
        lib.charge(4, 1.0)
    with pytest.raises(B.VfmError):
        lib.charge(0, -1.0)
    with pytest.raises(B.VfmError):
        lib.charge(0, float("nan"))
    assert np.array_equal(lib.state, lib_state)
