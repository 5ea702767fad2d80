"""Plain Python oracle of BFQ, the batch-aware fair queueing scheduler that
forms the mixed-task batches (paper Section 4.2, "Batch-aware Fair
Scheduling", Eq. 1-3, and the paragraph on the service-time mismatch).

TEST INFRASTRUCTURE ONLY.  Only ``tests/`` may import this module; the
product scheduler (``vfm_bfq_*`` in the C library) never calls it, and this
module imports nothing from the product package.

What it computes, step by step in the paper's order:

* Each task i has a weight w_i.  Request j of task i gets, on arrival, a
  start tag S = max(F of the task's previous request, v) and a finish tag
  F = S + l / w_i (Eq. 1, 2).  v is the global tag at arrival: the largest
  finish tag over the tasks' most recently dispatched requests (0 before any
  dispatch).  l is the expected service time of one request, T(1).
* A batch is formed from the queued requests in increasing start tag,
  extended one request at a time until it holds b_max requests, or until
  admitting the next request would make the batch's estimated completion
  time now + T(b) pass the deadline of any request in it.
* After the batch of b requests runs, every task that contributed to it has
  its tags recomputed with the batch-dependent per-request service time
  l(b) = T(b) / b (Eq. 3): the dispatched requests (their realised service)
  and then the task's queued ones, each chained as in Eq. 1 from its own
  arrival-time v.
* Token-based FMs are charged their token-level work in service-time units
  as it is realised (``charge``): it extends the task's last dispatched
  request, and the task's queued requests follow.

Readings where the paper is silent (each also a parameter of the C ABI):
T(b), the service time of a batch of b requests, is a caller-supplied table;
l(b) = T(b) / b is the same for every task (all requests share the backbone
and the per-task adapter difference is applied within the batch); ties in the
start tag go to the lower task id, then to the earlier request of that task;
the first request of a batch is always admitted, so the scheduler is
work-conserving; the scan stops at the first request that cannot be admitted.

``stfq_order`` is the textbook start-time fair queueing order of a set of
requests that are all queued at time 0 (every task backlogged), written
independently as the closed form S = (j - 1) * l / w_i; BFQ with b_max = 1
must dispatch in exactly that order (the reduction the paper starts from).
"""


class Request:
    __slots__ = ("req", "task", "arrival", "deadline", "va", "S", "F", "seq")

    def __init__(self, req, task, arrival, deadline, va, seq):
        self.req, self.task, self.arrival, self.deadline = req, task, arrival, deadline
        self.va, self.seq = va, seq
        self.S = self.F = 0.0


class BFQ:
    def __init__(self, weights, batch_time, b_max):
        self.w = [float(x) for x in weights]
        self.T = [float(x) for x in batch_time]   # T[b], b = 1..b_max (T[0] unused)
        self.b_max = int(b_max)
        n = len(self.w)
        self.queues = [[] for _ in range(n)]      # per task, arrival order
        self.f_last = [0.0] * n                   # F of the task's last request (queued or dispatched)
        self.f_disp = [0.0] * n                   # F of the task's most recently dispatched request
        self.dispatched = [False] * n
        self.seq = 0

    def v(self):
        """Global tag: the largest finish tag of the tasks' last dispatched requests."""
        tags = [f for f, d in zip(self.f_disp, self.dispatched) if d]
        return max(tags) if tags else 0.0

    def enqueue(self, task, req, arrival, deadline):
        r = Request(req, task, float(arrival), float(deadline), self.v(), self.seq)
        self.seq += 1
        r.S = max(self.f_last[task], r.va)                 # Eq. 1
        r.F = r.S + self.T[1] / self.w[task]               # Eq. 2, single-request service
        self.f_last[task] = r.F
        self.queues[task].append(r)

    def queued(self, task):
        return len(self.queues[task])

    def next_batch(self, now):
        """The next batch as [(request id, task id)], removed from the queues."""
        cand = sorted((r for q in self.queues for r in q), key=lambda r: (r.S, r.task, r.seq))
        batch = []
        for r in cand:
            if len(batch) == self.b_max:
                break
            done = now + self.T[len(batch) + 1]
            if batch and any(done > x.deadline for x in batch + [r]):
                break
            batch.append(r)
        if not batch:
            return []
        b = len(batch)
        l_b = self.T[b] / b                                # per-request service in this batch
        for t in sorted({r.task for r in batch}):
            mine = [r for r in batch if r.task == t]       # the task's first len(mine) queued
            q = self.queues[t]
            assert q[:len(mine)] == mine
            rest = q[len(mine):]
            prev = self.f_disp[t] if self.dispatched[t] else 0.0
            for r in mine + rest:                          # Eq. 3 re-tagging, chained as Eq. 1
                r.S = max(prev, r.va)
                r.F = r.S + l_b / self.w[t]
                prev = r.F
            self.f_disp[t] = mine[-1].F
            self.dispatched[t] = True
            self.f_last[t] = prev
            self.queues[t] = rest
        return [(r.req, r.task) for r in batch]


    def charge(self, task, service):
        """Token-based FMs (Section 4.2: token-level work charged in
        service-time units): `service` of realised work is added to the
        task's last dispatched request, whose finish tag moves by
        service / w; the task's queued requests keep their service lengths
        and are chained after it as in Eq. 1."""
        prev = (self.f_disp[task] if self.dispatched[task] else 0.0) + service / self.w[task]
        self.f_disp[task] = prev
        self.dispatched[task] = True
        for r in self.queues[task]:
            length = r.F - r.S
            r.S = max(prev, r.va)
            r.F = r.S + length
            prev = r.F
        self.f_last[task] = prev


def stfq_order(counts, weights, l=1.0):
    """Dispatch order (task ids) of textbook STFQ over counts[i] requests of
    task i, all backlogged from time 0: the k-th request of task i has start
    tag k * l / w_i; ties by task id, then k."""
    tags = [(k * l / float(weights[i]), i, k) for i in range(len(counts)) for k in range(counts[i])]
    return [i for _, i, _ in sorted(tags)]
