"""Host-side scheduling of the continuous-batching loop (no GPU): which
prompts join the running batch under the sequence slots, the per-step token
budget and the page commitments, FIFO and BFQ admission, and that a request
that can never fit is refused up front."""
import numpy as np
import pytest

from paper_2606_09643_amd import binding as B
from paper_2606_09643_amd import runner as R
from paper_2606_09643_amd import workloads as wl


class _StubModel:
    """Just what the batcher reads before a step runs."""

    def __init__(self):
        self.w = wl.WORKLOADS[5].replace(n_layers=1, d=256, n_heads=2, head_dim=128, d_ff=512, n_tasks=3)
        self.n_layers = 1
        self.cfg = R.cfg_for(self.w)


def _batcher(**kw):
    args = dict(page_size=16, n_pages=12, max_seqs=3, max_step_tokens=64, max_pages=6, device="cpu")
    args.update(kw)
    return R.ContinuousBatcher(_StubModel(), emb=None, **args)


def test_fifo_admission_respects_slots_tokens_and_pages():
    cb = _batcher()
    # budgets (pages of 16 for prompt + new - 1 tokens): 1, 2, 1, 3, 2
    for rid, (L, n) in enumerate([(5, 6), (17, 3), (1, 8), (33, 4), (9, 9)]):
        cb.submit(rid, rid % 3, np.zeros(L, np.int32), n)
    new = cb._admit(0.0)
    # slots: 3; tokens 5 + 17 + 1 = 23 <= 64; pages 1 + 2 + 1 = 4 <= 12
    assert [s.rid for s in new] == [0, 1, 2] and cb.committed == 4
    assert [s.rid for s in cb.waiting] == [3, 4]
    assert cb._admit(0.0) == []                      # no slot free
    # a finished sequence frees its slot and pages
    s0 = cb.running[0]
    cb.alloc.release(s0.slot)
    cb.free_slots.append(s0.slot)
    cb.committed -= s0.budget
    cb.running.remove(s0)
    new = cb._admit(0.0)                             # 2 decode rows + 33 prompt tokens <= 64
    assert [s.rid for s in new] == [3] and cb.committed == 6


def test_fifo_admission_stops_at_the_first_prompt_that_does_not_fit():
    cb = _batcher(max_step_tokens=40, chunk_prompts=False)
    for rid, L in enumerate([30, 20, 5]):
        cb.submit(rid, 0, np.zeros(L, np.int32), 2)
    assert [s.rid for s in cb._admit(0.0)] == [0]    # 30 + 20 > 40: FIFO does not skip ahead
    assert [s.rid for s in cb.waiting] == [1, 2]


def test_chunked_prompts_join_with_what_is_left_of_the_budget():
    cb = _batcher(max_step_tokens=40, max_pages=6)
    for rid, L in enumerate([30, 20, 5]):
        cb.submit(rid, 0, np.zeros(L, np.int32), 2)
    # 30 tokens, then 10 of the 20-token prompt; the third has no token left this step
    assert [s.rid for s in cb._admit(0.0)] == [0, 1]
    assert [s.rid for s in cb.waiting] == [2]


def test_page_commitment_holds_back_prompts():
    cb = _batcher(n_pages=4, max_pages=4, max_step_tokens=1000)
    cb.submit(0, 0, np.zeros(40, np.int32), 10)      # 49 tokens: 4 pages
    cb.submit(1, 1, np.zeros(3, np.int32), 2)        # 1 page
    assert [s.rid for s in cb._admit(0.0)] == [0]
    assert cb.committed == 4 and [s.rid for s in cb.waiting] == [1]


def test_bfq_admission_takes_whole_batches_in_tag_order():
    bfq = B.BFQ([1.0, 1.0, 1.0], [0.0, 1.0, 1.5], b_max=2)
    cb = _batcher(bfq=bfq, max_seqs=4)
    for rid, task in enumerate([0, 0, 1, 2]):
        cb.submit(rid, task, np.zeros(4, np.int32), 3)
    new = cb._admit(0.0)
    # start tags: task 0: 0, 1; task 1: 0; task 2: 0 -> batches (0, 2) then (3, 1)
    assert [s.rid for s in new] == [0, 2, 3, 1]
    assert cb.waiting == []


def test_requests_that_can_never_fit_are_refused():
    cb = _batcher(max_pages=2)
    with pytest.raises(ValueError):
        cb.submit(0, 0, np.zeros(40, np.int32), 1)   # 40 tokens need 3 pages of 16
    with pytest.raises(ValueError):
        cb.submit(1, 0, np.zeros(0, np.int32), 1)    # empty prompt
