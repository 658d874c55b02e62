"""Host-only tests of the scheduler (Sec. IV, "Isolated Prefill",
Algorithms 1 and 2) in dry-run mode: no engine, the same scheduling
decisions, tokens 0.  Checks the iteration trace the algorithms imply, the
concurrency limit, first-in-first-out admission with head-of-line blocking,
full-sequence KV admission and page accounting, and slot reuse."""
import numpy as np
import pytest

from paper_2608_14376_amd import corun

P, D = corun.Scheduler.PREFILL, corun.Scheduler.DECODE


def test_trace_of_isolated_prefill_and_decode():
    """max_num_reqs = 2, three requests of 3 output tokens: prefill 0, prefill
    1 (each alone: its first token), two decode steps finish both, then
    request 2 is prefilled alone and decoded twice."""
    s = corun.Scheduler(None, max_num_reqs=2, n_slots=4, max_seq_len=64)
    for i in range(3):
        s.add_request(i, [1] * 5, max_new_tokens=3)
    assert s.run_until_idle() == [P, P, D, D, P, D, D]
    for i in range(3):
        tok, lp, fin = s.output(i)
        assert len(tok) == 3 and fin


def test_concurrency_limit_and_fifo_admission():
    s = corun.Scheduler(None, max_num_reqs=3, n_slots=8, max_seq_len=256)
    rng = np.random.default_rng(1)
    n = 12
    for i in range(n):
        s.add_request(i, [2] * int(rng.integers(1, 30)), max_new_tokens=int(rng.integers(1, 9)))
    admitted, seen = [], set()
    while True:
        ev = s.step()
        st = s.state()
        assert st["running"] <= 3
        # a prefill step admits one request: the one whose first token appeared
        new = [i for i in range(n) if i not in seen and len(s.output(i)[0]) > 0]
        assert len(new) == (1 if ev == P else 0)
        for i in new:
            seen.add(i)
            admitted.append(i)
        if ev == corun.Scheduler.IDLE:
            break
    assert admitted == sorted(admitted) == list(range(n))     # first in, first out
    for i in range(n):
        assert s.output(i)[2]


def test_full_sequence_admission_blocks_the_head_and_frees_pages():
    """Six 16-token pages: A needs 4 (30 + 20 tokens), B 3 (20 + 20), C 1.
    After A is admitted only 2 pages are free: B waits although a slot is
    free, and C waits behind it (Algorithm 1 looks at the waiting head
    only).  When A finishes its pages return and B, then C, start."""
    s = corun.Scheduler(None, max_num_reqs=4, n_slots=4, page_size=16, num_pages=6, max_pages_per_seq=4)
    s.add_request(0, [1] * 30, max_new_tokens=20)
    s.add_request(1, [1] * 20, max_new_tokens=20)
    s.add_request(2, [1] * 5, max_new_tokens=5)
    assert s.step() == P
    st = s.state()
    assert st["free_pages"] == 2 and st["running"] == 1 and st["waiting"] == 2
    # A decodes alone until it finishes (19 more tokens); B and C wait
    for _ in range(19):
        assert s.step() == D
        st = s.state()
        assert st["free_pages"] + 4 * (st["running"] > 0) == 6 or st["running"] == 0
    st = s.state()
    assert st["running"] == 0 and st["free_pages"] == 6 and st["waiting"] == 2
    assert s.step() == P                                        # B
    assert s.state()["free_pages"] == 3
    assert s.step() == P                                        # C fits now (1 page)
    assert s.state()["free_pages"] == 2
    s.run_until_idle()
    st = s.state()
    assert st["free_pages"] == 6 and st["free_slots"] == 4


def test_lowest_free_slot_is_reused():
    s = corun.Scheduler(None, max_num_reqs=3, n_slots=3, max_seq_len=64)
    s.add_request(10, [1] * 4, max_new_tokens=1)     # finishes at its prefill
    s.add_request(11, [1] * 4, max_new_tokens=5)
    assert s.step() == P                             # 10 in slot 0, done at once
    assert list(s.state()["slot_owner"]) == [-1, -1, -1]
    assert s.step() == P                             # 11 takes slot 0 again
    assert list(s.state()["slot_owner"]) == [11, -1, -1]


def test_requests_that_can_never_fit_are_refused():
    s = corun.Scheduler(None, n_slots=2, max_seq_len=32)
    with pytest.raises(corun.CorunError):
        s.add_request(1, [1] * 30, max_new_tokens=3)
    s.add_request(2, [1] * 29, max_new_tokens=3)     # exactly 32
    with pytest.raises(corun.CorunError):
        s.add_request(2, [1] * 4, max_new_tokens=1)  # id reused
    sp = corun.Scheduler(None, n_slots=2, page_size=16, num_pages=3, max_pages_per_seq=2)
    with pytest.raises(corun.CorunError):
        sp.add_request(1, [1] * 30, max_new_tokens=3)  # 3 pages > 2 per sequence


def test_every_request_generates_its_output_length():
    s = corun.Scheduler(None, max_num_reqs=5, n_slots=6, max_seq_len=128)
    rng = np.random.default_rng(2)
    want = {}
    for i in range(30):
        want[i] = int(rng.integers(1, 12))
        s.add_request(i, [3] * int(rng.integers(1, 60)), max_new_tokens=want[i])
    events = s.run_until_idle()
    assert events.count(P) == 30
    for i, n in want.items():
        tok, lp, fin = s.output(i)
        assert len(tok) == n and fin


def test_chunked_prefill_runs_the_head_to_completion_first():
    """Algorithm 1's first branch: a running head whose prompt is not fully
    computed continues before anything else.  A (2-token prompt) is running;
    B's 10-token prompt in chunks of 4 takes three isolated iterations in a
    row -- no decode and no other admission in between -- and only its last
    chunk yields a token."""
    s = corun.Scheduler(None, max_num_reqs=3, n_slots=4, max_seq_len=64, prefill_chunk=4)
    s.add_request(0, [1] * 2, max_new_tokens=6)
    assert s.step() == P
    s.add_request(1, [1] * 10, max_new_tokens=2)
    s.add_request(2, [1] * 3, max_new_tokens=2)
    for k in range(3):
        assert s.step() == P
        assert len(s.output(0)[0]) == 1                       # A was not decoded
        assert len(s.output(1)[0]) == (1 if k == 2 else 0)    # B's token after its last chunk
        assert len(s.output(2)[0]) == 0                       # C not admitted meanwhile
    assert s.step() == P                                      # C: one chunk
    assert s.step() == D
    assert len(s.output(0)[0]) == 2 and len(s.output(1)[0]) == 2 and len(s.output(2)[0]) == 2


def test_chunk_count_per_prompt():
    s = corun.Scheduler(None, max_num_reqs=1, n_slots=2, max_seq_len=128, prefill_chunk=16)
    lens = [1, 15, 16, 17, 48, 100]
    for i, L in enumerate(lens):
        s.add_request(i, [5] * L, max_new_tokens=1)
    ev = s.run_until_idle()
    assert ev.count(P) == sum((L + 15) // 16 for L in lens) and ev.count(D) == 0
    with pytest.raises(corun.CorunError):
        corun.Scheduler(None, n_slots=2, max_seq_len=64, prefill_chunk=-1)


def test_batched_prefill_takes_the_fitting_requests_in_order():
    """prefill_batch_tokens = 25, prompts of 10 tokens: a prefill iteration
    takes the selected head and the next waiting requests while the prompts
    total at most 25 tokens (two at a time), within the concurrency limit;
    all of a batch get their first token in that iteration."""
    s = corun.Scheduler(None, max_num_reqs=5, n_slots=6, max_seq_len=64, prefill_batch_tokens=25)
    for i in range(6):
        s.add_request(i, [1] * 10, max_new_tokens=3)
    assert s.step() == P
    assert [len(s.output(i)[0]) for i in range(6)] == [1, 1, 0, 0, 0, 0]
    assert s.step() == P
    assert [len(s.output(i)[0]) for i in range(6)] == [1, 1, 1, 1, 0, 0]
    assert s.step() == P                                   # the limit of 5 cuts the third batch to one
    assert [len(s.output(i)[0]) for i in range(6)] == [1, 1, 1, 1, 1, 0]
    assert s.state()["running"] == 5
    assert s.step() == D
    s.run_until_idle()
    for i in range(6):
        assert s.output(i)[2] and len(s.output(i)[0]) == 3


def test_batched_prefill_respects_pages_and_fifo():
    """Eight 16-token pages: the head needs 4 (40 + 20 tokens), the next 3,
    the third 2: only the first two fit together, and the third waits
    although the token budget would allow it."""
    s = corun.Scheduler(None, max_num_reqs=4, n_slots=4, page_size=16, num_pages=8, max_pages_per_seq=4,
                        prefill_batch_tokens=1000)
    s.add_request(0, [1] * 40, max_new_tokens=20)
    s.add_request(1, [1] * 30, max_new_tokens=10)
    s.add_request(2, [1] * 20, max_new_tokens=10)
    assert s.step() == P
    st = s.state()
    assert st["running"] == 2 and st["waiting"] == 1 and st["free_pages"] == 1
    with pytest.raises(corun.CorunError):
        corun.Scheduler(None, n_slots=2, max_seq_len=64, prefill_chunk=16, prefill_batch_tokens=64)
