"""The serving engine (duet_engine_*): its steps against the trace's batch former, bit for bit, and
the page allocator's invariants over a whole trace."""
import numpy as np
import pytest

import paper_2511_04791_amd as duet
from paper_2511_04791_amd import workloads as wl

PS = 16


def _engine_trace(num_iters, warmup, *, num_pages=1 << 20, max_pages=2100, budget=8192, seed=1005, check=None):
    """Drives the engine with the trace's request stream and clock (50 ms per iteration; an idle
    engine jumps to the next arrival), as the batch former does."""
    arrivals, prompts, outputs = wl.trace_requests(seed)
    eng = duet.Engine(budget, num_pages, max_pages, shuffle_seed=7)
    clock, nxt, out = 0.0, 0, []
    for it in range(warmup + num_iters):
        while nxt < len(arrivals) and arrivals[nxt] <= clock:
            eng.add_request(int(prompts[nxt]), int(outputs[nxt]))
            nxt += 1
        w, r, _ = eng.stats()
        if w == 0 and r == 0 and nxt < len(arrivals):
            clock = float(arrivals[nxt])
            continue
        meta, table, ids = eng.step()
        if check:
            check(meta, table, ids)
        eng.complete()
        rows = [(int(k), int(q), int(c)) for k, _, q, c in meta]
        if it >= warmup and rows:
            out.append(rows)
        clock += 0.05
        if len(out) >= num_iters:
            break
    return out, eng


def test_engine_steps_equal_the_trace_batch_former():
    got, _ = _engine_trace(200, 200)
    want = wl.serving_trace(num_iters=200)
    assert len(got) == len(want) == 200
    for i, (g, w) in enumerate(zip(got, want)):
        assert g == [tuple(x) for x in w], f"iteration {i}"


def test_page_tables_over_a_trace():
    """Rows are packed, decodes first; each row holds exactly the pages its keys need; no page is
    held by two live requests; a request's pages never move."""
    owner = {}        # page -> request id
    pages_of = {}     # request id -> its pages so far

    def check(meta, table, ids):
        assert (meta[:, 1] == np.concatenate([[0], np.cumsum(meta[:-1, 2])])).all()
        kinds = meta[:, 0]
        n_dec = int((kinds == 1).sum())
        assert (kinds[:n_dec] == 1).all() and (kinds[n_dec:] == 0).all()
        live = set(int(i) for i in ids)
        for row, rid in enumerate(ids):
            rid = int(rid)
            n = -(-int(meta[row, 2] + meta[row, 3]) // PS)
            pages = [int(p) for p in table[row] if p >= 0]
            assert len(pages) == n and (table[row, n:] == -1).all()
            prev = pages_of.get(rid, [])
            assert pages[:len(prev)] == prev, "a request's pages moved"
            pages_of[rid] = pages
            for p in pages:
                o = owner.get(p)
                assert o is None or o == rid or o not in live, f"page {p} held by {o} and {rid}"
                owner[p] = rid

    _engine_trace(120, 60, num_pages=300000, check=check)


def test_out_of_pages_changes_nothing():
    eng = duet.Engine(256, 10, 8)
    eng.add_request(100, 4)           # 7 pages
    eng.add_request(60, 4)            # 4 more pages in the same step: 11 > 10
    before = eng.stats()
    with pytest.raises(duet.DuetError):
        eng.step()
    assert eng.stats() == before
    eng2 = duet.Engine(64, 10, 8)
    eng2.add_request(100, 1)
    meta, _, _ = eng2.step()          # 64 tokens of the prompt (budget)
    assert meta.tolist() == [[0, 0, 64, 0]]
    eng2.complete()
    meta, _, _ = eng2.step()
    assert meta.tolist() == [[0, 0, 36, 64]]
    eng2.complete()
    meta, table, _ = eng2.step()      # the decode of the only token, then the request ends
    assert meta.tolist() == [[1, 0, 1, 100]] and (table[0, :7] >= 0).all()
    eng2.complete()
    assert eng2.stats() == (0, 0, 10)


def test_engine_argument_checks():
    eng = duet.Engine(16, 100, 4)
    with pytest.raises(duet.DuetError):
        eng.add_request(60, 10)       # 70 tokens need 5 pages > 4
    with pytest.raises(duet.DuetError):
        eng.add_request(0, 1)
    eng.add_request(10, 1)
    eng.step()
    with pytest.raises(duet.DuetError):
        eng.step()                    # the previous step is not completed
    eng.complete()
    with pytest.raises(duet.DuetError):
        eng.complete()
    with pytest.raises(duet.DuetError):
        duet.Engine(0, 10, 4)


def test_lookahead_step_reserves_and_credits_k_tokens():
    """A look-ahead step (Section 4.3) reserves pages for k tokens of every decode and credits each
    decode min(k, its remaining output) tokens; a request whose output ends inside the step is
    released when the step completes."""
    eng = duet.Engine(64, 100, 8)
    a = eng.add_request(30, 10)        # decodes 10 tokens
    b = eng.add_request(20, 2)         # decodes 2 tokens
    meta, _, ids = eng.step()          # both prompts (50 tokens)
    assert meta[:, 0].tolist() == [0, 0]
    eng.complete()
    meta, table, ids = eng.step(decode_steps=4)
    assert meta.tolist() == [[1, 0, 1, 30], [1, 1, 1, 20]] and ids.tolist() == [a, b]
    for row, c in enumerate((30, 20)):
        n = -(-(c + 4) // PS)          # pages for the cached tokens and 4 new ones
        assert (table[row, :n] >= 0).all() and (table[row, n:] == -1).all()
    eng.complete()
    w, r, _ = eng.stats()
    assert (w, r) == (0, 1)            # b produced its 2 tokens and left
    meta, _, ids = eng.step(decode_steps=3)
    assert meta.tolist() == [[1, 0, 1, 34]] and ids.tolist() == [a]   # a gained 4 tokens
    eng.complete()
    meta, _, _ = eng.step(decode_steps=5)
    assert meta.tolist() == [[1, 0, 1, 37]]
    eng.complete()                     # 3 + 4 + 5 > 10: a is done
    assert eng.stats() == (0, 0, 100)


def test_lookahead_step_checks():
    eng = duet.Engine(64, 100, 3)      # rows of 3 pages: 48 tokens
    eng.add_request(40, 8)
    eng.step()
    eng.complete()
    before = eng.stats()
    with pytest.raises(duet.DuetError):
        eng.step(decode_steps=9)       # 40 + 9 tokens need 4 pages
    with pytest.raises(duet.DuetError):
        eng.step(decode_steps=0)
    assert eng.stats() == before
    meta, _, _ = eng.step(decode_steps=8)
    assert meta.tolist() == [[1, 0, 1, 40]]


def test_lookahead_step_completed_with_fewer_steps():
    eng = duet.Engine(64, 100, 8)
    eng.add_request(30, 10)
    eng.step()
    eng.complete()
    eng.step(decode_steps=6)           # pages for 6 tokens
    with pytest.raises(duet.DuetError):
        eng.complete(decode_steps_run=7)
    eng.complete(decode_steps_run=2)   # only 2 ran
    meta, table, _ = eng.step()
    assert meta.tolist() == [[1, 0, 1, 32]]
    assert (table[0, :3] >= 0).all()   # the page reserved for the 6 steps stays
    eng.complete()
