"""Host bookkeeping of the paged server (no device): page reservation, dense
slots, retirement by moving the last request, the block-table rows, and a
pending (asynchronously evicted) batch in the top slots."""
import random

import numpy as np
import pytest

from paper_2512_21859_amd.serving import PAGE, SlotTable


def _invariants(st: SlotTable):
    owned = [p for e in st.slots + st.pending for p in e.pages]
    assert len(owned) == len(set(owned)), "a page is owned twice"
    assert not set(owned) & set(st.free), "a page is both owned and free"
    assert sorted(owned + st.free) == list(range(st.n_pages)), "pages lost or invented"
    # the running slots [0, n) and the pending ones [max_seqs - p, max_seqs) are disjoint
    assert len(st.slots) + len(st.pending) <= st.max_seqs
    rows = st.table_rows()
    assert rows.shape == (len(st.slots), st.max_pages)
    for i, e in enumerate(st.slots):
        assert e.length + e.left <= len(e.pages) * PAGE, "reservation too small"
        assert rows[i, : len(e.pages)].tolist() == e.pages
        # every row decode can touch (tiles below the final length) is the request's own page
        last_tile = (e.length + e.left - 1) // PAGE
        assert set(rows[i, : last_tile + 1].tolist()) <= set(e.pages)
    assert st.lengths().tolist() == [e.length for e in st.slots]


def test_reserve_and_release():
    st = SlotTable(n_pages=9, max_seqs=3, max_pages=4)
    assert st.admit(7, n_keep=33, max_new=0) == 0          # 2 pages
    assert st.slots[0].pages == [0, 1]
    assert st.admit(8, n_keep=100, max_new=28) == 1        # 128 rows: 4 pages
    with pytest.raises(ValueError):
        st.admit(9, n_keep=100, max_new=29)                # 5 pages > max_pages
    with pytest.raises(ValueError):
        st.admit(7, n_keep=1, max_new=1)                   # already running
    with pytest.raises(MemoryError):
        st.admit(9, n_keep=120, max_new=8)                 # 4 pages needed, 3 free
    st.admit(9, n_keep=90, max_new=6)                      # takes the last 3 pages
    with pytest.raises(MemoryError):
        st.admit(10, n_keep=1, max_new=0)                  # no slot left
    _invariants(st)
    assert st.retire(7) == 2                               # the last slot moved into 0
    assert [e.rid for e in st.slots] == [9, 8]
    assert st.retire(8) is None                            # last slot: nothing moves
    _invariants(st)


def test_fits_counts_pages_and_slots():
    st = SlotTable(n_pages=8, max_seqs=4, max_pages=8)
    assert st.fits([32 * 4, 32 * 4])
    assert not st.fits([32 * 4, 32 * 4 + 1])
    assert not st.fits([1] * 5)
    assert not st.fits([32 * 9])


def test_advance_and_finish():
    st = SlotTable(n_pages=16, max_seqs=4, max_pages=4)
    st.admit(1, 31, 2)
    st.admit(2, 10, 1)
    st.advance()
    assert st.lengths().tolist() == [32, 11]
    assert st.finished() == [2]
    with pytest.raises(RuntimeError):
        st.advance()                                       # request 2 has no steps left
    st.retire(2)
    st.advance()
    assert st.lengths().tolist() == [33] and st.finished() == [1]
    _invariants(st)


def test_table_rows_pad_with_own_last_page():
    st = SlotTable(n_pages=6, max_seqs=2, max_pages=5)
    st.admit(0, 40, 0)                                     # pages 0, 1
    st.admit(1, 1, 0)                                      # page 2
    assert st.table_rows().tolist() == [[0, 1, 1, 1, 1], [2, 2, 2, 2, 2]]
    assert st.table_rows(1, 2).tolist() == [[2, 2, 2, 2, 2]]


def test_random_stream_keeps_invariants():
    rng = random.Random(5)
    st = SlotTable(n_pages=64, max_seqs=8, max_pages=12)
    rid = 0
    for _ in range(2000):
        op = rng.random()
        if op < 0.3:
            n_keep, max_new = rng.randint(1, 300), rng.randint(0, 80)
            if st.fits([n_keep + max_new]):
                st.admit(rid, n_keep, max_new)
                rid += 1
        elif op < 0.8 and st.slots:
            for r in st.finished():
                st.retire(r)
            if st.slots:
                st.advance()
        elif st.slots:
            st.retire(rng.choice(st.slots).rid)
        _invariants(st)
    assert rid > 100


def test_pending_batch_takes_top_slots_and_joins_at_the_end():
    st = SlotTable(n_pages=16, max_seqs=6, max_pages=4)
    st.admit(1, 40, 4)                                     # pages 0, 1
    st.admit(2, 10, 4)                                     # page 2
    top = st.admit_pending([5, 6], [31, 64], [1, 0], [0.5, 0.2], [62, 80])
    assert top == 4                                        # slots 4, 5
    assert st.pending_rows().tolist() == [[3, 3, 3, 3], [4, 5, 5, 5]]
    assert [e.rid for e in st.pending] == [5, 6]
    _invariants(st)
    with pytest.raises(RuntimeError):
        st.admit_pending([7], [1], [0], [0.0], [1])        # one pending batch at a time
    with pytest.raises(ValueError):
        st.admit(5, 1, 0)                                  # pending requests count as running
    assert st.fits([32, 32]) and not st.fits([32, 32, 32])  # 2 free slots left
    # the running batch keeps stepping and retiring meanwhile
    st.advance()
    assert st.retire(1) == 1                               # request 2 moves into slot 0
    assert [e.rid for e in st.slots] == [2]
    assert [e.length for e in st.pending] == [31, 64]      # untouched by advance
    _invariants(st)
    assert st.promote() == (1, 3)
    assert [e.rid for e in st.slots] == [2, 5, 6] and not st.pending
    assert st.lengths().tolist() == [11, 31, 64]
    assert st.table_rows(1, 3).tolist() == [[3, 3, 3, 3], [4, 5, 5, 5]]
    _invariants(st)


def test_pending_batch_cancel_frees_its_pages():
    st = SlotTable(n_pages=8, max_seqs=4, max_pages=4)
    st.admit(1, 40, 0)                                     # pages 0, 1
    free0 = list(st.free)
    st.admit_pending([2, 3], [64, 1], [0, 31], [0.0, 0.0], [64, 1])
    assert not set(free0) <= set(st.free)
    st.cancel_pending()
    assert not st.pending and sorted(st.free) == sorted(free0)
    _invariants(st)
    assert st.admit_pending([2], [1], [0], [0.0], [1]) == 3   # a new batch may follow


def test_pending_batch_checked_whole():
    st = SlotTable(n_pages=4, max_seqs=4, max_pages=4)
    with pytest.raises(MemoryError):
        st.admit_pending([1, 2], [64, 64], [32, 33], [0, 0], [64, 64])   # 3 + 4 pages > 4
    assert not st.pending and len(st.free) == 4            # nothing reserved
    with pytest.raises(ValueError):
        st.admit_pending([1, 1], [1, 1], [0, 0], [0, 0], [1, 1])         # duplicate request
    assert not st.pending and len(st.free) == 4


def test_random_stream_with_pending_batches():
    rng = random.Random(11)
    st = SlotTable(n_pages=64, max_seqs=8, max_pages=12)
    rid = joined = 0
    for _ in range(2000):
        op = rng.random()
        if op < 0.2 and not st.pending:
            b = rng.randint(1, 3)
            nk = [rng.randint(1, 300) for _ in range(b)]
            mn = [rng.randint(0, 80) for _ in range(b)]
            if st.fits([k + m for k, m in zip(nk, mn)]):
                st.admit_pending(list(range(rid, rid + b)), nk, mn, [0.0] * b, nk)
                rid += b
        elif op < 0.3 and st.pending:
            n0 = len(st.slots)
            lo, hi = st.promote()
            assert lo == n0 and hi - lo >= 1
            joined += hi - lo
        elif op < 0.8 and st.slots:
            for r in st.finished():
                st.retire(r)
            if st.slots:
                st.advance()
        elif st.slots:
            st.retire(rng.choice(st.slots).rid)
        _invariants(st)
    assert joined > 100


def test_budget_planning_follows_the_controller():
    """Admission by time budget hands every request the controller's alpha*
    and pessimistic length (checked against the oracle's closed forms), and a
    larger budget never asks for more eviction."""
    from oracle import controller as C
    from paper_2512_21859_amd.pipeline import TimeModel, plan_requests
    model = TimeModel(prefill_abc=(2e-9, 6e-5, 12.0), step_pq=(2.5e-4, 21.0), bucket=16, k=3,
                      n_max=512, t_predict=3.0, alpha_max=0.95)
    rng = random.Random(3)
    n_x = [rng.randint(500, 32000) for _ in range(40)]
    n_hat = [rng.randint(1, 40) for _ in range(40)]
    budgets = [rng.uniform(300.0, 15000.0) for _ in range(40)]
    plan = plan_requests(model, n_x, budgets, n_hat)
    for (a, feas, w), n, nh, T in zip(plan, n_x, n_hat, budgets):
        w_ref = C.pessimistic_length(C.predicted_length(nh, model.bucket, model.n_max), model.k,
                                     model.n_max)
        a_ref, f_ref = C.alpha_star(model.prefill_abc, model.step_pq, n, w_ref, T,
                                    model.t_predict, model.alpha_max)
        assert w == w_ref and feas == f_ref
        assert abs(a - a_ref) <= 1e-12
        if feas:
            t = model.t_predict + C.t_wcet(model.prefill_abc, model.step_pq, n, a, w)
            assert t <= T * (1 + 1e-9)
    assert any(f for _, f, _ in plan) and not all(f for _, f, _ in plan)
    more = plan_requests(model, n_x, [2 * T for T in budgets], n_hat)
    assert all(m[0] <= p[0] for m, p in zip(more, plan))
    with pytest.raises(ValueError):
        plan_requests(model, n_x, budgets[:-1], n_hat)
