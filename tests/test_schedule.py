"""Host scheduler (Algorithm 1, Eq. 1 admission, Eq. 2): the oracle's
reference pinned to the paper's closed forms and worked examples, and the
library's native scheduler checked decision by decision against it."""
import numpy as np
import pytest

import oracle
import synth
from oracle import schedule as osch
import paper_2607_08930_amd as bs


def cycle(s, eos=()):
    """One block boundary on the oracle scheduler: refill, then complete."""
    adm = s.admit()
    gone = s.complete_cycle(eos)
    return adm, gone


# ---------------------------------------------------------------- oracle pins
def test_eq1_cost_matches_bounding_box_definition():
    rng = np.random.default_rng(3)
    for _ in range(50):
        n, L = int(rng.integers(1, 9)), int(rng.choice([8, 16, 32]))
        p = rng.integers(0, 300, n); g = rng.integers(1, 200, n)
        reqs = [osch.Req(i, int(p[i]), int(g[i]), L, b=int(rng.integers(0, -(-int(g[i]) // L)))) for i in range(n)]
        desc = np.zeros(n, synth.REQ_DTYPE)
        desc["p"] = [r.p for r in reqs]; desc["g"] = [r.g for r in reqs]; desc["k"] = [r.b for r in reqs]
        assert osch.cost(reqs) == oracle.bbox_cost(desc, L) == n * max(r.p + (r.b + 1) * L for r in reqs)


def test_fig1_example1_eviction_and_refill():
    # Fixed batch of three; request 3 reaches its last block first, is evicted
    # at the block boundary and request 4 takes its slot from the queue.
    s = osch.Scheduler(L=32, policy=osch.FIXED, fixed_batch=3, rows=4, width=1024, order=osch.ARRIVAL)
    s.submit([(1, 100, 128), (2, 120, 128), (3, 90, 64), (4, 110, 96)])
    assert cycle(s) == ([1, 2, 3], [])
    row3 = next(r.row for r in s.active if r.id == 3)
    assert cycle(s) == ([], [3])                    # request 3: K = 2 blocks
    adm, _ = cycle(s)
    assert adm == [4]
    assert next(r.row for r in s.active if r.id == 4) == row3


def test_fig1_example2_bounding_box_shrink_expands_the_batch():
    # Budget admission: the wide request 1 bounds the box; when it completes,
    # the box shrinks and two queued requests fit (batch 3 -> 4).
    L = 32
    s = osch.Scheduler(L=L, policy=osch.BUDGET, budget=1300, rows=8, width=1024, order=osch.ARRIVAL)
    s.submit([(1, 400, 64), (2, 100, 256), (3, 100, 256), (4, 100, 256), (5, 100, 256)])
    assert s.admit() == [1, 2, 3]                  # 3 x 432 = 1296 <= 1300; a fourth would cost 1728
    assert s.cost() == 3 * (400 + L)
    s.complete_cycle()
    assert s.admit() == []                         # box now 464: 4 x 464 > 1300
    assert s.complete_cycle() == [1]               # request 1 finishes its K = 2 blocks
    box = max(r.width() for r in s.active)
    assert box == 100 + 3 * L                      # the box shrank to the survivors' rows
    assert s.admit() == [4, 5]                     # both are sand fills: 100 + 32 <= 196
    assert len(s.active) == 4 and s.cost() == 4 * box <= 1300


def test_eq2_effective_compute_ratio_hand_trace():
    # Fixed cap B = 2, blocks K = (1, 2, 3): active counts per cycle 2, 2, 1, 1
    s = osch.Scheduler(L=8, policy=osch.FIXED, fixed_batch=2, rows=2, width=64, order=osch.ARRIVAL)
    s.submit([(1, 4, 8), (2, 4, 16), (3, 4, 24)])
    while not s.done():
        cycle(s)
    assert s.active_counts == [2, 2, 1, 1]
    assert oracle.effective_compute_ratio(s.active_counts, 2) == pytest.approx(6 / 8)


def test_eos_evicts_at_the_block_boundary():
    s = osch.Scheduler(L=8, policy=osch.FIXED, fixed_batch=4, rows=4, width=128)
    s.submit([(1, 4, 64), (2, 4, 64)])
    s.admit()
    assert s.complete_cycle(eos_ids=[2]) == [2]
    assert [r.id for r in s.active] == [1] and s.active[0].b == 1


def _random_stream(rng, n, L):
    # prompt lengths spread like the benchmark statistics table (short and long prompts)
    p = np.where(rng.random(n) < 0.8, rng.integers(16, 200, n), rng.integers(300, 900, n))
    g = rng.choice([64, 128, 256], n)
    return [(i, int(p[i]), int(g[i])) for i in range(n)]


@pytest.mark.parametrize("order", [osch.ASCENDING, osch.DESCENDING, osch.ARRIVAL])
def test_admission_postconditions_and_completion(order):
    """After every refill: a refill that admits leaves the cost within budget
    (Algorithm 1 checks the budget only when admitting: the rows of admitted
    requests grow by L per block afterwards), no sand-filling candidate that
    would fit remains, and the queue head does not fit (or no row is free).
    Every request leaves after exactly K blocks when nobody reports EOS."""
    L, budget, rows = 32, 6000, 12
    rng = np.random.default_rng(10 + order)
    s = osch.Scheduler(L=L, policy=osch.BUDGET, budget=budget, rows=rows, width=1200, order=order)
    s.submit(_random_stream(rng, 60, L))
    blocks = {}
    while not s.done():
        before = s.cost()
        adm = s.admit()
        assert len(s.active) <= rows
        assert s.cost() <= max(budget, before)
        if adm:
            assert s.cost() <= budget
        if len(s.active) < rows:
            box = max((r.width() for r in s.active), default=0)
            for c in s.pending:
                if c.p + L <= box:
                    assert osch.cost(s.active, c) > budget
            if s.pending:
                assert osch.cost(s.active, s.pending[0]) > budget
        for r in s.active:
            blocks[r.id] = blocks.get(r.id, 0) + 1
        s.complete_cycle()
    assert sorted(r.id for r in s.finished) == list(range(60))
    assert all(blocks[r.id] == r.K for r in s.finished)


# ---------------------------------------------------------------- library vs oracle
@pytest.mark.parametrize("policy,order", [(osch.BUDGET, osch.ASCENDING), (osch.BUDGET, osch.DESCENDING),
                                          (osch.BUDGET, osch.ARRIVAL), (osch.FIXED, osch.ASCENDING)])
def test_native_scheduler_matches_reference(policy, order):
    L, rows, width = 32, 16, 1200
    budget, fixed = 9000, 10
    rng = np.random.default_rng(100 + 10 * policy + order)
    ref = osch.Scheduler(L=L, policy=policy, budget=budget, fixed_batch=fixed, rows=rows, width=width, order=order)
    nat = bs.Scheduler(L, policy=policy, budget=budget, fixed_batch=fixed, rows=rows, width=width, order=order)
    stream = _random_stream(rng, 120, L)
    for wave in range(3):                        # requests arrive in three waves
        part = stream[wave * 40:(wave + 1) * 40]
        ref.submit(part)
        nat.submit(part)
        for _ in range(4):
            adm_r = ref.admit()
            plan = nat.refill()
            assert plan["admitted"].tolist() == adm_r
            act = ref.active_sorted()
            assert plan["ids"].tolist() == [r.id for r in act]
            d = plan["descs"]
            assert d["p"].tolist() == [r.p for r in act] and d["g"].tolist() == [r.g for r in act]
            assert d["k"].tolist() == [r.b for r in act] and d["row"].tolist() == [r.row for r in act]
            assert (d["off"] == width - (d["p"] + d["g"])).all()
            oracle.validate_reqs(d, L, rows, width)
            assert plan["cost"] == ref.cost() == oracle.bbox_cost(d, L)
            for a, rid in enumerate(adm_r):
                seg = plan["segs"][a]
                r = next(x for x in act if x.id == rid)
                assert (seg["src_kind"], seg["src_row"], seg["src_col"], seg["dst_row"], seg["dst_col"],
                        seg["len"]) == (1, a, 0, r.row, width - r.p - r.g, r.p + r.g)
            eos = rng.random(len(act)) < 0.1
            gone_r = ref.complete_cycle([r.id for r, e in zip(act, eos) if e])
            assert nat.complete(eos.astype(np.uint8)).tolist() == gone_r
    while not ref.done():
        adm_r = ref.admit()
        assert nat.refill()["admitted"].tolist() == adm_r
        gone_r = ref.complete_cycle()
        assert nat.complete().tolist() == gone_r
    c = nat.counts()
    assert c["pending"] == 0 and c["active"] == 0 and c["finished"] == 120
    assert c["cycles"] == len(ref.active_counts) and c["sum_active"] == sum(ref.active_counts)


def test_native_scheduler_rejects_unservable_requests():
    s = bs.Scheduler(32, policy=bs.SCHED_BUDGET, budget=500, rows=4, width=600)
    with pytest.raises(bs.BlockServeError, match="width"):
        s.submit([(1, 500, 200)])
    with pytest.raises(bs.BlockServeError, match="budget"):
        s.submit([(2, 480, 64)])
    assert s.counts()["pending"] == 0
    s.submit([(3, 10, 64)])
    s.refill()
    with pytest.raises(bs.BlockServeError, match="active"):
        s.complete(np.zeros(5, np.uint8))
    with pytest.raises(bs.BlockServeError):
        bs.Scheduler(0, rows=1, width=1, budget=1)
