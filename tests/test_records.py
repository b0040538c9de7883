"""Host-side trajectory record H(x) (stride_records_*) on the CPU: the plan equals the oracle's
restart pick on the same records; records are replaced on put; a task without a record
restarts from K0 = 0 (Algorithm 1's else branch); concurrent puts are safe."""
import threading

import numpy as np

import paper_2609_14636_amd as P
from oracle import oracle as O


def test_plan_matches_oracle_restart_pick():
    rng = np.random.default_rng(3)
    rec = P.Records()
    tasks, recs = [], {}
    for task in range(300):
        n = int(rng.integers(0, 14))
        vals = rng.choice(np.array([-1.4, -1.0, -0.9, -0.8, -0.6, -0.3]), size=n)
        mask = (rng.random(n) < 0.85).astype(np.uint8) if rng.random() < 0.5 else None
        rec.put(task, vals, mask)
        recs[task] = (vals, mask)
        tasks.append(task)
    alpha = np.where(rng.random(len(tasks)) < 0.3, -np.inf, -0.8)
    ks, k0, km = rec.plan(tasks, alpha)
    for i, t in enumerate(tasks):
        vals, mask = recs[t]
        off = np.array([0, vals.size])
        o = O.restart(off, vals, None, np.array([alpha[i]]), mask)
        assert (ks[i], k0[i], km[i]) == (o[0][0], o[1][0], o[2][0]), (t, vals, mask)


def test_put_replaces_and_missing_task_restarts_from_zero():
    rec = P.Records()
    rec.put(5, [-0.5, -0.7, -0.6, -0.9, -0.4])
    assert rec.plan([5], -0.8)[1].tolist() == [1]
    rec.put(5, [-0.9, -0.5])
    v, m = rec.get(5)
    assert v.tolist() == [-0.9, -0.5] and m.tolist() == [1, 1]
    ks, k0, km = rec.plan([5, 6], -0.8)
    assert ks.tolist() == [-1, -1] and k0.tolist() == [0, 0] and km.tolist() == [0, 0]
    assert rec.get(6) is None and len(rec) == 1


def test_concurrent_puts():
    rec = P.Records()

    def work(base):
        for i in range(500):
            rec.put(base * 1000 + i, np.full(3, -0.1 * (i % 7)))
    th = [threading.Thread(target=work, args=(b,)) for b in range(8)]
    for t in th:
        t.start()
    for t in th:
        t.join()
    assert len(rec) == 4000
    assert rec.get(7 * 1000 + 13)[0].tolist() == [-0.1 * (13 % 7)] * 3
