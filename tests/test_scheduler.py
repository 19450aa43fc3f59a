"""Hybrid batch admission (Alg. 2) on toy latency estimates, and the simulated instance.

The estimator here is a plain sum of per-kind costs, so the admitted batch can be
worked out by hand from the algorithm's three ordered loops: each queue is admitted
in order until its first candidate that would take the batch past delta.
"""
from paper_2607_00151_amd import scheduler as S
from paper_2607_00151_amd import perf_model as pm

COST = {"decode": 1.0, "lc": 5.0, "be": 10.0}


def est(batch):
    return sum(COST[x.kind] * x.q for x in batch)


def items(kind, n, q=1):
    return [S.Item(kind, i, q, 100) for i in range(n)]


def test_admission_by_hand():
    b = S.hybrid_batch(items("decode", 4), items("lc", 2), items("be", 3), 25.0, est)
    assert [x.kind for x in b] == ["decode"] * 4 + ["lc"] * 2 + ["be"]      # 4 + 10 + 10 = 24 <= 25
    assert est(b) <= 25.0


def test_first_violation_ends_a_queue():
    be = [S.Item("be", 0, 2, 100), S.Item("be", 1, 1, 100)]               # costs 20, then 10
    b = S.hybrid_batch(items("decode", 4), [], be, 20.0, est)
    assert [x.kind for x in b] == ["decode"] * 4                            # 24 > 20: stop, the cheaper one is not tried


def test_each_queue_gets_its_own_loop():
    # the decode queue stops at its first misfit; a cheaper LC chunk behind it may still fit
    dec = [S.Item("decode", 0, 1, 10), S.Item("decode", 1, 8, 10)]          # 1, then 8
    b = S.hybrid_batch(dec, items("lc", 1), [], 6.0, est)
    assert [x.kind for x in b] == ["decode", "lc"]
    # nothing fits: empty batch
    assert S.hybrid_batch(items("decode", 1), [], [], 0.5, est) == []


def test_model_estimate_matches_eq1():
    coef = (0.01, 2e-8, 3e-10)
    batch = [S.Item("decode", 0, 1, 5000), S.Item("lc", 1, 256, 4096 + 256)]
    want = 0.01 + 2e-8 * 5000 + 3e-10 * pm.prefill_pairs(256, 4096)
    assert abs(S.est_batch_latency(coef, batch) - want) < 1e-15
    assert S.est_batch_latency(coef, []) == 0.0


def test_instance_advances_and_replaces_finished_requests():
    inst = S.make_instance(3, 1, 1, seed=1)
    ctx0 = list(inst.decode_ctx)
    dec, lc, be = inst.queues()
    assert [x.kv for x in dec] == [c + 1 for c in ctx0]
    assert lc[0].q == 256 and lc[0].kv == inst.lc_prefix + 256
    for _ in range(inst.segment // inst.chunk):
        dec, lc, be = inst.queues()
        inst.advance(dec + lc)                                              # BE never admitted
    assert inst.decode_ctx == [c + inst.segment // inst.chunk for c in ctx0]
    assert inst.lc[0][0] != 100 and inst.lc[0][1] == inst.lc_prefix       # replaced by a fresh request
    assert inst.be[0] == [200, inst.be_prefix, inst.segment]
