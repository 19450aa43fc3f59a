"""GPU runs of the latency model (Sec. 4, Eq. 1) and of hybrid batch admission
(Alg. 2) through the library, each launch's output checked against the oracle.

* A reduced version of the model's sweep: decode-only and prefill-only profiling
  launches and mixed batches of decode requests with 256-token prefill chunks (as in
  the paper's accuracy experiment), on seeded inputs; every launch is timed by the
  model's own timing function and its sampled rows (first and last row of every
  sequence, every head, plus random rows) compared with the oracle.  The fits must
  give positive per-key and per-pair costs, and the context-aware models must beat
  the token-count-only one on the mixed batches.
* One Alg. 2 iteration: decode requests, a latency-critical prefill chunk and
  best-effort lookahead chunks are admitted under delta with the launch-shape
  estimate; the admitted batch obeys the algorithm's rules (queues in priority
  order, each stopping at its first misfit, the estimate within delta) and its
  attention launch matches the oracle on sampled rows.
"""
import numpy as np
import pytest
import torch

import oracle
import paper_2607_00151_amd as sa
from paper_2607_00151_amd import perf_model as pm
from paper_2607_00151_amd import scheduler as S
from workloads.configs import build

from harness import build_cache, compare, dev_u16, host_u16, layout_of, sample_rows

pytestmark = pytest.mark.gpu

HQ, HKV, P = 32, 8, 16


def run_checked(ctx, name, seed, q_len, kv_len, reps=5, warmup=2):
    """Seeded inputs of these lengths; time the launch with the model's timing function
    and check sampled rows against the oracle.  Returns (ms, layout)."""
    pre = [int(k) - int(q) for q, k in zip(q_len, kv_len)]
    w = build(name, seed, HQ, HKV, 128, P, pre, list(q_len))
    L = layout_of(w)
    kp, vp, ip, ix = build_cache(w)
    T = int(w.qlen.sum())
    o = torch.empty((T, HQ, 128), dtype=torch.int16, device="cuda")
    ms = pm.time_launch(sa, ctx, L, dev_u16(w.q), (kp, vp), ip, ix, w.qlen, w.kv, o, reps, warmup)
    toks, heads = sample_rows(w, 8, seed)
    ref, _, _ = oracle.attention_rows(w.q, w.k, w.v, w.q_indptr, w.kv_indptr, HQ, HKV, w.scale, toks, heads)
    compare(host_u16(o)[toks, heads], ref, 2e-2, 2e-3)
    return ms


@pytest.mark.timeout(600)
def test_latency_model_sweep_through_the_library():
    prof_b = [(q, kv) for name, q, kv in pm.profiling_batches() if "32768" not in name and "16384" not in name]
    mix_b = [(q, kv) for name, q, kv in pm.mixed_batches() if "32768" not in name and "16384" not in name]
    L = sa.Layout(num_q_heads=HQ, num_kv_heads=HKV, head_dim=128, page_size=P, num_layers=1, num_slots=1)
    with sa.Context(0) as ctx:
        run_checked(ctx, "warm", 1, [256] * 4, [4096 + 256] * 4, reps=40, warmup=0)   # clock warm-up
        prof = [(q, kv, run_checked(ctx, f"prof{i}", 100 + i, q, kv)) for i, (q, kv) in enumerate(prof_b)]
        mixed = [(q, kv, run_checked(ctx, f"mix{i}", 200 + i, q, kv)) for i, (q, kv) in enumerate(mix_b)]
    for q, kv, t in prof + mixed:
        print(f"  q {len(q)} seqs, kv up to {max(kv)}: {t * 1e3:.1f} us", flush=True)
    ev = pm.evaluate(L, prof, mixed)
    print("  max relative error", ev["max_rel_error"], flush=True)
    c, ad, ap = ev["context_model"]
    assert ad > 0 and ap > 0
    err = ev["max_rel_error"]
    assert err["context_aware"] < err["token_only"] and err["launch_shape"] < err["token_only"]


@pytest.mark.timeout(300)
def test_alg2_iteration_through_the_library():
    inst = S.make_instance(16, 1, 8, seed=5)
    dec, lc, be = inst.queues()
    L = sa.Layout(num_q_heads=HQ, num_kv_heads=HKV, head_dim=128, page_size=P, num_layers=1, num_slots=1)
    # launch-shape estimate with coefficients of the size this kernel measures (ms)
    coef = (0.018, 6.7e-7, 1.4e-8, 2.0e-4, 0.01)
    est = lambda b: S.est_batch_latency(coef, b, L)   # noqa: E731
    delta = 0.3
    batch = S.hybrid_batch(dec, lc, be, delta, est)
    kinds = [x.kind for x in batch]
    print(f"  admitted {kinds.count('decode')} decode, {kinds.count('lc')} LC, {kinds.count('be')} BE chunks; "
          f"estimate {est(batch) * 1e3:.1f} us", flush=True)
    # Alg. 2's rules: priority order, each queue a prefix of itself cut at its first misfit
    order = {"decode": 0, "lc": 1, "be": 2}
    assert kinds == sorted(kinds, key=order.get)
    assert est(batch) <= delta
    prefix = []
    for queue in (dec, lc, be):
        n = sum(1 for x in batch if x.kind == queue[0].kind) if queue else 0
        assert [x.rid for x in batch if queue and x.kind == queue[0].kind] == [x.rid for x in queue[:n]]
        prefix += queue[:n]
        if n < len(queue):
            assert est(prefix + [queue[n]]) > delta
    assert kinds.count("decode") == len(dec) and kinds.count("be") < len(be)
    # the admitted batch's attention launch against the oracle
    with sa.Context(0) as ctx:
        run_checked(ctx, "alg2", 300, [x.q for x in batch], [x.kv for x in batch])
