"""The latency model of the attention terms (Sec. 4, Eq. 1): its work features and fits.

The pair count A_j = q prefix + q (q + 1) / 2 is pinned to the oracle, which counts the
keys each row actually attends to; decode requests (one query token) count their
whole KV length.  The least-squares fits recover known coefficients exactly, and a
token-count-only model cannot tell apart batches of equal token count -- the gap the
paper's accuracy experiment measures.
"""
import numpy as np

import oracle
from paper_2607_00151_amd import perf_model as pm
from workloads.configs import build


def test_pairs_match_the_oracles_key_counts():
    pre, q = [0, 5, 37, 300, 64], [1, 3, 17, 1, 64]
    w = build("pm", 31, 4, 2, 128, 16, pre, q)
    T = int(w.q_indptr[-1])
    toks = np.arange(T, dtype=np.int64)
    heads = np.zeros(T, dtype=np.int32)
    _, _, nk = oracle.attention_rows(w.q, w.k, w.v, w.q_indptr, w.kv_indptr, w.num_q_heads,
                                     w.num_kv_heads, w.scale, toks, heads)
    per_seq = [int(nk[w.q_indptr[b]: w.q_indptr[b + 1]].sum()) for b in range(w.batch)]
    for b in range(w.batch):
        assert per_seq[b] == pm.prefill_pairs(q[b], pre[b])      # q = 1 rows: A = pre + 1 = L
    f = pm.features(q, np.asarray(pre) + np.asarray(q))
    assert f.tokens == sum(q)
    assert f.decode_keys == sum(p + 1 for p, n in zip(pre, q) if n == 1)
    assert f.prefill_pairs == sum(per_seq[b] for b in range(w.batch) if q[b] > 1)


def test_context_fit_recovers_known_coefficients():
    c, ad, ap = 0.011, 3.0e-8, 2.5e-10
    works = [pm.features(qs, kvs) for _, qs, kvs in pm.profiling_batches()]
    t = [c + ad * x.decode_keys + ap * x.prefill_pairs for x in works]
    got = pm.fit_context_model(works, t)
    assert np.allclose(got, (c, ad, ap), rtol=1e-8, atol=1e-12)
    mixed = [pm.features(qs, kvs) for _, qs, kvs in pm.mixed_batches()]
    truth = [c + ad * x.decode_keys + ap * x.prefill_pairs for x in mixed]
    assert pm.max_rel_error(pm.predict_context(got, mixed), truth) < 1e-9


def test_token_model_is_blind_to_cached_context():
    mixed = pm.mixed_batches()
    works = [pm.features(qs, kvs) for _, qs, kvs in mixed]
    coef = pm.fit_token_model([pm.features([256], [256]), pm.features([256] * 4, [256] * 4)], [0.02, 0.05])
    pred = pm.predict_token(coef, works)
    for n_p in (2, 4):
        series = [p for (name, _, _), p in zip(mixed, pred) if f"{n_p}x256" in name]
        assert len(series) == 6 and np.ptp(series) == 0.0
    # same tokens, growing work: the context-aware features do grow
    two = [x for (name, _, _), x in zip(mixed, works) if "2x256" in name]
    assert all(b.prefill_pairs > a.prefill_pairs and b.decode_keys > a.decode_keys for a, b in zip(two, two[1:]))
    assert len({x.tokens for x in two}) == 1


def test_max_rel_error():
    assert abs(pm.max_rel_error([1.1, 2.0], [1.0, 2.0]) - 0.1) < 1e-12


def test_segment_roofline_bound_switches_at_the_ridge():
    from paper_2607_00151_amd import segments as sg
    # q x G rows per KV head = FLOP per K/V byte; the bf16 ridge is 2516.6e12 / 8e12 = 315
    for q, bound in ((16, "hbm"), (32, "hbm"), (256, "mfma"), (512, "mfma")):
        flop, byt, t, rows = sg.attention_roofline(32, q, 8192, 32, 8)
        assert rows == 4 * q
        got = "hbm" if byt / (sg.PEAK_GBS * 1e9) > flop / (sg.PEAK_TFLOPS * 1e12) else "mfma"
        assert got == bound, q
        assert abs(flop - 4 * 128 * 32 * 32 * pm.prefill_pairs(q, 8192)) < 1e-3 * flop


def _layout():
    import paper_2607_00151_amd as sa
    return sa.Layout(num_q_heads=32, num_kv_heads=8, head_dim=128, page_size=16, num_layers=1, num_slots=1 << 20)


def test_launch_shape_terms_come_from_the_planner():
    """The planner's own view of a launch (host only): a single short segment underfills
    the slots (makespan far above an even spread, no split); a few long decode requests
    are split by key range; the c2 shape fills one round whose longest item outlasts the
    mean (the causal imbalance)."""
    import paper_2607_00151_amd as sa
    L = _layout()
    st = sa.sa_attn_plan_stats(L, [2048], [8192 + 2048])
    assert st["items"] == 512 and st["parts"] == 0
    # 8 KV heads x 64 row tiles of 32 tokens; tile k sees 8192 + 32 (k + 1) keys
    assert st["tiles"] == 8 * sum(-(-(8192 + 32 * (k + 1)) // 64) for k in range(64))
    assert st["makespan_tiles"] == (8192 + 2048) // 64            # the longest row tile
    w = pm.features([2048], [10240], L)
    assert abs(w.excess_tiles - (160 - st["tiles"] / 512)) < 1e-9 and w.split == 0
    w = pm.features([1] * 4, [32768] * 4, L)
    assert w.split == 1
    w = pm.features([256], [256], L)
    assert w.excess_tiles > 0 and w.split == 0


def test_shape_fit_recovers_known_coefficients():
    L = _layout()
    coef = (0.012, 3.0e-8, 2.5e-10, 4.0e-4, 0.009)
    works = [pm.features(qs, kvs, L) for _, qs, kvs in pm.profiling_batches()]
    t = pm.predict_shape(coef, works)
    got = pm.fit_shape_model(works, t)
    assert np.allclose(got, coef, rtol=1e-6, atol=1e-12)
