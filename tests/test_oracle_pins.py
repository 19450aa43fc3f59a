"""Pins for the CPU oracle: it is checked against things other than itself.

* brute force: a masked full-matrix softmax on tiny inputs (different route:
  one score matrix per head, an explicit boolean mask, scipy's softmax);
* closed forms: hand-derived two- and three-key cases that fix the scale,
  the exponential base and the mask offset; K = 0 gives running means; a
  constant V is returned unchanged; a first row with no prefix returns v_0;
* invariants: causality, grouped-query head mapping, shift invariance of
  softmax, the per-row key count summing to the paper's A_j (Sec. 4);
* segment decomposability (Sec. 3.1): prefilling a segment in chunks over the
  growing prefix gives the one-shot outputs exactly;
* page operations: hand-worked fixtures and round-trip properties.
"""
import json
import math
import os

import numpy as np
import pytest
from scipy.special import softmax

import oracle
from oracle import pages
from workloads import rng

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def bf16(x):
    return rng.f32_to_bf16_bits(np.asarray(x, dtype=np.float32))


def f32(b):
    return rng.bf16_bits_to_f32(b).astype(np.float64)


def run(q, k, v, qlen, kvlen, Hq, Hkv, scale):
    qi = np.concatenate([[0], np.cumsum(qlen)])
    ki = np.concatenate([[0], np.cumsum(kvlen)])
    return oracle.attention_all(q, k, v, qi, ki, Hq, Hkv, scale)


def brute_force(q, k, v, qlen, kvlen, Hq, Hkv, scale):
    """Full score matrix per (sequence, head) with an explicit causal mask."""
    G = Hq // Hkv
    head_to_kv = np.repeat(np.arange(Hkv), G)        # heads 0..G-1 -> kv head 0, ...
    outs, lses = [], []
    qo = ko = 0
    for ql, kl in zip(qlen, kvlen):
        Q = f32(q[qo:qo + ql])                          # [ql][Hq][D]
        K = f32(k[ko:ko + kl])[:, head_to_kv]            # [kl][Hq][D]
        V = f32(v[ko:ko + kl])[:, head_to_kv]
        S = np.einsum("ihd,jhd->hij", Q, K) * scale      # [Hq][ql][kl]
        row_pos = (kl - ql) + np.arange(ql)[:, None]      # absolute position of each query
        visible = np.arange(kl)[None, :] <= row_pos       # [ql][kl]
        S = np.where(visible[None], S, -np.inf)
        Pm = softmax(S, axis=-1)
        outs.append(np.einsum("hij,jhd->ihd", Pm, V))
        mx = S.max(axis=-1)
        lses.append((mx + np.log(np.exp(S - mx[..., None]).sum(-1))).T)
        qo += ql
        ko += kl
    return np.concatenate(outs), np.concatenate(lses)


CASES = [
    # Hq, Hkv, D, prefix lengths, segment lengths
    (1, 1, 4, [0], [1]),
    (2, 1, 8, [1], [2]),
    (4, 2, 8, [3], [5]),
    (8, 2, 128, [17], [33]),
    (8, 4, 4, [0, 3, 17], [33, 1, 5]),
    (4, 1, 128, [1, 0], [2, 5]),
    (8, 8, 8, [3], [2]),
]


@pytest.mark.parametrize("Hq,Hkv,D,pre,ql", CASES)
def test_brute_force(Hq, Hkv, D, pre, ql):
    seed = Hq * 1000 + Hkv * 100 + D + len(pre)
    pre, ql = np.array(pre), np.array(ql)
    kvl = pre + ql
    q = rng.normal_bf16(seed, 0, (ql.sum(), Hq, D))
    k = rng.normal_bf16(seed, 1, (kvl.sum(), Hkv, D))
    v = rng.normal_bf16(seed, 2, (kvl.sum(), Hkv, D))
    scale = 1.0 / math.sqrt(D)
    out, lse, nk = run(q, k, v, ql, kvl, Hq, Hkv, scale)
    ref, ref_lse = brute_force(q, k, v, ql, kvl, Hq, Hkv, scale)
    np.testing.assert_allclose(out, ref, rtol=1e-10, atol=1e-12)
    np.testing.assert_allclose(lse, ref_lse, rtol=1e-10, atol=1e-12)


def test_two_key_closed_form():
    """prefix 1, segment 1, D 4, scale 1/2: scores (0, 1) -> O = (v0 + e v1)/(1 + e)."""
    q = bf16([[[1, 0, 0, 0]]])
    k = bf16([[[0, 0, 0, 0]], [[2, 0, 0, 0]]])
    v = bf16([[[1, 0, 0, 0]], [[0, 1, 0, 0]]])
    out, lse, nk = run(q, k, v, [1], [2], 1, 1, 0.5)
    e = math.e
    np.testing.assert_allclose(out[0, 0], [1 / (1 + e), e / (1 + e), 0, 0], rtol=1e-14, atol=1e-15)
    assert lse[0, 0] == pytest.approx(math.log(1 + e), rel=1e-14)
    assert nk[0, 0] == 2


def test_three_key_causal_closed_form():
    """prefix 1, segment 2: row 0 sees keys 0..1 (scores 0, 1), row 1 sees 0..2
    (scores 0, 0, 4); the scale 1/2 multiplies q.k."""
    q = bf16([[[1, 0, 0, 0]], [[0, 2, 0, 0]]])
    k = bf16([[[0, 0, 0, 0]], [[2, 0, 0, 0]], [[0, 4, 0, 0]]])
    v = bf16([[[1, 0, 0, 0]], [[0, 1, 0, 0]], [[0, 0, 1, 0]]])
    out, lse, nk = run(q, k, v, [2], [3], 1, 1, 0.5)
    e, e4 = math.e, math.exp(4.0)
    np.testing.assert_allclose(out[0, 0], [1 / (1 + e), e / (1 + e), 0, 0], rtol=1e-14, atol=1e-15)
    np.testing.assert_allclose(out[1, 0], [1 / (2 + e4), 1 / (2 + e4), e4 / (2 + e4), 0],
                               rtol=1e-13, atol=1e-15)
    assert lse[1, 0] == pytest.approx(math.log(2 + e4), rel=1e-14)
    assert list(nk[:, 0]) == [2, 3]


def test_zero_keys_give_running_mean():
    """K = 0 makes every visible score equal, so row i returns the mean of V
    rows 0..prefix+i."""
    Hq, Hkv, D, pre, ql = 4, 2, 8, 5, 7
    v = rng.normal_bf16(7, 2, (pre + ql, Hkv, D))
    k = np.zeros((pre + ql, Hkv, D), dtype=np.uint16)
    q = rng.normal_bf16(7, 0, (ql, Hq, D))
    out, _, _ = run(q, k, v, [ql], [pre + ql], Hq, Hkv, 0.3)
    V = f32(v)
    for i in range(ql):
        for h in range(Hq):
            mean = V[: pre + i + 1, h // (Hq // Hkv)].mean(axis=0)
            np.testing.assert_allclose(out[i, h], mean, rtol=1e-12, atol=1e-14)


def test_constant_values_returned():
    Hq, Hkv, D, pre, ql = 8, 2, 16, 9, 4
    c = bf16(np.linspace(-1, 1, D))
    v = np.broadcast_to(c, (pre + ql, Hkv, D)).copy()
    q = rng.normal_bf16(9, 0, (ql, Hq, D))
    k = rng.normal_bf16(9, 1, (pre + ql, Hkv, D))
    out, _, _ = run(q, k, v, [ql], [pre + ql], Hq, Hkv, 1 / 4)
    np.testing.assert_allclose(out, np.broadcast_to(f32(c), out.shape), rtol=1e-14, atol=1e-15)


def test_first_row_without_prefix_is_v0():
    Hq, Hkv, D, ql = 4, 4, 128, 3
    q = rng.normal_bf16(11, 0, (ql, Hq, D))
    k = rng.normal_bf16(11, 1, (ql, Hkv, D))
    v = rng.normal_bf16(11, 2, (ql, Hkv, D))
    out, lse, _ = run(q, k, v, [ql], [ql], Hq, Hkv, 1 / math.sqrt(D))
    assert np.array_equal(out[0], f32(v[0]))        # exactly v_0


def test_causality_future_rows_do_not_matter():
    """Changing K/V at positions after a row's own leaves that row bit-identical."""
    Hq, Hkv, D, pre, ql = 8, 2, 32, 6, 9
    q = rng.normal_bf16(13, 0, (ql, Hq, D))
    k = rng.normal_bf16(13, 1, (pre + ql, Hkv, D))
    v = rng.normal_bf16(13, 2, (pre + ql, Hkv, D))
    base, _, _ = run(q, k, v, [ql], [pre + ql], Hq, Hkv, 0.2)
    for i in range(ql):
        k2, v2 = k.copy(), v.copy()
        k2[pre + i + 1:] = rng.normal_bf16(100 + i, 1, k2[pre + i + 1:].shape)
        v2[pre + i + 1:] = rng.normal_bf16(200 + i, 2, v2[pre + i + 1:].shape)
        out, _, _ = run(q, k2, v2, [ql], [pre + ql], Hq, Hkv, 0.2)
        assert np.array_equal(out[: i + 1], base[: i + 1])
        if i + 1 < ql:
            assert not np.array_equal(out[i + 1:], base[i + 1:])


def test_grouped_query_mapping():
    """Query head h reads kv head floor(h / G): heads of other groups ignore it."""
    Hq, Hkv, D, pre, ql = 8, 4, 16, 5, 3
    G = Hq // Hkv
    q = rng.normal_bf16(17, 0, (ql, Hq, D))
    k = rng.normal_bf16(17, 1, (pre + ql, Hkv, D))
    v = rng.normal_bf16(17, 2, (pre + ql, Hkv, D))
    base, _, _ = run(q, k, v, [ql], [pre + ql], Hq, Hkv, 0.25)
    for g in range(Hkv):
        k2, v2 = k.copy(), v.copy()
        k2[:, g] = rng.normal_bf16(300 + g, 1, k2[:, g].shape)
        v2[:, g] = rng.normal_bf16(400 + g, 2, v2[:, g].shape)
        out, _, _ = run(q, k2, v2, [ql], [pre + ql], Hq, Hkv, 0.25)
        for h in range(Hq):
            same = np.array_equal(out[:, h], base[:, h])
            assert same == (h // G != g), (g, h)


def test_shift_invariance_of_keys():
    """Adding one vector c to every key shifts all scores of a row by the same
    amount, which softmax ignores (inputs chosen so k + c is exact in bf16)."""
    Hq, Hkv, D, pre, ql = 4, 2, 8, 7, 5
    g = rng.generator(19, 0)
    kint = g.integers(-8, 8, size=(pre + ql, Hkv, D))
    c = g.integers(-4, 4, size=(Hkv, D))
    q = bf16(g.integers(-4, 4, size=(ql, Hq, D)) / 8.0)
    v = rng.normal_bf16(19, 2, (pre + ql, Hkv, D))
    out1, _, _ = run(q, bf16(kint / 8.0), v, [ql], [pre + ql], Hq, Hkv, 0.1)
    out2, _, _ = run(q, bf16((kint + c) / 8.0), v, [ql], [pre + ql], Hq, Hkv, 0.1)
    np.testing.assert_allclose(out1, out2, rtol=1e-11, atol=1e-13)


def test_key_counts_sum_to_paper_work():
    """Sec. 4 prefill-attention term: a chunk of q tokens over a prefix of p
    tokens does A = q*p + q(q+1)/2 (query, key) pairs per head."""
    pre, ql = [0, 7, 100, 1], [1, 13, 31, 64]
    Hq, Hkv, D = 2, 1, 4
    kvl = np.array(pre) + np.array(ql)
    q = rng.normal_bf16(23, 0, (sum(ql), Hq, D))
    k = rng.normal_bf16(23, 1, (kvl.sum(), Hkv, D))
    out, lse, nk = run(q, k, k, ql, kvl, Hq, Hkv, 0.5)
    off = 0
    for p, n in zip(pre, ql):
        assert nk[off:off + n, 0].sum() == n * p + n * (n + 1) // 2
        assert list(nk[off:off + n, 1]) == [p + i + 1 for i in range(n)]
        off += n


@pytest.mark.parametrize("cuts", [[1], [3, 11], [5, 6, 20]])
def test_segment_decomposability(cuts):
    """Sec. 3.1/3.2: building the segment's outputs chunk by chunk, each chunk
    over everything before it, equals the one-shot prefill row for row."""
    Hq, Hkv, D, pre, ql = 8, 2, 64, 13, 29
    q = rng.normal_bf16(29, 0, (ql, Hq, D))
    k = rng.normal_bf16(29, 1, (pre + ql, Hkv, D))
    v = rng.normal_bf16(29, 2, (pre + ql, Hkv, D))
    one, one_lse, _ = run(q, k, v, [ql], [pre + ql], Hq, Hkv, 0.125)
    bounds = [0] + cuts + [ql]
    for a, b in zip(bounds[:-1], bounds[1:]):
        kv_end = pre + b
        part, part_lse, _ = run(q[a:b], k[:kv_end], v[:kv_end], [b - a], [kv_end], Hq, Hkv, 0.125)
        assert np.array_equal(part, one[a:b])
        assert np.array_equal(part_lse, one_lse[a:b])


def test_rejects_bad_inputs():
    q = rng.normal_bf16(1, 0, (2, 2, 4))
    k = rng.normal_bf16(1, 1, (1, 1, 4))
    with pytest.raises(ValueError):
        run(q, k, k, [2], [1], 2, 1, 1.0)       # q_len > kv_len


# ---------------------------------------------------------------- page ops

def _load(name):
    with open(os.path.join(GOLDEN, name)) as f:
        return json.load(f)


def test_assemble_worked_example():
    g = _load("assemble_worked.json")
    r = pages.assemble(g["src_len"], g["src_indptr"], g["src_indices"], g["keep_indptr"],
                       g["keep_spans"], g["reserve"], g["fresh"], g["page_size"])
    assert r["dst_indptr"].tolist() == g["expect_dst_indptr"]
    assert r["dst_indices"].tolist() == g["expect_dst_indices"]
    assert r["dst_len"].tolist() == g["expect_dst_len"]
    assert [list(x) for x in zip(r["copy_src"].tolist(), r["copy_dst"].tolist())] == g["expect_copies"]


def test_append_worked_example():
    g = _load("append_worked.json")
    s, r = pages.append_destinations(g["start"], g["new_len"], g["indptr"], g["indices"],
                                     g["page_size"])
    assert s.tolist() == g["expect_slot"]
    assert r.tolist() == g["expect_row"]


def test_append_then_read_back_round_trip():
    P, Hkv, D, S = 16, 2, 8, 40
    lengths = [37, 5, 64]
    starts = [0, 17, 20]
    npg = [pages.pages_for(s + n, P) for s, n in zip(starts, lengths)]
    indptr = np.concatenate([[0], np.cumsum(npg)])
    indices = rng.permutation(3, 0, S)[: indptr[-1]]
    pool = rng.normal_bf16(3, 1, (S, Hkv, P, D))
    before = pool.copy()
    new = rng.normal_bf16(3, 2, (sum(lengths), Hkv, D))
    sl, ro = pages.append_destinations(starts, lengths, indptr, indices, P)
    pages.apply_append(pool, new, sl, ro)
    off = 0
    for b, (s, n) in enumerate(zip(starts, lengths)):
        got = pages.gather_logical(pool, indptr[b:], indices, [s + n], P, 0)
        assert np.array_equal(got[s:], new[off:off + n])
        off += n
    touched = np.zeros((S, P), dtype=bool)
    touched[sl, ro] = True
    assert np.array_equal(pool.transpose(0, 2, 1, 3)[~touched], before.transpose(0, 2, 1, 3)[~touched])


def test_assemble_keeps_exactly_the_surviving_tokens():
    """Reading the replacement cache back gives the source tokens with the
    dropped pages cut out, in order; dropped tokens = whole dropped pages."""
    P, Hkv, D, S = 8, 2, 4, 200
    src_len = [61, 16, 9, 30]
    spans = [[(0, 2), (5, 8)], [(1, 2)], [(0, 2)], []]
    reserve = [10, 0, 7, 3]
    npg = [pages.pages_for(n, P) for n in src_len]
    src_indptr = np.concatenate([[0], np.cumsum(npg)])
    perm = rng.permutation(5, 0, S)
    src_indices = perm[: src_indptr[-1]]
    fresh = perm[src_indptr[-1]:]
    keep_indptr = np.concatenate([[0], np.cumsum([len(s) for s in spans])])
    keep_spans = [x for s in spans for x in s]
    pool = rng.normal_bf16(5, 1, (S, Hkv, P, D))
    r = pages.assemble(src_len, src_indptr, src_indices, keep_indptr, keep_spans, reserve, fresh, P)
    for a, d in zip(r["copy_src"], r["copy_dst"]):
        pool[d] = pool[a]
    for b in range(len(src_len)):
        src = pages.gather_logical(pool, src_indptr[b:], src_indices, [src_len[b]], P, 0)
        want = np.concatenate([src[p0 * P: min(p1 * P, src_len[b])] for p0, p1 in spans[b]]
                              or [src[:0]])
        got = pages.gather_logical(pool, r["dst_indptr"][b:], r["dst_indices"], [r["dst_len"][b]],
                                   P, 0)
        assert np.array_equal(got, want)
        n_dst = r["dst_indptr"][b + 1] - r["dst_indptr"][b]
        assert n_dst == pages.pages_for(r["dst_len"][b] + reserve[b], P)
    assert r["dst_indices"].tolist() == list(fresh[: r["dst_indptr"][-1]])


def test_assemble_rejects_overlapping_spans():
    with pytest.raises(ValueError):
        pages.assemble([32], [0, 4], [0, 1, 2, 3], [0, 2], [(0, 2), (1, 3)], [0], [9, 8, 7, 6], 8)
    with pytest.raises(ValueError):
        pages.assemble([32], [0, 4], [0, 1, 2, 3], [0, 1], [(0, 5)], [0], [9, 8, 7, 6, 5], 8)
    with pytest.raises(ValueError):
        pages.assemble([32], [0, 4], [0, 1, 2, 3], [0, 1], [(0, 4)], [0], [9, 8, 7], 8)


def test_alias_splice_reads_back_the_surviving_tokens_without_copying():
    """The zero-copy splice: reading the replacement cache through its table
    gives the source tokens with the dropped pages cut out, from the untouched
    pool; its table is the copy splice's with every surviving entry replaced by
    the page's source slot, and only reserved pages consume the free list."""
    P, Hkv, D, S = 8, 2, 4, 200
    src_len = [61, 16, 9, 30]
    spans = [[(0, 2), (5, 8)], [(1, 2)], [(0, 2)], []]
    reserve = [10, 0, 7, 3]
    npg = [pages.pages_for(n, P) for n in src_len]
    src_indptr = np.concatenate([[0], np.cumsum(npg)])
    perm = rng.permutation(7, 0, S)
    src_indices = perm[: src_indptr[-1]]
    fresh = perm[src_indptr[-1]:]
    keep_indptr = np.concatenate([[0], np.cumsum([len(s) for s in spans])])
    keep_spans = [x for s in spans for x in s]
    pool = rng.normal_bf16(7, 1, (S, Hkv, P, D))
    before = pool.copy()
    r = pages.splice_alias(src_len, src_indptr, src_indices, keep_indptr, keep_spans, reserve, fresh, P)
    c = pages.assemble(src_len, src_indptr, src_indices, keep_indptr, keep_spans, reserve, fresh, P)
    assert r["dst_indptr"].tolist() == c["dst_indptr"].tolist()
    assert r["dst_len"].tolist() == c["dst_len"].tolist()
    n_fresh = 0
    for b in range(len(src_len)):
        src = pages.gather_logical(pool, src_indptr[b:], src_indices, [src_len[b]], P, 0)
        want = np.concatenate([src[p0 * P: min(p1 * P, src_len[b])] for p0, p1 in spans[b]]
                              or [src[:0]])
        got = pages.gather_logical(pool, r["dst_indptr"][b:], r["dst_indices"], [r["dst_len"][b]], P, 0)
        assert np.array_equal(got, want)
        kept_pages = [p for p0, p1 in spans[b] for p in range(p0, p1)]
        ent = r["dst_indices"][r["dst_indptr"][b]: r["dst_indptr"][b + 1]].tolist()
        assert ent[: len(kept_pages)] == [int(src_indices[src_indptr[b] + p]) for p in kept_pages]
        assert ent[len(kept_pages):] == list(fresh[n_fresh: n_fresh + len(ent) - len(kept_pages)])
        n_fresh += len(ent) - len(kept_pages)
    assert r["fresh_used"] == n_fresh
    assert np.array_equal(pool, before)
    with pytest.raises(ValueError):
        pages.splice_alias([32], [0, 4], [0, 1, 2, 3], [0, 2], [(0, 2), (1, 3)], [0], [9], 8)
