"""GPU parity of the single-launch append + attention.

sa_segment_prefill_attn_append with fusion on (sa_set_fused_append) is one attention
launch that takes the segment's keys and values straight from k_new / v_new
and writes each new row to its page once (paper Sec. 3.2: the segment's KV is
built on the transformed prefix).  For every case:

* both pools end bit for bit as the oracle's append leaves them (layer 1 of
  two, canary everywhere nothing is written);
* every output row and LSE matches the fp64 oracle (sampled rows at the full
  c2 size);
* where both forms take the same kernel steps -- every prefix a multiple of 4
  keys and no request of at most 32 query rows -- output and LSE equal
  those of the two-launch form (sa_set_fused_append(ctx, 0): append kernel,
  then attention) bit for bit; elsewhere both meet the oracle's bar.
"""
import numpy as np
import pytest
import torch

import oracle
import paper_2607_00151_amd as sa
import workloads
from oracle import pages as opages
from workloads.configs import build

from harness import compare, dev_i32, dev_u16, host_u16, layout_of, new_pool, place_range, sample_rows
from test_gpu_parity import MAX_TOL, MEAN_TOL, check_lse, oracle_all, random_case, small, SMALL

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def ctx():
    print("creating context", flush=True)
    c = sa.Context(0)
    yield c
    c.close()


def run(ctx, w, fused, num_layers=2, layer=1):
    """One sa_segment_prefill_attn_append call over pools holding only the prefix.
    Returns the pools, the output, the LSE and the pools as they were."""
    L = layout_of(w, num_layers=num_layers)
    ip, ix = dev_i32(w.pages_indptr), dev_i32(w.pages)
    kp, vp = new_pool(w, num_layers), new_pool(w, num_layers)
    for pool, full in ((kp, w.k), (vp, w.v)):
        place_range(pool, layer, w, lambda b, full=full: full[w.prefix_rows(b)], w.pages_indptr,
                    w.pages, w.pre)
    before = (kp.clone(), vp.clone())
    T = int(w.q_indptr[-1])
    o = torch.empty((T, w.num_q_heads, 128), dtype=torch.int16, device="cuda")
    lse = torch.empty((T, w.num_q_heads), dtype=torch.float32, device="cuda")
    sa.sa_set_fused_append(ctx, fused)
    try:
        sa.sa_segment_prefill_attn_append(ctx, L, layer, dev_u16(w.q), kp, vp, dev_u16(w.k_seg()),
                                          dev_u16(w.v_seg()), w.qlen, w.kv, ip, ix, w.scale, o, lse)
        sa.sa_sync_check(ctx)
    finally:
        sa.sa_set_fused_append(ctx, False)
    return kp, vp, o, lse, before


def check_pools(w, kp, vp, before, layer=1):
    """The pools are the oracle's append applied to the pools as they were, every bit."""
    sl, ro = opages.append_destinations(w.pre, w.qlen, w.pages_indptr, w.pages, w.page_size)
    for got, was, seg in ((kp, before[0], w.k_seg()), (vp, before[1], w.v_seg())):
        want = was.clone()
        if len(sl):
            view = want[layer].permute(0, 2, 1, 3)                  # [slot][row][head][d]
            view[torch.from_numpy(sl).cuda(), torch.from_numpy(ro).cuda()] = dev_u16(seg)
        assert torch.equal(got, want)


def same_steps(w):
    """Both forms run the same kernel steps: prefixes are multiples of 4 keys (no group
    of four keys mixes prefix and segment rows) and no request has at most 32 query rows
    (the fused form sends the later key-range parts of such a request, when the plan
    splits it, through the general path)."""
    G = w.num_q_heads // w.num_kv_heads
    decode = [b for b in range(w.batch) if 0 < int(w.qlen[b]) * G <= 32]
    return all(int(p) % 4 == 0 for p in w.pre) and not decode


def check_case(ctx, w, folded=False):
    print(f"fused append {w.name}: B {w.batch} Hq {w.num_q_heads} Hkv {w.num_kv_heads} P {w.page_size} "
          f"pre {list(w.pre)[:8]} q {list(w.qlen)[:8]} folded {folded}", flush=True)
    sa.sa_set_exact_scale(ctx, not folded)
    try:
        kp, vp, o, lse, before = run(ctx, w, True)
        check_pools(w, kp, vp, before)
        del kp, vp, before
        ref, ref_lse, _ = oracle_all(w)
        mx, mean = compare(host_u16(o), ref, MAX_TOL, MEAN_TOL)
        check_lse(w, lse.cpu().numpy(), ref_lse, folded=folded)
        k2, v2, o2, lse2, before2 = run(ctx, w, False)
        check_pools(w, k2, v2, before2)
        if same_steps(w):
            assert torch.equal(o, o2)
            assert torch.equal(lse, lse2)
        else:
            compare(host_u16(o2), ref, MAX_TOL, MEAN_TOL)
            check_lse(w, lse2.cpu().numpy(), ref_lse, folded=folded)
    finally:
        sa.sa_set_exact_scale(ctx, True)
    print(f"  max {mx:.3e} mean {mean:.3e} bitwise-vs-two-launch {same_steps(w)}", flush=True)


@pytest.mark.parametrize("name", SMALL)
def test_fused_small(ctx, name):
    check_case(ctx, small(name))


@pytest.mark.parametrize("k", range(14))
def test_fused_random(ctx, k):
    check_case(ctx, random_case(k))


@pytest.mark.parametrize("seed", range(3))
def test_fused_aligned_prefixes(ctx, seed):
    """Prefixes that are multiples of 4 but not of the 64-key tile: the boundary tile
    takes page rows and segment rows group by group on the interleaved path, and the
    result equals the two-launch form bit for bit."""
    r = np.random.default_rng(9300 + seed)
    B = int(r.integers(1, 5))
    pre = [4 * int(x) for x in r.integers(1, 600, B)]
    ql = [int(x) for x in r.integers(40, 400, B)]
    w = build(f"al4_{seed}", 9300 + seed, 16, 4, 128, 16 if seed != 1 else 32, pre, ql)
    assert same_steps(w)
    check_case(ctx, w)


def test_fused_split_and_decode(ctx):
    """Key-range split items (few long requests), some of at most 32 rows that read the
    rows they wrote, and later parts that hold segment keys."""
    check_case(ctx, build("split", 21, 8, 1, 128, 16, [5000, 3000, 70, 0], [1, 1, 3, 1]))


@pytest.mark.parametrize("k", range(3))
def test_fused_mixed_decode_prefill(ctx, k):
    r = np.random.default_rng(9100 + k)
    B = int(r.integers(2, 7))
    pre = [int(x) for x in r.integers(0, 4001, B)]
    ql = [1 if r.random() < 0.5 else int(r.integers(2, 201)) for _ in range(B)]
    check_case(ctx, build("amix%d" % k, 9100 + k, 16, 4, 128, 16, pre, ql))


def test_fused_empty_segments(ctx):
    """Sequences with no new rows first, in the middle and last: they write nothing and
    produce no output rows."""
    check_case(ctx, build("empty", 9200, 8, 2, 128, 16, [40, 300, 0, 64, 17], [0, 90, 0, 130, 0]))


@pytest.mark.parametrize("name", ["ragged_g4_p16", "g8_p32_outliers", "g3_p16"])
def test_fused_folded_scale(ctx, name):
    """The same single launch with the softmax scale folded into the query rows."""
    check_case(ctx, small(name), folded=True)


def test_fused_c2_full(ctx):
    """The c2 step's append + attention at full size (8192-key prefix, 2048-token
    segment, 8 KV heads): the whole pool against the oracle's append, 128 sampled rows
    per sequence against the oracle, and the whole output and LSE against the
    two-launch form bit for bit."""
    w = workloads.make("c2")
    print("fused append c2 full", flush=True)
    kp, vp, o, lse, before = run(ctx, w, True, num_layers=1, layer=0)
    check_pools(w, kp, vp, before, layer=0)
    del kp, vp, before
    toks, heads = sample_rows(w, 128)
    ref, ref_lse, _ = oracle.attention_rows(w.q, w.k, w.v, w.q_indptr, w.kv_indptr, w.num_q_heads,
                                            w.num_kv_heads, w.scale, toks, heads)
    mx, mean = compare(host_u16(o)[toks, heads], ref, MAX_TOL, MEAN_TOL)
    check_lse(w, lse.cpu().numpy()[toks, heads], ref_lse, toks, heads)
    assert same_steps(w)
    _, _, o2, lse2, _ = run(ctx, w, False, num_layers=1, layer=0)
    assert torch.equal(o, o2)
    assert torch.equal(lse, lse2)
    print(f"  {len(toks)} rows, max {mx:.3e} mean {mean:.3e}", flush=True)


def test_fused_missing_page_is_reported(ctx):
    """A new row whose page is not in the table is skipped and reported by the fused
    launch too, and the next fused launch on the context is whole."""
    w = build("short", 51, 8, 2, 128, 16, [20], [40])
    L = layout_of(w)
    ip = dev_i32([0, 2])                          # 60 tokens need 4 pages; the table has 2
    ix = dev_i32(w.pages[:2])
    T = int(w.qlen.sum())
    kp, vp = new_pool(w), new_pool(w)
    o = torch.empty((T, w.num_q_heads, 128), dtype=torch.int16, device="cuda")
    sa.sa_set_fused_append(ctx, True)
    try:
        sa.sa_segment_prefill_attn_append(ctx, L, 0, dev_u16(w.q), kp, vp, dev_u16(w.k_seg()),
                                          dev_u16(w.v_seg()), w.qlen, w.kv, ip, ix, w.scale, o)
        with pytest.raises(sa.SaError) as e:
            sa.sa_sync_check(ctx)
        assert e.value.name == "SA_ERR_RANGE"
        sa.sa_sync_check(ctx)
    finally:
        sa.sa_set_fused_append(ctx, False)
    check_case(ctx, workloads.make("c1"))
