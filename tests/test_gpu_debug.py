"""GPU checks of the debug and sizing calls.

* SA_DEBUG=1 (read once per process, so in a child process): a valid splice,
  splice + append and append run and match the oracle's page definitions; a
  free list that repeats a slot, one that hands out a surviving source slot,
  and two sequences appending to the same rows are refused with
  SA_ERR_OVERLAP before anything is launched (the pools are unchanged).
* sa_reserve: after reserving, plans small and large (attention with and
  without key-range splits, splices) give the same bits as on a fresh context.
"""
import os
import subprocess
import sys

import numpy as np
import pytest
import torch

import paper_2607_00151_amd as sa
import workloads
from oracle import pages as opages
from workloads.configs import build

from harness import (attention, build_cache, build_source_cache, dev_i32, dev_u16, host_u16, layout_of,
                     new_pool, place_range)

pytestmark = pytest.mark.gpu

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))

CHILD = r"""
import sys
sys.path.insert(0, {root!r}); sys.path.insert(0, {tests!r})
import numpy as np, torch
import paper_2607_00151_amd as sa
from oracle import pages as opages
from workloads.configs import build
from harness import build_source_cache, dev_i32, dev_u16, host_u16, layout_of, new_pool, place_range
ctx = sa.Context(0)
w = build("dbg", 81, 8, 2, 128, 16, [300, 40, 77], [100, 33, 5], assemble=True)
a = w.asm
L = layout_of(w)

def splice(fresh, append):
    kp, vp, sip, sid, _ = build_source_cache(w)
    before = (host_u16(kp), host_u16(vp))
    dip = torch.zeros(w.batch + 1, dtype=torch.int32, device="cuda")
    did = torch.full((len(a.fresh),), -1, dtype=torch.int32, device="cuda")
    try:
        if append:
            sa.sa_kv_assemble_append(ctx, L, kp, vp, kp, vp, a.src_len, a.keep_indptr, a.keep_spans, a.reserve,
                                     sip, sid, dev_i32(fresh), dip, did, 0, dev_u16(w.k_seg()), dev_u16(w.v_seg()),
                                     w.qlen)
        else:
            sa.sa_kv_assemble(ctx, L, kp, vp, kp, vp, a.src_len, a.keep_indptr, a.keep_spans, a.reserve, sip, sid,
                              dev_i32(fresh), dip, did)
        sa.sa_sync_check(ctx)
        return None, kp, vp, dip, did
    except sa.SaError as e:
        torch.cuda.synchronize()
        assert np.array_equal(host_u16(kp), before[0]) and np.array_equal(host_u16(vp), before[1])
        return e.name, kp, vp, dip, did

for append in (False, True):
    err, kp, vp, dip, did = splice(a.fresh, append)
    assert err is None, err
    r = opages.assemble(a.src_len, a.src_indptr, a.src_indices, a.keep_indptr, a.keep_spans, a.reserve,
                        a.fresh, w.page_size)
    assert np.array_equal(did.cpu().numpy()[: r["dst_indptr"][-1]], r["dst_indices"])
    print("debug: valid splice (append %s) ok" % append, flush=True)
    bad = a.fresh.copy(); bad[3] = bad[1]
    assert splice(bad, append)[0] == "SA_ERR_OVERLAP"
    print("debug: repeated free slot refused", flush=True)
    bad = a.fresh.copy(); bad[0] = a.src_indices[0]
    assert splice(bad, append)[0] == "SA_ERR_OVERLAP"
    print("debug: surviving slot in the free list refused", flush=True)
    bad = a.fresh.copy(); bad[2] = w.num_slots + 3
    assert splice(bad, append)[0] == "SA_ERR_RANGE"
    print("debug: free slot out of range refused", flush=True)

# append: two sequences on the same rows of one slot
kp, vp = new_pool(w), new_pool(w)
ip = dev_i32(w.pages_indptr)
good = w.pages.copy()
sa.sa_kv_append(ctx, L, 0, kp, vp, dev_u16(w.k_seg()), dev_u16(w.v_seg()), w.pre, w.qlen, ip, dev_i32(good))
sa.sa_sync_check(ctx)
clash = good.copy()
p1 = int(w.pages_indptr[1]) + int(w.pre[1]) // 16     # the page sequence 1 appends to
p0 = int(w.pages_indptr[0]) + int(w.pre[0]) // 16     # the page sequence 0 appends to
clash[p1] = clash[p0]
try:
    sa.sa_kv_append(ctx, L, 0, kp, vp, dev_u16(w.k_seg()), dev_u16(w.v_seg()), w.pre, w.qlen, ip, dev_i32(clash))
    raise AssertionError("overlapping append accepted")
except sa.SaError as e:
    assert e.name == "SA_ERR_OVERLAP", e.name
print("debug: overlapping append refused", flush=True)
ctx.close()
print("ALL-OK", flush=True)
"""


@pytest.mark.timeout(300)
def test_debug_checks_refuse_overlapping_slots():
    code = CHILD.format(root=ROOT, tests=os.path.join(ROOT, "tests"))
    env = dict(os.environ, SA_DEBUG="1")
    r = subprocess.run([sys.executable, "-u", "-c", code], env=env, cwd=ROOT, capture_output=True, text=True,
                       timeout=280)
    print(r.stdout[-4000:])
    print(r.stderr[-3000:])
    assert r.returncode == 0 and "ALL-OK" in r.stdout


def test_reserve_then_plans_of_every_size():
    """sa_reserve sizes the buffers; plans below and above the reservation, and a split
    launch, give the bits a fresh context gives."""
    print("reserve", flush=True)
    cases = [build("res_small", 91, 8, 2, 128, 16, [100], [20]),
             build("res_split", 92, 8, 1, 128, 16, [5000, 3000, 70, 0], [1, 1, 3, 1]),
             workloads.make("c1"),
             build("res_big", 93, 32, 8, 128, 16, [4000, 700], [1500, 900])]
    with sa.Context(0) as fresh_ctx, sa.Context(0) as ctx:
        sa.sa_reserve(ctx, 1 << 16, 1 << 20)
        for w in cases:
            L = layout_of(w)
            kp, vp, ip, ix = build_cache(w)
            o1, l1 = attention(fresh_ctx, w, L, dev_u16(w.q), kp, vp, ip, ix)
            o2, l2 = attention(ctx, w, L, dev_u16(w.q), kp, vp, ip, ix)
            sa.sa_sync_check(ctx)
            assert torch.equal(o1, o2) and torch.equal(l1, l2), w.name
        with pytest.raises(sa.SaError):
            sa.sa_reserve(ctx, -1, 0)


@pytest.mark.parametrize("where", ["first", "middle", "last", "all_but_one"])
def test_empty_sequences_in_a_batch(where):
    """Sequences with q_len = 0 (nothing to prefill) at the front, in the middle, at the
    end: attention skips them, the others match the oracle; append and splice + append
    leave their pages alone (pools compared whole against the oracle's definitions)."""
    import oracle
    pre = [300, 40, 900, 0, 77]
    ql = [100, 33, 60, 20, 5]
    empty = {"first": [0], "middle": [2], "last": [4], "all_but_one": [0, 1, 2, 4]}[where]
    for b in empty:
        ql[b] = 0
    w = build(f"empty_{where}", 95, 8, 2, 128, 16, pre, ql, assemble=True)
    print(f"empty sequences {where}: q {ql}", flush=True)
    L = layout_of(w)
    with sa.Context(0) as ctx:
        kp, vp, ip, ix = build_cache(w)
        o, lse = attention(ctx, w, L, dev_u16(w.q), kp, vp, ip, ix)
        sa.sa_sync_check(ctx)
        ref, ref_lse, _ = oracle.attention_all(w.q, w.k, w.v, w.q_indptr, w.kv_indptr, w.num_q_heads,
                                               w.num_kv_heads, w.scale)
        from harness import compare
        compare(host_u16(o), ref, 2e-2, 2e-3)
        assert np.abs(lse.cpu().numpy() - ref_lse).max() <= 1e-3
        # append of the segments onto the prefixes: whole pools bit for bit
        kp2, vp2 = new_pool(w), new_pool(w)
        for pool, full in ((kp2, w.k), (vp2, w.v)):
            place_range(pool, 0, w, lambda b, full=full: full[w.prefix_rows(b)], w.pages_indptr, w.pages, w.pre)
        want = [host_u16(kp2), host_u16(vp2)]
        sa.sa_kv_append(ctx, L, 0, kp2, vp2, dev_u16(w.k_seg()), dev_u16(w.v_seg()), w.pre, w.qlen, ip, ix)
        sa.sa_sync_check(ctx)
        sl, ro = opages.append_destinations(w.pre, w.qlen, w.pages_indptr, w.pages, w.page_size)
        for wa, new, got in ((want[0], w.k_seg(), kp2), (want[1], w.v_seg(), vp2)):
            opages.apply_append(wa[0], new, sl, ro)
            assert np.array_equal(host_u16(got), wa)
        # splice + append in one launch: whole pools and the destination table
        a = w.asm
        kp3, vp3, sip, sid, fresh = build_source_cache(w)
        want = [host_u16(kp3).copy(), host_u16(vp3).copy()]
        dip = torch.zeros(w.batch + 1, dtype=torch.int32, device="cuda")
        did = torch.full((len(a.fresh),), -1, dtype=torch.int32, device="cuda")
        kept = sa.sa_kv_assemble_append(ctx, L, kp3, vp3, kp3, vp3, a.src_len, a.keep_indptr, a.keep_spans,
                                        a.reserve, sip, sid, fresh, dip, did, 0, dev_u16(w.k_seg()),
                                        dev_u16(w.v_seg()), w.qlen)
        sa.sa_sync_check(ctx)
        r = opages.assemble(a.src_len, a.src_indptr, a.src_indices, a.keep_indptr, a.keep_spans, a.reserve,
                            a.fresh, w.page_size)
        assert np.array_equal(kept, r["dst_len"])
        assert np.array_equal(dip.cpu().numpy(), r["dst_indptr"])
        assert np.array_equal(did.cpu().numpy()[: r["dst_indptr"][-1]], r["dst_indices"])
        sl, ro = opages.append_destinations(r["dst_len"], w.qlen, r["dst_indptr"], r["dst_indices"], w.page_size)
        for wa, seg, got in ((want[0], w.k_seg(), kp3), (want[1], w.v_seg(), vp3)):
            for s_, d_ in zip(r["copy_src"], r["copy_dst"]):
                wa[0, d_] = wa[0, s_]
            opages.apply_append(wa[0], seg, sl, ro)
            assert np.array_equal(host_u16(got), wa)
