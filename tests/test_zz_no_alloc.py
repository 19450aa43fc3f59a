"""The allocation-free attention entry point (sa_segment_prefill_attn_noalloc)
against sa_segment_prefill_attn, through the C ABI.

Two calls in a row, the second on a smaller input, each compared bit for bit
with the allocating entry point on the same inputs (same plan, same kernels),
and against the oracle.  The cases include launches that split long items by
key range, whose partials then live in the fixed scratch array, and a decode +
prefill batch.  The second call's smaller plan and fewer partials overwrite the
first's: nothing of the first may leak into it.
"""
import numpy as np
import pytest
import torch

import oracle
import paper_2607_00151_amd as sa
import workloads
from workloads.configs import build

from harness import build_cache, compare, dev_u16, host_u16, layout_of

pytestmark = pytest.mark.gpu


def run(fn, ctx, w, L, kp, vp, ip, ix):
    T = int(w.qlen.sum())
    o = torch.full((T, w.num_q_heads, 128), -1, dtype=torch.int16, device="cuda")
    lse = torch.full((T, w.num_q_heads), float("nan"), dtype=torch.float32, device="cuda")
    fn(ctx, L, 0, dev_u16(w.q), kp, vp, w.qlen, w.kv, ip, ix, w.scale, o, lse)
    return o, lse


@pytest.mark.parametrize("first,second", [
    ("split_big", "split_small"),      # key-range splits both times, fewer parts the second time
    ("mixed", "c1"),                   # decode + prefill rows, then a small prefill
    ("c1", "split_small"),             # whole items, then split items
])
def test_noalloc_matches_allocating_entry_point(first, second):
    cases = {
        "split_big": lambda: build("na_split_big", 101, 8, 1, 128, 16, [9000, 6000, 70, 0, 3000],
                                   [1, 1, 3, 1, 2]),
        "split_small": lambda: build("na_split_small", 102, 8, 1, 128, 16, [5000, 20], [1, 1]),
        "mixed": lambda: build("na_mixed", 103, 16, 4, 128, 16, [3000, 1200, 40, 5000], [1, 300, 1, 64]),
        "c1": lambda: workloads.make("c1"),
    }
    with sa.Context(0) as ctx:
        for name in (first, second):
            w = cases[name]()
            print(f"no-alloc {name}: pre {list(w.pre)} q {list(w.qlen)}", flush=True)
            L = layout_of(w)
            kp, vp, ip, ix = build_cache(w)
            o_ref, lse_ref = run(sa.sa_segment_prefill_attn, ctx, w, L, kp, vp, ip, ix)
            o_na, lse_na = run(sa.sa_segment_prefill_attn_noalloc, ctx, w, L, kp, vp, ip, ix)
            sa.sa_sync_check(ctx)
            assert torch.equal(o_na, o_ref), name
            assert torch.equal(lse_na, lse_ref), name
            ref, ref_lse, _ = oracle.attention_all(w.q, w.k, w.v, w.q_indptr, w.kv_indptr, w.num_q_heads,
                                                   w.num_kv_heads, w.scale)
            mx, mean = compare(host_u16(o_na), ref, 2e-2, 2e-3)
            assert np.abs(lse_na.cpu().numpy() - ref_lse).max() <= 1e-3
            print(f"  bit-equal to sa_segment_prefill_attn; max {mx:.3e} mean {mean:.3e}", flush=True)


def test_noalloc_rejects_a_plan_beyond_its_scratch():
    """More work items than the fixed plan area holds: refused before any launch."""
    # 2 MiB / 40 B = 52428 items; 840 single-token sequences x 64 KV heads = 53760 items
    B = 840
    L = sa.Layout(num_q_heads=64, num_kv_heads=64, head_dim=128, page_size=16, num_layers=1, num_slots=64)
    ql = np.ones(B, dtype=np.int32)
    kv = ql.copy()
    with sa.Context(0) as ctx:
        q = torch.zeros((int(ql.sum()), 64, 128), dtype=torch.int16, device="cuda")
        o = torch.zeros_like(q)
        pool = torch.zeros((1, 64, 64, 16, 128), dtype=torch.int16, device="cuda")
        ip = torch.zeros(B + 1, dtype=torch.int32, device="cuda")
        ix = torch.zeros(1, dtype=torch.int32, device="cuda")
        with pytest.raises(sa.SaError) as e:
            sa.sa_segment_prefill_attn_noalloc(ctx, L, 0, q, pool, pool, ql, kv, ip, ix, 0.088, o)
        assert e.value.name == "SA_ERR_SHAPE" and "scratch" in str(e.value)
