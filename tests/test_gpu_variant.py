"""GPU parity of the alternative attention kernels and of the single-launch
append + attention.

The library picks its attention kernel once per process (the
SA_ATTN_VARIANT environment variable; variant 0 is the software-pipelined
default the other GPU tests use, 1 the phase-separated kernel, 2 the
pipelined kernel with two key-splitting groups per block).  This test runs
the small attention parity cases, a split/merge case and the append-with-
attention entry point (a separate append launch for these kernels) in a
child process per variant, against the same oracle and tolerances.  The
single-launch form of sa_segment_prefill_attn_append (SA_APPEND_IN_ATTN=1,
also chosen once per process) gets the same append-with-attention checks as
the default two-launch form, the full c2 step and the mixed c5 batch, in a
child process of its own.
"""
import os
import subprocess
import sys

import pytest

pytestmark = pytest.mark.gpu

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))

CHILD = r"""
import sys
import numpy as np
sys.path.insert(0, {root!r}); sys.path.insert(0, {tests!r})
import oracle, workloads
import paper_2607_00151_amd as sa
from workloads.configs import build
from harness import attention, build_cache, compare, dev_u16, host_u16, layout_of
from test_gpu_parity import small, SMALL, MAX_TOL, MEAN_TOL, check_lse
ctx = sa.Context(0)
cases = [(n, small(n)) for n in SMALL]
cases.append(("split", build("split", 21, 8, 1, 128, 16, [5000, 3000, 70, 0], [1, 1, 3, 1])))
for name, w in cases:
    print("variant {variant} attention", name, flush=True)
    L = layout_of(w)
    kp, vp, ip, ix = build_cache(w)
    o, lse = attention(ctx, w, L, dev_u16(w.q), kp, vp, ip, ix)
    sa.sa_sync_check(ctx)
    ref, ref_lse, _ = oracle.attention_all(w.q, w.k, w.v, w.q_indptr, w.kv_indptr,
                                           w.num_q_heads, w.num_kv_heads, w.scale)
    mx, mean = compare(host_u16(o), ref, MAX_TOL, MEAN_TOL)
    check_lse(w, lse.cpu().numpy(), ref_lse, folded={folded})
    print("  ok max %.3e mean %.3e" % (mx, mean), flush=True)
from test_gpu_parity import check_attention_append
print("variant {variant} attention with append (separate append launch)", flush=True)
check_attention_append(ctx, small("ragged_g4_p16"), folded={folded})
ctx.close()
print("ALL-OK", flush=True)
"""


@pytest.mark.timeout(300)
@pytest.mark.parametrize("variant", [1, 2])
def test_variant_kernel_parity(variant):
    # variant 1 always scales each score in fp32, variant 2 always folds the scale into q
    code = CHILD.format(root=ROOT, tests=os.path.join(ROOT, "tests"), variant=variant, folded=variant == 2)
    env = dict(os.environ, SA_ATTN_VARIANT=str(variant))
    r = subprocess.run([sys.executable, "-u", "-c", code], env=env, cwd=ROOT,
                       capture_output=True, text=True, timeout=280)
    print(r.stdout[-4000:])
    print(r.stderr[-2000:])
    assert r.returncode == 0 and "ALL-OK" in r.stdout


CHILD_APPEND = r"""
import sys
sys.path.insert(0, {root!r}); sys.path.insert(0, {tests!r})
import workloads
import paper_2607_00151_amd as sa
from workloads.configs import build
from test_gpu_parity import (small, SMALL, check_attention_append, check_step, check_direct,
                             test_append_inside_attention_missing_page_is_reported)
ctx = sa.Context(0)
sa.sa_set_exact_scale(ctx, False)      # the single-launch append runs in the folded-scale mode
for n in SMALL:
    print("append in attention", n, flush=True)
    check_attention_append(ctx, small(n), folded=True)
print("append in attention, split", flush=True)
check_attention_append(ctx, build("split", 21, 8, 1, 128, 16, [5000, 3000, 70, 0], [1, 1, 3, 1]), folded=True)
print("append in attention, missing page", flush=True)
test_append_inside_attention_missing_page_is_reported(ctx, folded=True)
from test_gpu_parity import random_case
import numpy as np
for k in range(6):
    print("append in attention, random shape", k, flush=True)
    check_attention_append(ctx, random_case(k), launches=1, folded=True)
for k in range(4):
    r = np.random.default_rng(9100 + k)
    B = int(r.integers(2, 7))
    pre = [int(x) for x in r.integers(0, 4001, B)]
    ql = [1 if r.random() < 0.5 else int(r.integers(2, 201)) for _ in range(B)]
    print("append in attention, mixed decode/prefill", k, pre, ql, flush=True)
    check_attention_append(ctx, build("amix%d" % k, 9100 + k, 16, 4, 128, 16, pre, ql), launches=1, folded=True)
print("append in attention, c2 step", flush=True)
check_step(ctx, workloads.make("c2"), per_seq_rows=128, mode="attn_append", folded=True)
print("append in attention, c5", flush=True)
check_direct(ctx, workloads.make("c5"), per_seq_rows=16, fused=True, folded=True)
ctx.close()
print("ALL-OK", flush=True)
"""


@pytest.mark.timeout(400)
def test_append_in_attention_kernel_parity():
    code = CHILD_APPEND.format(root=ROOT, tests=os.path.join(ROOT, "tests"))
    env = dict(os.environ, SA_APPEND_IN_ATTN="1")
    r = subprocess.run([sys.executable, "-u", "-c", code], env=env, cwd=ROOT,
                       capture_output=True, text=True, timeout=380)
    print(r.stdout[-4000:])
    print(r.stderr[-2000:])
    assert r.returncode == 0 and "ALL-OK" in r.stdout
