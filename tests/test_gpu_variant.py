"""GPU parity of the alternative attention kernels.

The library picks its attention kernel once per process (the
SA_ATTN_VARIANT environment variable; variant 0 is the software-pipelined
default the other GPU tests use, 1 the phase-separated kernel, 2 the
pipelined kernel with two key-splitting groups per block).  This test runs
the small attention parity cases, a split/merge case and the append-with-
attention entry point (a separate append launch for these kernels) in a
child process per variant, against the same oracle and tolerances.
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
