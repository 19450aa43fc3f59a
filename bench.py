"""Benchmark of one segment re-prefill step on one MI355X.

Workload (Llama-3-8B-shaped attention layer): 32 query heads, 8 KV heads,
head_dim 128, bf16, page size 16.  A cached context of 683 pages (10928
tokens) is spliced by dropping a contiguous run of 171 pages (25%), leaving an
8192-token prefix; a 2048-token transformed segment is appended after it and
its causal grouped-query attention is computed over prefix + segment.

One step = splice, append of the segment's K/V, attention, all on the current
stream with inputs resident in HBM.  --fuse picks the entry points:
"splice" (default): sa_kv_assemble_append (splice and append in one launch)
-> sa_segment_prefill_attn; "attn": sa_kv_assemble ->
sa_segment_prefill_attn_append with sa_set_fused_append on (the attention
launch writes the segment's rows and reads the segment's keys from k_new /
v_new); "none": sa_kv_assemble
-> sa_kv_append -> sa_segment_prefill_attn.  Every step uses one of R
disjoint copies of the cache (default 8 x 128 MB per pool), so the 256 MB
Infinity Cache cannot hold the data a step reads from its previous use.

Prints one JSON line.  `value` is segment tokens per second over K whole
steps timed between two events on the launch stream; per-kernel averages come
from HIP events recorded on that stream around every call in a second pass of
K steps (`ms_per_step_instrumented` is that pass's step time); the attention
kernel's time comes from a pair of events the library binds to the kernel
launch itself (sa_set_kernel_events), the time rocprofv3's kernel trace
reports; the page kernels of the step are timed the same way.  The timed
steps plan the attention with the XCD speeds the run measures on its own
launches (sa_set_xcd_weights); `attn.without_xcd_weights` is the same kernel
placed without them.  Context measured in the same run: torch's bf16 GEMM
(`gemm_reference`, the practical MFMA rate) and plain device copies of the
step's and the 32-layer splice's bytes (`copy_reference`, the practical HBM
rate).
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_BF16_TFLOPS = 2516.6      # MI355X dense bf16 MFMA: 256 CU x 4096 flop/clk x 2.4 GHz
PEAK_HBM_GBS = 8000.0


def parse():
    p = argparse.ArgumentParser()
    p.add_argument("--gpus", type=int, default=1)
    p.add_argument("--steps", type=int, default=50)
    p.add_argument("--warmup", type=int, default=100,
                   help="untimed steps first (the clock takes tens of steps to settle)")
    p.add_argument("--rotate", type=int, default=8, help="disjoint cache copies cycled per step")
    p.add_argument("--fuse", choices=("attn", "splice", "none"), default="splice",
                   help="which launch carries the append (see the module docstring)")
    p.add_argument("--folded-scale", action="store_true",
                   help="fast mode: fold the softmax scale into the bf16 query rows "
                        "(sa_set_exact_scale(ctx, 0)); the default applies it to each fp32 score")
    p.add_argument("--no-cpu-baseline", action="store_true")
    p.add_argument("--no-xcd-weights", action="store_true",
                   help="skip measuring the XCDs' speeds and weighing the attention planner by them")
    p.add_argument("--no-gemm-reference", action="store_true",
                   help="skip timing torch's bf16 GEMM (context for the MFMA roofline)")
    p.add_argument("--cpu-stride", type=int, default=1, help="oracle sample: every n-th token")
    p.add_argument("--assemble-layers", type=int, default=32,
                   help="layers of the separate all-layer assemble measurement (0: skip)")
    p.add_argument("--config", choices=("c1", "c2", "c3", "c4", "c5"), default="c2",
                   help="workload; c2 is the benchmark line, the others are measured the same way "
                        "(splice where the configuration has one, append, attention) without rotation")
    p.add_argument("--assemble-only", choices=("shuffled", "contiguous"), default=None,
                   help="time only the c2 commit splice over --assemble-layers layers, on the shuffled page "
                        "placement of the workload or on an identity placement (surviving pages and fresh "
                        "slots each one contiguous run): the same kernel and bytes, with and without the "
                        "address spread")
    p.add_argument("--copy-bytes", type=int, default=0,
                   help="instead of the step, time a plain device copy of this many bytes "
                        "(calibrates the FETCH_SIZE / WRITE_SIZE counters)")
    return p.parse_args()


def dev_u16(a):
    """uint16 bit patterns -> int16 device tensor (same bits)."""
    import torch
    return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).cuda()


def dev_i32(a):
    import torch
    return torch.from_numpy(np.ascontiguousarray(np.asarray(a, dtype=np.int32))).cuda()


def new_pool(num_slots, Hkv, P, layers=1):
    import torch
    return torch.zeros((layers, num_slots, Hkv, P, 128), dtype=torch.int16, device="cuda")


def fill_cache(ctx, L, kp, vp, k_rows, v_rows, lengths, indptr, indices):
    """Write each sequence's first lengths[b] cache rows (k_rows / v_rows, sequences
    back to back) at its logical positions 0.. through the page table, with the
    library's own append kernel (set-up, outside every timed region)."""
    import paper_2607_00151_amd as sa
    sa.sa_kv_append(ctx, L, 0, kp, vp, dev_u16(k_rows), dev_u16(v_rows), np.zeros(len(lengths), np.int32),
                    lengths, indptr, indices)
    sa.sa_sync_check(ctx)


def source_cache(ctx, L, w, kp, vp, src_indices_dev):
    """The splice's source cache (kept prefix with the dropped pages in place)."""
    from workloads.configs import source_rows
    a = w.asm
    k = np.concatenate([source_rows(w, b, "k") for b in range(w.batch)])
    v = np.concatenate([source_rows(w, b, "v") for b in range(w.batch)])
    fill_cache(ctx, L, kp, vp, k, v, a.src_len, dev_i32(a.src_indptr), src_indices_dev)


def source_digest() -> str:
    """Hash of the attention kernel sources and of the planner that places its
    work items (which decides how often K/V cross an XCD's L2); counter figures
    taken for another version of either are not reported."""
    import hashlib
    h = hashlib.sha256()
    for f in ("attn_kernel.h", "attn_pipe.h", "common.h", "plan.h"):
        with open(os.path.join(ROOT, "paper_2607_00151_amd", "csrc", f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


def stored_traffic(kernel: str, algorithmic: float):
    """HBM bytes per launch from the committed counter summary, if it was taken
    on the current kernel sources (else None)."""
    path = os.path.join(ROOT, "profiles", "traffic.json")
    if not os.path.exists(path):
        return None
    with open(path) as f:
        t = json.load(f)
    k = t.get("kernels", {}).get(kernel)
    if not k or k.get("source_digest") != source_digest():
        return None
    fetch = k["fetch_kib_per_launch"] * 1024 * t["copy_calibration"]["fetch_factor"]
    write = k["write_kib_per_launch"] * 1024 * t["copy_calibration"]["write_factor"]
    return {"bytes": fetch + write, "fetch_bytes": fetch, "write_bytes": write,
            "algorithmic_bytes": algorithmic, "ratio_to_algorithmic": (fetch + write) / algorithmic}


def calibrate_xcds(ctx, run, launches: int = 5, settle: int = 20, refine: int = 2):
    """This GPU's XCD speeds, handed to the attention planner (sa_set_xcd_weights).
    In the configurations timed here every XCD runs the same work (the KV heads
    map one to one onto the 8 XCDs), so each XCD's mean workgroup time over a
    few launches, from the device clock each workgroup records
    (sa_set_block_clock), is inversely proportional to its speed; `refine`
    rounds then scale each XCD's speed by how late its last workgroup ends
    under the weights.  run(i) runs one step; the steps after the weights are
    set let the new plan settle."""
    import torch
    import paper_2607_00151_amd as sa
    cbuf = torch.full((4 * 65536,), -1, dtype=torch.int64, device="cuda")
    sa.sa_set_block_clock(ctx, cbuf)
    acc = np.zeros(8)
    for i in range(launches):
        cbuf.fill_(-1)
        run(i)
        torch.cuda.synchronize()
        r = cbuf.view(-1, 4).cpu().numpy()
        ids = np.nonzero((r[:, 0] != -1) & ((r[:, 3] & 0xffffffff) != 0))[0]
        acc += [float(np.mean(r[ids[ids % 8 == x], 1] - r[ids[ids % 8 == x], 0])) for x in range(8)]
    speed = acc.mean() / acc
    sa.sa_set_xcd_weights(ctx, speed)
    # then correct the estimate on what the weights are for, the time each XCD's
    # last workgroup ends: an XCD that still ends late gets less speed credit
    n = launches
    for _ in range(refine):
        ends = np.zeros(8)
        for i in range(launches):
            cbuf.fill_(-1)
            run(n)
            n += 1
            torch.cuda.synchronize()
            r = cbuf.view(-1, 4).cpu().numpy()
            ids = np.nonzero((r[:, 0] != -1) & ((r[:, 3] & 0xffffffff) != 0))[0]
            t0 = r[ids, 0].min()
            ends += [float(r[ids[ids % 8 == x], 1].max() - t0) for x in range(8)]
        speed = speed * (ends.mean() / ends)
        speed = speed / speed.mean()
        sa.sa_set_xcd_weights(ctx, speed)
    sa.sa_set_block_clock(ctx, None)
    for i in range(settle):
        run(n + i)
    sa.sa_sync_check(ctx)
    torch.cuda.synchronize()
    return speed


def gemm_reference(n: int = 8192, reps: int = 30):
    """Context for the MFMA roofline: torch's own bf16 GEMM (hipBLASLt) of
    n x n x n on the same GPU, in the same run."""
    import torch
    a = torch.randn(n, n, device="cuda", dtype=torch.bfloat16)
    b = torch.randn(n, n, device="cuda", dtype=torch.bfloat16)
    for _ in range(10):
        c = a @ b
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
    torch.cuda.synchronize()
    ev[0].record()
    for _ in range(reps):
        c = a @ b
    ev[1].record()
    torch.cuda.synchronize()
    ms = ev[0].elapsed_time(ev[1]) / reps
    tflops = 2.0 * n ** 3 / (ms * 1e-3) / 1e12
    del a, b, c
    return {"kind": f"torch.matmul bf16 {n}x{n}x{n} (hipBLASLt)", "ms": ms, "tflops": tflops,
            "frac_of_bf16_peak": tflops / PEAK_BF16_TFLOPS}


def copy_rate(nbytes: int, steps: int = 30, warmup: int = 10) -> dict:
    """A plain device copy (torch's copy kernel) of nbytes, the practical rate for the page
    kernels at the same byte count.  Enough source / destination pairs rotate that their
    footprint exceeds the 256 MB Infinity Cache (1 GiB or more); each copy is timed by its
    own events and the median reported."""
    import torch
    n = nbytes // 2
    pairs = max(2, -(-(1 << 30) // (2 * nbytes)))
    src = [torch.empty(n, dtype=torch.int16, device="cuda").fill_(1) for _ in range(pairs)]
    dst = [torch.empty_like(src[0]) for _ in range(pairs)]
    for i in range(warmup):
        dst[i % pairs].copy_(src[i % pairs])
    torch.cuda.synchronize()
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(steps)]
    for i, (a, b) in enumerate(ev):
        a.record()
        dst[i % pairs].copy_(src[(i + 1) % pairs])
        b.record()
    torch.cuda.synchronize()
    ms = float(np.median([a.elapsed_time(b) for a, b in ev]))
    del src, dst
    gbs = 4 * n / (ms * 1e-3) / 1e9
    return {"bytes_read": 2 * n, "bytes_written": 2 * n, "buffer_pairs": pairs, "ms": ms, "gbs": gbs,
            "frac_of_hbm": gbs / PEAK_HBM_GBS}


def copy_mode(nbytes: int, steps: int, warmup: int):
    print(json.dumps({"mode": "copy", **copy_rate(nbytes, steps, warmup)}), flush=True)


def assemble_mode(args):
    """The c2 commit splice of every layer in one launch, timed by kernel events, on
    the workload's shuffled page placement or on a contiguous one."""
    import torch
    import paper_2607_00151_amd as sa
    import workloads
    w = workloads.make("c2")
    a = w.asm
    NL, Hkv, P = max(1, args.assemble_layers), w.num_kv_heads, w.page_size
    n_src = int(a.src_indptr[-1])
    if args.assemble_only == "contiguous":
        src_ix = np.arange(n_src, dtype=np.int32)
        fresh = np.arange(n_src, n_src + len(a.fresh), dtype=np.int32)
        slots = n_src + len(a.fresh)
    else:
        src_ix, fresh, slots = a.src_indices, a.fresh, w.num_slots
    L = sa.Layout(num_q_heads=w.num_q_heads, num_kv_heads=Hkv, head_dim=128, page_size=P, num_layers=NL,
                  num_slots=slots)
    kl = torch.zeros((NL, slots, Hkv, P, 128), dtype=torch.int16, device="cuda")
    vl = torch.zeros_like(kl)
    sip, sid, fr = dev_i32(a.src_indptr), dev_i32(src_ix), dev_i32(fresh)
    dip = torch.zeros(w.batch + 1, dtype=torch.int32, device="cuda")
    did = torch.zeros(len(a.fresh), dtype=torch.int32, device="cuda")
    ctx = sa.Context(0)
    stream = torch.cuda.current_stream()

    def run():
        sa.sa_kv_assemble(ctx, L, kl, vl, kl, vl, a.src_len, a.keep_indptr, a.keep_spans, a.reserve, sip, sid,
                          fr, dip, did)
    for _ in range(args.warmup):
        run()
    torch.cuda.synchronize()
    ev = [[torch.cuda.Event(enable_timing=True) for _ in range(2)] for _ in range(args.steps)]
    for e in ev:
        e[0].record(stream)
        e[1].record(stream)
    torch.cuda.synchronize()
    for e in ev:
        sa.sa_set_kernel_events(ctx, sa.TIMED_PAGES, e[0].cuda_event, e[1].cuda_event)
        run()
    sa.sa_set_kernel_events(ctx, sa.TIMED_PAGES)
    torch.cuda.synchronize()
    sa.sa_sync_check(ctx)
    ms = float(np.median([e[0].elapsed_time(e[1]) for e in ev]))
    kept_pages = int(sum(e - b for b, e in a.keep_spans))
    n_dst = int(sum(-(-int(x + y) // P) for x, y in zip(w.pre, w.qlen)))
    nbytes = 2 * kept_pages * 2 * Hkv * P * 128 * 2 * NL + 4 * (n_dst + kept_pages + w.batch + 1)
    ctx.close()
    print(json.dumps({"mode": "assemble", "placement": args.assemble_only, "layers": NL, "pages": kept_pages,
                      "bytes": nbytes, "ms": ms, "gbs": nbytes / (ms * 1e-3) / 1e9,
                      "frac_of_hbm": nbytes / (ms * 1e-3) / 1e9 / PEAK_HBM_GBS}), flush=True)


def config_mode(args):
    """One configuration other than the benchmark line: each step is the splice with
    the append (configurations with an assembly step) or the append alone, then the
    attention, on one cache (these caches exceed the 256 MB Infinity Cache, c1 aside)."""
    import torch
    import paper_2607_00151_amd as sa
    if not os.path.exists(sa.library_path()):
        from paper_2607_00151_amd import build
        build.build()
    import workloads

    w = workloads.make(args.config)
    L = sa.Layout(num_q_heads=w.num_q_heads, num_kv_heads=w.num_kv_heads, head_dim=128,
                  page_size=w.page_size, num_layers=1, num_slots=w.num_slots)
    T = int(w.qlen.sum())
    Hkv, P, Hq = w.num_kv_heads, w.page_size, w.num_q_heads
    q, ks, vs = dev_u16(w.q), dev_u16(w.k_seg()), dev_u16(w.v_seg())
    o = torch.empty((T, Hq, 128), dtype=torch.int16, device="cuda")
    lse = torch.empty((T, Hq), dtype=torch.float32, device="cuda")
    ctx = sa.Context(0)
    if args.folded_scale:
        sa.sa_set_exact_scale(ctx, False)
    stream = torch.cuda.current_stream()
    app_bytes = 2 * T * Hkv * 128 * 2 * 2
    a = w.asm
    kp, vp = new_pool(w.num_slots, Hkv, P), new_pool(w.num_slots, Hkv, P)
    if a is not None:
        sip, sid, fresh = dev_i32(a.src_indptr), dev_i32(a.src_indices), dev_i32(a.fresh)
        source_cache(ctx, L, w, kp, vp, sid)
        dip = torch.zeros(w.batch + 1, dtype=torch.int32, device="cuda")
        did = torch.zeros(len(a.fresh), dtype=torch.int32, device="cuda")
        kept_pages = int(sum(e - b for b, e in a.keep_spans))
        n_dst = int(sum(-(-int(x + y) // P) for x, y in zip(w.pre, w.qlen)))
        splice_bytes = 2 * kept_pages * 2 * Hkv * P * 128 * 2 + 4 * (n_dst + kept_pages + w.batch + 1)
        if args.fuse == "none":
            # the splice alone is timed; the append follows it in the attention's window
            first_bytes, first_name = splice_bytes, "assemble"

            def first():
                kept = sa.sa_kv_assemble(ctx, L, kp, vp, kp, vp, a.src_len, a.keep_indptr, a.keep_spans,
                                         a.reserve, sip, sid, fresh, dip, did)
                return kept
        else:
            first_bytes, first_name = splice_bytes + app_bytes, "splice_append"

            def first():
                return sa.sa_kv_assemble_append(ctx, L, kp, vp, kp, vp, a.src_len, a.keep_indptr,
                                                a.keep_spans, a.reserve, sip, sid, fresh, dip, did, 0, ks, vs,
                                                w.qlen)
        pages = (dip, did)
    else:
        ip, ix = dev_i32(w.pages_indptr), dev_i32(w.pages)
        pre_k = np.concatenate([w.k[w.prefix_rows(b)] for b in range(w.batch)])
        pre_v = np.concatenate([w.v[w.prefix_rows(b)] for b in range(w.batch)])
        fill_cache(ctx, L, kp, vp, pre_k, pre_v, w.pre, ip, ix)
        first_bytes, first_name = app_bytes, "append"

        def first():
            sa.sa_kv_append(ctx, L, 0, kp, vp, ks, vs, w.pre, w.qlen, ip, ix)
            return w.pre
        pages = (ip, ix)

    def step(ev=None):
        if ev is not None:
            ev[0].record(stream)
        kept = first()
        if ev is not None:
            ev[1].record(stream)
        if a is not None and args.fuse == "none":
            sa.sa_kv_append(ctx, L, 0, kp, vp, ks, vs, kept, w.qlen, pages[0], pages[1])
        sa.sa_segment_prefill_attn(ctx, L, 0, q, kp, vp, w.qlen, kept + w.qlen, pages[0], pages[1], w.scale, o, lse)
        if ev is not None:
            ev[2].record(stream)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    sa.sa_sync_check(ctx)
    # the XCD-speed weights are for launches of at most two rounds of workgroups
    # (c2); these configurations launch many rounds, which the planner leaves as
    # placed
    xcd_speed = None
    K = args.steps
    t0, t1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    t0.record(stream)
    for _ in range(K):
        step()
    t1.record(stream)
    torch.cuda.synchronize()
    ms_per_step = t0.elapsed_time(t1) / K
    evs = [[torch.cuda.Event(enable_timing=True) for _ in range(3)] for _ in range(K)]
    # kernel events bound to the attention kernel and to the first page kernel
    # of the step (sa_set_kernel_events): their execution on the device
    kev = [[torch.cuda.Event(enable_timing=True) for _ in range(4)] for _ in range(K)]
    for e in kev:
        for x in e:
            x.record(stream)
    torch.cuda.synchronize()
    one_page_kernel = not (a is not None and args.fuse == "none")
    for e, k in zip(evs, kev):
        sa.sa_set_kernel_events(ctx, sa.TIMED_ATTN, k[0].cuda_event, k[1].cuda_event)
        if one_page_kernel:
            sa.sa_set_kernel_events(ctx, sa.TIMED_PAGES, k[2].cuda_event, k[3].cuda_event)
        step(e)
    sa.sa_set_kernel_events(ctx, sa.TIMED_ATTN)
    sa.sa_set_kernel_events(ctx, sa.TIMED_PAGES)
    torch.cuda.synchronize()
    sa.sa_sync_check(ctx)
    first_call_ms = float(np.mean([e[0].elapsed_time(e[1]) for e in evs]))
    first_ms = float(np.mean([k[2].elapsed_time(k[3]) for k in kev])) if one_page_kernel else first_call_ms
    attn_call_ms = float(np.mean([e[1].elapsed_time(e[2]) for e in evs]))
    attn_kernel_ms = float(np.mean([k[0].elapsed_time(k[1]) for k in kev]))
    attn_ms = attn_kernel_ms
    flops = w.attn_flops()
    tflops = flops / (attn_ms * 1e-3) / 1e12
    rec = {
        "metric": "segment-prefill tokens/s + attn TFLOP/s (% MFMA peak); KV assemble GB/s (% HBM)",
        "value": T / (ms_per_step * 1e-3), "unit": "tokens/s", "n_gpus": 1, "steps": K, "warmup": args.warmup,
        "ms_per_step": ms_per_step, "higher_is_better": True, "dtype": "bf16", "data": "synthetic",
        "config": {"workload": f"{w.name}: batch {w.batch}, Hq {Hq} / Hkv {Hkv} / d 128, page {P}, "
                               f"prefix {int(w.pre.min())}..{int(w.pre.max())}, segment {int(w.qlen.min())}.."
                               f"{int(w.qlen.max())}", "segment_tokens": T, "cached_keys": int(w.kv.sum())},
        "attn": {"ms": attn_ms, "timing": "kernel events (the attention kernel; a split launch's merge not "
                                          "included)", "call_ms": attn_call_ms,
                 "xcd_speeds": None if xcd_speed is None else [round(float(x), 4) for x in xcd_speed],
                 "gflop": flops / 1e9, "tflops": tflops, "frac_of_bf16_peak": tflops / PEAK_BF16_TFLOPS},
        first_name: {"ms": first_ms, "timing": "kernel events" if one_page_kernel else "call events",
                     "call_ms": first_call_ms, "bytes": first_bytes, "gbs": first_bytes / (first_ms * 1e-3) / 1e9,
                     "frac_of_hbm": first_bytes / (first_ms * 1e-3) / 1e9 / PEAK_HBM_GBS},
    }
    dec = w.qlen == 1
    if dec.any() and not dec.all():
        # the same launch over only the decode rows, and over only the prefill segments
        for name, sel in (("decode_only", dec), ("prefill_only", ~dec)):
            rows = np.concatenate([np.arange(w.q_indptr[b], w.q_indptr[b + 1]) for b in np.nonzero(sel)[0]])
            qs = dev_u16(w.q[rows])
            os_ = torch.empty((len(rows), Hq, 128), dtype=torch.int16, device="cuda")
            ql = np.where(sel, w.qlen, 0)
            sub = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(K)]
            for x, y in sub:
                x.record(stream)
                y.record(stream)
            for i in range(args.warmup + K):
                if i >= args.warmup:
                    x, y = sub[i - args.warmup]
                    sa.sa_set_kernel_events(ctx, sa.TIMED_ATTN, x.cuda_event, y.cuda_event)
                sa.sa_segment_prefill_attn(ctx, L, 0, qs, kp, vp, ql, np.where(sel, w.kv, 0), pages[0], pages[1],
                                           w.scale, os_)
            sa.sa_set_kernel_events(ctx, sa.TIMED_ATTN)
            torch.cuda.synchronize()
            sa.sa_sync_check(ctx)
            keys = int(w.kv[sel].sum())
            rec[name] = {"ms": float(np.mean([x.elapsed_time(y) for x, y in sub])), "rows": int(len(rows)),
                         "cached_keys": keys}
        d = rec["decode_only"]
        d["kv_gbs"] = d["cached_keys"] * Hkv * 128 * 2 * 2 / (d["ms"] * 1e-3) / 1e9
        # inside the mixed launch: when the decode rows' workgroups end, from the
        # per-workgroup clock the kernel writes (sa_set_block_clock)
        buf = torch.full((4 * 65536,), -1, dtype=torch.int64, device="cuda")
        khz = sa.sa_set_block_clock(ctx, buf)
        spans, dec_done, pre_done = [], [], []
        for _ in range(K):
            buf.fill_(-1)
            sa.sa_segment_prefill_attn(ctx, L, 0, q, kp, vp, w.qlen, w.kv, pages[0], pages[1], w.scale, o, lse)
            torch.cuda.synchronize()
            r = buf.view(-1, 4).cpu().numpy()
            r = r[(r[:, 0] != -1) & ((r[:, 3] & 0xffffffff) != 0)]
            t0c = r[:, 0].min()
            to_ms = 1.0 / khz
            spans.append((r[:, 1].max() - t0c) * to_ms)
            dec_done.append((r[(r[:, 3] & 0xffffffff) == 1, 1].max() - t0c) * to_ms)
            pre_done.append((r[(r[:, 3] & 0xffffffff) > 1, 1].max() - t0c) * to_ms)
        sa.sa_set_block_clock(ctx, None)
        sa.sa_sync_check(ctx)
        rec["mixed_launch_clock"] = {
            "about": "one launch over decode rows and prefill segments; per-workgroup device clock "
                     f"({khz} kHz): time from the first workgroup's start",
            "decode_rows_done_ms": float(np.mean(dec_done)), "prefill_done_ms": float(np.mean(pre_done)),
            "span_ms": float(np.mean(spans)),
            "prefill_tokens_per_s": float(int(w.qlen[w.qlen > 1].sum()) / (np.mean(pre_done) * 1e-3))}
    ctx.close()
    print(json.dumps(rec), flush=True)


def main():
    args = parse()
    if args.gpus != 1:
        print(json.dumps({"error": "this benchmark runs on one GPU only; --gpus must be 1",
                          "n_gpus": args.gpus}))
        sys.exit(2)
    if args.copy_bytes:
        copy_mode(args.copy_bytes, args.steps, args.warmup)
        return
    if args.assemble_only:
        assemble_mode(args)
        return
    if args.config != "c2":
        config_mode(args)
        return

    import torch
    import paper_2607_00151_amd as sa
    if not os.path.exists(sa.library_path()):
        from paper_2607_00151_amd import build
        build.build()
    import workloads

    w = workloads.make("c2")
    a = w.asm
    R = max(1, args.rotate)
    base_slots = w.num_slots
    L = sa.Layout(num_q_heads=w.num_q_heads, num_kv_heads=w.num_kv_heads, head_dim=128,
                  page_size=w.page_size, num_layers=1, num_slots=base_slots * R)

    ctx = sa.Context(0)
    if args.folded_scale:
        sa.sa_set_exact_scale(ctx, False)
    if args.fuse == "attn":
        sa.sa_set_fused_append(ctx, True)
    kp, vp = new_pool(base_slots * R, w.num_kv_heads, w.page_size), new_pool(base_slots * R, w.num_kv_heads,
                                                                              w.page_size)
    copies = []
    for r in range(R):
        off = r * base_slots
        sid = dev_i32(a.src_indices + off)
        source_cache(ctx, L, w, kp, vp, sid)
        copies.append(dict(sip=dev_i32(a.src_indptr), sid=sid, fresh=dev_i32(a.fresh + off),
                           dip=torch.zeros(w.batch + 1, dtype=torch.int32, device="cuda"),
                           did=torch.zeros(len(a.fresh), dtype=torch.int32, device="cuda")))
    q = dev_u16(w.q)
    ks, vs = dev_u16(w.k_seg()), dev_u16(w.v_seg())
    T = int(w.qlen.sum())
    o = torch.empty((T, w.num_q_heads, 128), dtype=torch.int16, device="cuda")
    lse = torch.empty((T, w.num_q_heads), dtype=torch.float32, device="cuda")
    stream = torch.cuda.current_stream()
    fuse = args.fuse

    def step(r, ev=None, pages_ev=None):
        """One step; ev: four events recorded around the calls; pages_ev: kernel
        events for the step's first page kernel and (fuse "none") the append."""
        c = copies[r % R]
        if ev is not None:
            ev[0].record(stream)
        if pages_ev is not None:
            sa.sa_set_kernel_events(ctx, sa.TIMED_PAGES, pages_ev[0][0].cuda_event, pages_ev[0][1].cuda_event)
        if fuse == "splice":
            kept = sa.sa_kv_assemble_append(ctx, L, kp, vp, kp, vp, a.src_len, a.keep_indptr,
                                            a.keep_spans, a.reserve, c["sip"], c["sid"], c["fresh"],
                                            c["dip"], c["did"], 0, ks, vs, w.qlen)
            if ev is not None:
                ev[1].record(stream)
        else:
            kept = sa.sa_kv_assemble(ctx, L, kp, vp, kp, vp, a.src_len, a.keep_indptr, a.keep_spans,
                                     a.reserve, c["sip"], c["sid"], c["fresh"], c["dip"], c["did"])
            if ev is not None:
                ev[1].record(stream)
            if fuse == "none":
                if pages_ev is not None:
                    sa.sa_set_kernel_events(ctx, sa.TIMED_PAGES, pages_ev[1][0].cuda_event,
                                            pages_ev[1][1].cuda_event)
                sa.sa_kv_append(ctx, L, 0, kp, vp, ks, vs, kept, w.qlen, c["dip"], c["did"])
        if ev is not None:
            ev[2].record(stream)
        if fuse == "attn":
            sa.sa_segment_prefill_attn_append(ctx, L, 0, q, kp, vp, ks, vs, w.qlen, kept + w.qlen, c["dip"],
                                              c["did"], w.scale, o, lse)
        else:
            sa.sa_segment_prefill_attn(ctx, L, 0, q, kp, vp, w.qlen, kept + w.qlen, c["dip"], c["did"],
                                       w.scale, o, lse)
        if ev is not None:
            ev[3].record(stream)
        return kept

    for i in range(args.warmup):
        step(i)
    sa.sa_sync_check(ctx)
    torch.cuda.synchronize()

    def attn_kernel_pass(n, base):
        """Mean attention kernel time (kernel events) over n steps."""
        ev = [[torch.cuda.Event(enable_timing=True) for _ in range(2)] for _ in range(n)]
        for e in ev:
            e[0].record(stream)
            e[1].record(stream)
        torch.cuda.synchronize()
        for i in range(n):
            sa.sa_set_kernel_events(ctx, sa.TIMED_ATTN, ev[i][0].cuda_event, ev[i][1].cuda_event)
            step(base + i)
        sa.sa_set_kernel_events(ctx, sa.TIMED_ATTN)
        torch.cuda.synchronize()
        sa.sa_sync_check(ctx)
        return float(np.mean([e[0].elapsed_time(e[1]) for e in ev]))

    # the attention kernel as planned without XCD speeds, for comparison
    unweighted_ms = attn_kernel_pass(args.steps, args.warmup)
    xcd_speed = None
    if not args.no_xcd_weights:
        xcd_speed = calibrate_xcds(ctx, lambda i: step(args.warmup + args.steps + i))

    # The timed region: K whole steps, bracketed by two events and nothing in
    # between.  Per-kernel times come from a second pass of K steps with an
    # event around every call (instrumentation that the first pass leaves out,
    # since each event adds a marker between the launches).
    K = args.steps
    t_start = torch.cuda.Event(enable_timing=True)
    t_end = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    t_start.record(stream)
    for i in range(K):
        step(args.warmup + i)
    t_end.record(stream)
    torch.cuda.synchronize()
    sa.sa_sync_check(ctx)
    total_ms = t_start.elapsed_time(t_end)
    evs = [[torch.cuda.Event(enable_timing=True) for _ in range(4)] for _ in range(K)]
    # kernel events: bound by the library to the attention kernel (kev) and to
    # the step's page kernel (pev) themselves (sa_set_kernel_events), so they
    # time their execution on the device; recorded once here so that the HIP
    # events exist
    kev = [[torch.cuda.Event(enable_timing=True) for _ in range(2)] for _ in range(K)]
    pev = [[[torch.cuda.Event(enable_timing=True) for _ in range(2)] for _ in range(2)] for _ in range(K)]
    for e in [x for p in pev for x in p] + kev:
        e[0].record(stream)
        e[1].record(stream)
    torch.cuda.synchronize()
    ev_start = torch.cuda.Event(enable_timing=True)
    ev_end = torch.cuda.Event(enable_timing=True)
    ev_start.record(stream)
    for i in range(K):
        sa.sa_set_kernel_events(ctx, sa.TIMED_ATTN, kev[i][0].cuda_event, kev[i][1].cuda_event)
        step(args.warmup + K + i, evs[i], pev[i])
    sa.sa_set_kernel_events(ctx, sa.TIMED_ATTN)
    sa.sa_set_kernel_events(ctx, sa.TIMED_PAGES)
    ev_end.record(stream)
    torch.cuda.synchronize()
    sa.sa_sync_check(ctx)
    instrumented_ms = ev_start.elapsed_time(ev_end) / K
    asm_ms = float(np.mean([e[0].elapsed_time(e[1]) for e in evs]))
    app_ms = float(np.mean([e[1].elapsed_time(e[2]) for e in evs]))
    # the attention kernel's own duration (kernel events) and that of the call
    # (events around it on the stream, including the dispatch gap)
    attn_ms = float(np.mean([e[0].elapsed_time(e[1]) for e in kev]))
    attn_call_ms = float(np.mean([e[2].elapsed_time(e[3]) for e in evs]))
    ms_per_step = total_ms / K

    Hkv, P, D = w.num_kv_heads, w.page_size, 128
    page_bytes = 2 * Hkv * P * D * 2                      # K and V of one slot
    kept_pages = int(sum(e - b for b, e in a.keep_spans))
    n_dst = int(sum(-(-int(x + y) // P) for x, y in zip(w.pre, w.qlen)))
    asm_bytes = 2 * kept_pages * page_bytes + 4 * (n_dst + kept_pages + w.batch + 1)
    app_bytes = 2 * T * Hkv * D * 2 * 2                   # K and V rows, read + write
    flops = w.attn_flops()
    attn_tflops = flops / (attn_ms * 1e-3) / 1e12
    # compulsory attention bytes: Q, the cache rows it reads, O and LSE
    attn_bytes = (T * w.num_q_heads * 128 * 2 + int(w.kv.sum()) * Hkv * 128 * 2 * 2
                  + T * w.num_q_heads * 128 * 2 + T * w.num_q_heads * 4)

    rec = {
        "metric": "segment-prefill tokens/s + attn TFLOP/s (% MFMA peak); KV assemble GB/s (% HBM)",
        "value": T / (ms_per_step * 1e-3),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": K,
        "warmup": args.warmup,
        "ms_per_step": ms_per_step,
        "ms_per_step_instrumented": instrumented_ms,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {
            "workload": "segment re-prefill, Llama-3-8B-shaped layer: Hq 32 / Hkv 8 / d 128, "
                        "page 16; splice 683 -> 512 pages (drop 171), append 2048-token segment, "
                        "causal GQA over 8192 + 2048",
            "batch": 1, "prefix": int(w.pre[0]), "segment": T, "page_size": P,
            "cache_copies_rotated": R,
            "softmax_scale": "folded into q (bf16)" if args.folded_scale else "per score, fp32",
        },
        "attn": {"ms": attn_ms, "timing": "kernel events (hipExtLaunchKernelGGL)", "call_ms": attn_call_ms,
                 "gflop": flops / 1e9, "tflops": attn_tflops,
                 "frac_of_bf16_peak": attn_tflops / PEAK_BF16_TFLOPS,
                 "tokens_per_s": T / (attn_ms * 1e-3),
                 "without_xcd_weights": {
                     "ms": unweighted_ms,
                     "frac_of_bf16_peak": flops / (unweighted_ms * 1e-3) / 1e12 / PEAK_BF16_TFLOPS}},
        "roofline": {"bound": "mfma", "achieved": attn_tflops, "peak": PEAK_BF16_TFLOPS,
                     "unit": "TFLOP/s", "frac": attn_tflops / PEAK_BF16_TFLOPS,
                     "traffic": None},
        "paper_context": "paper reports up to 11.9x transform-point TTFT reduction end to end on "
                         "H100 80GB (SGLang, Qwen3-8B); no kernel-level numbers",
    }

    traffic = stored_traffic("attn_pipe_kernel", attn_bytes)
    if traffic is not None:
        rec["roofline"]["traffic"] = traffic["bytes"]
        rec["roofline"]["traffic_detail"] = traffic
    if not args.no_gemm_reference:
        rec["gemm_reference"] = gemm_reference()
        # the practical HBM rate for the page kernels: plain copies of the step's bytes and of
        # the 32-layer splice's
        rec["copy_reference"] = {"kind": "torch Tensor.copy_ between contiguous buffers (median of 30)",
                                 "step_bytes": copy_rate(42 * (1 << 20)), "all_layers_bytes": copy_rate(1 << 30)}

    rec["config"]["launches"] = {"attn": "splice | append + attention (one launch, segment rows read from k_new/v_new)",
                                 "splice": "splice + append | attention",
                                 "none": "splice | append | attention"}[fuse]
    # each page kernel's own time (kernel events)
    first_ms = float(np.mean([p[0][0].elapsed_time(p[0][1]) for p in pev]))
    kernels_ms = first_ms + attn_ms
    if fuse == "splice":
        sp_bytes = asm_bytes + app_bytes
        rec["splice_append"] = {"ms": first_ms, "timing": "kernel events (hipExtLaunchKernelGGL)",
                                "call_ms": asm_ms + app_ms, "bytes": sp_bytes,
                                "gbs": sp_bytes / (first_ms * 1e-3) / 1e9,
                                "frac_of_hbm": sp_bytes / (first_ms * 1e-3) / 1e9 / PEAK_HBM_GBS}
    else:
        rec["assemble"] = {"ms": first_ms, "timing": "kernel events (hipExtLaunchKernelGGL)",
                           "call_ms": asm_ms, "bytes": asm_bytes, "gbs": asm_bytes / (first_ms * 1e-3) / 1e9,
                           "frac_of_hbm": asm_bytes / (first_ms * 1e-3) / 1e9 / PEAK_HBM_GBS}
    if fuse == "attn":
        rec["attn"]["includes_append"] = {"bytes_written": app_bytes // 2}
    if fuse == "none":
        ap_ms = float(np.mean([p[1][0].elapsed_time(p[1][1]) for p in pev]))
        kernels_ms += ap_ms
        rec["append"] = {"ms": ap_ms, "timing": "kernel events (hipExtLaunchKernelGGL)", "call_ms": app_ms,
                         "bytes": app_bytes, "gbs": app_bytes / (ap_ms * 1e-3) / 1e9}
    rec["kernels_ms_per_step"] = kernels_ms

    # where the attention launch's time goes across the chip: each workgroup's
    # start and end on the device clock (sa_set_block_clock), over 10 launches;
    # workgroup i runs on XCD i % 8
    buf = torch.full((4 * 8192,), -1, dtype=torch.int64, device="cuda")
    khz = sa.sa_set_block_clock(ctx, buf)
    spans, xcd_end, xcd_start, xcd_wg, busy = [], [], [], [], []
    for i in range(10):
        buf.fill_(-1)
        step(args.warmup + 2 * K + i)
        torch.cuda.synchronize()
        r = buf.view(-1, 4).cpu().numpy()
        ids = np.nonzero(r[:, 0] != -1)[0]
        r = r[ids]
        t0c, t1c = r[:, 0].min(), r[:, 1].max()
        us = 1e3 / khz
        spans.append((t1c - t0c) * us)
        xcd_end.append([(r[ids % 8 == x, 1].max() - t0c) * us for x in range(8)])
        xcd_start.append([(r[ids % 8 == x, 0].max() - t0c) * us for x in range(8)])
        xcd_wg.append([float(np.mean(r[ids % 8 == x, 1] - r[ids % 8 == x, 0])) * us for x in range(8)])
        busy.append(float((r[:, 1] - r[:, 0]).sum()) / (2 * 256 * (t1c - t0c)))
    sa.sa_set_block_clock(ctx, None)
    sa.sa_sync_check(ctx)
    xe = np.mean(np.array(xcd_end), axis=0)
    rec["attn"]["xcd_speeds"] = None if xcd_speed is None else [round(float(x), 4) for x in xcd_speed]
    rec["attn"]["workgroup_clock"] = {
        "about": "device clock per workgroup, mean of 10 launches: launch span; per XCD when its last "
                 "workgroup ended, when its last one started, its mean workgroup time; and the share of "
                 "the 512 workgroup slots' time spent in a workgroup",
        "span_us": float(np.mean(spans)), "xcd_last_end_us": [round(float(x), 1) for x in xe],
        "xcd_last_start_us": [round(float(x), 1) for x in np.mean(np.array(xcd_start), axis=0)],
        "xcd_mean_workgroup_us": [round(float(x), 1) for x in np.mean(np.array(xcd_wg), axis=0)],
        "slot_busy_frac": float(np.mean(busy))}

    if args.assemble_layers > 0:
        # the commit splice of every layer of the model in one launch: the same
        # page plan applied to pools that hold num_layers layers
        NL = args.assemble_layers
        L2 = sa.Layout(num_q_heads=w.num_q_heads, num_kv_heads=w.num_kv_heads, head_dim=128,
                       page_size=w.page_size, num_layers=NL, num_slots=base_slots)
        kl = torch.empty((NL, base_slots, Hkv, P, D), dtype=torch.int16, device="cuda")
        vl = torch.empty_like(kl)
        kl[:] = kp[0, :base_slots]
        vl[:] = vp[0, :base_slots]
        c0 = copies[0]
        evl = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
        for i in range(3):
            sa.sa_kv_assemble(ctx, L2, kl, vl, kl, vl, a.src_len, a.keep_indptr, a.keep_spans,
                              a.reserve, c0["sip"], c0["sid"], c0["fresh"], c0["dip"], c0["did"])
        torch.cuda.synchronize()
        reps = 10
        evl[0].record(stream)
        for i in range(reps):
            sa.sa_kv_assemble(ctx, L2, kl, vl, kl, vl, a.src_len, a.keep_indptr, a.keep_spans,
                              a.reserve, c0["sip"], c0["sid"], c0["fresh"], c0["dip"], c0["did"])
        evl[1].record(stream)
        torch.cuda.synchronize()
        sa.sa_sync_check(ctx)
        ms_l = evl[0].elapsed_time(evl[1]) / reps
        bytes_l = 2 * kept_pages * page_bytes * NL + 4 * (n_dst + kept_pages + w.batch + 1)
        rec["assemble_all_layers"] = {
            "layers": NL, "ms": ms_l, "bytes": bytes_l, "gbs": bytes_l / (ms_l * 1e-3) / 1e9,
            "frac_of_hbm": bytes_l / (ms_l * 1e-3) / 1e9 / PEAK_HBM_GBS}
        del kl, vl

    if not args.no_cpu_baseline:
        import oracle
        stride = max(1, args.cpu_stride)
        toks = np.arange(0, T, stride, dtype=np.int64)
        tok_rows = np.repeat(toks, w.num_q_heads)
        heads = np.tile(np.arange(w.num_q_heads, dtype=np.int32), len(toks))
        t0 = time.perf_counter()
        oracle.attention_rows(w.q, w.k, w.v, w.q_indptr, w.kv_indptr, w.num_q_heads,
                              w.num_kv_heads, w.scale, tok_rows, heads)
        dt = time.perf_counter() - t0
        rec["cpu_baseline"] = {
            "value": len(toks) / dt, "unit": "tokens/s", "cores": oracle.num_threads(),
            "kind": "oracle",
            "sample": f"attention of every {stride}th segment token ({len(toks)} tokens x "
                      f"{w.num_q_heads} heads) of the same workload; {dt:.2f} s",
        }
    ctx.close()
    print(json.dumps(rec), flush=True)


if __name__ == "__main__":
    main()
