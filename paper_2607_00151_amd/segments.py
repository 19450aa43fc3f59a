"""Streaming short segments over long prefixes (Sec. 3.5 isolation's streamed instruction chunks).

A batch of sub-agent contexts, each with a long cached prefix, receives a short
segment of q new tokens; the step is zero-copy splice (the prefix pages stay where
they are), append of the segment, and the segment's causal attention.  With q x G
query rows per KV head, the attention does q x G FLOP per byte of K/V it reads: below
q ~ 80 (G = 4) that is under the bf16 ridge of MI355X (2.5166 PFLOP/s over 8 TB/s),
so short segments are bound by HBM, long ones by the matrix cores.  `run()` sweeps
q and reports each step's kernels against the roofline of their own bound:
python -m paper_2607_00151_amd.segments [--out FILE]
"""
from __future__ import annotations

import json
import sys

import numpy as np

PEAK_TFLOPS = 2516.6
PEAK_GBS = 8000.0


def attention_roofline(B, q, prefix, Hq, Hkv, D=128):
    """(FLOP, compulsory bytes, time bound in ms) of one attention launch."""
    G = Hq // Hkv
    pairs = B * (q * prefix + q * (q + 1) // 2)                   # per head
    flop = 4.0 * D * Hq * pairs
    kv = B * (prefix + q) * Hkv * D * 2 * 2                       # K and V rows read once
    qo = 2 * B * q * Hq * D * 2                                   # Q read, O written
    bytes_ = kv + qo + B * q * Hq * 4
    t = max(flop / (PEAK_TFLOPS * 1e12), bytes_ / (PEAK_GBS * 1e9)) * 1e3
    return flop, bytes_, t, q * G


def run(out_path=None, B=32, prefix=8192, qs=(16, 32, 64, 128, 256, 512), reps=10, warmup=3):
    import torch
    import paper_2607_00151_amd as sa

    Hq, Hkv, D, P = 32, 8, 128, 16
    pages_src = prefix // P
    max_pages = pages_src + (max(qs) + P - 1) // P + 1
    L = sa.Layout(num_q_heads=Hq, num_kv_heads=Hkv, head_dim=D, page_size=P, num_layers=1,
                  num_slots=B * max_pages + 16)
    g = torch.Generator(device="cuda").manual_seed(11)
    shape = (L.num_slots, Hkv, P, D)
    kp = (torch.randn(shape, generator=g, device="cuda") * 0.5).to(torch.bfloat16).view(torch.int16)
    vp = (torch.randn(shape, generator=g, device="cuda") * 0.5).to(torch.bfloat16).view(torch.int16)
    perm = torch.randperm(L.num_slots, generator=g, device="cuda").to(torch.int32)
    src_ix = perm[: B * pages_src].contiguous()
    fresh = perm[B * pages_src:].contiguous()
    src_ip = torch.arange(0, B * pages_src + 1, pages_src, dtype=torch.int32, device="cuda")
    src_len = np.full(B, prefix, dtype=np.int32)
    keep_indptr = np.arange(B + 1, dtype=np.int32)
    keep_spans = np.array([[0, pages_src]] * B, dtype=np.int32)
    stream = torch.cuda.current_stream()
    rec = {"batch": B, "prefix": prefix, "layout": "Hq 32 / Hkv 8 / d 128, page 16, bf16", "rows": []}
    with sa.Context(0) as ctx:
        for q in qs:
            T = B * q
            qt = (torch.randn((T, Hq, D), generator=g, device="cuda") * 0.5).to(torch.bfloat16).view(torch.int16)
            kn = (torch.randn((T, Hkv, D), generator=g, device="cuda") * 0.5).to(torch.bfloat16).view(torch.int16)
            vn = (torch.randn((T, Hkv, D), generator=g, device="cuda") * 0.5).to(torch.bfloat16).view(torch.int16)
            o = torch.empty((T, Hq, D), dtype=torch.int16, device="cuda")
            reserve = np.full(B, q, dtype=np.int32)
            n_dst = B * ((prefix + q + P - 1) // P)
            dip = torch.zeros(B + 1, dtype=torch.int32, device="cuda")
            did = torch.zeros(n_dst, dtype=torch.int32, device="cuda")
            qlen = np.full(B, q, dtype=np.int32)

            def step(ev=None):
                if ev:
                    ev[0].record(stream)
                kept = sa.sa_kv_splice_alias(ctx, L, src_len, keep_indptr, keep_spans, reserve, src_ip,
                                             src_ix, fresh, dip, did)
                if ev:
                    ev[1].record(stream)
                sa.sa_kv_append(ctx, L, 0, kp, vp, kn, vn, kept, qlen, dip, did)
                if ev:
                    ev[2].record(stream)
                sa.sa_segment_prefill_attn(ctx, L, 0, qt, kp, vp, qlen, kept + qlen, dip, did, D ** -0.5, o)
                if ev:
                    ev[3].record(stream)

            # the first size also carries the clock's warm-up (tens of milliseconds of load)
            for _ in range(warmup if q != qs[0] else 200):
                step()
            evs = [[torch.cuda.Event(enable_timing=True) for _ in range(4)] for _ in range(reps)]
            for ev in evs:
                step(ev)
            torch.cuda.synchronize()
            sa.sa_sync_check(ctx)
            t_spl = float(np.median([e[0].elapsed_time(e[1]) for e in evs]))
            t_app = float(np.median([e[1].elapsed_time(e[2]) for e in evs]))
            t_att = float(np.median([e[2].elapsed_time(e[3]) for e in evs]))
            flop, byt, t_bound, rows = attention_roofline(B, q, prefix, Hq, Hkv, D)
            r = {"q": q, "rows_per_kv_head": rows, "splice_ms": t_spl, "append_ms": t_app, "attn_ms": t_att,
                 "attn_tflops": flop / (t_att * 1e-3) / 1e12, "attn_gbs": byt / (t_att * 1e-3) / 1e9,
                 "attn_bound": "hbm" if byt / (PEAK_GBS * 1e9) > flop / (PEAK_TFLOPS * 1e12) else "mfma",
                 "attn_roofline_frac": t_bound / t_att, "tokens_per_s": T / ((t_spl + t_app + t_att) * 1e-3)}
            rec["rows"].append(r)
            print(f"q {q:4d}: splice {t_spl * 1e3:6.1f} us  append {t_app * 1e3:6.1f} us  attention "
                  f"{t_att * 1e3:7.1f} us ({r['attn_tflops']:6.1f} TFLOP/s, {r['attn_gbs']:6.0f} GB/s, "
                  f"{r['attn_bound']}-bound, {100 * r['attn_roofline_frac']:4.1f}% of its roofline)", flush=True)
    if out_path:
        with open(out_path, "w") as f:
            json.dump(rec, f, indent=1)
    return rec


if __name__ == "__main__":
    out = sys.argv[sys.argv.index("--out") + 1] if "--out" in sys.argv else None
    run(out)
