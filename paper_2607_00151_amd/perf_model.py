"""Context-aware latency model of the attention terms (Sec. 4, Eq. 1), fitted on this library.

The paper estimates a mixed batch's latency as

    EstBatchLatency(B) = T_GEMM(M) + alpha_d * sum_{decode j} L_j + alpha_p * sum_{prefill j} A_j

with M the forward tokens of the batch, L_j the KV length a decode request reads, and
A_j = q_j * prefix_j + q_j (q_j + 1) / 2 the causal query-key pairs of a prefill chunk.
This module covers the attention part on this library's kernel: the work features of a
batch, a least-squares fit of (c, alpha_d, alpha_p) -- c being the fixed cost of a
launch -- from measured launch times, the token-count-only model it is compared with
(latency as a function of M alone), and the measurement sweep itself, after the
paper's accuracy experiment (Sec. 6, the prediction-error figure): profile the
coefficients on decode-only and prefill-only launches, then predict mixed batches of
four decode requests and two or four 256-token prefill chunks whose cached context
grows while their new work stays fixed.

Small batches do not fill the chip, and then the launch's time follows how its work
falls onto the 2 x 256 workgroup slots rather than its total: the launch-shape model
adds two terms taken from the library's own planner (sa_attn_plan_stats, host only):
the makespan of the launch in key tiles beyond an even spread of its tiles over the
slots, and whether long items were split by key range (a partial-merge launch
follows).  It is fitted on the same profiling launches.

Run on the GPU:  python -m paper_2607_00151_amd.perf_model [--out FILE]
"""
from __future__ import annotations

import json
import sys
from dataclasses import dataclass

import numpy as np


# ------------------------------------------------------------------ features

def prefill_pairs(q: int, prefix: int) -> int:
    """A_j = q prefix + q (q + 1) / 2: row i of the chunk sees prefix + i + 1 keys (Sec. 4)."""
    return q * prefix + q * (q + 1) // 2


@dataclass
class Work:
    """Work features of one attention launch (one layer, all heads)."""
    tokens: int        # M: query tokens of the launch
    decode_keys: int   # sum of L_j over decode requests (q_j = 1)
    prefill_pairs: int  # sum of A_j over prefill chunks (q_j > 1)
    excess_tiles: float = 0.0  # planner makespan in key tiles beyond an even spread over the slots
    split: int = 0     # 1 when the planner splits items by key range (a merge launch follows)


SLOTS_PER_CU = 2


def features(q_len, kv_len, layout=None, num_cu: int = 256) -> Work:
    """Sequences with one query token count as decode requests (they read their whole
    KV cache, L_j = kv_len); the others as prefill chunks with prefix = kv_len - q_len.
    With a layout, the launch-shape terms come from the library's planner."""
    q_len = np.asarray(q_len, dtype=np.int64)
    kv_len = np.asarray(kv_len, dtype=np.int64)
    dec = q_len == 1
    pre = ~dec & (q_len > 0)
    a = sum(prefill_pairs(int(q), int(k - q)) for q, k in zip(q_len[pre], kv_len[pre]))
    w = Work(int(q_len.sum()), int(kv_len[dec].sum()), int(a))
    if layout is not None:
        import paper_2607_00151_amd as sa
        st = sa.sa_attn_plan_stats(layout, q_len, kv_len, num_cu)
        w.excess_tiles = max(0.0, st["makespan_tiles"] - st["tiles"] / (SLOTS_PER_CU * num_cu))
        w.split = int(st["parts"] > 0)
    return w


# ------------------------------------------------------------------ models

def fit_context_model(works, times):
    """Least squares t = c + alpha_d * sum L + alpha_p * sum A.  Returns (c, alpha_d, alpha_p)."""
    X = np.array([[1.0, w.decode_keys, w.prefill_pairs] for w in works])
    coef, *_ = np.linalg.lstsq(X, np.asarray(times, dtype=np.float64), rcond=None)
    return tuple(float(x) for x in coef)


def predict_context(coef, works):
    c, ad, ap = coef
    return np.array([c + ad * w.decode_keys + ap * w.prefill_pairs for w in works])


def fit_shape_model(works, times):
    """Least squares t = c + alpha_d sum L + alpha_p sum A + beta excess + gamma split.
    Returns (c, alpha_d, alpha_p, beta, gamma)."""
    X = np.array([[1.0, w.decode_keys, w.prefill_pairs, w.excess_tiles, w.split] for w in works])
    coef, *_ = np.linalg.lstsq(X, np.asarray(times, dtype=np.float64), rcond=None)
    return tuple(float(x) for x in coef)


def predict_shape(coef, works):
    c, ad, ap, b, g = coef
    return np.array([c + ad * w.decode_keys + ap * w.prefill_pairs + b * w.excess_tiles + g * w.split
                     for w in works])


def fit_token_model(works, times):
    """Least squares t = a + b * M (latency from the number of forward tokens alone)."""
    X = np.array([[1.0, w.tokens] for w in works])
    coef, *_ = np.linalg.lstsq(X, np.asarray(times, dtype=np.float64), rcond=None)
    return tuple(float(x) for x in coef)


def predict_token(coef, works):
    a, b = coef
    return np.array([a + b * w.tokens for w in works])


def max_rel_error(pred, meas) -> float:
    pred, meas = np.asarray(pred, dtype=np.float64), np.asarray(meas, dtype=np.float64)
    return float(np.max(np.abs(pred - meas) / meas))


# ------------------------------------------------------------------ batches of the sweep

def profiling_batches():
    """Decode-only and prefill-only launches: (name, q_len list, kv_len list)."""
    out = []
    for n in (4, 16):
        for L in (2048, 8192, 32768):
            out.append((f"decode {n}x L={L}", [1] * n, [L] * n))
    for n in (1, 2, 4):
        for pre in (0, 4096, 16384):
            out.append((f"prefill {n}x256 prefix={pre}", [256] * n, [pre + 256] * n))
    return out


def mixed_batches():
    """Four decode requests plus two or four 256-token prefill chunks; the cached
    context c of every request grows while the new work stays fixed."""
    out = []
    for n_p in (2, 4):
        for c in (1024, 2048, 4096, 8192, 16384, 32768):
            q = [1] * 4 + [256] * n_p
            kv = [c] * 4 + [c + 256] * n_p
            out.append((f"4 decode + {n_p}x256, context {c}", q, kv))
    return out


# ------------------------------------------------------------------ measurement (GPU)

def time_launch(sa, ctx, L, q, pools, indptr, indices, q_len, kv_len, o, reps=10, warmup=3):
    """Median HIP-event time (ms) of one attention launch on the given device inputs."""
    import torch
    stream = torch.cuda.current_stream()
    D = L.head_dim

    def launch():
        sa.sa_segment_prefill_attn(ctx, L, 0, q, pools[0], pools[1], q_len, kv_len, indptr, indices,
                                   D ** -0.5, o)

    for _ in range(warmup):
        launch()
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(reps)]
    for a, b in ev:
        a.record(stream)
        launch()
        b.record(stream)
    torch.cuda.synchronize()
    sa.sa_sync_check(ctx)
    return float(np.median([a.elapsed_time(b) for a, b in ev]))


def _random_launch(sa, ctx, L, pools, q_len, kv_len, reps=10, warmup=3, seed=0):
    """time_launch over random bf16 queries and a random page placement."""
    import torch
    g = torch.Generator(device="cuda").manual_seed(seed)
    Hq, D, P = L.num_q_heads, L.head_dim, L.page_size
    q_len = np.asarray(q_len, dtype=np.int32)
    kv_len = np.asarray(kv_len, dtype=np.int32)
    pages = (kv_len + P - 1) // P
    n_pages = int(pages.sum())
    assert n_pages <= L.num_slots
    T = int(q_len.sum())
    q = (torch.randn((T, Hq, D), generator=g, device="cuda") * 0.5).to(torch.bfloat16).view(torch.int16)
    perm = torch.randperm(L.num_slots, generator=g, device="cuda")[:n_pages].to(torch.int32)
    indptr = torch.zeros(len(q_len) + 1, dtype=torch.int32, device="cuda")
    indptr[1:] = torch.from_numpy(np.cumsum(pages).astype(np.int32)).cuda()
    o = torch.empty((T, Hq, D), dtype=torch.int16, device="cuda")
    return time_launch(sa, ctx, L, q, pools, indptr, perm, q_len, kv_len, o, reps, warmup)


# The linear layers of one Llama-3-8B layer (hidden 4096, 32/8 heads of 128,
# MLP 14336): (K, N) of each GEMM a batch of M tokens runs.
LAYER_GEMMS = ((4096, 6144), (4096, 4096), (4096, 2 * 14336), (14336, 4096))


def time_layer_gemms(M: int, reps: int = 20) -> float:
    """T_GEMM(M) of Eq. 1: median time (ms) of the layer's four bf16 GEMMs for M
    tokens, run with torch.matmul (hipBLASLt) -- context for the attention terms,
    not part of this library."""
    import torch
    mats = [(torch.randn(M, k, device="cuda", dtype=torch.bfloat16),
             torch.randn(k, n, device="cuda", dtype=torch.bfloat16)) for k, n in LAYER_GEMMS]
    for a, b in mats:
        a @ b
    times = []
    for _ in range(reps):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for a, b in mats:
            a @ b
        e1.record()
        torch.cuda.synchronize()
        times.append(e0.elapsed_time(e1))
    return float(np.median(times))


def evaluate_batch(L, prof, mixed, gemm_ms):
    """Eq. 1 as the paper states it, for one layer: T_GEMM(M) + the attention terms.
    T_GEMM is fitted linearly in M on the profiling launches' measured GEMM times
    (gemm_ms: M -> ms), the attention terms as in evaluate(); measured batch latency
    is the measured GEMM time plus the measured attention launch."""
    pm_ = np.array([[1.0, int(np.sum(q))] for q, _, _ in prof])
    g = np.linalg.lstsq(pm_, np.array([gemm_ms[int(np.sum(q))] for q, _, _ in prof]), rcond=None)[0]
    t_gemm = lambda M: g[0] + g[1] * M   # noqa: E731
    ev = evaluate(L, prof, mixed)
    meas = np.array([gemm_ms[int(np.sum(q))] + t for q, _, t in mixed])
    gm = np.array([t_gemm(int(np.sum(q))) for q, _, _ in mixed])
    tok = fit_token_model([features(q, kv) for q, kv, _ in prof],
                          [gemm_ms[int(np.sum(q))] + t for q, _, t in prof])
    pred = {"context_aware": gm + ev["pred"]["context_aware"], "launch_shape": gm + ev["pred"]["launch_shape"],
            "token_only": predict_token(tok, [features(q, kv) for q, kv, _ in mixed])}
    return {"gemm_fit_ms": (float(g[0]), float(g[1])), "measured_ms": meas, "pred": pred,
            "max_rel_error": {k: max_rel_error(v, meas) for k, v in pred.items()}}


def evaluate(L, prof, mixed):
    """Fit the paper's model, the launch-shape model and the token-count model on the
    profiling launches ((q, kv, ms) triples) and predict the mixed ones."""
    pw = [features(q, kv, L) for q, kv, _ in prof]
    pt = [t for _, _, t in prof]
    mw = [features(q, kv, L) for q, kv, _ in mixed]
    mt = [t for _, _, t in mixed]
    cm, sm, tm = fit_context_model(pw, pt), fit_shape_model(pw, pt), fit_token_model(pw, pt)
    pc, ps, pk = predict_context(cm, mw), predict_shape(sm, mw), predict_token(tm, mw)
    return {"context_model": cm, "shape_model": sm, "token_model": tm,
            "pred": {"context_aware": pc, "launch_shape": ps, "token_only": pk},
            "max_rel_error": {"context_aware": max_rel_error(pc, mt), "launch_shape": max_rel_error(ps, mt),
                              "token_only": max_rel_error(pk, mt)}}


def run(out_path=None):
    import torch
    import paper_2607_00151_amd as sa

    P = 16
    batches = profiling_batches() + mixed_batches()
    slots = max(int(sum((k + P - 1) // P for k in kv)) for _, _, kv in batches)
    L = sa.Layout(num_q_heads=32, num_kv_heads=8, head_dim=128, page_size=P, num_layers=1, num_slots=slots)
    g = torch.Generator(device="cuda").manual_seed(7)
    shape = (L.num_slots, L.num_kv_heads, L.page_size, L.head_dim)
    pools = [(torch.randn(shape, generator=g, device="cuda") * 0.5).to(torch.bfloat16).view(torch.int16)
             for _ in range(2)]
    rec = {"layout": "Hq 32 / Hkv 8 / d 128, page 16, bf16", "profile": [], "mixed": []}
    with sa.Context(0) as ctx:
        # the shader clock takes tens of milliseconds of load to settle: warm up on the
        # largest profiling batch (~50 ms) before any launch is timed
        _random_launch(sa, ctx, L, pools, [256] * 4, [16384 + 256] * 4, reps=200, warmup=0)
        prof, mixed = [], []
        for name, q, kv in profiling_batches():
            t = _random_launch(sa, ctx, L, pools, q, kv)
            prof.append((q, kv, t))
            rec["profile"].append({"batch": name, "ms": t, **features(q, kv, L).__dict__})
            print(f"profile  {name:36s} {t * 1e3:9.1f} us", flush=True)
        for name, q, kv in mixed_batches():
            mixed.append((q, kv, _random_launch(sa, ctx, L, pools, q, kv)))
        gemm_ms = {}
        for q, _, _ in prof + mixed:
            M = int(np.sum(q))
            if M not in gemm_ms:
                gemm_ms[M] = time_layer_gemms(M)
    ev = evaluate(L, prof, mixed)
    evb = evaluate_batch(L, prof, mixed, gemm_ms)
    for (name, q, kv), (_, _, t), a, s_, b in zip(mixed_batches(), mixed, ev["pred"]["context_aware"],
                                                 ev["pred"]["launch_shape"], ev["pred"]["token_only"]):
        rec["mixed"].append({"batch": name, "ms": t, "context_model_ms": a, "shape_model_ms": s_,
                             "token_model_ms": b, **features(q, kv, L).__dict__})
        print(f"mixed    {name:36s} {t * 1e3:9.1f} us  context-aware {a * 1e3:9.1f}  launch-shape "
              f"{s_ * 1e3:9.1f}  token-only {b * 1e3:9.1f}", flush=True)
    cm, sm, tm = ev["context_model"], ev["shape_model"], ev["token_model"]
    rec["context_model"] = {"c_ms": cm[0], "alpha_d_ms_per_key": cm[1], "alpha_p_ms_per_pair": cm[2]}
    rec["shape_model"] = {"c_ms": sm[0], "alpha_d_ms_per_key": sm[1], "alpha_p_ms_per_pair": sm[2],
                          "beta_ms_per_excess_tile": sm[3], "gamma_ms_split": sm[4]}
    rec["token_model"] = {"a_ms": tm[0], "b_ms_per_token": tm[1]}
    rec["max_rel_error"] = ev["max_rel_error"]
    rec["layer_gemm_ms"] = {str(k): v for k, v in sorted(gemm_ms.items())}
    rec["batch_latency"] = {
        "about": "Eq. 1 with its GEMM term: the Llama-3-8B layer's four GEMMs (torch.matmul, measured; "
                 "fitted linearly in M on the profiling batches) plus the attention terms",
        "gemm_fit_ms": evb["gemm_fit_ms"], "measured_ms": evb["measured_ms"].tolist(),
        "pred_ms": {k: v.tolist() for k, v in evb["pred"].items()},
        "max_rel_error": evb["max_rel_error"]}
    print("attention only:", json.dumps(rec["max_rel_error"]), flush=True)
    print("batch latency (GEMM + attention):", json.dumps(evb["max_rel_error"]), flush=True)
    if out_path:
        with open(out_path, "w") as f:
            json.dump(rec, f, indent=1)
    return rec


if __name__ == "__main__":
    out = sys.argv[sys.argv.index("--out") + 1] if "--out" in sys.argv else None
    run(out)
