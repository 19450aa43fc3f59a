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


def features(q_len, kv_len) -> Work:
    """Sequences with one query token count as decode requests (they read their whole
    KV cache, L_j = kv_len); the others as prefill chunks with prefix = kv_len - q_len."""
    q_len = np.asarray(q_len, dtype=np.int64)
    kv_len = np.asarray(kv_len, dtype=np.int64)
    dec = q_len == 1
    pre = ~dec & (q_len > 0)
    a = sum(prefill_pairs(int(q), int(k - q)) for q, k in zip(q_len[pre], kv_len[pre]))
    return Work(int(q_len.sum()), int(kv_len[dec].sum()), int(a))


# ------------------------------------------------------------------ models

def fit_context_model(works, times):
    """Least squares t = c + alpha_d * sum L + alpha_p * sum A.  Returns (c, alpha_d, alpha_p)."""
    X = np.array([[1.0, w.decode_keys, w.prefill_pairs] for w in works])
    coef, *_ = np.linalg.lstsq(X, np.asarray(times, dtype=np.float64), rcond=None)
    return tuple(float(x) for x in coef)


def predict_context(coef, works):
    c, ad, ap = coef
    return np.array([c + ad * w.decode_keys + ap * w.prefill_pairs for w in works])


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

def _time_launch(sa, ctx, L, pools, q_len, kv_len, reps=10, warmup=3, seed=0):
    """Median HIP-event time (ms) of one attention launch over random bf16 inputs."""
    import torch
    g = torch.Generator(device="cuda").manual_seed(seed)
    Hq, Hkv, D, P = L.num_q_heads, L.num_kv_heads, L.head_dim, L.page_size
    q_len = np.asarray(q_len, dtype=np.int32)
    kv_len = np.asarray(kv_len, dtype=np.int32)
    pages = (kv_len + P - 1) // P
    n_pages = int(pages.sum())
    assert n_pages <= L.num_slots
    T = int(q_len.sum())
    q = (torch.randn((T, Hq, D), generator=g, device="cuda") * 0.5).to(torch.bfloat16)
    perm = torch.randperm(L.num_slots, generator=g, device="cuda")[:n_pages].to(torch.int32)
    indptr = torch.zeros(len(q_len) + 1, dtype=torch.int32, device="cuda")
    indptr[1:] = torch.from_numpy(np.cumsum(pages).astype(np.int32)).cuda()
    o = torch.empty((T, Hq, D), dtype=torch.bfloat16, device="cuda")
    stream = torch.cuda.current_stream()

    def launch():
        sa.sa_segment_prefill_attn(ctx, L, 0, q.view(torch.int16), pools[0], pools[1], q_len, kv_len,
                                   indptr, perm, D ** -0.5, o.view(torch.int16))

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
        _time_launch(sa, ctx, L, pools, [256] * 4, [16384 + 256] * 4, reps=200, warmup=0)
        prof_w, prof_t = [], []
        for name, q, kv in profiling_batches():
            t = _time_launch(sa, ctx, L, pools, q, kv)
            w = features(q, kv)
            prof_w.append(w)
            prof_t.append(t)
            rec["profile"].append({"batch": name, "ms": t, **w.__dict__})
            print(f"profile  {name:36s} {t * 1e3:9.1f} us", flush=True)
        cm = fit_context_model(prof_w, prof_t)
        tm = fit_token_model(prof_w, prof_t)
        mix_w, mix_t = [], []
        for name, q, kv in mixed_batches():
            t = _time_launch(sa, ctx, L, pools, q, kv)
            w = features(q, kv)
            mix_w.append(w)
            mix_t.append(t)
        pc, pt = predict_context(cm, mix_w), predict_token(tm, mix_w)
        for (name, _, _), w, t, a, b in zip(mixed_batches(), mix_w, mix_t, pc, pt):
            rec["mixed"].append({"batch": name, "ms": t, "context_model_ms": a, "token_model_ms": b,
                                 **w.__dict__})
            print(f"mixed    {name:36s} {t * 1e3:9.1f} us  context-aware {a * 1e3:9.1f}  "
                  f"token-only {b * 1e3:9.1f}", flush=True)
    rec["context_model"] = {"c_ms": cm[0], "alpha_d_ms_per_key": cm[1], "alpha_p_ms_per_pair": cm[2]}
    rec["token_model"] = {"a_ms": tm[0], "b_ms_per_token": tm[1]}
    rec["max_rel_error"] = {"context_aware": max_rel_error(pc, mix_t), "token_only": max_rel_error(pt, mix_t)}
    print(json.dumps(rec["max_rel_error"]), flush=True)
    if out_path:
        with open(out_path, "w") as f:
            json.dump(rec, f, indent=1)
    return rec


if __name__ == "__main__":
    out = sys.argv[sys.argv.index("--out") + 1] if "--out" in sys.argv else None
    run(out)
