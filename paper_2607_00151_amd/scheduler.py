"""Hybrid batch admission for a co-located instance (Alg. 2), driven by the fitted latency model.

Each iteration builds one hybrid batch in priority order: decode requests first, then
latency-critical (LC) prefill chunks, then best-effort (BE) lookahead chunks.  A
candidate is admitted only while the estimated latency of the batch with it stays
within the iteration bound delta (the TBT SLO); the first candidate of a queue that
would exceed it ends that queue's admission (Sec. 4, Alg. 2).  The estimate is Eq. 1
restricted to attention, with coefficients fitted on this library's kernel
(`perf_model`).

`run()` drives the attention kernel on the GPU through a stream of iterations and
measures the decode iteration latency as BE lookahead load grows, against naive
piggybacking that admits every queued BE chunk:
python -m paper_2607_00151_amd.scheduler [--out FILE]
"""
from __future__ import annotations

import json
import sys
from dataclasses import dataclass, field

import numpy as np

from . import perf_model as pm


@dataclass
class Item:
    """One schedulable unit: a decode request (q = 1) or the next chunk of a prefill."""
    kind: str          # "decode", "lc" or "be"
    rid: int           # request id
    q: int             # query tokens of this unit
    kv: int            # KV length once the unit has run (prefix + q)


def est_batch_latency(coef, batch, layout=None) -> float:
    """Eq. 1 without the GEMM term: c + alpha_d * sum L_j + alpha_p * sum A_j (ms); with a
    layout and the five coefficients of the launch-shape model, also its two launch-shape
    terms, taken from the library's planner for this batch."""
    if not batch:
        return 0.0
    w = pm.features([x.q for x in batch], [x.kv for x in batch], layout if len(coef) == 5 else None)
    return float((pm.predict_shape if len(coef) == 5 else pm.predict_context)(coef, [w])[0])


def hybrid_batch(dec_q, lc_q, be_q, delta, est):
    """Alg. 2: admit decode requests, then LC chunks, then BE chunks, each queue in
    order, stopping a queue at its first candidate that would push est(batch) past delta."""
    batch = []
    for queue in (dec_q, lc_q, be_q):
        for cand in queue:
            if est(batch + [cand]) > delta:
                break
            batch.append(cand)
    return batch


# ------------------------------------------------------------------ simulated instance

@dataclass
class Instance:
    """Requests of a co-located instance.  Decode requests grow by one token per
    iteration they run; prefill requests advance by one chunk per admitted chunk and
    are replaced by a fresh request of the same kind when their segment is done."""
    decode_ctx: list
    lc: list = field(default_factory=list)        # [rid, prefix, remaining]
    be: list = field(default_factory=list)
    chunk: int = 256
    segment: int = 2048
    lc_prefix: int = 4096
    be_prefix: int = 16384
    next_rid: int = 1000

    def queues(self):
        dec = [Item("decode", i, 1, L + 1) for i, L in enumerate(self.decode_ctx)]
        lc = [Item("lc", r[0], min(self.chunk, r[2]), r[1] + min(self.chunk, r[2])) for r in self.lc]
        be = [Item("be", r[0], min(self.chunk, r[2]), r[1] + min(self.chunk, r[2])) for r in self.be]
        return dec, lc, be

    def advance(self, batch):
        for x in batch:
            if x.kind == "decode":
                self.decode_ctx[x.rid] += 1
                continue
            reqs = self.lc if x.kind == "lc" else self.be
            for r in reqs:
                if r[0] == x.rid:
                    r[1] += x.q
                    r[2] -= x.q
                    if r[2] <= 0:       # segment done: a new request of the same kind takes its place
                        r[0] = self.next_rid
                        self.next_rid += 1
                        r[1] = self.lc_prefix if x.kind == "lc" else self.be_prefix
                        r[2] = self.segment
                    break


def make_instance(n_decode, n_lc, n_be, seed=0):
    rng = np.random.default_rng(seed)
    inst = Instance(decode_ctx=[int(x) for x in rng.integers(4096, 16385, n_decode)])
    inst.lc = [[100 + i, inst.lc_prefix, inst.segment] for i in range(n_lc)]
    inst.be = [[200 + i, inst.be_prefix, inst.segment] for i in range(n_be)]
    return inst


# ------------------------------------------------------------------ measurement (GPU)

def run(out_path=None, iters=24, delta_ms=0.4, be_loads=(0, 2, 4, 8, 16), n_decode=16, n_lc=1):
    import torch
    import paper_2607_00151_amd as sa

    P, Hq, Hkv, D = 16, 32, 8, 128
    # coefficients of the latency model (Eq. 1's attention terms and the launch
    # shape), profiled on this kernel first: fitted on every launch of the model
    # sweep (decode-only, prefill-only and mixed batches)
    prof = pm.run()
    launches = prof["profile"] + prof["mixed"]
    coef = pm.fit_shape_model([pm.Work(x["tokens"], x["decode_keys"], x["prefill_pairs"], x["excess_tiles"],
                                       x["split"]) for x in launches], [x["ms"] for x in launches])

    max_kv = 16384 + iters + 1 + 16384 + 2048 + 4096
    pages_per_req = (max_kv + P - 1) // P
    n_req = n_decode + n_lc + max(be_loads)
    L = sa.Layout(num_q_heads=Hq, num_kv_heads=Hkv, head_dim=D, page_size=P, num_layers=1,
                  num_slots=pages_per_req * (n_req + 4))
    est = lambda b: est_batch_latency(coef, b, L)   # noqa: E731
    g = torch.Generator(device="cuda").manual_seed(3)
    shape = (L.num_slots, Hkv, P, D)
    pools = [(torch.randn(shape, generator=g, device="cuda") * 0.5).to(torch.bfloat16).view(torch.int16)
             for _ in range(2)]
    perm = torch.randperm(L.num_slots, generator=g, device="cuda").to(torch.int32)
    q_all = (torch.randn((n_decode + 64 * 256, Hq, D), generator=g, device="cuda") * 0.5).to(torch.bfloat16)
    o_all = torch.empty_like(q_all)
    stream = torch.cuda.current_stream()
    rec = {"delta_ms": delta_ms, "model": {"c_ms": coef[0], "alpha_d": coef[1], "alpha_p": coef[2],
                                           "beta_excess_tile": coef[3], "gamma_split": coef[4]},
           "runs": []}

    with sa.Context(0) as ctx:
        def launch(batch):
            """One attention launch over the batch; each request gets its own run of slots."""
            q_len = np.array([x.q for x in batch], dtype=np.int32)
            kv_len = np.array([x.kv for x in batch], dtype=np.int32)
            pages = (kv_len + P - 1) // P
            slot_of = {}
            idx = []
            for x, n in zip(batch, pages):
                key = (x.kind, x.rid)
                base = slot_of.setdefault(key, len(slot_of) * pages_per_req)
                idx.append(perm[base: base + int(n)])
            indices = torch.cat(idx)
            indptr = torch.zeros(len(batch) + 1, dtype=torch.int32, device="cuda")
            indptr[1:] = torch.from_numpy(np.cumsum(pages).astype(np.int32)).cuda()
            T = int(q_len.sum())
            a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            a.record(stream)
            sa.sa_segment_prefill_attn(ctx, L, 0, q_all[:T].view(torch.int16), pools[0], pools[1], q_len,
                                       kv_len, indptr, indices, D ** -0.5, o_all[:T].view(torch.int16))
            b.record(stream)
            return a, b

        # warm-up: one unmeasured pass of the heaviest admit-all run
        inst = make_instance(n_decode, n_lc, max(be_loads))
        for it in range(iters):
            dec, lc, be = inst.queues()
            launch(dec + lc + be)
            inst.advance(dec + lc + be)
        torch.cuda.synchronize()
        for policy in ("alg2", "naive"):
            for n_be in be_loads:
                inst = make_instance(n_decode, n_lc, n_be)
                evs, stats = [], []
                for it in range(iters):
                    dec, lc, be = inst.queues()
                    if policy == "alg2":
                        batch = hybrid_batch(dec, lc, be, delta_ms, est)
                    else:
                        batch = dec + lc + be
                    evs.append(launch(batch))
                    stats.append((sum(x.kind == "be" for x in batch), sum(x.kind == "lc" for x in batch),
                                  sum(x.kind == "decode" for x in batch), est(batch)))
                    inst.advance(batch)
                torch.cuda.synchronize()
                sa.sa_sync_check(ctx)
                ms = np.array([a.elapsed_time(b) for a, b in evs])[2:]     # first two: warm-up
                st = np.array(stats)[2:]
                r = {"policy": policy, "be_requests": n_be, "iter_ms_mean": float(ms.mean()),
                     "iter_ms_p95": float(np.percentile(ms, 95)), "iter_ms_max": float(ms.max()),
                     "be_chunks_per_iter": float(st[:, 0].mean()), "lc_chunks_per_iter": float(st[:, 1].mean()),
                     "decode_per_iter": float(st[:, 2].mean()), "est_ms_mean": float(st[:, 3].mean()),
                     "over_delta": int((ms > delta_ms).sum()), "iters": int(len(ms))}
                rec["runs"].append(r)
                print(f"{policy:5s} BE requests {n_be:2d}: iteration {r['iter_ms_mean'] * 1e3:7.1f} us mean, "
                      f"{r['iter_ms_max'] * 1e3:7.1f} max (est {r['est_ms_mean'] * 1e3:7.1f}); "
                      f"BE chunks/iter {r['be_chunks_per_iter']:.2f}; over delta {r['over_delta']}/{r['iters']}",
                      flush=True)
    if out_path:
        with open(out_path, "w") as f:
            json.dump(rec, f, indent=1)
    return rec


if __name__ == "__main__":
    out = sys.argv[sys.argv.index("--out") + 1] if "--out" in sys.argv else None
    run(out)
