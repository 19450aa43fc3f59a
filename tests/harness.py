"""Device-side set-up shared by the GPU tests, the smoke check and the bench.

Torch is used only to hold device memory: pools, page tables and inputs are
torch tensors whose addresses go through the C ABI.  Initial cache contents
are placed with torch indexing at the (slot, row) positions that the oracle's
paging definition gives, so the attention tests do not depend on the append
kernel.
"""
from __future__ import annotations

import numpy as np
import torch

import paper_2607_00151_amd as sa
from oracle import pages as opages
from workloads import Workload
from workloads.configs import source_rows

CANARY = 0x7FC1          # a bf16 NaN pattern: any stray read or write shows up


def dev_u16(a: np.ndarray, device="cuda") -> torch.Tensor:
    """uint16 bit patterns -> int16 device tensor (same bits)."""
    return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).to(device)


def host_u16(t: torch.Tensor) -> np.ndarray:
    return t.cpu().numpy().view(np.uint16)


def dev_i32(a, device="cuda") -> torch.Tensor:
    return torch.from_numpy(np.ascontiguousarray(np.asarray(a, dtype=np.int32))).to(device)


def bf16_to_f64(bits: np.ndarray) -> np.ndarray:
    return (bits.astype(np.uint32) << 16).view(np.float32).astype(np.float64)


def layout_of(w: Workload, num_layers: int = 1) -> sa.Layout:
    return sa.Layout(num_q_heads=w.num_q_heads, num_kv_heads=w.num_kv_heads, head_dim=w.head_dim,
                     page_size=w.page_size, num_layers=num_layers, num_slots=w.num_slots)


def new_pool(w: Workload, num_layers: int = 1, fill: int = CANARY) -> torch.Tensor:
    t = torch.empty((num_layers, w.num_slots, w.num_kv_heads, w.page_size, w.head_dim),
                    dtype=torch.int16, device="cuda")
    t.fill_(np.int16(np.uint16(fill).view(np.int16)))
    return t


def place(pool: torch.Tensor, layer: int, rows: np.ndarray, slots: np.ndarray, prow: np.ndarray):
    """pool[layer, slot_t, :, row_t, :] = rows[t] for every t."""
    if len(slots) == 0:
        return
    s = torch.from_numpy(slots.astype(np.int64)).cuda()
    r = torch.from_numpy(prow.astype(np.int64)).cuda()
    view = pool[layer].permute(0, 2, 1, 3)          # [slot][row][head][d]
    view[s, r] = dev_u16(rows)


def place_range(pool, layer, w: Workload, rows_of, indptr, indices, lengths, starts=None):
    """Place rows_of(b) ([n_b][Hkv][D]) of every sequence at logical positions
    starts[b] .. starts[b] + n_b - 1 through the page lists (indptr, indices)."""
    B = len(lengths)
    starts = np.zeros(B, dtype=np.int64) if starts is None else np.asarray(starts)
    sl, ro = opages.append_destinations(starts, lengths, indptr, indices, w.page_size)
    rows = np.concatenate([rows_of(b) for b in range(B)], axis=0) if B else None
    place(pool, layer, rows, sl, ro)


def build_cache(w: Workload, num_layers: int = 1, layer: int = 0, with_segment: bool = True):
    """Pools holding each sequence's prefix (and segment, unless with_segment
    is False) at its direct page list.  Returns (k_pool, v_pool, indptr, indices)."""
    kp, vp = new_pool(w, num_layers), new_pool(w, num_layers)
    lengths = w.kv if with_segment else w.pre
    for pool, full in ((kp, w.k), (vp, w.v)):
        def rows_of(b, full=full):
            s = int(w.kv_indptr[b])
            return full[s: s + int(lengths[b])]
        place_range(pool, layer, w, rows_of, w.pages_indptr, w.pages, lengths)
    return kp, vp, dev_i32(w.pages_indptr), dev_i32(w.pages)


def build_source_cache(w: Workload, num_layers: int = 1):
    """Pools holding every sequence's assembly source (kept prefix with the
    dropped pages inserted), in every layer (layer l holds the same rows with
    bit 0 of each value flipped l times, so layers are distinguishable)."""
    a = w.asm
    kp, vp = new_pool(w, num_layers), new_pool(w, num_layers)
    for pool, which in ((kp, "k"), (vp, "v")):
        for layer in range(num_layers):
            def rows_of(b, which=which, layer=layer):
                r = source_rows(w, b, which)
                return r ^ np.uint16(layer & 1) if layer else r
            place_range(pool, layer, w, rows_of, a.src_indptr, a.src_indices, a.src_len)
    return kp, vp, dev_i32(a.src_indptr), dev_i32(a.src_indices), dev_i32(a.fresh)


def run_assemble(ctx, w: Workload, L, kp, vp, src_indptr, src_indices, fresh, stream=None):
    a = w.asm
    n_dst_cap = int(len(a.fresh))
    dst_indptr = torch.zeros(w.batch + 1, dtype=torch.int32, device="cuda")
    dst_indices = torch.full((n_dst_cap,), -1, dtype=torch.int32, device="cuda")
    dst_len = sa.sa_kv_assemble(ctx, L, kp, vp, kp, vp, a.src_len, a.keep_indptr, a.keep_spans,
                                a.reserve, src_indptr, src_indices, fresh, dst_indptr,
                                dst_indices, stream=stream)
    return dst_indptr, dst_indices, dst_len


def attention(ctx, w: Workload, L, q_dev, kp, vp, indptr, indices, layer=0, with_lse=True,
              stream=None):
    T = int(w.qlen.sum())
    o = torch.empty((T, w.num_q_heads, w.head_dim), dtype=torch.int16, device="cuda")
    lse = torch.empty((T, w.num_q_heads), dtype=torch.float32, device="cuda") if with_lse else None
    sa.sa_segment_prefill_attn(ctx, L, layer, q_dev, kp, vp, w.qlen, w.kv, indptr, indices,
                               w.scale, o, lse, stream=stream)
    return o, lse


def sample_rows(w: Workload, per_seq: int, seed: int = 0):
    """(token, head) rows: first and last row of every segment, every head of
    the first and last token, and per_seq random rows per sequence."""
    g = np.random.Generator(np.random.Philox(key=[seed + 77, 5]))
    toks, heads = [], []
    qi = w.q_indptr
    for b in range(w.batch):
        n = int(w.qlen[b])
        if n == 0:
            continue
        for t in {0, n - 1}:
            toks += [int(qi[b]) + t] * w.num_q_heads
            heads += list(range(w.num_q_heads))
        for _ in range(per_seq):
            toks.append(int(qi[b]) + int(g.integers(0, n)))
            heads.append(int(g.integers(0, w.num_q_heads)))
    return np.asarray(toks, dtype=np.int64), np.asarray(heads, dtype=np.int32)


def score_shift_bound(w: Workload, toks: np.ndarray, heads: np.ndarray) -> np.ndarray:
    """max_j sum_d |c q_d k_jd| over each row's visible keys (c = scale log2 e): the
    bf16 rounding of c q moves that row's exponents by at most 2^-8 times this."""
    return lse_tolerance(w, toks, heads, slack=0.0) / (np.log(2.0) * 2.0 ** -8)


def lse_tolerance(w: Workload, toks: np.ndarray, heads: np.ndarray, slack: float = 1e-4) -> np.ndarray:
    """Per-row bound on the device LSE error (natural log).

    The kernel rounds c q (c = scale log2 e) to bf16 once, so each exponent
    x_j = c q.k_j moves by at most 2^-8 sum_d |c q_d k_jd| (the unit roundoff
    of bf16's 8-bit significand); the log-sum-exp of
    the row moves by no more than the largest such shift over its visible
    keys (it is monotone and commutes with a common shift), times ln 2 to go
    back from base 2.  slack covers the fp32 arithmetic of the rest.
    """
    c = w.scale * np.log2(np.e)
    G = w.num_q_heads // w.num_kv_heads
    qf = np.abs(bf16_to_f64(w.q[toks, heads]))               # [n][D]
    kf = w.k
    bound = np.zeros(len(toks))
    seq = np.searchsorted(w.q_indptr, toks, side="right") - 1
    for b in np.unique(seq):
        kv0 = int(w.kv_indptr[b])
        pre = int(w.kv[b]) - int(w.qlen[b])
        for g in np.unique(heads[seq == b] // G):
            sel = np.nonzero((seq == b) & (heads // G == g))[0]
            pos = pre + (toks[sel] - int(w.q_indptr[b]))       # last visible key of each row
            kb = np.abs(bf16_to_f64(kf[kv0: kv0 + int(pos.max()) + 1, g]))   # [keys][D]
            s = (qf[sel] * abs(c)) @ kb.T                      # sum_d |c q_d k_jd|
            s[np.arange(kb.shape[0])[None, :] > pos[:, None]] = 0.0
            bound[sel] = s.max(axis=1)
    return np.log(2.0) * 2.0 ** -8 * bound + slack


def compare(got_bits: np.ndarray, ref: np.ndarray, max_tol=2e-2, mean_tol=2e-3):
    """bf16 device output vs float64 oracle: returns (max_abs, mean_abs)."""
    got = bf16_to_f64(got_bits)
    err = np.abs(got - ref)
    assert np.isfinite(got).all(), "non-finite output"
    mx, mean = float(err.max()), float(err.mean())
    assert mx <= max_tol and mean <= mean_tol, (mx, mean)
    return mx, mean
