"""Workload recipes.

All values are N(0, 1) * 0.5 rounded to bf16, softmax scale 1/sqrt(head_dim),
pages placed by a seeded permutation of the slot pool.  Each named stream
(queries, keys, values, dropped pages, slots, lengths, drop positions,
outliers) has its own Philox key, so changing one recipe knob leaves the
others' draws alone.

Per sequence b a workload holds
  pre[b]   cached prefix tokens the segment attends to (after any assembly)
  qlen[b]  new segment tokens; kv = pre + qlen
and the CONTIGUOUS logical contents q [sum q][Hq][D], k/v [sum kv][Hkv][D]
(sequence b's rows: its prefix, then its segment).  ``pages`` is a page list
for the whole kv range of each sequence (used when the cache is built
directly).  Configurations with an assembly step also carry ``asm``: a source
cache that holds the kept prefix with whole pages of other tokens inserted at
an interior run, which the commit splice must drop again.

The named configurations:
  c1  1 x (512 + 256), 8/2 heads, P 16                  small correctness case
  c2  1 x (8192 + 2048), 32/8 heads, P 16; the 8192-token prefix is what
      survives assembling a 683-page source cache after dropping a contiguous
      run of 171 pages (25%, never page 0)
  c3  16 ragged contexts, prefix U[4096, 32768], segment U[512, 4096], 32/8,
      P 16, one shared pool of 131072 slots, same 25% drop per sequence
  c4  1 x (65536 + 8192), 64/8 heads, P 32, 1% of key rows scaled by 8
  c5  4 x (16384 + 2048) prefills plus 64 single-token decode rows with
      context U[4096, 16384], 32/8 heads, P 16
"""
from __future__ import annotations

import math
from dataclasses import dataclass, field
from typing import Optional

import numpy as np

from . import rng

# stream ids
S_Q, S_K, S_V, S_KDROP, S_VDROP, S_SLOTS, S_PRE, S_Q_LEN, S_DROP_AT, S_OUTLIER = range(10)


@dataclass
class AssembleInputs:
    src_len: np.ndarray          # [B] int64 tokens in the source cache
    src_indptr: np.ndarray       # [B+1] int32
    src_indices: np.ndarray      # [sum src pages] int32
    keep_indptr: np.ndarray      # [B+1] int32
    keep_spans: np.ndarray       # [n, 2] int32 [begin, end) logical source pages
    reserve: np.ndarray          # [B] int64 tokens to reserve after the kept ones
    fresh: np.ndarray            # [n_fresh] int32 free slots
    drop_at: np.ndarray          # [B] first dropped page
    n_drop: np.ndarray           # [B] dropped pages
    k_drop: np.ndarray           # [sum dropped tokens][Hkv][D] uint16 contents of dropped pages
    v_drop: np.ndarray


@dataclass
class Workload:
    name: str
    seed: int
    num_q_heads: int
    num_kv_heads: int
    head_dim: int
    page_size: int
    num_slots: int
    pre: np.ndarray              # [B] int64
    qlen: np.ndarray             # [B] int64
    q: np.ndarray                # uint16 [sum q][Hq][D]
    k: np.ndarray                # uint16 [sum kv][Hkv][D]
    v: np.ndarray
    pages_indptr: np.ndarray     # [B+1] int32
    pages: np.ndarray            # [sum pages] int32
    scale: float
    asm: Optional[AssembleInputs] = None
    outlier_rows: Optional[np.ndarray] = None   # [n] flat (token row, kv head) indices scaled x8
    notes: dict = field(default_factory=dict)

    @property
    def batch(self) -> int:
        return len(self.qlen)

    @property
    def kv(self) -> np.ndarray:
        return self.pre + self.qlen

    @property
    def q_indptr(self) -> np.ndarray:
        return np.concatenate([[0], np.cumsum(self.qlen)]).astype(np.int64)

    @property
    def kv_indptr(self) -> np.ndarray:
        return np.concatenate([[0], np.cumsum(self.kv)]).astype(np.int64)

    def seg_rows(self, b: int):
        """Rows of k/v holding sequence b's segment."""
        s = int(self.kv_indptr[b] + self.pre[b])
        return slice(s, s + int(self.qlen[b]))

    def prefix_rows(self, b: int):
        s = int(self.kv_indptr[b])
        return slice(s, s + int(self.pre[b]))

    def k_seg(self) -> np.ndarray:
        """Concatenated segment K rows [sum q][Hkv][D] (the append input)."""
        return np.concatenate([self.k[self.seg_rows(b)] for b in range(self.batch)], axis=0)

    def v_seg(self) -> np.ndarray:
        return np.concatenate([self.v[self.seg_rows(b)] for b in range(self.batch)], axis=0)

    def attn_pairs(self) -> int:
        """Unmasked (query, key) pairs per query head: sum_b q*pre + q(q+1)/2."""
        q = self.qlen.astype(np.int64)
        return int(np.sum(q * self.pre + q * (q + 1) // 2))

    def attn_flops(self) -> float:
        """Algorithmic attention FLOPs: 2 flops per MAC for QK^T and PV."""
        return 4.0 * self.head_dim * self.num_q_heads * self.attn_pairs()


def _pages(n, P):
    return -(-int(n) // P)


def build(name: str, seed: int, Hq: int, Hkv: int, D: int, P: int,
          pre, qlen, *, num_slots: Optional[int] = None, assemble: bool = False,
          outlier_frac: float = 0.0, outlier_scale: float = 8.0, std: float = 0.5,
          keep_page0: bool = True) -> Workload:
    """Build a workload from explicit per-sequence prefix and segment lengths."""
    pre = np.asarray(pre, dtype=np.int64)
    qlen = np.asarray(qlen, dtype=np.int64)
    B = len(qlen)
    kv = pre + qlen
    Tq, Tkv = int(qlen.sum()), int(kv.sum())
    q = rng.normal_bf16(seed, S_Q, (Tq, Hq, D), std)
    k = rng.normal_bf16(seed, S_K, (Tkv, Hkv, D), std)
    v = rng.normal_bf16(seed, S_V, (Tkv, Hkv, D), std)

    outliers = None
    if outlier_frac > 0:
        n_rows = Tkv * Hkv
        n_out = int(round(outlier_frac * n_rows))
        outliers = rng.choice(seed, S_OUTLIER, n_rows, n_out)
        kf = k.reshape(n_rows, D)
        vals = rng.bf16_bits_to_f32(kf[outliers]) * np.float32(outlier_scale)
        kf[outliers] = rng.f32_to_bf16_bits(vals)   # exact: power-of-two scale

    direct_pages = [_pages(x, P) for x in kv]
    asm_src_len = asm_drop_at = asm_n_drop = None
    n_src_pages = []
    if assemble:
        n_full = pre // P
        asm_n_drop = np.array([-(-int(f) // 3) for f in n_full], dtype=np.int64)
        lo = 1 if keep_page0 else 0
        asm_drop_at = np.array([int(rng.integers(seed, S_DROP_AT + 16 * b, 1, lo, max(lo, int(f)))[0])
                                for b, f in enumerate(n_full)], dtype=np.int64)
        asm_src_len = pre + asm_n_drop * P
        n_src_pages = [_pages(x, P) for x in asm_src_len]
        n_dst_pages = [_pages(x, P) for x in kv]
    need = sum(direct_pages) + (sum(n_src_pages) + sum(n_dst_pages) if assemble else 0)
    if num_slots is None:
        num_slots = max(16, 2 * need)
    if need > num_slots:
        raise ValueError(f"{name}: pool of {num_slots} slots cannot hold {need} pages")
    perm = rng.permutation(seed, S_SLOTS, num_slots)
    cur = 0
    pages_indptr = np.concatenate([[0], np.cumsum(direct_pages)]).astype(np.int32)
    pages = perm[cur: cur + sum(direct_pages)].copy()
    cur += sum(direct_pages)

    asm = None
    if assemble:
        src_indptr = np.concatenate([[0], np.cumsum(n_src_pages)]).astype(np.int32)
        src_indices = perm[cur: cur + sum(n_src_pages)].copy()
        cur += sum(n_src_pages)
        fresh = perm[cur: cur + sum(n_dst_pages)].copy()
        cur += sum(n_dst_pages)
        spans, keep_indptr = [], [0]
        for b in range(B):
            a, nd, ns = int(asm_drop_at[b]), int(asm_n_drop[b]), n_src_pages[b]
            if nd == 0:                       # too short to drop a whole page
                if ns > 0:
                    spans.append((0, ns))
            else:
                if a > 0:
                    spans.append((0, a))
                if a + nd < ns:
                    spans.append((a + nd, ns))
            keep_indptr.append(len(spans))
        n_drop_tok = int((asm_n_drop * P).sum())
        asm = AssembleInputs(
            src_len=asm_src_len, src_indptr=src_indptr, src_indices=src_indices,
            keep_indptr=np.asarray(keep_indptr, dtype=np.int32),
            keep_spans=np.asarray(spans, dtype=np.int32).reshape(-1, 2),
            reserve=qlen.copy(), fresh=fresh, drop_at=asm_drop_at, n_drop=asm_n_drop,
            k_drop=rng.normal_bf16(seed, S_KDROP, (n_drop_tok, Hkv, D), std),
            v_drop=rng.normal_bf16(seed, S_VDROP, (n_drop_tok, Hkv, D), std))

    return Workload(name=name, seed=seed, num_q_heads=Hq, num_kv_heads=Hkv, head_dim=D,
                    page_size=P, num_slots=int(num_slots), pre=pre, qlen=qlen, q=q, k=k, v=v,
                    pages_indptr=pages_indptr, pages=pages, scale=1.0 / math.sqrt(D), asm=asm,
                    outlier_rows=outliers)


def source_rows(w: Workload, b: int, which: str = "k") -> np.ndarray:
    """Logical contents of sequence b's source cache (kept prefix with the
    dropped pages inserted at their run), [src_len][Hkv][D]."""
    a = w.asm
    P = w.page_size
    full = w.k if which == "k" else w.v
    drop = a.k_drop if which == "k" else a.v_drop
    pre_rows = full[w.prefix_rows(b)]
    d0 = int((a.n_drop[:b] * P).sum())
    dropped = drop[d0: d0 + int(a.n_drop[b]) * P]
    cut = int(a.drop_at[b]) * P
    return np.concatenate([pre_rows[:cut], dropped, pre_rows[cut:]], axis=0)


CONFIG_SEEDS = {"c1": 1001, "c2": 1002, "c3": 1003, "c4": 1004, "c5": 1005}


def make(name: str, seed: Optional[int] = None) -> Workload:
    """The named configurations c1..c5 (see module docstring)."""
    s = CONFIG_SEEDS[name] if seed is None else seed
    if name == "c1":
        return build("c1", s, 8, 2, 128, 16, [512], [256])
    if name == "c2":
        # 8192 kept tokens = 512 pages; the source held 683 pages (171 dropped)
        return build("c2", s, 32, 8, 128, 16, [8192], [2048], assemble=True)
    if name == "c3":
        pre = rng.integers(s, S_PRE, 16, 4096, 32768)
        ql = rng.integers(s, S_Q_LEN, 16, 512, 4096)
        return build("c3", s, 32, 8, 128, 16, pre, ql, num_slots=131072, assemble=True)
    if name == "c4":
        return build("c4", s, 64, 8, 128, 32, [65536], [8192], outlier_frac=0.01)
    if name == "c5":
        ctx = rng.integers(s, S_PRE, 64, 4096, 16384)
        pre = np.concatenate([[16384] * 4, ctx - 1])
        ql = np.concatenate([[2048] * 4, [1] * 64])
        return build("c5", s, 32, 8, 128, 16, pre, ql)
    raise KeyError(name)


CONFIGS = ("c1", "c2", "c3", "c4", "c5")
