"""Oracle for the paged-cache operations (test infrastructure only).

Only the tests, the smoke check and the CPU-baseline leg of the benchmark use
this module; the product path never imports it.

The paper leaves the cache layout to the serving system (Sec. 5 builds on a
paged, prefix-cached KV store; Sec. 7 names paged attention and prefix
caching).  The readings written out here are:

* Paging.  A sequence's logical token x lives in page x // P of its page list,
  at row x % P of that page's slot.  Every page is full except possibly the
  last.
* Append.  Writing a new segment of n tokens at logical start s puts token t
  (0 <= t < n) at position s + t, i.e. at (slot of page (s + t) // P,
  row (s + t) % P).  Nothing else changes.
* Assemble (the commit splice of Sec. 3.2, where the transformed prefix
  replaces the old one; for keep-recent-K, Sec. 3.4, the head of the context
  and the recent turns survive while an interior run is dropped).  The caller
  names the surviving source pages as ascending, disjoint [begin, end) spans
  of logical page numbers.  The replacement cache of a sequence is those pages
  in ascending order, renumbered densely from 0, followed by as many new pages
  as ``reserve`` further tokens need.  Its slots are taken from the front of a
  caller-supplied free list, sequence after sequence; each surviving page is
  copied whole (all P rows) from its source slot to its new slot.

Each function is the definition, one page or token at a time.
"""
from __future__ import annotations

import numpy as np


def pages_for(n_tokens: int, P: int) -> int:
    """Pages needed to hold n_tokens tokens."""
    return -(-int(n_tokens) // P)


def append_destinations(start, new_len, indptr, indices, P):
    """(slot, row) of every appended token, in input order.

    start, new_len: per-sequence logical start and count of new tokens.
    indptr, indices: the sequence page lists (CSR).
    Returns int64 arrays slot[sum new_len], row[sum new_len].
    """
    slots, rows = [], []
    for b in range(len(new_len)):
        base = int(indptr[b])
        n_pages = int(indptr[b + 1]) - base
        for t in range(int(new_len[b])):
            x = int(start[b]) + t
            page = x // P
            if page >= n_pages:
                raise ValueError(f"sequence {b}: token {x} needs page {page}, only {n_pages}")
            slots.append(int(indices[base + page]))
            rows.append(x % P)
    return np.asarray(slots, dtype=np.int64), np.asarray(rows, dtype=np.int64)


def apply_append(pool, new_rows, slots, rows):
    """Expected pool after an append: pool[slot][:, row, :] = new token's rows.

    pool: array [num_slots][Hkv][P][D] (modified in place and returned).
    new_rows: [sum new_len][Hkv][D] in input order.
    """
    for t in range(len(slots)):
        pool[slots[t], :, rows[t], :] = new_rows[t]
    return pool


def kept_tokens_of_page(src_len: int, page: int, P: int) -> int:
    """Tokens held by logical page `page` of a sequence of src_len tokens."""
    return min(P, int(src_len) - page * P)


def assemble(src_len, src_indptr, src_indices, keep_indptr, keep_spans, reserve, fresh, P):
    """Replacement-cache plan and destination page table.

    src_len[b]              tokens in sequence b's source cache
    src_indptr/src_indices  source page lists
    keep_indptr[b+1], keep_spans[n][2]   surviving [begin, end) page spans
    reserve[b]              tokens to leave room for after the kept ones
    fresh                   free slots, consumed from the front

    Returns dict with dst_indptr [B+1], dst_indices [sum dst pages],
    dst_len [B] (kept tokens), copy_src / copy_dst slot pairs (whole pages).
    """
    B = len(src_len)
    dst_indptr = [0]
    dst_indices, dst_len, copy_src, copy_dst = [], [], [], []
    cursor = 0
    for b in range(B):
        n_src_pages = pages_for(src_len[b], P)
        if int(src_indptr[b + 1]) - int(src_indptr[b]) < n_src_pages:
            raise ValueError(f"sequence {b}: page list shorter than its length")
        kept_pages = []
        prev_end = 0
        for s in range(int(keep_indptr[b]), int(keep_indptr[b + 1])):
            begin, end = int(keep_spans[s][0]), int(keep_spans[s][1])
            if not (prev_end <= begin < end <= n_src_pages):
                raise ValueError(f"sequence {b}: bad keep span [{begin}, {end})")
            prev_end = end
            kept_pages.extend(range(begin, end))
        kept = sum(kept_tokens_of_page(src_len[b], p, P) for p in kept_pages)
        n_dst = max(len(kept_pages), pages_for(kept + int(reserve[b]), P))
        if cursor + n_dst > len(fresh):
            raise ValueError("free list exhausted")
        for j in range(n_dst):
            slot = int(fresh[cursor + j])
            dst_indices.append(slot)
            if j < len(kept_pages):
                copy_src.append(int(src_indices[int(src_indptr[b]) + kept_pages[j]]))
                copy_dst.append(slot)
        cursor += n_dst
        dst_indptr.append(cursor)
        dst_len.append(kept)
    return {
        "dst_indptr": np.asarray(dst_indptr, dtype=np.int32),
        "dst_indices": np.asarray(dst_indices, dtype=np.int32),
        "dst_len": np.asarray(dst_len, dtype=np.int64),
        "copy_src": np.asarray(copy_src, dtype=np.int64),
        "copy_dst": np.asarray(copy_dst, dtype=np.int64),
    }


def splice_alias(src_len, src_indptr, src_indices, keep_indptr, keep_spans, reserve, fresh, P):
    """Zero-copy form of the splice: the replacement cache of a sequence is its
    surviving source pages, in order, left in their source slots, followed by
    as many new pages as ``reserve`` further tokens need, whose slots are taken
    from the front of the free list, sequence after sequence.  Nothing is copied.

    Returns dict with dst_indptr [B+1], dst_indices, dst_len [B] (kept tokens)
    and fresh_used (free-list entries consumed).
    """
    B = len(src_len)
    dst_indptr, dst_indices, dst_len = [0], [], []
    cursor = 0
    for b in range(B):
        n_src_pages = pages_for(src_len[b], P)
        if int(src_indptr[b + 1]) - int(src_indptr[b]) < n_src_pages:
            raise ValueError(f"sequence {b}: page list shorter than its length")
        kept_pages, prev_end = [], 0
        for s in range(int(keep_indptr[b]), int(keep_indptr[b + 1])):
            begin, end = int(keep_spans[s][0]), int(keep_spans[s][1])
            if not (prev_end <= begin < end <= n_src_pages):
                raise ValueError(f"sequence {b}: bad keep span [{begin}, {end})")
            prev_end = end
            kept_pages.extend(range(begin, end))
        kept = sum(kept_tokens_of_page(src_len[b], p, P) for p in kept_pages)
        n_dst = max(len(kept_pages), pages_for(kept + int(reserve[b]), P))
        for p in kept_pages:
            dst_indices.append(int(src_indices[int(src_indptr[b]) + p]))
        n_new = n_dst - len(kept_pages)
        if cursor + n_new > len(fresh):
            raise ValueError("free list exhausted")
        dst_indices.extend(int(x) for x in fresh[cursor: cursor + n_new])
        cursor += n_new
        dst_indptr.append(len(dst_indices))
        dst_len.append(kept)
    return {
        "dst_indptr": np.asarray(dst_indptr, dtype=np.int32),
        "dst_indices": np.asarray(dst_indices, dtype=np.int32),
        "dst_len": np.asarray(dst_len, dtype=np.int64),
        "fresh_used": cursor,
    }


def gather_logical(pool, indptr, indices, lengths, P, b):
    """Contiguous [len][Hkv][D] rows of sequence b read back through its page list."""
    n = int(lengths[b])
    base = int(indptr[b])
    out = np.empty((n,) + pool.shape[1:2] + pool.shape[3:], dtype=pool.dtype)
    for x in range(n):
        out[x] = pool[int(indices[base + x // P]), :, x % P, :]
    return out
