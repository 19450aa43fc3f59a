"""The seeded input generator: determinism, rounding, and the recipes' shapes."""
import numpy as np
import torch

import workloads
from workloads import rng


def test_bf16_rounding_matches_torch():
    """Round-to-nearest-even to bf16, checked against torch's conversion,
    including exact ties."""
    g = rng.generator(1, 0)
    x = g.standard_normal(100000).astype(np.float32) * np.float32(3.0)
    ties = (np.arange(0, 128, dtype=np.uint32) << np.uint32(16)) | np.uint32(0x8000)
    ties = (ties + np.uint32(0x3F000000)).view(np.float32)   # mantissa halfway cases
    x = np.concatenate([x, ties, np.array([0.0, -0.0, 1e-30, -1e30], dtype=np.float32)])
    ours = rng.f32_to_bf16_bits(x)
    theirs = torch.from_numpy(x).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(ours, theirs)


def test_streams_are_deterministic_and_chunk_invariant():
    a = rng.normal_bf16(5, 3, (3, 1 << 20))          # spans several internal chunks
    b = rng.normal_bf16(5, 3, (3 << 20,))
    assert np.array_equal(a.reshape(-1), b)
    c = rng.normal_bf16(5, 4, (10,))
    assert not np.array_equal(b[:10], c)


def test_value_distribution():
    x = rng.bf16_bits_to_f32(rng.normal_bf16(9, 0, (1 << 20,))).astype(np.float64)
    assert abs(x.mean()) < 2e-3
    assert abs(x.std() - 0.5) < 2e-3


def test_c1_c2_recipes():
    w = workloads.make("c1")
    assert (w.num_q_heads, w.num_kv_heads, w.head_dim, w.page_size) == (8, 2, 128, 16)
    assert w.pre.tolist() == [512] and w.qlen.tolist() == [256]
    assert w.pages_indptr.tolist() == [0, 48]
    assert len(set(w.pages.tolist())) == 48
    w = workloads.make("c2")
    assert w.attn_flops() == 4 * 128 * 32 * (2048 * 8192 + 2048 * 2049 // 2)
    a = w.asm
    assert a.src_len.tolist() == [8192 + 171 * 16]
    assert 1 <= a.drop_at[0] <= 512 and a.n_drop.tolist() == [171]
    # source slots, fresh slots and the direct page list are disjoint
    s = set(a.src_indices.tolist()); f = set(a.fresh.tolist()); d = set(w.pages.tolist())
    assert not (s & f) and not (s & d) and not (f & d)
    src = workloads.configs.source_rows(w, 0, "k")
    P = w.page_size
    cut = int(a.drop_at[0]) * P
    kept = np.concatenate([src[:cut], src[cut + 171 * P:]])
    assert np.array_equal(kept, w.k[w.prefix_rows(0)])
