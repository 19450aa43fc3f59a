"""GPU parity: the HIP path through the C ABI against the CPU oracle.

Page operations and page tables must match bit for bit (pools are filled with
a NaN canary first, so stray writes show); attention must be within max-abs
2e-2 and mean-abs 2e-3 of the double-precision oracle, on every row for small
cases and on sampled rows at the full configuration sizes.
"""
import numpy as np
import pytest
import torch

import oracle
import paper_2607_00151_amd as sa
import workloads
from oracle import pages as opages
from workloads.configs import build, source_rows

from harness import (attention, build_cache, build_source_cache, compare, dev_i32, dev_u16,
                     host_u16, layout_of, lse_tolerance, new_pool, place_range, run_assemble,
                     sample_rows, score_shift_bound)


LSE_TOL = 1e-3      # natural-log units, every row of the default (exact-scale) path


def check_lse(w, got, ref, toks=None, heads=None, folded=False):
    """Device LSE against the oracle's: within LSE_TOL on the default path, where the
    scale is applied to each fp32 score; with the scale folded into the bf16 query
    (sa_set_exact_scale(ctx, 0)), within the per-row shift that rounding allows."""
    if not folded:
        err = np.abs(np.asarray(got, dtype=np.float64) - ref)
        assert np.isfinite(got).all() and float(err.max()) <= LSE_TOL, float(err.max())
        return
    if toks is None:
        T = int(w.q_indptr[-1])
        toks = np.repeat(np.arange(T, dtype=np.int64), w.num_q_heads)
        heads = np.tile(np.arange(w.num_q_heads, dtype=np.int32), T)
        got, ref = got.reshape(-1), ref.reshape(-1)
    tol = lse_tolerance(w, toks, heads)
    err = np.abs(got - ref)
    assert (err <= tol).all(), (float(err.max()), float((err - tol).max()))

pytestmark = pytest.mark.gpu

MAX_TOL, MEAN_TOL = 2e-2, 2e-3


@pytest.fixture(scope="module")
def ctx():
    print("creating context", flush=True)
    c = sa.Context(0)
    yield c
    c.close()


def small(name):
    if name == "c1":
        return workloads.make("c1")
    if name == "ragged_g4_p16":
        return build(name, 7, 8, 2, 128, 16, [0, 1, 37, 700, 16, 129], [1, 300, 64, 5, 17, 1],
                     assemble=True)
    if name == "g8_p32_outliers":
        return build(name, 8, 16, 2, 128, 32, [0, 513, 31], [77, 200, 1], outlier_frac=0.01,
                     assemble=True)
    if name == "g1_p16":
        return build(name, 9, 4, 4, 128, 16, [33, 0], [40, 130], assemble=True)
    if name == "g2_p32":
        return build(name, 10, 8, 4, 128, 32, [100], [100])
    if name == "g16_p16":
        return build(name, 11, 32, 2, 128, 16, [64, 3], [50, 9])
    if name == "g3_p16":
        return build(name, 12, 6, 2, 128, 16, [45, 0, 300], [43, 70, 2], assemble=True)
    if name == "zero_len":
        # sequences with no new tokens first, in the middle (one with no cache at all)
        # and last, beside a decode row and segments over partial pages
        return build(name, 13, 8, 2, 128, 16, [40, 300, 0, 64, 17, 5], [0, 90, 0, 130, 0, 1],
                     assemble=True)
    raise KeyError(name)


SMALL = ["c1", "ragged_g4_p16", "g8_p32_outliers", "g1_p16", "g2_p32", "g16_p16", "g3_p16", "zero_len"]
WITH_ASM = ["ragged_g4_p16", "g8_p32_outliers", "g1_p16", "g3_p16", "zero_len"]


def oracle_all(w):
    return oracle.attention_all(w.q, w.k, w.v, w.q_indptr, w.kv_indptr, w.num_q_heads,
                                w.num_kv_heads, w.scale)


# ------------------------------------------------------------------ append

@pytest.mark.parametrize("name", SMALL)
def test_append_bitexact(ctx, name):
    print(f"append {name}", flush=True)
    w = small(name)
    L = layout_of(w, num_layers=2)
    kp, vp = new_pool(w, 2), new_pool(w, 2)
    layer = 1
    # prefix placed by the harness, segment appended by the kernel
    for pool, full in ((kp, w.k), (vp, w.v)):
        place_range(pool, layer, w, lambda b, full=full: full[w.prefix_rows(b)], w.pages_indptr,
                    w.pages, w.pre)
    before_k, before_v = host_u16(kp), host_u16(vp)
    indptr, indices = dev_i32(w.pages_indptr), dev_i32(w.pages)
    sa.sa_kv_append(ctx, L, layer, kp, vp, dev_u16(w.k_seg()), dev_u16(w.v_seg()), w.pre, w.qlen,
                    indptr, indices)
    sa.sa_sync_check(ctx)
    sl, ro = opages.append_destinations(w.pre, w.qlen, w.pages_indptr, w.pages, w.page_size)
    for before, new, got in ((before_k, w.k_seg(), kp), (before_v, w.v_seg(), vp)):
        want = before.copy()
        opages.apply_append(want[layer], new, sl, ro)
        assert np.array_equal(host_u16(got), want)


# ---------------------------------------------------------------- assemble

@pytest.mark.parametrize("name", WITH_ASM)
def test_assemble_bitexact(ctx, name):
    print(f"assemble {name}", flush=True)
    w = small(name)
    a = w.asm
    L = layout_of(w, num_layers=2)
    kp, vp, sip, sid, fresh = build_source_cache(w, num_layers=2)
    before_k, before_v = host_u16(kp), host_u16(vp)
    dip, did, dst_len = run_assemble(ctx, w, L, kp, vp, sip, sid, fresh)
    sa.sa_sync_check(ctx)
    r = opages.assemble(a.src_len, a.src_indptr, a.src_indices, a.keep_indptr, a.keep_spans,
                        a.reserve, a.fresh, w.page_size)
    assert np.array_equal(dst_len, r["dst_len"])
    assert np.array_equal(dip.cpu().numpy(), r["dst_indptr"])
    n = int(r["dst_indptr"][-1])
    assert np.array_equal(did.cpu().numpy()[:n], r["dst_indices"])
    assert (did.cpu().numpy()[n:] == -1).all()
    for before, got in ((before_k, kp), (before_v, vp)):
        want = before.copy()
        want[:, r["copy_dst"]] = before[:, r["copy_src"]]
        assert np.array_equal(host_u16(got), want)
    # the kept prefix reads back as the workload's prefix rows
    g = host_u16(kp)[0]
    for b in range(w.batch):
        got = opages.gather_logical(g, r["dst_indptr"][b:], r["dst_indices"], [r["dst_len"][b]],
                                    w.page_size, 0)
        assert np.array_equal(got, w.k[w.prefix_rows(b)])


# --------------------------------------------------------------- attention

@pytest.mark.parametrize("name", SMALL)
def test_attention_all_rows(ctx, name):
    print(f"attention {name}", flush=True)
    w = small(name)
    L = layout_of(w)
    kp, vp, ip, ix = build_cache(w)
    o, lse = attention(ctx, w, L, dev_u16(w.q), kp, vp, ip, ix)
    sa.sa_sync_check(ctx)
    ref, ref_lse, _ = oracle_all(w)
    mx, mean = compare(host_u16(o), ref, MAX_TOL, MEAN_TOL)
    print(f"  max {mx:.3e} mean {mean:.3e}")
    check_lse(w, lse.cpu().numpy(), ref_lse)


def test_split_kv_and_merge(ctx):
    """Few long work items force key-range splits and the LSE merge."""
    w = build("split", 21, 8, 1, 128, 16, [5000, 3000, 70, 0], [1, 1, 3, 1])
    L = layout_of(w)
    kp, vp, ip, ix = build_cache(w)
    o, lse = attention(ctx, w, L, dev_u16(w.q), kp, vp, ip, ix)
    sa.sa_sync_check(ctx)
    ref, ref_lse, _ = oracle_all(w)
    compare(host_u16(o), ref, MAX_TOL, MEAN_TOL)
    check_lse(w, lse.cpu().numpy(), ref_lse)


def check_attention_append(ctx, w, launches=2, folded=False):
    """sa_segment_prefill_attn_append over a cache holding only the prefix (layer 1 of
    two): both pools end exactly as the oracle's append leaves them, and every output
    row and LSE matches the oracle.  Each launch starts from fresh pools, so the second
    also shows the launch left its counters ready for the next."""
    L = layout_of(w, num_layers=2)
    layer = 1
    ip, ix = dev_i32(w.pages_indptr), dev_i32(w.pages)
    ref, ref_lse, _ = oracle_all(w)
    sl, ro = opages.append_destinations(w.pre, w.qlen, w.pages_indptr, w.pages, w.page_size)
    T = int(w.q_indptr[-1])
    for n in range(launches):
        kp, vp = new_pool(w, 2), new_pool(w, 2)
        for pool, full in ((kp, w.k), (vp, w.v)):
            place_range(pool, layer, w, lambda b, full=full: full[w.prefix_rows(b)], w.pages_indptr,
                        w.pages, w.pre)
        want = [host_u16(kp), host_u16(vp)]
        o = torch.empty((T, w.num_q_heads, 128), dtype=torch.int16, device="cuda")
        lse = torch.empty((T, w.num_q_heads), dtype=torch.float32, device="cuda")
        sa.sa_segment_prefill_attn_append(ctx, L, layer, dev_u16(w.q), kp, vp, dev_u16(w.k_seg()),
                                          dev_u16(w.v_seg()), w.qlen, w.kv, ip, ix, w.scale, o, lse)
        sa.sa_sync_check(ctx)
        for wa, new, got in ((want[0], w.k_seg(), kp), (want[1], w.v_seg(), vp)):
            opages.apply_append(wa[layer], new, sl, ro)
            assert np.array_equal(host_u16(got), wa), n
        mx, mean = compare(host_u16(o), ref, MAX_TOL, MEAN_TOL)
        check_lse(w, lse.cpu().numpy(), ref_lse, folded=folded)
    print(f"  {w.name}: max {mx:.3e} mean {mean:.3e}", flush=True)


@pytest.mark.parametrize("name", SMALL)
def test_append_inside_attention_all_rows(ctx, name):
    print(f"attention with append {name}", flush=True)
    check_attention_append(ctx, small(name))


def test_append_inside_attention_split_kv(ctx):
    """Key-range split items: some end before the new keys, some start inside them."""
    print("attention with append, split", flush=True)
    check_attention_append(ctx, build("split", 21, 8, 1, 128, 16, [5000, 3000, 70, 0], [1, 1, 3, 1]))


def test_append_inside_attention_missing_page_is_reported(ctx, folded=False):
    """A new row whose page is not in the table is skipped and reported."""
    print("attention with append, missing page", flush=True)
    w = build("short", 51, 8, 2, 128, 16, [20], [40])
    L = layout_of(w)
    ip = dev_i32([0, 2])                          # 60 tokens need 4 pages; the table has 2
    ix = dev_i32(w.pages[:2])
    T = int(w.qlen.sum())
    kp, vp = new_pool(w), new_pool(w)
    o = torch.empty((T, w.num_q_heads, 128), dtype=torch.int16, device="cuda")
    sa.sa_segment_prefill_attn_append(ctx, L, 0, dev_u16(w.q), kp, vp, dev_u16(w.k_seg()), dev_u16(w.v_seg()),
                                      w.qlen, w.kv, ip, ix, w.scale, o)
    with pytest.raises(sa.SaError) as e:
        sa.sa_sync_check(ctx)
    assert e.value.name == "SA_ERR_RANGE"
    sa.sa_sync_check(ctx)
    check_attention_append(ctx, workloads.make("c1"), launches=1, folded=folded)   # the next launch is whole


def test_first_row_without_prefix_is_v0_bitwise(ctx):
    """With no cached prefix, segment row 0 sees only key 0: its output is v_0 bit for bit
    (p = 2^0 = 1 on both sides of the division), for every query head of the group."""
    w = build("v0", 61, 8, 2, 128, 16, [0, 0, 37], [5, 70, 3])
    L = layout_of(w)
    kp, vp, ip, ix = build_cache(w)
    o, _ = attention(ctx, w, L, dev_u16(w.q), kp, vp, ip, ix)
    sa.sa_sync_check(ctx)
    got = host_u16(o)
    G = w.num_q_heads // w.num_kv_heads
    for b in (0, 1):
        t, kv0 = int(w.q_indptr[b]), int(w.kv_indptr[b])
        for h in range(w.num_q_heads):
            assert np.array_equal(got[t, h], w.v[kv0, h // G]), (b, h)


def test_constant_values_and_zero_keys_closed_forms(ctx):
    """V = c everywhere gives O = c; K = 0 gives each row the mean of the values it sees."""
    w = build("closed", 62, 8, 2, 128, 16, [300, 0], [90, 130])
    L = layout_of(w)
    c = 0.375
    w.v[:] = workloads.rng.f32_to_bf16_bits(np.full(w.v.shape, c, dtype=np.float32))
    kp, vp, ip, ix = build_cache(w)
    o, _ = attention(ctx, w, L, dev_u16(w.q), kp, vp, ip, ix)
    sa.sa_sync_check(ctx)
    got = (host_u16(o).astype(np.uint32) << 16).view(np.float32)
    assert np.abs(got - c).max() <= c * 2.0 ** -8          # P rounded to bf16 in the numerator only

    w = build("closed", 63, 8, 2, 128, 16, [300, 0], [90, 130])
    w.k[:] = 0
    kp, vp, ip, ix = build_cache(w)
    o, _ = attention(ctx, w, L, dev_u16(w.q), kp, vp, ip, ix)
    sa.sa_sync_check(ctx)
    bits = host_u16(o)
    vf = (w.v.astype(np.uint32) << 16).view(np.float32).astype(np.float64)
    G = w.num_q_heads // w.num_kv_heads
    for b in range(w.batch):
        k0, pre = int(w.kv_indptr[b]), int(w.pre[b])
        run = np.cumsum(vf[k0: k0 + int(w.kv[b])], axis=0) / np.arange(1, int(w.kv[b]) + 1)[:, None, None]
        for i in range(int(w.qlen[b])):
            want = np.repeat(run[pre + i], G, axis=0)            # [Hq][D]
            compare(bits[int(w.q_indptr[b]) + i], want, MAX_TOL, MEAN_TOL)


@pytest.mark.parametrize("scale,std", [(1.0, 1.0), (2.0, 1.0), (1e-4, 1.0), (128 ** -0.5, 2.0)])
def test_large_and_tiny_softmax_scales(ctx, scale, std):
    """Scores spread over tens of powers of two (the running max keeps moving past the
    lazy-rescale threshold), nearly uniform weights, and inputs four times wider than the
    configurations' at their scale: every output within max 2e-2 / mean 2e-3 of the
    oracle and every LSE within 1e-3 (a missed rescale or an overflow would be off by
    factors of 2^8 or not finite)."""
    w = build(f"scale{scale}", 64, 8, 2, 128, 16, [700, 0, 33], [150, 90, 1], std=std)
    w.scale = scale
    L = layout_of(w)
    kp, vp, ip, ix = build_cache(w)
    o, lse = attention(ctx, w, L, dev_u16(w.q), kp, vp, ip, ix)
    sa.sa_sync_check(ctx)
    ref, ref_lse, _ = oracle_all(w)
    mx, mean = compare(host_u16(o), ref, MAX_TOL, MEAN_TOL)
    print(f"  scale {scale} std {std}: max {mx:.3e} mean {mean:.3e}", flush=True)
    check_lse(w, lse.cpu().numpy(), ref_lse)


def _bf16_bits(x):
    """bf16 bits of float values that bf16 holds exactly."""
    b = np.asarray(x, dtype=np.float32).view(np.uint32)
    assert ((b & 0xFFFF) == 0).all()
    return (b >> 16).astype(np.uint16)


def test_dominant_key_weight_is_exact(ctx):
    """The default path's normaliser carries the bf16 rounding of each row's record key.
    Every query row is e_0; key 0 scores 0 (it sets the row's offset in the first tile),
    key 100 (second tile) scores 39.25 * scale * log2 e = 5.005 above it (no rescale, under
    2^8), every other key about -30, and all V rows are one vector of entries in [1.5, 2).
    Key 100's probability 2^5.005 = 32.11 is packed to bf16 as 32.0; with numerator and
    denominator carrying the same value every output row is exactly the V row, bit for
    bit -- an fp32 denominator alone would scale it by 33.0 / 33.11 (over half an ulp)."""
    w = build("dominant", 41, 8, 2, 128, 16, [200, 0], [8, 5])
    G = w.num_q_heads // w.num_kv_heads
    rng = np.random.default_rng(41)
    q = np.zeros((int(w.q_indptr[-1]), w.num_q_heads, 128), dtype=np.float32)
    q[:, :, 0] = 1.0
    k = np.zeros((int(w.kv_indptr[-1]), w.num_kv_heads, 128), dtype=np.float32)
    k[:, :, 0] = -235.0
    vrow = (rng.choice([-1.0, 1.0], size=128) * (1.5 + rng.integers(0, 64, size=128) / 128.0)).astype(np.float32)
    v = np.broadcast_to(vrow, (int(w.kv_indptr[-1]), w.num_kv_heads, 128)).copy()
    s0 = int(w.kv_indptr[0])
    k[s0 + 0, :, 0] = 0.0
    k[s0 + 100, :, 0] = 39.25
    w.q, w.k, w.v = _bf16_bits(q), _bf16_bits(k), _bf16_bits(v)
    L = layout_of(w)
    kp, vp, ip, ix = build_cache(w)
    o, lse = attention(ctx, w, L, dev_u16(w.q), kp, vp, ip, ix)
    sa.sa_sync_check(ctx)
    got = host_u16(o)
    n0 = int(w.qlen[0])
    assert np.array_equal(got[:n0], np.broadcast_to(_bf16_bits(vrow), (n0, w.num_q_heads, 128)))
    # against the oracle too (the second sequence, no prefix, is plain causal attention)
    ref, ref_lse, _ = oracle_all(w)
    compare(got, ref, MAX_TOL, MEAN_TOL)
    check_lse(w, lse.cpu().numpy(), ref_lse)
    assert G == 4


@pytest.fixture(scope="module")
def ctx_folded():
    """A context in the fast mode that folds the scale into the bf16 query rows."""
    c = sa.Context(0)
    sa.sa_set_exact_scale(c, False)
    yield c
    c.close()


@pytest.mark.parametrize("name", SMALL)
def test_folded_scale_all_rows(ctx_folded, name):
    """Folded-scale mode: outputs within the same bars, the LSE within the per-row shift
    the bf16 rounding of the scaled query allows."""
    w = small(name)
    L = layout_of(w)
    kp, vp, ip, ix = build_cache(w)
    o, lse = attention(ctx_folded, w, L, dev_u16(w.q), kp, vp, ip, ix)
    sa.sa_sync_check(ctx_folded)
    ref, ref_lse, _ = oracle_all(w)
    compare(host_u16(o), ref, MAX_TOL, MEAN_TOL)
    check_lse(w, lse.cpu().numpy(), ref_lse, folded=True)


@pytest.mark.parametrize("scale", [1.0, 2.0, 1e-4])
def test_folded_scale_at_large_and_tiny_scales(ctx_folded, scale):
    """Folded-scale mode at large logits: each row's exponents may move by
    eps = 2^-8 max_j sum_d |c q_d k_jd|, so its LSE must stay within ln 2 eps of the
    oracle's and each output within (2^(2 eps) - 1) max|v| plus the bf16 roundings of P
    and O (2^-7 max|v|).  This is the mode's documented accuracy, not the default's."""
    w = build(f"fscale{scale}", 64, 8, 2, 128, 16, [700, 0, 33], [150, 90, 1], std=1.0)
    w.scale = scale
    L = layout_of(w)
    kp, vp, ip, ix = build_cache(w)
    o, lse = attention(ctx_folded, w, L, dev_u16(w.q), kp, vp, ip, ix)
    sa.sa_sync_check(ctx_folded)
    ref, ref_lse, _ = oracle_all(w)
    got = (host_u16(o).astype(np.uint32) << 16).view(np.float32).astype(np.float64)
    assert np.isfinite(got).all() and np.isfinite(lse.cpu().numpy()).all()
    check_lse(w, lse.cpu().numpy(), ref_lse, folded=True)
    T = int(w.q_indptr[-1])
    toks = np.repeat(np.arange(T, dtype=np.int64), w.num_q_heads)
    heads = np.tile(np.arange(w.num_q_heads, dtype=np.int32), T)
    eps = 2.0 ** -8 * score_shift_bound(w, toks, heads)
    vmax = np.abs((w.v.astype(np.uint32) << 16).view(np.float32)).max()
    tol = (2.0 ** (2 * eps) - 1.0) * vmax + 2.0 ** -7 * vmax + 1e-3
    err = np.abs(got - ref).reshape(T * w.num_q_heads, -1).max(axis=1)
    assert (err <= tol).all(), float((err - tol).max())
    if scale < 1e-3:
        compare(host_u16(o), ref, MAX_TOL, MEAN_TOL)


@pytest.mark.timeout(600)
def test_folded_scale_step_c2_full(ctx_folded):
    print("c2 full step, folded scale", flush=True)
    check_step(ctx_folded, workloads.make("c2"), per_seq_rows=128, folded=True)


def test_attention_kernel_events(ctx):
    """The timing hook (sa_set_kernel_events) launches the same kernel: same bits,
    and its two events span a positive time no longer than events around the call."""
    print("attention kernel events c1", flush=True)
    w = workloads.make("c1")
    L = layout_of(w)
    kp, vp, ip, ix = build_cache(w)
    o1, _ = attention(ctx, w, L, dev_u16(w.q), kp, vp, ip, ix)
    stream = torch.cuda.current_stream()
    kev = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
    cev = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
    for e in kev:
        e.record(stream)
    torch.cuda.synchronize()
    sa.sa_set_kernel_events(ctx, sa.TIMED_ATTN, kev[0].cuda_event, kev[1].cuda_event)
    try:
        cev[0].record(stream)
        o2, _ = attention(ctx, w, L, dev_u16(w.q), kp, vp, ip, ix)
        cev[1].record(stream)
    finally:
        sa.sa_set_kernel_events(ctx, sa.TIMED_ATTN)
    torch.cuda.synchronize()
    sa.sa_sync_check(ctx)
    assert torch.equal(o1, o2)
    k_ms, c_ms = kev[0].elapsed_time(kev[1]), cev[0].elapsed_time(cev[1])
    print(f"  kernel {k_ms * 1e3:.1f} us, call {c_ms * 1e3:.1f} us")
    assert 0.0 < k_ms <= c_ms
    # the page kernels: an append timed by its own events writes the same bits
    kp2, vp2 = new_pool(w, 1), new_pool(w, 1)
    indptr, indices = dev_i32(w.pages_indptr), dev_i32(w.pages)
    pev = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
    for e in pev:
        e.record(stream)
    torch.cuda.synchronize()
    sa.sa_set_kernel_events(ctx, sa.TIMED_PAGES, pev[0].cuda_event, pev[1].cuda_event)
    try:
        sa.sa_kv_append(ctx, L, 0, kp2, vp2, dev_u16(w.k_seg()), dev_u16(w.v_seg()), w.pre, w.qlen,
                        indptr, indices)
    finally:
        sa.sa_set_kernel_events(ctx, sa.TIMED_PAGES)
    torch.cuda.synchronize()
    sa.sa_sync_check(ctx)
    assert pev[0].elapsed_time(pev[1]) > 0.0
    kp3, vp3 = new_pool(w, 1), new_pool(w, 1)
    sa.sa_kv_append(ctx, L, 0, kp3, vp3, dev_u16(w.k_seg()), dev_u16(w.v_seg()), w.pre, w.qlen,
                    indptr, indices)
    sa.sa_sync_check(ctx)
    assert torch.equal(kp2, kp3) and torch.equal(vp2, vp3)


def test_page_permutation_invariance(ctx):
    """Where the pages sit in the pool does not change a single output bit."""
    w = workloads.make("c1")
    L = layout_of(w)
    kp, vp, ip, ix = build_cache(w)
    o1, _ = attention(ctx, w, L, dev_u16(w.q), kp, vp, ip, ix)
    w2 = workloads.make("c1")
    w2.pages = np.arange(len(w.pages), dtype=np.int32)[::-1].copy()
    kp2, vp2, ip2, ix2 = build_cache(w2)
    o2, _ = attention(ctx, w2, L, dev_u16(w.q), kp2, vp2, ip2, ix2)
    assert torch.equal(o1, o2)


def test_causality(ctx):
    """Changing the K/V of segment tokens after t leaves rows <= t bit-identical."""
    w = build("causal", 31, 8, 2, 128, 16, [40], [100])
    L = layout_of(w)
    kp, vp, ip, ix = build_cache(w)
    q = dev_u16(w.q)
    base, _ = attention(ctx, w, L, q, kp, vp, ip, ix)
    for t in (0, 37, 63, 98):
        w2 = build("causal", 31, 8, 2, 128, 16, [40], [100])
        cut = int(w.pre[0]) + t + 1
        w2.k[cut:] = workloads.rng.normal_bf16(500 + t, 1, w2.k[cut:].shape)
        w2.v[cut:] = workloads.rng.normal_bf16(600 + t, 2, w2.v[cut:].shape)
        kp2, vp2, _, _ = build_cache(w2)
        o2, _ = attention(ctx, w2, L, q, kp2, vp2, ip, ix)
        assert torch.equal(o2[: t + 1], base[: t + 1]), t
        assert not torch.equal(o2[t + 1:], base[t + 1:]), t


def test_chunked_prefill_matches_one_shot(ctx):
    """Segment decomposability on the device: append + attend chunk by chunk
    over the growing cache gives the one-shot rows (within tolerance of the
    oracle, and of each other)."""
    w = build("chunks", 41, 8, 2, 128, 16, [200], [300])
    L = layout_of(w)
    kp, vp, ip, ix = build_cache(w, with_segment=False)
    q = dev_u16(w.q)
    seg_k, seg_v = w.k_seg(), w.v_seg()
    outs = []
    for a, b in ((0, 77), (77, 200), (200, 300)):
        sa.sa_kv_append(ctx, L, 0, kp, vp, dev_u16(seg_k[a:b]), dev_u16(seg_v[a:b]),
                        [200 + a], [b - a], ip, ix)
        o = torch.empty((b - a, 8, 128), dtype=torch.int16, device="cuda")
        sa.sa_segment_prefill_attn(ctx, L, 0, q[a:b].contiguous(), kp, vp, [b - a], [200 + b], ip,
                                   ix, w.scale, o)
        outs.append(o)
    chunked = torch.cat(outs)
    one, _ = attention(ctx, w, L, q, kp, vp, ip, ix)
    sa.sa_sync_check(ctx)
    ref, _, _ = oracle_all(w)
    compare(host_u16(chunked), ref, MAX_TOL, MEAN_TOL)
    compare(host_u16(one), ref, MAX_TOL, MEAN_TOL)


def test_out_of_range_slot_is_reported(ctx):
    """A slot id beyond the pool is skipped by the kernels and reported."""
    w = workloads.make("c1")
    L = layout_of(w)
    kp, vp, ip, ix = build_cache(w)
    bad = w.pages.copy()
    bad[3] = w.num_slots + 5
    o, _ = attention(ctx, w, L, dev_u16(w.q), kp, vp, ip, dev_i32(bad))
    with pytest.raises(sa.SaError) as e:
        sa.sa_sync_check(ctx)
    assert e.value.name == "SA_ERR_RANGE"
    sa.sa_sync_check(ctx)           # flag cleared


# ------------------------------------------------------ whole step, full size

def run_step(ctx, w, L, state, mode="copy"):
    """assemble (commit splice; zero-copy in mode "alias") -> append (segment) -> attention;
    mode "splice_append" runs the first two as one launch (as the bench does), mode
    "attn_append" the last two."""
    kp, vp, sip, sid, fresh, dip, did, q, ks, vs, o, lse = state
    a = w.asm
    if mode == "splice_append":
        dst_len = sa.sa_kv_assemble_append(ctx, L, kp, vp, kp, vp, a.src_len, a.keep_indptr, a.keep_spans,
                                           a.reserve, sip, sid, fresh, dip, did, 0, ks, vs, w.qlen)
        sa.sa_segment_prefill_attn(ctx, L, 0, q, kp, vp, w.qlen, dst_len + w.qlen, dip, did, w.scale, o, lse)
        return dst_len
    if mode == "attn_append":
        dst_len = sa.sa_kv_assemble(ctx, L, kp, vp, kp, vp, a.src_len, a.keep_indptr, a.keep_spans,
                                    a.reserve, sip, sid, fresh, dip, did)
        sa.sa_segment_prefill_attn_append(ctx, L, 0, q, kp, vp, ks, vs, w.qlen, dst_len + w.qlen, dip, did,
                                          w.scale, o, lse)
        return dst_len
    alias = mode == "alias"
    if alias:
        dst_len = sa.sa_kv_splice_alias(ctx, L, a.src_len, a.keep_indptr, a.keep_spans, a.reserve, sip,
                                        sid, fresh, dip, did)
    else:
        dst_len = sa.sa_kv_assemble(ctx, L, kp, vp, kp, vp, a.src_len, a.keep_indptr, a.keep_spans,
                                    a.reserve, sip, sid, fresh, dip, did)
    sa.sa_kv_append(ctx, L, 0, kp, vp, ks, vs, dst_len, w.qlen, dip, did)
    sa.sa_segment_prefill_attn(ctx, L, 0, q, kp, vp, w.qlen, dst_len + w.qlen, dip, did, w.scale,
                               o, lse)
    return dst_len


def check_step(ctx, w, per_seq_rows, mode="copy", folded=False):
    alias = mode == "alias"
    L = layout_of(w)
    kp, vp, sip, sid, fresh = build_source_cache(w)
    if alias:
        # slots outside the source pages and the segment's pages must stay untouched
        k_before, v_before = kp.clone(), vp.clone()
    n_dst = len(w.asm.fresh)
    dip = torch.zeros(w.batch + 1, dtype=torch.int32, device="cuda")
    did = torch.full((n_dst,), -1, dtype=torch.int32, device="cuda")
    T = int(w.qlen.sum())
    o = torch.empty((T, w.num_q_heads, 128), dtype=torch.int16, device="cuda")
    lse = torch.empty((T, w.num_q_heads), dtype=torch.float32, device="cuda")
    state = (kp, vp, sip, sid, fresh, dip, did, dev_u16(w.q), dev_u16(w.k_seg()),
             dev_u16(w.v_seg()), o, lse)
    if not alias:
        pools_before = (kp.clone(), vp.clone())
    dst_len = run_step(ctx, w, L, state, mode)
    sa.sa_sync_check(ctx)
    assert np.array_equal(dst_len, w.pre)
    # the assembled cache reads back as prefix ++ segment, bit for bit (sampled sequences)
    splice = opages.splice_alias if alias else opages.assemble
    r = splice(w.asm.src_len, w.asm.src_indptr, w.asm.src_indices, w.asm.keep_indptr,
               w.asm.keep_spans, w.asm.reserve, w.asm.fresh, w.page_size)
    if alias:
        # no page was copied: only the rows the segment was appended to changed
        sl, ro = opages.append_destinations(w.pre, w.qlen, r["dst_indptr"], r["dst_indices"], w.page_size)
        touched = torch.zeros((L.num_slots, w.page_size), dtype=torch.bool, device="cuda")
        touched[torch.from_numpy(sl).cuda(), torch.from_numpy(ro).cuda()] = True
        for after, before in ((kp, k_before), (vp, v_before)):
            keep = ~touched[:, None, :, None].expand_as(after[0])
            assert torch.equal(after[0][keep], before[0][keep])
    assert np.array_equal(dip.cpu().numpy(), r["dst_indptr"])
    assert np.array_equal(did.cpu().numpy()[: r["dst_indptr"][-1]], r["dst_indices"])
    if not alias:
        # the whole pools, every slot and row: the oracle's splice (surviving pages copied
        # whole to their fresh slots) then its append, applied to the pools as they were;
        # canary-filled slots nobody writes must come out unchanged
        sl, ro = opages.append_destinations(r["dst_len"], w.qlen, r["dst_indptr"], r["dst_indices"],
                                            w.page_size)
        csrc = torch.from_numpy(np.asarray(r["copy_src"], dtype=np.int64)).cuda()
        cdst = torch.from_numpy(np.asarray(r["copy_dst"], dtype=np.int64)).cuda()
        for after, before, seg in ((kp, pools_before[0], w.k_seg()), (vp, pools_before[1], w.v_seg())):
            want = before.clone()
            want[0, cdst] = before[0, csrc]
            if len(sl):
                view = want[0].permute(0, 2, 1, 3)                  # [slot][row][head][d]
                view[torch.from_numpy(sl).cuda(), torch.from_numpy(ro).cuda()] = dev_u16(seg)
            assert torch.equal(after, want)
            del want
        del pools_before
    ip_h, ix_h = r["dst_indptr"], r["dst_indices"]
    for b in range(w.batch):
        pages_b = ix_h[ip_h[b]: ip_h[b + 1]]
        kv_b = int(w.kv[b])
        for pool, full in ((kp, w.k), (vp, w.v)):
            got = pool[0][torch.from_numpy(pages_b.astype(np.int64)).cuda()]
            got = host_u16(got)                               # [pages][Hkv][P][D]
            got = got.transpose(0, 2, 1, 3).reshape(-1, w.num_kv_heads, 128)[:kv_b]
            assert np.array_equal(got, full[int(w.kv_indptr[b]): int(w.kv_indptr[b]) + kv_b]), b
    # attention on sampled rows
    toks, heads = sample_rows(w, per_seq_rows)
    ref, ref_lse, _ = oracle.attention_rows(w.q, w.k, w.v, w.q_indptr, w.kv_indptr,
                                            w.num_q_heads, w.num_kv_heads, w.scale, toks, heads)
    got = host_u16(o)[toks, heads]
    mx, mean = compare(got, ref, MAX_TOL, MEAN_TOL)
    print(f"  {w.name}: {len(toks)} rows, max {mx:.3e} mean {mean:.3e}", flush=True)
    check_lse(w, lse.cpu().numpy()[toks, heads], ref_lse, toks, heads, folded=folded)
    assert torch.isfinite(o.view(torch.bfloat16).float()).all()


@pytest.mark.parametrize("name", WITH_ASM)
def test_step_small(ctx, name):
    check_step(ctx, small(name), per_seq_rows=64)


@pytest.mark.parametrize("name", WITH_ASM)
def test_step_small_zero_copy_splice(ctx, name):
    check_step(ctx, small(name), per_seq_rows=64, mode="alias")


@pytest.mark.parametrize("mode", ["splice_append", "attn_append"])
@pytest.mark.parametrize("name", WITH_ASM)
def test_step_small_fused(ctx, name, mode):
    print(f"step {mode} {name}", flush=True)
    check_step(ctx, small(name), per_seq_rows=64, mode=mode)


@pytest.mark.parametrize("layers,layer", [(1, 0), (2, 1)])
@pytest.mark.parametrize("name", WITH_ASM)
def test_splice_and_append_in_one_launch(ctx, name, layers, layer):
    """sa_kv_assemble_append leaves both pools exactly as the oracle's splice (whole
    pages copied, in every layer) followed by its append (in the given layer only) --
    including the rows of a partial last surviving page that the segment fills and
    those it does not.  With the append in layer 0 the attention over the result is
    checked too (the other layers hold bit-flipped copies of the rows)."""
    print(f"splice+append {name}, {layers} layers, append in layer {layer}", flush=True)
    w = small(name)
    a = w.asm
    L = layout_of(w, num_layers=layers)
    kp, vp, sip, sid, fresh = build_source_cache(w, num_layers=layers)
    want_k, want_v = host_u16(kp).copy(), host_u16(vp).copy()
    dip = torch.zeros(w.batch + 1, dtype=torch.int32, device="cuda")
    did = torch.full((len(a.fresh),), -1, dtype=torch.int32, device="cuda")
    kept = sa.sa_kv_assemble_append(ctx, L, kp, vp, kp, vp, a.src_len, a.keep_indptr, a.keep_spans,
                                    a.reserve, sip, sid, fresh, dip, did, layer, dev_u16(w.k_seg()),
                                    dev_u16(w.v_seg()), w.qlen)
    sa.sa_sync_check(ctx)
    r = opages.assemble(a.src_len, a.src_indptr, a.src_indices, a.keep_indptr, a.keep_spans,
                        a.reserve, a.fresh, w.page_size)
    assert np.array_equal(kept, r["dst_len"])
    assert np.array_equal(dip.cpu().numpy(), r["dst_indptr"])
    assert np.array_equal(did.cpu().numpy()[: r["dst_indptr"][-1]], r["dst_indices"])
    sl, ro = opages.append_destinations(r["dst_len"], w.qlen, r["dst_indptr"], r["dst_indices"],
                                        w.page_size)
    for want, seg in ((want_k, w.k_seg()), (want_v, w.v_seg())):
        for lay in range(layers):
            for s_, d_ in zip(r["copy_src"], r["copy_dst"]):
                want[lay, d_] = want[lay, s_]
        opages.apply_append(want[layer], seg, sl, ro)
    assert np.array_equal(host_u16(kp), want_k)
    assert np.array_equal(host_u16(vp), want_v)
    assert any(int(x) % w.page_size for x in r["dst_len"])    # a partial last page was exercised
    if layer != 0:
        return
    o, lse = attention(ctx, w, L, dev_u16(w.q), kp, vp, dip, did)
    sa.sa_sync_check(ctx)
    ref, ref_lse, _ = oracle_all(w)
    compare(host_u16(o), ref, MAX_TOL, MEAN_TOL)
    check_lse(w, lse.cpu().numpy(), ref_lse)

@pytest.mark.parametrize("k", range(4))
def test_random_page_batches(ctx, k):
    """Seeded larger page batches: up to 16 sequences over prefixes up to 8000 tokens, a fifth
    of them with no new tokens, 1-4 layers with the append in a random one, the splice and
    append in one launch or as two calls -- both pools, every layer and slot, bit for bit
    against the oracle's splice then append."""
    r = np.random.default_rng(60000 + k)
    B = int(r.integers(1, 17))
    Hkv = int(r.choice([1, 2, 4, 8]))
    P = int(r.choice([16, 32]))
    pre = [int(x) for x in r.integers(0, 8001, B)]
    ql = [int(x) if r.random() < 0.8 else 0 for x in r.integers(1, 2001, B)]
    layers = int(r.integers(1, 5))
    layer = int(r.integers(0, layers))
    fused = bool(r.random() < 0.5)
    print(f"random pages {k}: B {B} Hkv {Hkv} P {P} layers {layers} append layer {layer} fused {fused}",
          flush=True)
    w = build(f"pages{k}", 60000 + k, Hkv, Hkv, 128, P, pre, ql, assemble=True)
    a = w.asm
    L = layout_of(w, num_layers=layers)
    kp, vp, sip, sid, fresh = build_source_cache(w, num_layers=layers)
    want_k, want_v = host_u16(kp).copy(), host_u16(vp).copy()
    dip = torch.zeros(w.batch + 1, dtype=torch.int32, device="cuda")
    did = torch.full((len(a.fresh),), -1, dtype=torch.int32, device="cuda")
    if fused:
        kept = sa.sa_kv_assemble_append(ctx, L, kp, vp, kp, vp, a.src_len, a.keep_indptr, a.keep_spans,
                                        a.reserve, sip, sid, fresh, dip, did, layer, dev_u16(w.k_seg()),
                                        dev_u16(w.v_seg()), w.qlen)
    else:
        kept = sa.sa_kv_assemble(ctx, L, kp, vp, kp, vp, a.src_len, a.keep_indptr, a.keep_spans,
                                 a.reserve, sip, sid, fresh, dip, did)
        sa.sa_kv_append(ctx, L, layer, kp, vp, dev_u16(w.k_seg()), dev_u16(w.v_seg()), kept, w.qlen,
                        dip, did)
    sa.sa_sync_check(ctx)
    res = opages.assemble(a.src_len, a.src_indptr, a.src_indices, a.keep_indptr, a.keep_spans,
                          a.reserve, a.fresh, w.page_size)
    assert np.array_equal(kept, res["dst_len"])
    assert np.array_equal(dip.cpu().numpy(), res["dst_indptr"])
    assert np.array_equal(did.cpu().numpy()[: res["dst_indptr"][-1]], res["dst_indices"])
    sl, ro = opages.append_destinations(res["dst_len"], w.qlen, res["dst_indptr"], res["dst_indices"],
                                        w.page_size)
    src = np.asarray(res["copy_src"], dtype=np.int64)
    dst = np.asarray(res["copy_dst"], dtype=np.int64)
    for want, seg in ((want_k, w.k_seg()), (want_v, w.v_seg())):
        for lay in range(layers):
            for s_, d_ in zip(src, dst):
                want[lay, d_] = want[lay, s_]
        opages.apply_append(want[layer], seg, sl, ro)
    assert np.array_equal(host_u16(kp), want_k)
    assert np.array_equal(host_u16(vp), want_v)


def random_case(k):
    """Seeded small workload k: 1-5 sequences, prefixes 0..700 (partial pages included),
    segments 1..300, 1-4 KV heads with G in {1, 2, 4, 8}, page 16 or 32; case 12 has no
    prefixes, case 13 only whole-page ones."""
    r = np.random.default_rng(7000 + k)
    B = int(r.integers(1, 6))
    Hkv = int(r.choice([1, 2, 4]))
    G = int(r.choice([1, 2, 4, 8]))
    P = int(r.choice([16, 32]))
    pre = [int(x) for x in r.integers(0, 701, B)]
    ql = [int(x) for x in r.integers(1, 301, B)]
    if k == 12:
        pre = [0] * B                                   # nothing cached: plain causal prefill
    if k == 13:
        pre = [P * int(x) for x in r.integers(1, 20, B)]  # prefixes that end on a page boundary
    return build(f"rand{k}", 7000 + k, Hkv * G, Hkv, 128, P, pre, ql, assemble=True)


@pytest.mark.parametrize("k", range(14))
def test_random_small_steps(ctx, k):
    """The benchmark step's launches (splice with the append in one launch, then the
    attention) on seeded random shapes: destination table and kept lengths exact, every
    output row and LSE against the oracle."""
    w = random_case(k)
    print(f"random step {k}: B {w.batch} Hq {w.num_q_heads} Hkv {w.num_kv_heads} P {w.page_size} "
          f"pre {list(w.pre)} q {list(w.qlen)}", flush=True)
    a = w.asm
    L = layout_of(w)
    kp, vp, sip, sid, fresh = build_source_cache(w)
    dip = torch.zeros(w.batch + 1, dtype=torch.int32, device="cuda")
    did = torch.full((len(a.fresh),), -1, dtype=torch.int32, device="cuda")
    kept = sa.sa_kv_assemble_append(ctx, L, kp, vp, kp, vp, a.src_len, a.keep_indptr, a.keep_spans,
                                    a.reserve, sip, sid, fresh, dip, did, 0, dev_u16(w.k_seg()),
                                    dev_u16(w.v_seg()), w.qlen)
    o, lse = attention(ctx, w, L, dev_u16(w.q), kp, vp, dip, did)
    sa.sa_sync_check(ctx)
    r = opages.assemble(a.src_len, a.src_indptr, a.src_indices, a.keep_indptr, a.keep_spans,
                        a.reserve, a.fresh, w.page_size)
    assert np.array_equal(kept, w.pre) and np.array_equal(kept, r["dst_len"])
    assert np.array_equal(dip.cpu().numpy(), r["dst_indptr"])
    assert np.array_equal(did.cpu().numpy()[: r["dst_indptr"][-1]], r["dst_indices"])
    ref, ref_lse, _ = oracle_all(w)
    compare(host_u16(o), ref, MAX_TOL, MEAN_TOL)
    check_lse(w, lse.cpu().numpy(), ref_lse)


@pytest.mark.parametrize("k", range(8))
def test_random_mixed_attention(ctx, k):
    """Seeded batches mixing decode rows (q = 1) and prefill segments over prefixes up to 6000
    tokens; with few work items the planner splits long ones by key range and merges the
    parts, so both paths meet shapes no fixed case has.  Every row and LSE vs the oracle."""
    r = np.random.default_rng(9000 + k)
    B = int(r.integers(1, 7))
    Hkv = int(r.choice([1, 2, 4]))
    G = int(r.choice([1, 2, 4, 8]))
    P = int(r.choice([16, 32]))
    pre = [int(x) for x in r.integers(0, 6001, B)]
    ql = [1 if r.random() < 0.5 else int(r.integers(2, 201)) for _ in range(B)]
    w = build(f"mixed{k}", 9000 + k, Hkv * G, Hkv, 128, P, pre, ql)
    print(f"random mixed {k}: Hq {w.num_q_heads} Hkv {Hkv} P {P} pre {pre} q {ql}", flush=True)
    L = layout_of(w)
    kp, vp, ip, ix = build_cache(w)
    o, lse = attention(ctx, w, L, dev_u16(w.q), kp, vp, ip, ix)
    sa.sa_sync_check(ctx)
    ref, ref_lse, _ = oracle_all(w)
    compare(host_u16(o), ref, MAX_TOL, MEAN_TOL)
    check_lse(w, lse.cpu().numpy(), ref_lse)


@pytest.mark.parametrize("k", range(6))
def test_random_large_batches(ctx, k):
    """Seeded larger batches: up to 24 sequences over prefixes up to 20000 tokens, 40% decode
    rows, G up to 16, page 16 or 32, half of them planned under random XCD speeds -- the
    planner's multi-round, pairing, split and weighting paths on shapes no fixed case has.
    Sampled rows (first and last token of every sequence in all heads, 8 random ones per
    sequence) and their LSE against the oracle."""
    r = np.random.default_rng(50000 + k)
    B = int(r.integers(1, 25))
    Hkv = int(r.choice([1, 2, 4, 8]))
    G = int(r.choice([1, 2, 4, 8, 16]))
    while Hkv * G > 64:
        G //= 2
    P = int(r.choice([16, 32]))
    pre = [int(x) for x in r.integers(0, 20001, B)]
    ql = [1 if r.random() < 0.4 else int(r.integers(1, 3001)) for _ in range(B)]
    weighted = r.random() < 0.5
    print(f"random large {k}: B {B} Hq {Hkv * G} Hkv {Hkv} P {P} sum pre {sum(pre)} sum q {sum(ql)} "
          f"weighted {weighted}", flush=True)
    w = build(f"large{k}", 50000 + k, Hkv * G, Hkv, 128, P, pre, ql)
    L = layout_of(w)
    kp, vp, ip, ix = build_cache(w)
    try:
        if weighted:
            sa.sa_set_xcd_weights(ctx, 0.9 + 0.2 * r.random(8))
        o, lse = attention(ctx, w, L, dev_u16(w.q), kp, vp, ip, ix)
        sa.sa_sync_check(ctx)
    finally:
        sa.sa_set_xcd_weights(ctx, None)
    toks, heads = sample_rows(w, 8, seed=k)
    ref, ref_lse, _ = oracle.attention_rows(w.q, w.k, w.v, w.q_indptr, w.kv_indptr, w.num_q_heads,
                                            w.num_kv_heads, w.scale, toks, heads)
    mx, mean = compare(host_u16(o)[toks, heads], ref, MAX_TOL, MEAN_TOL)
    print(f"  {len(toks)} rows, max {mx:.3e} mean {mean:.3e}", flush=True)
    check_lse(w, lse.cpu().numpy()[toks, heads], ref_lse, toks, heads)


def test_block_clock_records(ctx):
    """sa_set_block_clock: one record per workgroup, start <= end, the item's sequence and
    q_len, and the same output bits as without it; decode rows and prefill rows mixed."""
    w = build("clock", 77, 16, 4, 128, 16, [3000, 1200, 40, 5000], [1, 300, 1, 64])
    print("block clock: pre [3000, 1200, 40, 5000] q [1, 300, 1, 64]", flush=True)
    L = layout_of(w)
    kp, vp, ip, ix = build_cache(w)
    o1, _ = attention(ctx, w, L, dev_u16(w.q), kp, vp, ip, ix)
    buf = torch.full((4 * 4096,), -1, dtype=torch.int64, device="cuda")
    khz = sa.sa_set_block_clock(ctx, buf)
    try:
        o2, _ = attention(ctx, w, L, dev_u16(w.q), kp, vp, ip, ix)
    finally:
        sa.sa_set_block_clock(ctx, None)
    torch.cuda.synchronize()
    sa.sa_sync_check(ctx)
    assert torch.equal(o1, o2)
    assert khz > 0
    rec = buf.view(-1, 4).cpu().numpy()
    n = int((rec[:, 0] != -1).sum())
    assert n > 0 and (rec[n:] == -1).all()          # one record per workgroup, nothing beyond
    rec = rec[:n]
    assert (rec[:, 1] >= rec[:, 0]).all()
    it = clock_items(rec)
    live = it["q_len"] != 0                          # workgroups of padding items report q_len 0
    assert set(it["seq"][live].tolist()) == set(range(w.batch))
    assert np.array_equal(it["q_len"][live], w.qlen[it["seq"][live]])
    assert (it["kvh"][live] < w.num_kv_heads).all()
    G = w.num_q_heads // w.num_kv_heads
    assert (it["row0"][live] % 32 == 0).all() and (it["row0"][live] < w.qlen[it["seq"][live]] * G).all()
    span_us = (rec[:, 1].max() - rec[:, 0].min()) / khz * 1e3
    print(f"  {n} workgroups, clock {khz} kHz, span {span_us:.1f} us", flush=True)
    # a buffer too small for the launch is refused before anything runs
    small_buf = torch.zeros(4, dtype=torch.int64, device="cuda")
    sa.sa_set_block_clock(ctx, small_buf)
    try:
        with pytest.raises(sa.SaError):
            attention(ctx, w, L, dev_u16(w.q), kp, vp, ip, ix)
    finally:
        sa.sa_set_block_clock(ctx, None)


def clock_items(rec):
    """The work item of each sa_set_block_clock record: sequence, KV head, first key
    tile (mod 2^16), q_len and first packed query row."""
    w2, w3 = rec[:, 2], rec[:, 3]
    return {"seq": w2 & 0xFFFFFFFF, "kvh": (w2 >> 32) & 0xFFFF, "tile": (w2 >> 48) & 0xFFFF,
            "q_len": w3 & 0xFFFFFFFF, "row0": (w3 >> 32) & 0xFFFFFFFF}


def test_xcd_weights_two_rounds_every_item_once(ctx):
    """A launch of 512 work items (two per CU: the planner's swap search between XCDs),
    weighted twice in a row (the second call reuses the first's weighting): output and LSE
    equal the unweighted launch's bit for bit; every launch runs each (sequence, KV head,
    row tile, key tile) item exactly once; the second weighted launch places the items as
    the first did; and the XCD given 0.8 of the others' speed gets fewer key tiles."""
    w = build("xcdw2", 33, 32, 8, 128, 16, [3000], [2048])
    print("xcd weights, two rounds: Hq 32 / Hkv 8, pre 3000, q 2048", flush=True)
    L = layout_of(w)
    kp, vp, ip, ix = build_cache(w)
    buf = torch.full((4 * 4096,), -1, dtype=torch.int64, device="cuda")
    G = w.num_q_heads // w.num_kv_heads
    pre, kv = int(w.pre[0]), int(w.kv[0])

    def run():
        buf.fill_(-1)
        sa.sa_set_block_clock(ctx, buf)
        try:
            o, lse = attention(ctx, w, L, dev_u16(w.q), kp, vp, ip, ix)
        finally:
            sa.sa_set_block_clock(ctx, None)
        torch.cuda.synchronize()
        rec = buf.view(-1, 4).cpu().numpy().copy()
        n = int((rec[:, 0] != -1).sum())
        return o, lse, clock_items(rec[:n])

    def items(it):
        live = np.nonzero(it["q_len"] != 0)[0]
        keys = [(int(it["seq"][i]), int(it["kvh"][i]), int(it["row0"][i]), int(it["tile"][i])) for i in live]
        assert len(keys) == len(set(keys))                         # no item twice
        return keys, live

    def xcd_tiles(it, x):
        keys, live = items(it)
        tiles = 0
        for (s_, h, r0, t0), i in zip(keys, live):
            if i % 8 != x:
                continue
            end = min(kv, pre + (r0 + 128 + G - 1) // G)           # the row tile's last visible key + 1
            tiles += (end + 63) // 64 - t0
        return tiles

    o1, lse1, r1 = run()
    sa.sa_set_xcd_weights(ctx, [1, 1, 1, 1, 1, 1, 1, 0.8])
    try:
        o2, lse2, r2 = run()
        o3, lse3, r3 = run()
    finally:
        sa.sa_set_xcd_weights(ctx, None)
    sa.sa_sync_check(ctx)
    for o_, l_ in ((o2, lse2), (o3, lse3)):
        assert torch.equal(o1, o_) and torch.equal(lse1, l_)
    k1, _ = items(r1)
    k2, l2 = items(r2)
    k3, l3 = items(r3)
    assert len(k1) == 512 and set(k1) == set(k2) == set(k3)
    assert [(int(i), k) for i, k in zip(l2, k2)] == [(int(i), k) for i, k in zip(l3, k3)]
    t_before, t_after = xcd_tiles(r1, 7), xcd_tiles(r2, 7)
    others = [xcd_tiles(r2, x) for x in range(7)]
    print(f"  XCD 7 key tiles {t_before} -> {t_after}; others {min(others)}..{max(others)}", flush=True)
    assert t_after < t_before and t_after < min(others)
    toks, heads = sample_rows(w, 64)
    ref, ref_lse, _ = oracle.attention_rows(w.q, w.k, w.v, w.q_indptr, w.kv_indptr,
                                            w.num_q_heads, w.num_kv_heads, w.scale, toks, heads)
    compare(host_u16(o2)[toks, heads], ref, MAX_TOL, MEAN_TOL)


def test_xcd_weights_move_work_not_results(ctx):
    """sa_set_xcd_weights re-places work items across the XCDs: the output is the same bit
    for bit (and matches the oracle on sampled rows), and the slow XCD gets fewer key tiles."""
    w = build("xcdw", 31, 32, 8, 128, 16, [2000], [1024])
    print("xcd weights: Hq 32 / Hkv 8, pre 2000, q 1024", flush=True)
    L = layout_of(w)
    kp, vp, ip, ix = build_cache(w)
    buf = torch.full((4 * 4096,), -1, dtype=torch.int64, device="cuda")

    def run():
        sa.sa_set_block_clock(ctx, buf)
        try:
            o, lse = attention(ctx, w, L, dev_u16(w.q), kp, vp, ip, ix)
        finally:
            sa.sa_set_block_clock(ctx, None)
        torch.cuda.synchronize()
        return o, lse, buf.view(-1, 4).cpu().numpy().copy()

    o1, lse1, r1 = run()
    sa.sa_set_xcd_weights(ctx, [1, 1, 1, 1, 1, 1, 1, 0.8])
    try:
        o2, lse2, r2 = run()
    finally:
        sa.sa_set_xcd_weights(ctx, None)
    sa.sa_sync_check(ctx)
    assert torch.equal(o1, o2) and torch.equal(lse1, lse2)
    n = int((r1[:, 0] != -1).sum())
    assert n == int((r2[:, 0] != -1).sum()) and n % 8 == 0
    # XCD 7 (workgroups i % 8 == 7) spends less time on its items than before
    t1 = (r1[:n, 1] - r1[:n, 0])[7::8].sum()
    t2 = (r2[:n, 1] - r2[:n, 0])[7::8].sum()
    print(f"  XCD 7 workgroup time {t1} -> {t2} clock ticks", flush=True)
    assert t2 < t1
    toks, heads = sample_rows(w, 64)
    ref, ref_lse, _ = oracle.attention_rows(w.q, w.k, w.v, w.q_indptr, w.kv_indptr,
                                            w.num_q_heads, w.num_kv_heads, w.scale, toks, heads)
    compare(host_u16(o2)[toks, heads], ref, MAX_TOL, MEAN_TOL)


@pytest.mark.timeout(600)
def test_step_c2_full(ctx):
    print("c2 full step", flush=True)
    check_step(ctx, workloads.make("c2"), per_seq_rows=512)


@pytest.mark.timeout(600)
@pytest.mark.parametrize("mode", ["splice_append", "attn_append"])
def test_step_c2_full_fused(ctx, mode):
    print(f"c2 full step, {mode}", flush=True)
    check_step(ctx, workloads.make("c2"), per_seq_rows=256, mode=mode)


@pytest.mark.timeout(900)
def test_step_c3_full(ctx):
    print("c3 full step", flush=True)
    check_step(ctx, workloads.make("c3"), per_seq_rows=192)


def check_direct(ctx, w, per_seq_rows, extra_rows=None, fused=False, folded=False):
    L = layout_of(w)
    kp, vp, ip, ix = build_cache(w, with_segment=False)
    if fused:
        T = int(w.qlen.sum())
        o = torch.empty((T, w.num_q_heads, 128), dtype=torch.int16, device="cuda")
        lse = torch.empty((T, w.num_q_heads), dtype=torch.float32, device="cuda")
        sa.sa_segment_prefill_attn_append(ctx, L, 0, dev_u16(w.q), kp, vp, dev_u16(w.k_seg()),
                                          dev_u16(w.v_seg()), w.qlen, w.kv, ip, ix, w.scale, o, lse)
    else:
        sa.sa_kv_append(ctx, L, 0, kp, vp, dev_u16(w.k_seg()), dev_u16(w.v_seg()), w.pre, w.qlen,
                        ip, ix)
        o, lse = attention(ctx, w, L, dev_u16(w.q), kp, vp, ip, ix)
    sa.sa_sync_check(ctx)
    toks, heads = sample_rows(w, per_seq_rows)
    if extra_rows is not None:
        toks = np.concatenate([toks, extra_rows[0]])
        heads = np.concatenate([heads, extra_rows[1]])
    ref, ref_lse, _ = oracle.attention_rows(w.q, w.k, w.v, w.q_indptr, w.kv_indptr,
                                            w.num_q_heads, w.num_kv_heads, w.scale, toks, heads)
    mx, mean = compare(host_u16(o)[toks, heads], ref, MAX_TOL, MEAN_TOL)
    print(f"  {w.name}: {len(toks)} rows, max {mx:.3e} mean {mean:.3e}", flush=True)
    check_lse(w, lse.cpu().numpy()[toks, heads], ref_lse, toks, heads, folded=folded)
    assert torch.isfinite(o.view(torch.bfloat16).float()).all()


@pytest.mark.timeout(600)
def test_c1_full(ctx):
    check_direct(ctx, workloads.make("c1"), per_seq_rows=256)


@pytest.mark.timeout(900)
def test_c4_full_outliers(ctx):
    print("c4 full", flush=True)
    w = workloads.make("c4")
    # rows whose own position is right after an outlier key: those keys dominate their softmax
    out_tok = (w.outlier_rows // w.num_kv_heads) - int(w.pre[0])
    out_kvh = w.outlier_rows % w.num_kv_heads
    sel = (out_tok >= 0) & (out_tok < int(w.qlen[0]))
    G = w.num_q_heads // w.num_kv_heads
    extra = (out_tok[sel][:64].astype(np.int64), (out_kvh[sel][:64] * G).astype(np.int32))
    check_direct(ctx, w, per_seq_rows=640, extra_rows=extra)


@pytest.mark.timeout(600)
@pytest.mark.parametrize("fused", [False, True])
def test_c5_full_mixed(ctx, fused):
    print(f"c5 full, append inside attention {fused}", flush=True)
    check_direct(ctx, workloads.make("c5"), per_seq_rows=96, fused=fused)
