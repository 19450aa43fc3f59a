"""C-ABI library checks that need no GPU: it loads, exports every function
include/sa.h declares, and rejects bad arguments on the host before any HIP
call (the context argument is checked last, so a NULL context reaches the
shape checks)."""
import ctypes
import os
import re

import numpy as np
import pytest

import paper_2607_00151_amd as sa

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(sa.library_path()):
        from paper_2607_00151_amd import build
        build.build()
    return sa.load_library()


def declared_functions():
    text = open(os.path.join(ROOT, "include", "sa.h")).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(sa_[a-z_]+)\s*\(", text)))


def test_header_and_library_agree(lib):
    names = declared_functions()
    assert names == sorted(sa.EXPORTED_SYMBOLS)
    for n in names:
        assert hasattr(lib, n), n


def test_status_strings(lib):
    for code in range(10):
        assert lib.sa_status_string(code)
    assert lib.sa_status_string(99) == b"unknown status"


FAKE = 0x100000   # aligned non-null stand-in device address; never dereferenced


def layout(**kw):
    d = dict(num_q_heads=32, num_kv_heads=8, head_dim=128, page_size=16, num_layers=1,
             num_slots=1024)
    d.update(kw)
    return sa.Layout(**d)


def attn(lib, L, q_len, kv_len, q=FAKE, o=FAKE, layer=0, scale=0.1, lse=None, ctx=None):
    ql = np.asarray(q_len, dtype=np.int32)
    kl = np.asarray(kv_len, dtype=np.int32)
    return lib.sa_segment_prefill_attn(ctx, ctypes.byref(L), layer, q, FAKE, FAKE, len(ql),
                                       ql.ctypes.data, kl.ctypes.data,
                                       sa._Pages(FAKE, FAKE), scale, o, lse, None)


def test_attn_validation(lib):
    assert attn(lib, layout(), [4], [8]) == 1                     # all valid -> NULL ctx
    assert attn(lib, layout(head_dim=64), [4], [8]) == 3
    assert attn(lib, layout(page_size=8), [4], [8]) == 3
    assert attn(lib, layout(num_q_heads=12, num_kv_heads=8), [4], [8]) == 2
    assert attn(lib, layout(), [9], [8]) == 2                     # q_len > kv_len
    assert attn(lib, layout(), [-1], [8]) == 2
    assert attn(lib, layout(), [4], [8], layer=1) == 2
    assert attn(lib, layout(), [4], [8], q=FAKE + 8) == 4        # misaligned
    assert attn(lib, layout(), [4], [8], o=None) == 1
    assert attn(lib, layout(), [4], [8], scale=float("inf")) == 2
    assert attn(lib, layout(), [0], [8], q=None, o=None) == 1     # nothing to do, still needs ctx
    assert b"context" in lib.sa_last_error()


def attn_append(lib, L, q_len, kv_len, k_new=FAKE, v_new=FAKE, layer=0):
    ql = np.asarray(q_len, dtype=np.int32)
    kl = np.asarray(kv_len, dtype=np.int32)
    return lib.sa_segment_prefill_attn_append(None, ctypes.byref(L), layer, FAKE, FAKE, FAKE, k_new, v_new,
                                              len(ql), ql.ctypes.data, kl.ctypes.data,
                                              sa._Pages(FAKE, FAKE), 0.1, FAKE, None, None)


def test_exact_scale_needs_a_context(lib):
    assert lib.sa_set_exact_scale(None, 1) == 1
    assert b"context" in lib.sa_last_error()


def test_xcd_weights_need_a_context(lib):
    assert lib.sa_set_xcd_weights(None, None) == 1
    assert b"context" in lib.sa_last_error()


def test_block_clock_needs_a_context(lib):
    assert lib.sa_set_block_clock(None, None, 0, None) == 1
    assert b"context" in lib.sa_last_error()


def test_kernel_events_need_a_context(lib):
    assert lib.sa_set_kernel_events(None, 0, None, None) == 1
    assert b"context" in lib.sa_last_error()


def test_attn_append_validation(lib):
    assert attn_append(lib, layout(), [4], [8]) == 1                # all valid -> NULL ctx
    assert b"context" in lib.sa_last_error()
    assert attn_append(lib, layout(), [4], [8], k_new=None) == 1
    assert b"k_new" in lib.sa_last_error()
    assert attn_append(lib, layout(), [4], [8], v_new=FAKE + 4) == 4
    assert attn_append(lib, layout(), [9], [8]) == 2
    assert attn_append(lib, layout(), [4], [8], layer=1) == 2
    assert attn_append(lib, layout(), [0], [8], k_new=None, v_new=None) == 1   # no new rows: still needs ctx
    assert b"context" in lib.sa_last_error()


def append(lib, L, start, new_len, k_new=FAKE, layer=0):
    st = np.asarray(start, dtype=np.int32)
    nl = np.asarray(new_len, dtype=np.int32)
    return lib.sa_kv_append(None, ctypes.byref(L), layer, FAKE, FAKE, k_new, FAKE, len(st),
                            st.ctypes.data, nl.ctypes.data, sa._Pages(FAKE, FAKE), None)


def test_append_validation(lib):
    assert append(lib, layout(), [0, 5], [3, 1]) == 1
    assert append(lib, layout(), [-1], [3]) == 2
    assert append(lib, layout(), [0], [-3]) == 2
    assert append(lib, layout(), [0], [3], k_new=None) == 1
    assert append(lib, layout(), [0], [3], k_new=FAKE + 2) == 4
    assert append(lib, layout(num_layers=2), [0], [3], layer=2) == 2


def assemble(lib, L, src_len, keep_indptr, spans, reserve, num_fresh=100, cap=100):
    a = [np.asarray(x, dtype=np.int32) for x in (src_len, keep_indptr, np.asarray(spans).reshape(-1),
                                                  reserve)]
    out = np.zeros(len(a[0]), dtype=np.int32)
    rc = lib.sa_kv_assemble(None, ctypes.byref(L), FAKE, FAKE, FAKE, FAKE, len(a[0]),
                            a[0].ctypes.data, a[1].ctypes.data, a[2].ctypes.data if a[2].size else None,
                            a[3].ctypes.data, sa._Pages(FAKE, FAKE), FAKE, num_fresh, FAKE, FAKE,
                            cap, out.ctypes.data, None)
    return rc


def test_assemble_validation(lib):
    L = layout(page_size=16)
    assert assemble(lib, L, [100], [0, 2], [[0, 2], [4, 7]], [10]) == 1
    assert assemble(lib, L, [100], [0, 2], [[0, 2], [1, 7]], [10]) == 5      # overlap
    assert assemble(lib, L, [100], [0, 1], [[0, 8]], [10]) == 5              # past the last page
    assert assemble(lib, L, [100], [0, 1], [[3, 3]], [10]) == 5              # empty span
    assert assemble(lib, L, [100], [0, 1], [[0, 7]], [20], num_fresh=7) == 6  # 120 tokens: 8 pages
    assert assemble(lib, L, [100], [0, 1], [[0, 7]], [20], cap=7) == 6
    assert assemble(lib, L, [100], [0, 1], [[0, 7]], [12], num_fresh=7, cap=7) == 1  # 112: 7 pages
    assert assemble(lib, L, [100], [1, 1], [[0, 7]], [10]) == 2              # indptr[0] != 0
    assert assemble(lib, L, [-1], [0, 0], [], [0]) == 2


def splice_alias(lib, L, src_len, keep_indptr, spans, reserve, num_fresh=100, cap=100, fresh=FAKE):
    a = [np.asarray(x, dtype=np.int32) for x in (src_len, keep_indptr, np.asarray(spans).reshape(-1),
                                                  reserve)]
    out = np.zeros(len(a[0]), dtype=np.int32)
    rc = lib.sa_kv_splice_alias(None, ctypes.byref(L), len(a[0]), a[0].ctypes.data, a[1].ctypes.data,
                                a[2].ctypes.data if a[2].size else None, a[3].ctypes.data,
                                sa._Pages(FAKE, FAKE), fresh, num_fresh, FAKE, FAKE, cap, out.ctypes.data,
                                None)
    return rc, out


def test_splice_alias_validation(lib):
    L = layout(page_size=16)
    assert splice_alias(lib, L, [100], [0, 2], [[0, 2], [4, 7]], [10])[0] == 1   # host checks pass; no context
    assert splice_alias(lib, L, [100], [0, 2], [[0, 2], [1, 7]], [10])[0] == 5   # overlap
    assert splice_alias(lib, L, [100], [0, 1], [[0, 8]], [10])[0] == 5           # past the last page
    # only reserved pages take fresh slots: 7 kept pages + 20 tokens -> 8 pages, 1 fresh
    assert splice_alias(lib, L, [100], [0, 1], [[0, 7]], [20], num_fresh=1)[0] == 1
    assert splice_alias(lib, L, [100], [0, 1], [[0, 7]], [20], num_fresh=0)[0] == 6
    assert splice_alias(lib, L, [100], [0, 1], [[0, 7]], [20], cap=7)[0] == 6
    assert splice_alias(lib, L, [100], [0, 1], [[0, 7]], [12], num_fresh=0, fresh=None)[0] == 1  # no page reserved
    assert splice_alias(lib, L, [100], [0, 1], [[0, 7]], [20], fresh=None)[0] == 1   # a NULL list is caught later
    assert splice_alias(lib, L, [100], [1, 1], [[0, 7]], [10])[0] == 2           # indptr[0] != 0


def assemble_append(lib, L, src_len, keep_indptr, spans, reserve, new_len, layer=0, k_new=FAKE, src_indices=FAKE):
    a = [np.asarray(x, dtype=np.int32) for x in (src_len, keep_indptr, np.asarray(spans).reshape(-1),
                                                  reserve, new_len)]
    out = np.zeros(len(a[0]), dtype=np.int32)
    return lib.sa_kv_assemble_append(None, ctypes.byref(L), FAKE, FAKE, FAKE, FAKE, len(a[0]),
                                     a[0].ctypes.data, a[1].ctypes.data,
                                     a[2].ctypes.data if a[2].size else None, a[3].ctypes.data,
                                     sa._Pages(FAKE, src_indices), FAKE, 100, FAKE, FAKE, 100, out.ctypes.data,
                                     layer, k_new, FAKE, a[4].ctypes.data, None)


def test_assemble_append_validation(lib):
    L = layout(page_size=16)
    # 100 tokens on 7 pages, 7 pages kept (100 tokens), room for 12 more: 112 = 7 pages
    assert assemble_append(lib, L, [100], [0, 1], [[0, 7]], [12], [12]) == 1   # host checks pass; no context
    assert assemble_append(lib, L, [100], [0, 1], [[0, 7]], [12], [13]) == 2   # 113 tokens need an 8th page
    assert assemble_append(lib, L, [100], [0, 1], [[0, 7]], [12], [-1]) == 2
    assert assemble_append(lib, L, [100], [0, 1], [[0, 7]], [12], [4], layer=1) == 2
    assert assemble_append(lib, L, [100], [0, 1], [[0, 7]], [12], [4], k_new=None) == 1
    assert assemble_append(lib, L, [100], [0, 1], [[0, 7]], [12], [4], k_new=FAKE + 2) == 4
    assert assemble_append(lib, L, [100], [0, 2], [[0, 2], [1, 7]], [12], [4]) == 5   # overlap
    # nothing cached: no source page is read, so the source slot list may be absent
    assert assemble_append(lib, L, [0, 0], [0, 0, 0], [], [40, 3], [40, 3], src_indices=None) == 1
    assert b"context" in lib.sa_last_error()
    assert assemble_append(lib, L, [100], [0, 1], [[0, 7]], [12], [4], src_indices=None) == 1
    assert b"NULL" in lib.sa_last_error()


def test_context_creation_without_gpu(lib):
    import torch
    if torch.cuda.is_available():
        pytest.skip("a GPU is present")
    h = ctypes.c_void_p()
    assert lib.sa_create(0, ctypes.byref(h)) == 8       # SA_ERR_DEVICE
    assert not h.value
