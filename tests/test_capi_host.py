"""Host-side checks of the C ABI that need no GPU: the library loads, exports every
entry point the header declares, and rejects bad arguments before touching the device."""
import ctypes
import os
import re

import pytest

from paper_2502_21231_amd import bs_attn as B

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "bs_attn.h")


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(bs_\w+)\s*\(", text)))


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(B.LIB_PATH):
        pytest.fail("libbs_attn.so is not built (run __graft_entry__.build())")
    return B.load_library()


def test_exports_every_declared_symbol(lib):
    names = declared_functions()
    assert len(names) == 19, names
    assert set(names) == set(B.EXPORTS)
    for n in names:
        assert hasattr(lib, n), n


FAKE = 4096  # a non-null, aligned address that the validation rejects before any use


def dims(**kw):
    d = dict(total_q=128, total_k=128, hq=4, hkv=2, head_dim=128, dtype=B.BS_BF16)
    d.update(kw)
    return B.bs_dims(**d)


def fwd(lib, d, ws_bytes=1 << 30, scale=0.1, q=FAKE, cu=FAKE):
    return lib.bs_attn_varlen_fwd(ctypes.byref(d), q, FAKE, FAKE, cu, cu, 1, 128, 1, scale, FAKE,
                                  FAKE, FAKE, ws_bytes, None)


def test_rejects_bad_arguments_without_device(lib):
    assert fwd(lib, dims(head_dim=96)) == B.BS_ERR_UNSUPPORTED
    assert "head_dim" in B.bs_last_error()
    assert fwd(lib, dims(dtype=7)) == B.BS_ERR_UNSUPPORTED
    assert fwd(lib, dims(hq=6, hkv=4)) == B.BS_ERR_INVALID_ARG
    assert fwd(lib, dims(hkv=0)) == B.BS_ERR_INVALID_ARG
    assert fwd(lib, dims(hq=8192, hkv=8)) == B.BS_ERR_INVALID_ARG  # above the 4096-head limit
    assert fwd(lib, dims(total_q=-1)) == B.BS_ERR_INVALID_ARG
    assert fwd(lib, dims(), q=None) == B.BS_ERR_INVALID_ARG
    assert "q is NULL" in B.bs_last_error()
    assert fwd(lib, dims(), q=FAKE + 2) == B.BS_ERR_INVALID_ARG
    assert fwd(lib, dims(), scale=float("nan")) == B.BS_ERR_INVALID_ARG
    assert fwd(lib, dims(), scale=-1.0) == B.BS_ERR_INVALID_ARG
    assert fwd(lib, dims(), cu=None) == B.BS_ERR_INVALID_ARG
    assert fwd(lib, dims(), ws_bytes=16) == B.BS_ERR_WORKSPACE
    assert "smaller" in B.bs_last_error()
    d = dims()
    assert lib.bs_lse_merge(ctypes.byref(d), FAKE, FAKE, 0, FAKE, FAKE, None) == B.BS_ERR_INVALID_ARG
    # the packed chunk ops need the per-segment positions as well as cu_seqlens
    assert lib.bs_attn_packed_chunk_fwd(ctypes.byref(d), FAKE, FAKE, FAKE, FAKE, FAKE, None, FAKE, 1,
                                        128, 1, 0.1, FAKE, FAKE, FAKE, 1 << 30, None) == B.BS_ERR_INVALID_ARG
    assert "q_pos" in B.bs_last_error()
    assert lib.bs_attn_packed_chunk_bwd(ctypes.byref(d), FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE,
                                        FAKE, FAKE, FAKE, 1, 128, 1, 0.1, None, FAKE, FAKE, 0, FAKE,
                                        1 << 30, None) == B.BS_ERR_INVALID_ARG
    assert "dq_accum" in B.bs_last_error()
    assert lib.bs_read_device_status(None, None) == B.BS_ERR_WORKSPACE
    assert lib.bs_copy_async(None, FAKE, 64, None) == B.BS_ERR_INVALID_ARG
    assert lib.bs_copy_async(FAKE, FAKE + 32, 64, None) == B.BS_ERR_INVALID_ARG
    assert "overlap" in B.bs_last_error()
    assert lib.bs_copy_async(None, None, 0, None) == B.BS_OK  # nothing to copy: nothing enqueued


def test_softmax_xent_rejects_bad_arguments(lib):
    def xent(rows=4, vocab=1000, dtype=B.BS_BF16, logits=FAKE, labels=FAKE, g=1.0, loss=FAKE,
             dlogits=None):
        return lib.bs_softmax_xent(rows, vocab, dtype, logits, labels, -100, g, loss, None,
                                   dlogits, None)

    assert xent(dtype=5) == B.BS_ERR_UNSUPPORTED
    assert xent(rows=-1) == B.BS_ERR_INVALID_ARG
    assert xent(rows=1 << 30) == B.BS_ERR_INVALID_ARG
    assert xent(vocab=0) == B.BS_ERR_INVALID_ARG
    assert xent(vocab=1 << 31) == B.BS_ERR_INVALID_ARG
    assert xent(g=float("inf")) == B.BS_ERR_INVALID_ARG
    assert xent(logits=None) == B.BS_ERR_INVALID_ARG
    assert xent(loss=None) == B.BS_ERR_INVALID_ARG
    assert xent(logits=FAKE + 1) == B.BS_ERR_INVALID_ARG  # bf16 needs 2-byte alignment
    assert "aligned" in B.bs_last_error()
    assert xent(labels=FAKE + 4) == B.BS_ERR_INVALID_ARG  # int64 labels need 8-byte alignment
    assert xent(loss=FAKE + 2) == B.BS_ERR_INVALID_ARG
    # a gradient buffer that overlaps the logits without being them
    assert xent(dlogits=FAKE + 64) == B.BS_ERR_INVALID_ARG
    assert "overlaps" in B.bs_last_error()
    assert xent(rows=0, logits=None, labels=None, loss=None) == B.BS_OK  # nothing to do


def test_running_merge_rejects_bad_state(lib):
    """The forward steps that fold into a running (O, LSE) need both running buffers; the
    optional final output must not overlap the running O."""
    d = dims()
    qn = 128 * 4 * 128  # total_q * hq * head_dim

    def chunk(o_run=FAKE, lse_run=FAKE, out=None, ws_bytes=1 << 30):
        return lib.bs_attn_chunk_fwd_merge(ctypes.byref(d), FAKE, FAKE, FAKE, 0, 0, 1, 0.1, o_run,
                                           lse_run, 1, out, FAKE, ws_bytes, None)

    assert chunk(o_run=None) == B.BS_ERR_INVALID_ARG
    assert "o_run is NULL" in B.bs_last_error()
    assert chunk(lse_run=None) == B.BS_ERR_INVALID_ARG
    assert "lse_run is NULL" in B.bs_last_error()
    assert chunk(o_run=FAKE + 8) == B.BS_ERR_INVALID_ARG
    assert "aligned" in B.bs_last_error()
    # bf16 out of qn * 2 bytes starting inside the float32 o_run, or o_run starting inside out
    assert chunk(o_run=1 << 20, out=(1 << 20) + qn * 4 - 16) == B.BS_ERR_INVALID_ARG
    assert "overlaps" in B.bs_last_error()
    assert chunk(o_run=(1 << 20) + qn * 2 - 16, out=1 << 20) == B.BS_ERR_INVALID_ARG
    # adjacent buffers pass that check and stop at the (too small) workspace, enqueueing nothing
    assert chunk(o_run=1 << 20, out=(1 << 20) + qn * 4, ws_bytes=16) == B.BS_ERR_WORKSPACE
    assert chunk(o_run=(1 << 20) + qn * 2, out=1 << 20, ws_bytes=16) == B.BS_ERR_WORKSPACE
    assert lib.bs_attn_packed_chunk_fwd_merge(ctypes.byref(d), FAKE, FAKE, FAKE, FAKE, FAKE, None,
                                              FAKE, 1, 128, 1, 0.1, FAKE, FAKE, 0, None, FAKE,
                                              1 << 30, None) == B.BS_ERR_INVALID_ARG
    assert "q_pos" in B.bs_last_error()
    assert lib.bs_attn_packed_chunk_fwd_merge(ctypes.byref(d), FAKE, FAKE, FAKE, FAKE, FAKE, FAKE,
                                              FAKE, 1, 128, 1, 0.1, None, FAKE, 0, None, FAKE,
                                              1 << 30, None) == B.BS_ERR_INVALID_ARG
    assert "o_run is NULL" in B.bs_last_error()


def test_workspace_size_grows_with_problem(lib):
    small = B.bs_attn_workspace_size(B.BS_OP_VARLEN_FWD, dims(), 1, 128)
    big = B.bs_attn_workspace_size(B.BS_OP_VARLEN_FWD, dims(total_q=4096, total_k=4096), 1, 4096)
    bwd = B.bs_attn_workspace_size(B.BS_OP_VARLEN_BWD, dims(total_q=4096, total_k=4096), 1, 4096)
    assert 0 < small < big < bwd
    # the backward holds D [hq, T]; the float32 varlen backward also a dQ accumulator [T, hq, d]
    assert bwd >= 4 * 4096 * 4
    f32 = B.bs_attn_workspace_size(B.BS_OP_VARLEN_BWD,
                                   dims(total_q=4096, total_k=4096, dtype=B.BS_F32), 1, 4096)
    assert f32 >= bwd + 4096 * 4 * 128 * 4
    assert lib.bs_attn_workspace_size(9, ctypes.byref(dims()), 1, 1) == 0
    # the packed chunk backward adds into the caller's dQ accumulator: no dQ buffer of its own
    pk = B.bs_attn_workspace_size(B.BS_OP_PACKED_CHUNK_BWD,
                                  dims(total_q=4096, total_k=4096, dtype=B.BS_F32), 1, 4096)
    assert bwd <= pk < f32


def test_noalloc_forward_rejects_sizes_beyond_its_scratch(lib):
    """The allocation-free forward checks the plan size against its fixed scratch array on the
    host and enqueues nothing: 2^28 bf16 query tokens need 2M work items of 48 B."""
    def call(d, n=1, cu=FAKE):
        return lib.bs_attn_varlen_fwd_noalloc(ctypes.byref(d), FAKE, FAKE, FAKE, cu, cu, n, 1 << 28,
                                              1, 0.1, FAKE, FAKE, None)
    assert call(dims(total_q=1 << 28, total_k=1 << 28)) == B.BS_ERR_WORKSPACE
    assert "allocation-free" in B.bs_last_error()
    assert call(dims(head_dim=96)) == B.BS_ERR_UNSUPPORTED
    assert call(dims(), cu=None) == B.BS_ERR_INVALID_ARG
    assert call(dims(), n=-1) == B.BS_ERR_INVALID_ARG
