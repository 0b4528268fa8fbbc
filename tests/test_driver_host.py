"""Host-side checks of the decode-then-GEMM driver's C ABI: workspace sizing
and argument validation.  Every call here is rejected before anything is
enqueued, so no device is touched (the pointers are never dereferenced)."""
import ctypes

import numpy as np
import pytest

from paper_2504_11651_amd import codec, synth

def llama_mats():
    mats, off = [], 0
    for _, r, c in synth.LLAMA3_8B_BLOCK:
        mats.append((off, r, c))
        off += r * c
    return mats, off


def test_workspace_closed_form():
    # up to 8 tokens every matrix is split into k ranges of 1024 columns
    # (4 for the 4096-column matrices, 14 for down); partial sums of rows x
    # ranges x tokens floats
    mats, _ = llama_mats()
    few = 4 * (4096 + 1024 + 1024 + 4096 + 14336 + 14336) + 14 * 4096
    for t in (1, 7, 8):
        assert codec.gemm_workspace_bytes(mats, t) == 4 * few * t
    # from 9 tokens the base ranges are 4096 columns (1 per 4096-column
    # matrix, 4 for down) and a device may double any matrix's ranges to
    # balance its CUs: the workspace covers the doubled split of every matrix
    many = 2 * (4096 + 1024 + 1024 + 4096 + 14336 + 14336) + 8 * 4096
    for t in (9, 16, 33, 64):
        assert codec.gemm_workspace_bytes(mats, t) == 4 * many * t
    assert codec.gemm_workspace_bytes([(0, 16, 1024)], 5) == 0
    assert codec.gemm_workspace_bytes([(0, 16, 256)], 40) == 0
    assert codec.gemm_workspace_bytes([(0, 16, 4096)], 40) == 4 * 16 * 2 * 40
    assert codec.gemm_workspace_bytes([(0, 16, 4096)], 5) == 4 * 16 * 4 * 5
    # 8192 columns -> 8 ranges (few tokens) or up to 4; 28672 -> 28 or up to 14
    assert codec.gemm_workspace_bytes([(0, 32, 8192)], 3) == 4 * 32 * 8 * 3
    assert codec.gemm_workspace_bytes([(0, 32, 8192)], 40) == 4 * 32 * 4 * 40
    assert codec.gemm_workspace_bytes([(0, 32, 28672)], 2) == 4 * 32 * 28 * 2
    assert codec.gemm_workspace_bytes([(0, 32, 28672)], 64) == 4 * 32 * 14 * 64


@pytest.mark.parametrize("mats,tokens,rc", [
    ([(0, 16, 64)], 0, -6),        # no tokens
    ([(0, 16, 64)], 65, -6),       # more than 64 tokens
    ([(0, 15, 64)], 1, -6),        # rows not a multiple of 16
    ([(0, 16, 96)], 1, -6),        # cols not a multiple of 64
    ([(4, 16, 64)], 1, -6),        # offset not 16-byte aligned
    ([(0, 0, 64)], 1, -1),         # empty matrix
    ([], 1, -1),                   # no matrices
    ([(0, 16, 64)] * 9, 1, -1),    # more than 8 matrices
])
def test_shape_rejections(mats, tokens, rc):
    L = codec.lib()
    m = codec._mats(mats) if mats else None
    out = ctypes.c_uint64()
    assert L.df11_gemm_workspace_bytes(m, len(mats), tokens, ctypes.byref(out)) == rc


def _call_gemm(weights, n_weights, mats, xs, ys, tokens, ws, ws_bytes):
    L = codec.lib()
    m = codec._mats(mats)
    xp = (ctypes.c_void_p * len(xs))(*xs)
    yp = (ctypes.c_void_p * len(ys))(*ys)
    return L.df11_block_gemm(ctypes.c_void_p(weights), n_weights, m, len(mats), xp, tokens, yp,
                             ctypes.c_void_p(ws), ws_bytes, ctypes.c_void_p(0))


A = 1 << 20  # a 16-byte aligned stand-in address (never dereferenced)


def test_argument_rejections():
    mats = [(0, 16, 64)]
    assert _call_gemm(0, 1024, mats, [A], [A], 1, 0, 0) == -1           # null weights
    assert _call_gemm(A + 2, 1024, mats, [A], [A], 1, 0, 0) == -1       # misaligned weights
    assert _call_gemm(A, 1023, mats, [A], [A], 1, 0, 0) == -1           # matrix past the block
    assert _call_gemm(A, 1024, mats, [A + 8], [A], 1, 0, 0) == -1       # misaligned x
    assert _call_gemm(A, 1024, mats, [A], [A + 2], 1, 0, 0) == -1       # misaligned y
    assert _call_gemm(A, 1024, mats, [0], [A], 1, 0, 0) == -1           # null x
    # with many tokens too (the per-device choice of k ranges comes after
    # every argument check)
    assert _call_gemm(A, 1023, mats, [A], [A], 64, 0, 0) == -1          # matrix past the block
    assert _call_gemm(A, 1024, mats, [A + 8], [A], 64, 0, 0) == -1      # misaligned x
    assert _call_gemm(A, 1024, mats, [A], [0], 64, 0, 0) == -1          # null y
    # a split matrix needs a workspace
    big = [(0, 16, 8192)]
    need = codec.gemm_workspace_bytes(big, 2)
    assert _call_gemm(A, 16 * 8192, big, [A], [A], 2, A, need - 4) == -3
    assert _call_gemm(A, 16 * 8192, big, [A], [A], 2, 0, need) == -1    # null workspace
    assert _call_gemm(A, 16 * 8192, big, [A], [A], 2, A + 4, need) == -1


def test_block_forward_checks_gemm_arguments_before_decoding():
    # an invalid matrix list is rejected before the decode is enqueued
    L = codec.lib()
    st = codec.Stream()
    st.sizes.n_elems = 1024
    st.layout.bytes_per_thread, st.layout.threads_per_block, st.layout.lut_bits = 8, 64, 11
    m = codec._mats([(0, 16, 64)])
    xp = (ctypes.c_void_p * 1)(A)
    yp = (ctypes.c_void_p * 1)(A)
    rc = L.df11_block_forward(ctypes.byref(st), ctypes.c_void_p(A), m, 1, xp, 65, yp,
                              ctypes.c_void_p(0), 0, ctypes.c_void_p(0))
    assert rc == -6
    rc = L.df11_block_forward(ctypes.byref(st), ctypes.c_void_p(A + 2), m, 1, xp, 1, yp,
                              ctypes.c_void_p(0), 0, ctypes.c_void_p(0))
    assert rc == -1
    assert L.df11_block_forward(None, ctypes.c_void_p(A), m, 1, xp, 1, yp, ctypes.c_void_p(0), 0,
                                ctypes.c_void_p(0)) == -1


# ---- fused decode-and-multiply: argument checks (rejected before launch)
def _stream_desc(n=1 << 20, T=64):
    st = codec.Stream()
    st.sizes.n_elems = n
    st.sizes.num_blocks = 4
    st.layout.bytes_per_thread, st.layout.threads_per_block, st.layout.lut_bits = 8, T, 11
    return st


def _call_gemv(st, mats, xs, ys, ws, ws_bytes):
    L = codec.lib()
    m = codec._mats(mats)
    xp = (ctypes.c_void_p * len(xs))(*xs)
    yp = (ctypes.c_void_p * len(ys))(*ys)
    return L.df11_block_gemv(ctypes.byref(st), m, len(mats), xp, yp, ctypes.c_void_p(ws),
                             ws_bytes, ctypes.c_void_p(0))


@pytest.mark.parametrize("mats,rc", [
    ([(0, 16, 1024)], -6),                  # fewer than 2048 columns
    ([(0, 4, 2048 + 32)], -6),              # columns not a multiple of 64
    ([(8, 1, 2048)], -6),                   # fewer than 4096 weights
    ([(4, 16, 2048)], -6),                  # offset not 16-byte aligned
    ([(65536, 16, 2048), (0, 16, 2048)], -6),  # not sorted by offset
    ([(0, 16, 2048), (16 * 2048 - 8, 16, 2048)], -6),  # overlapping
    ([(0, 1024, 2048)], -1),                # past the end of the stream
])
def test_gemv_shape_rejections(mats, rc):
    st = _stream_desc()
    # null stream buffers make check_stream fail first for a non-empty
    # stream, so give them stand-in addresses (never dereferenced)
    _fill_valid_sizes(st)
    n = len(mats)
    assert _call_gemv(st, mats, [A] * n, [A] * n, A, 1 << 20) == rc


def _fill_valid_sizes(st):
    """Stand-in addresses and sizes consistent with the layout, so that the
    stream descriptor itself passes the decoder's checks."""
    T, B, n = int(st.layout.threads_per_block), int(st.sizes.num_blocks), int(st.sizes.n_elems)
    st.exp = st.sm = st.gaps = st.tables = A
    st.block_pos = A
    st.sizes.max_code_len = 20
    st.sizes.num_chunks = B * T
    st.sizes.exp_bytes = B * 8 * T + 16
    st.sizes.gap_bytes = 4 * ((5 * (B * T + 1) + 31) // 32 + 2)
    st.sizes.sm_bytes = ((n + 15) & ~15) + 16
    st.sizes.max_elems_per_block = 4096
    st.sizes.table_bytes = codec.lib() and _table_bytes(int(st.layout.lut_bits))


def _table_bytes(K):
    cb = codec.codebook_from_counts(np.array([1, 1] + [0] * 254, np.uint64))
    return codec.build_tables(cb, K).size


def test_gemv_rejects_other_layouts_and_bad_buffers():
    mats = [(0, 16, 2048)]
    st = _stream_desc(T=256)
    _fill_valid_sizes(st)
    assert _call_gemv(st, mats, [A], [A], A, 1 << 20) == -6      # needs T = 64
    st = _stream_desc()
    _fill_valid_sizes(st)
    assert _call_gemv(st, mats, [A + 8], [A], A, 1 << 20) == -1  # misaligned x
    assert _call_gemv(st, mats, [A], [A + 2], A, 1 << 20) == -1  # misaligned y
    assert _call_gemv(st, mats, [0], [A], A, 1 << 20) == -1      # null x
    need = 4 * 8 * 4 + 8 * 16  # 8 floats per block (4 blocks), two indices per row (16 rows)
    assert _call_gemv(st, mats, [A], [A], A, need - 4) == -3     # short workspace
    assert _call_gemv(st, mats, [A], [A], 0, need) == -1         # null workspace
    out = ctypes.c_uint64()
    assert codec.lib().df11_gemv_workspace_bytes(ctypes.byref(st), codec._mats(mats), 1,
                                                 ctypes.byref(out)) == 0
    assert out.value == need


def test_binding_refuses_host_tensors():
    # the library dereferences every pointer on the GPU; the binding refuses
    # host tensors before calling it
    import torch
    w = np.zeros(4096, np.uint16)
    hs = codec.encode(w)
    with pytest.raises(ValueError):
        codec.to_device(hs, "cpu")
    weights = torch.zeros(1024, dtype=torch.bfloat16)
    x = torch.zeros((1, 64), dtype=torch.bfloat16)
    y = torch.zeros((1, 16), dtype=torch.float32)
    with pytest.raises(ValueError):
        codec.block_gemm(weights, [(0, 16, 64)], [x], [y])
    with pytest.raises(ValueError):
        codec.block_gemm(weights, [], [], [])
