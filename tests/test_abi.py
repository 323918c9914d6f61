"""The C-ABI library loads and exports every function include/duet.h declares; host-side
argument checks return the documented codes without touching a GPU."""
import ctypes
import os
import re

import pytest

from paper_2511_04791_amd import _native as N

HEADER = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "include", "duet.h")


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(duet_[a-z_0-9]+)\s*\(", text)))


def test_every_declared_symbol_is_exported(native):
    names = declared_functions()
    assert len(names) >= 20
    for name in names:
        assert hasattr(native, name), name
        assert name in N._SIGS, f"{name} missing from the Python binding"


def _shape(**kw):
    base = dict(num_q_heads=32, num_kv_heads=8, head_dim=128, page_size=16, dtype=N.BF16, num_layers=1)
    base.update(kw)
    return N.Shape(**base)


def _batch(rows):
    arr = (N.SeqMeta * len(rows))(*[N.SeqMeta(*r) for r in rows])
    return arr, N.Batch(arr, len(rows))


@pytest.mark.parametrize("kw,code", [(dict(head_dim=96), -2), (dict(page_size=32), -2), (dict(num_kv_heads=5), -2),
                                     (dict(dtype=7), -2), (dict(num_q_heads=0), -1), (dict(num_layers=0), -1)])
def test_shape_validation(native, kw, code):
    arr, b = _batch([(0, 0, 16, 0)])
    n = ctypes.c_size_t()
    assert native.duet_workspace_bytes(ctypes.byref(_shape(**kw)), ctypes.byref(b), ctypes.byref(n)) == code
    assert native.duet_last_error()


@pytest.mark.parametrize("row", [(1, 0, 2, 5), (0, 0, 0, 5), (0, 0, 4, -1), (3, 0, 1, 1)])
def test_batch_validation(native, row):
    arr, b = _batch([row])
    n = ctypes.c_size_t()
    assert native.duet_workspace_bytes(ctypes.byref(_shape()), ctypes.byref(b), ctypes.byref(n)) == -1


def test_split_validation(native):
    arr, b = _batch([(0, 0, 128, 0), (1, 128, 1, 100)])
    us = ctypes.c_double()
    for sp in [N.CuSplit(1, 100, 100, 1), N.CuSplit(1, 248, 16, 1), N.CuSplit(1, 128, 128, 0), N.CuSplit(5, 0, 0, 1),
               N.CuSplit(1, 0, 256, 1)]:
        assert native.duet_predict_iter_latency(None, ctypes.byref(_shape()), ctypes.byref(b), sp, ctypes.byref(us)) == -1
    assert native.duet_predict_iter_latency(None, ctypes.byref(_shape()), ctypes.byref(b), N.CuSplit(1, 128, 128, 1),
                                            ctypes.byref(us)) == 0


def test_attn_rejects_null_context(native):
    arr, b = _batch([(1, 0, 1, 10)])
    rc = native.duet_attn_mixed_batch(None, ctypes.byref(_shape()), 1, 1, 1, 10, 1, 4, ctypes.byref(b),
                                      N.CuSplit(0, 256, 0, 1), 1, 1 << 20, 1, None)
    assert rc == -1 and b"ctx" in native.duet_last_error()


def test_workspace_grows_with_decode_splits(native):
    small_arr, small = _batch([(1, 0, 1, 100)])
    big_arr, big = _batch([(1, 0, 1, 30000)])
    a, c = ctypes.c_size_t(), ctypes.c_size_t()
    assert native.duet_workspace_bytes(ctypes.byref(_shape()), ctypes.byref(small), ctypes.byref(a)) == 0
    assert native.duet_workspace_bytes(ctypes.byref(_shape()), ctypes.byref(big), ctypes.byref(c)) == 0
    # 30001 keys = 1876 pages = 59 splits of 32 pages (the library's fixed bf16 split length);
    # each split stores 4 heads x (128 + 2) floats per kv head
    assert c.value - a.value >= (59 - 1) * 8 * 4 * 130 * 4


def test_iteration_rejects_bad_layer_arguments(native):
    arr, b = _batch([(1, 0, 1, 10)])
    ptrs = (ctypes.c_void_p * 2)(1, 1)
    args = (1, 1, ctypes.byref(b), N.CuSplit(0, 256, 0, 1), 1, 1 << 20, ptrs, None)
    assert native.duet_attn_iteration(None, ctypes.byref(_shape(num_layers=2)), ptrs, ptrs, ptrs, 10, *args) == -1
    assert b"ctx" in native.duet_last_error()
    assert native.duet_attn_iteration(None, None, ptrs, ptrs, ptrs, 10, *args) == -1
    assert b"shape" in native.duet_last_error()
    assert native.duet_attn_iteration(None, ctypes.byref(_shape(num_layers=2)), None, ptrs, ptrs, 10, *args) == -1
    assert b"array" in native.duet_last_error()


def test_workspace_does_not_grow_with_layers(native):
    # the layers of a call share the decode queue counters (each reduce kernel clears them for the
    # next layer's partial kernel) and the split-K partials
    arr, b = _batch([(1, 0, 1, 100)])
    one, many = ctypes.c_size_t(), ctypes.c_size_t()
    assert native.duet_workspace_bytes(ctypes.byref(_shape(num_layers=1)), ctypes.byref(b), ctypes.byref(one)) == 0
    assert native.duet_workspace_bytes(ctypes.byref(_shape(num_layers=200)), ctypes.byref(b), ctypes.byref(many)) == 0
    assert many.value == one.value


def test_model_rejects_concurrent_control_mode(native):
    arr, b = _batch([(1, 0, 1, 10)])
    us = ctypes.c_double()
    assert native.duet_predict_iter_latency(None, ctypes.byref(_shape()), ctypes.byref(b), N.CuSplit(N.CONCURRENT, 256, 256, 1),
                                            ctypes.byref(us)) == -1


def test_lookahead_workspace_and_step_validation(native):
    arr, b = _batch([(0, 0, 100, 20), (1, 100, 1, 500), (1, 101, 1, 31)])
    one, four = ctypes.c_size_t(), ctypes.c_size_t()
    plain = ctypes.c_size_t()
    sh = ctypes.byref(_shape(num_layers=3))
    assert native.duet_workspace_bytes(sh, ctypes.byref(b), ctypes.byref(plain)) == 0
    assert native.duet_lookahead_workspace_bytes(sh, ctypes.byref(b), 1, ctypes.byref(one)) == 0
    assert native.duet_lookahead_workspace_bytes(sh, ctypes.byref(b), 4, ctypes.byref(four)) == 0
    assert one.value == plain.value
    # three more steps: three more copies of the metadata (3 rows of 16 bytes) and work lists
    assert four.value >= one.value + 3 * 3 * 16
    for k in (0, 65):
        assert native.duet_lookahead_workspace_bytes(sh, ctypes.byref(b), k, ctypes.byref(four)) == -1


def test_lookahead_rejects_null_context_and_bad_steps(native):
    arr, b = _batch([(1, 0, 1, 10)])
    ptrs = (ctypes.c_void_p * 1)(1)
    rc = native.duet_attn_lookahead(None, ctypes.byref(_shape()), ptrs, ptrs, ptrs, ptrs, ptrs, ptrs, 10, 1, 4,
                                    ctypes.byref(b), N.CuSplit(0, 256, 0, 2), 1, 1 << 20, ptrs, ptrs, None)
    assert rc == -1 and b"ctx" in native.duet_last_error()
    rc = native.duet_attn_lookahead(None, ctypes.byref(_shape()), ptrs, ptrs, ptrs, ptrs, ptrs, ptrs, 10, 1, 4,
                                    ctypes.byref(b), N.CuSplit(0, 256, 0, 0), 1, 1 << 20, ptrs, ptrs, None)
    assert rc == -1
    assert native.duet_set_decode_graphs(None, 1) == -1


def test_block_workspace_and_validation(native):
    arr, b = _batch([(0, 0, 100, 20), (1, 100, 1, 500)])
    attn, blk = ctypes.c_size_t(), ctypes.c_size_t()
    full = N.BlockShape(1024, 0, 3)
    assert native.duet_workspace_bytes(ctypes.byref(_shape()), ctypes.byref(b), ctypes.byref(attn)) == 0
    assert native.duet_block_workspace_bytes(ctypes.byref(_shape()), ctypes.byref(full), ctypes.byref(b), 1,
                                             ctypes.byref(blk)) == 0
    T, d, d_qkv, m = 101, 4096, 6144, 1024
    # the attention workspace, six activation buffers and two 32 MiB GEMM workspaces
    assert blk.value >= attn.value + T * 2 * (3 * d + d_qkv + 2 * m + m) + 2 * (32 << 20)
    for bad, code in ((N.BlockShape(1024, 0, 0), -2), (N.BlockShape(1020, 0, 3), -1), (N.BlockShape(0, 0, 3), -1)):
        assert native.duet_block_workspace_bytes(ctypes.byref(_shape()), ctypes.byref(bad), ctypes.byref(b), 1,
                                                 ctypes.byref(blk)) == code
    assert native.duet_block_workspace_bytes(ctypes.byref(_shape(dtype=N.F32, head_dim=64, num_q_heads=4,
                                                                 num_kv_heads=2)), ctypes.byref(full),
                                             ctypes.byref(b), 1, ctypes.byref(blk)) == -2
    assert native.duet_block_workspace_bytes(ctypes.byref(_shape()), ctypes.byref(full), ctypes.byref(b), 0,
                                             ctypes.byref(blk)) == -1


def test_block_forward_rejects_bad_arguments_before_any_launch(native):
    arr, b = _batch([(0, 0, 10, 0)])
    w = (N.BlockWeights * 1)(N.BlockWeights(1, 1, 1, 1, 1, 1))
    caches = (ctypes.c_void_p * 1)(16)
    # no context
    assert native.duet_block_forward(None, ctypes.byref(_shape()), ctypes.byref(N.BlockShape(1024, 0, 3)), w, 1e-5,
                                     32, None, caches, caches, 10, 64, 1, ctypes.byref(b), N.CuSplit(N.AGG, 256, 0, 1), 48,
                                     1 << 30, None) == -1
