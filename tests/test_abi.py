"""The C-ABI library loads and exports every entry point include/int2kv.h declares; host-side
argument validation rejects bad calls without touching a GPU (CPU only)."""
import ctypes
import os
import re

import pytest

from paper_2608_02691_amd import int2kv as K

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _declared():
    src = open(os.path.join(ROOT, "include", "int2kv.h")).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(int2kv_[a-z_]+)\s*\(", src)))


def test_header_declares_the_binding_names():
    assert _declared() == sorted(K.EXPORTED)


def test_library_exports_every_declared_symbol():
    lib = K.load_library()
    for name in _declared():
        assert hasattr(lib, name), name


def test_version_and_sizes():
    assert "gfx950" in K.int2kv_version()
    assert K.int2kv_pool_bytes(10, 8) == 10 * 8 * 1536
    assert K.int2kv_pool_bytes(10, 8, 32) == 10 * 8 * 1536
    assert K.int2kv_pool_bytes(10, 8, 128) == 10 * 8 * 1152
    assert K.int2kv_pool_bytes(10, 8, 64) == 0
    assert K.int2kv_pool_bytes(0, 8) == 0
    assert K.int2kv_decode_workspace_bytes(64, 40, 8, 32768, 5120) > 0
    assert K.int2kv_decode_workspace_bytes(2, 5, 2, 100, 0) == 0  # 5 % 2 != 0


def test_null_cache_and_bad_arguments_return_errors_without_launch():
    lib = K.load_library()
    st = lib.int2kv_decode(None, None, 1, 8, None, 1, None, 16, None, None, None, 0, 0, None, None, 0, None)
    assert st == K.INT2KV_EINVAL
    assert b"cache" in lib.int2kv_last_error()
    # a descriptor with an unsupported block size is refused before any pointer is used
    bad = K._Cache(16, 4, 2, 8, 128, 32)
    st = lib.int2kv_quantize_append(ctypes.byref(bad), None, None, None, 4, None, None, None, 1.0, 1.0, None)
    assert st == K.INT2KV_EUNSUPPORTED
    bad = K._Cache(16, 4, 2, 16, 128, 32)
    st = lib.int2kv_quantize_append(ctypes.byref(bad), None, None, None, 4, None, None, None, 1.0, 1.0, None)
    assert st == K.INT2KV_EINVAL  # NULL tensors
    st = lib.int2kv_quantize_pack_rotated(ctypes.byref(bad), 16, 16, 16, 1, 1.5, 1.0, None)
    assert st == K.INT2KV_EINVAL  # clip ratio out of range
    st = lib.int2kv_decode(ctypes.byref(bad), 16, 1, 3, 16, 1, 16, 16, 16, 16, None, 0, 0, 16, 256, 0, None)
    assert st == K.INT2KV_EINVAL  # 3 query heads over 2 KV heads
    st = lib.int2kv_decode(ctypes.byref(bad), 16, 1, 4, 16, 1, 16, 16, 16, 16, None, 0, 0, 16, 256, 0, None)
    assert st == K.INT2KV_EWORKSPACE
    assert lib.int2kv_set_decode_tuning(100, 0) == K.INT2KV_EINVAL
    assert lib.int2kv_set_decode_tuning(0, 7) == K.INT2KV_EINVAL
    assert lib.int2kv_set_decode_tuning(0, 0) == K.INT2KV_OK


def test_prepared_wo_sizes_and_argument_errors():
    lib = K.load_library()
    # rows padded to a multiple of 128, fp16
    assert K.int2kv_prepared_wo_bytes(5120, 40) == 5120 * 5120 * 2
    assert K.int2kv_prepared_wo_bytes(200, 2) == 256 * 256 * 2
    assert K.int2kv_prepared_wo_bytes(0, 2) == 0
    assert lib.int2kv_prepare_wo(None, None, 4096, 128, 1, 1, None) == K.INT2KV_EINVAL  # NULL W_o
    assert lib.int2kv_prepare_wo(4096, None, 1 << 20, 128, 3, 2, None) == K.INT2KV_EINVAL  # 3 % 2
    assert lib.int2kv_prepare_wo(4096, None, 4104, 128, 1, 1, None) == K.INT2KV_EINVAL  # misaligned output
    assert b"aligned" in lib.int2kv_last_error()
    assert lib.int2kv_prepare_wo(4096, None, 4096 + 1024, 128, 1, 1, None) == K.INT2KV_EINVAL  # overlap
    assert b"overlap" in lib.int2kv_last_error()


def test_decode_rejects_unknown_weight_format_without_launch():
    lib = K.load_library()
    good = K._Cache(16, 4, 2, 16, 128, 32)
    st = lib.int2kv_decode(ctypes.byref(good), 16, 1, 4, 16, 1, 16, 16, 16, 16, 16, 256, 4, 16, 256, 1 << 30, None)
    assert st == K.INT2KV_EINVAL
    assert b"wo_format" in lib.int2kv_last_error()


def test_record_bytes_and_group_sizes():
    assert K.int2kv_record_bytes(32) == 1536 == K.RECORD_BYTES_BY_GROUP[32]
    assert K.int2kv_record_bytes(128) == 1152 == K.RECORD_BYTES_BY_GROUP[128]
    assert K.int2kv_record_bytes(64) == 0
    lib = K.load_library()
    bad = K._Cache(16, 4, 2, 16, 128, 64)
    st = lib.int2kv_quantize_append(ctypes.byref(bad), None, None, None, 4, None, None, None, 1.0, 1.0, None)
    assert st == K.INT2KV_EUNSUPPORTED and b"group_size" in lib.int2kv_last_error()


def test_append_decode_rejects_bad_arguments_without_launch():
    lib = K.load_library()
    good = K._Cache(16, 4, 2, 16, 128, 32)
    # tokens given but no key rows
    st = lib.int2kv_append_decode(ctypes.byref(good), None, 16, 16, 4, 16, 1.0, 1.0, 16, 1, 4, 16, 1, 16, 16,
                                  16, 16, None, 0, 0, 16, 256, 1 << 30, None)
    assert st == K.INT2KV_EINVAL and b"NULL" in lib.int2kv_last_error()
    # clip ratio out of range
    st = lib.int2kv_append_decode(ctypes.byref(good), 16, 16, 16, 4, 16, 1.5, 1.0, 16, 1, 4, 16, 1, 16, 16,
                                  16, 16, None, 0, 0, 16, 256, 1 << 30, None)
    assert st == K.INT2KV_EINVAL and b"clip" in lib.int2kv_last_error()
    # negative token count
    st = lib.int2kv_append_decode(ctypes.byref(good), 16, 16, 16, -1, 16, 1.0, 1.0, 16, 1, 4, 16, 1, 16, 16,
                                  16, 16, None, 0, 0, 16, 256, 1 << 30, None)
    assert st == K.INT2KV_EINVAL
    # decode arguments are checked too: a workspace that is too small
    st = lib.int2kv_append_decode(ctypes.byref(good), 16, 16, 16, 4, 16, 1.0, 1.0, 16, 1, 4, 16, 1, 16, 16,
                                  16, 16, None, 0, 0, 16, 256, 16, None)
    assert st == K.INT2KV_EWORKSPACE


def test_tuning_knobs_are_per_thread():
    """int2kv_set_decode_tuning on one thread does not change another thread's workspace plan."""
    import threading
    lib = K.load_library()
    assert lib.int2kv_set_decode_tuning(0, 0) == K.INT2KV_OK
    base = lib.int2kv_decode_workspace_bytes(4, 8, 2, 4096, 0)
    seen = {}

    def other():
        assert lib.int2kv_set_decode_tuning(64, 1) == K.INT2KV_OK  # vector-ALU scan, 64-token chunks
        seen["other"] = lib.int2kv_decode_workspace_bytes(4, 8, 2, 4096, 0)

    t = threading.Thread(target=other)
    t.start()
    t.join()
    assert seen["other"] != base
    assert lib.int2kv_decode_workspace_bytes(4, 8, 2, 4096, 0) == base


def test_noalloc_rejects_workspace_beyond_the_static_scratch_without_launch():
    """A decode whose workspace exceeds the 64 MiB static scratch is refused before any HIP call."""
    lib = K.load_library()
    cache = K._Cache(16, 1 << 20, 8, 16, 128, 32)  # pool pointer never dereferenced
    st = lib.int2kv_append_decode_noalloc(ctypes.byref(cache), None, None, None, 0, None, 1.0, 1.0, 16, 4096, 40,
                                          16, 1, 16, 1 << 20, 16, 16, None, 0, 0, 16, None)
    assert st == K.INT2KV_EWORKSPACE
    assert b"static scratch" in lib.int2kv_last_error()


def test_rope_write_rejects_bad_arguments_without_launch():
    """int2kv_quantize_append_rope validates flags, rotations and the RoPE table on the host."""
    lib = K.load_library()
    cache = K._Cache(16, 1 << 20, 8, 16, 128, 32)  # pool pointer never dereferenced
    p = 1 << 20  # aligned stand-in pointers, never dereferenced on a rejected call

    def call(R_k, R_v, positions, cos_sin, max_pos, flags, k_out=None):
        return lib.int2kv_quantize_append_rope(ctypes.byref(cache), p, p, p, positions, 4, cos_sin, max_pos, R_k, R_v,
                                               p, 1.0, 1.0, flags, k_out, None)

    assert call(p, p, None, None, 0, 4) == K.INT2KV_EINVAL                      # unknown flag
    assert b"flags" in lib.int2kv_last_error()
    assert call(None, p, None, None, 0, 0) == K.INT2KV_EINVAL                   # R_K missing, no flag
    assert call(p, None, None, None, 0, K.INT2KV_HADAMARD_K) == K.INT2KV_EINVAL  # R_V missing
    assert call(p, p, p, None, 16, 0) == K.INT2KV_EINVAL                        # positions without table
    assert call(p, p, p, p, 0, 0) == K.INT2KV_EINVAL                            # empty table
    assert call(p, p, None, None, 0, 0, k_out=p) == K.INT2KV_EINVAL             # k_rope_out without RoPE
    assert call(p, p, p, p + 4, 16, 0) == K.INT2KV_EINVAL                       # misaligned table


def test_optr_workspace_query_validates_on_the_host():
    """int2kv_optr_workspace_bytes reads only the host tables: 0 for bad settings or sequences,
    a positive size otherwise (the device pointers are stand-ins, never dereferenced)."""
    import numpy as np
    lib = K.load_library()
    starts = np.array([0, 100, 250], np.int32)
    tr = K._OptrTraces(1 << 20, 1 << 20, 1 << 20, starts.ctypes.data_as(ctypes.POINTER(ctypes.c_int32)), 2)
    cfg = K.optr_config(2, 8, 64)
    assert lib.int2kv_optr_workspace_bytes(ctypes.byref(cfg), ctypes.byref(tr), None) > 0
    assert lib.int2kv_optr_workspace_bytes(ctypes.byref(cfg), ctypes.byref(tr), ctypes.byref(tr)) > \
        lib.int2kv_optr_workspace_bytes(ctypes.byref(cfg), ctypes.byref(tr), None)
    for bad in (K.optr_config(2, 7, 64), K.optr_config(2, 8, 64, group_size=64), K.optr_config(2, 8, 64, clip_k=0.0),
                K.optr_config(2, 8, 64, n_last=0), K.optr_config(2, 8, 64, eval_every=0),
                K.optr_config(2, 8, 64, lr=0.0)):
        assert lib.int2kv_optr_workspace_bytes(ctypes.byref(bad), ctypes.byref(tr), None) == 0
    long_starts = np.array([0, 5000], np.int32)  # a sequence beyond 4096 tokens
    tr2 = K._OptrTraces(1 << 20, 1 << 20, 1 << 20, long_starts.ctypes.data_as(ctypes.POINTER(ctypes.c_int32)), 1)
    assert lib.int2kv_optr_workspace_bytes(ctypes.byref(cfg), ctypes.byref(tr2), None) == 0
    assert b"4096" in lib.int2kv_last_error()
