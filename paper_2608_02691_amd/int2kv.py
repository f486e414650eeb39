"""Thin Python binding of libint2kv (ctypes). Argument marshalling only.

Every function has the name of the C entry point it calls (include/int2kv.h). Tensors must be
torch tensors already on the GPU; work is enqueued on torch's current stream. bf16 tensors may
be passed as torch.bfloat16 or as int16/uint16 bit patterns. There is no CPU fallback: if the
HIP library is missing, importing any entry point raises.
"""
from __future__ import annotations

import ctypes
import math
import os
from typing import Optional

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libint2kv.so")

HEAD_DIM = 128
BLOCK_SIZE = 16
GROUP_SIZE = 32
RECORD_BYTES = 1536
RECORD_BYTES_BY_GROUP = {32: 1536, 128: 1152}

INT2KV_OK = 0
INT2KV_EINVAL = -1
INT2KV_EUNSUPPORTED = -2
INT2KV_EWORKSPACE = -3
INT2KV_EHIP = -4

INT2KV_WO_PLAIN = 0
INT2KV_WO_FOLDED = 1
INT2KV_WO_PREPARED = 2
INT2KV_WO_PREPARED_FOLDED = 3

EXPORTED = (
    "int2kv_last_error", "int2kv_version", "int2kv_pool_bytes", "int2kv_record_bytes", "int2kv_prepare_mu_rot",
    "int2kv_fold_wo",
    "int2kv_prepared_wo_bytes", "int2kv_prepare_wo",
    "int2kv_quantize_pack_rotated", "int2kv_quantize_append", "int2kv_decode_workspace_bytes",
    "int2kv_decode", "int2kv_append_decode", "int2kv_append_decode_noalloc", "int2kv_window_write",
    "int2kv_decode_window",
    "int2kv_set_decode_tuning", "int2kv_set_decode_events", "int2kv_quantize_append_error",
    "int2kv_output_error_workspace_bytes", "int2kv_output_error", "int2kv_quantize_append_rope",
    "int2kv_optr_workspace_bytes", "int2kv_optr_key_mean", "int2kv_optr_key_loss", "int2kv_optr_value_loss",
    "int2kv_optr_calibrate",
)


class _Cache(ctypes.Structure):
    _fields_ = [("pool", ctypes.c_void_p), ("num_blocks", ctypes.c_int32), ("num_kv_heads", ctypes.c_int32),
                ("block_size", ctypes.c_int32), ("head_dim", ctypes.c_int32), ("group_size", ctypes.c_int32)]


class _OptrTraces(ctypes.Structure):
    _fields_ = [("k", ctypes.c_void_p), ("v", ctypes.c_void_p), ("q", ctypes.c_void_p),
                ("seq_starts", ctypes.POINTER(ctypes.c_int32)), ("num_seqs", ctypes.c_int32)]


class _OptrConfig(ctypes.Structure):
    _fields_ = [("num_kv_heads", ctypes.c_int32), ("num_q_heads", ctypes.c_int32), ("d_model", ctypes.c_int32),
                ("group_size", ctypes.c_int32), ("clip_k", ctypes.c_float), ("clip_v", ctypes.c_float),
                ("lambda_k", ctypes.c_double), ("n_last", ctypes.c_int32), ("sink", ctypes.c_int32),
                ("recent", ctypes.c_int32), ("steps", ctypes.c_int32), ("eval_every", ctypes.c_int32),
                ("lr", ctypes.c_double)]


_lib = None


def load_library(path: str = LIB_PATH):
    """Load the HIP library (raises if it has not been built)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise RuntimeError(f"{path} is missing: build it with __graft_entry__.build() "
                           "(there is no CPU fallback)")
    lib = ctypes.CDLL(path)
    P, I, F, S, Z = ctypes.c_void_p, ctypes.c_int, ctypes.c_float, ctypes.c_void_p, ctypes.c_size_t
    sig = {
        "int2kv_last_error": ([], ctypes.c_char_p),
        "int2kv_version": ([], ctypes.c_char_p),
        "int2kv_pool_bytes": ([I, I, I], Z),
        "int2kv_record_bytes": ([I], Z),
        "int2kv_prepare_mu_rot": ([P, P, P, I, S], I),
        "int2kv_fold_wo": ([P, P, P, I, I, I, S], I),
        "int2kv_prepared_wo_bytes": ([I, I], Z),
        "int2kv_prepare_wo": ([P, P, P, I, I, I, S], I),
        "int2kv_quantize_pack_rotated": ([ctypes.POINTER(_Cache), P, P, P, I, F, F, S], I),
        "int2kv_quantize_append": ([ctypes.POINTER(_Cache), P, P, P, I, P, P, P, F, F, S], I),
        "int2kv_decode_workspace_bytes": ([I, I, I, I, I], Z),
        "int2kv_decode": ([ctypes.POINTER(_Cache), P, I, I, P, I, P, I, P, P, P, I, I, P, P, Z, S], I),
        "int2kv_append_decode": ([ctypes.POINTER(_Cache), P, P, P, I, P, F, F, P, I, I, P, I, P, I, P, P, P, I, I, P,
                                  P, Z, S], I),
        "int2kv_append_decode_noalloc": ([ctypes.POINTER(_Cache), P, P, P, I, P, F, F, P, I, I, P, I, P, I, P, P, P,
                                          I, I, P, S], I),
        "int2kv_window_write": ([P, P, P, I, I, P, P, P, I, S], I),
        "int2kv_decode_window": ([ctypes.POINTER(_Cache), P, I, I, P, I, P, I, P, P, P, I, I, P, P, P, I, P, P, Z,
                                  S], I),
        "int2kv_set_decode_tuning": ([I, I], I),
        "int2kv_quantize_append_error": ([ctypes.POINTER(_Cache), P, P, P, I, P, P, P, F, F, P, S], I),
        "int2kv_output_error_workspace_bytes": ([I, I, I, I, I], Z),
        "int2kv_optr_workspace_bytes": ([ctypes.POINTER(_OptrConfig), ctypes.POINTER(_OptrTraces),
                                         ctypes.POINTER(_OptrTraces)], Z),
        "int2kv_optr_key_mean": ([P, I, I, P, S], I),
        "int2kv_optr_key_loss": ([ctypes.POINTER(_OptrConfig), ctypes.POINTER(_OptrTraces), P, P, P, P, P, P, P, Z, S],
                                 I),
        "int2kv_optr_value_loss": ([ctypes.POINTER(_OptrConfig), ctypes.POINTER(_OptrTraces), P, P, P, P, P, P, P, P,
                                    P, Z, S], I),
        "int2kv_optr_calibrate": ([ctypes.POINTER(_OptrConfig), ctypes.POINTER(_OptrTraces),
                                   ctypes.POINTER(_OptrTraces), P, P, P, P, P, P, P, P, P, P, Z, S], I),
        "int2kv_quantize_append_rope": ([ctypes.POINTER(_Cache), P, P, P, P, I, P, I, P, P, P, F, F, I, P, S], I),
        "int2kv_output_error": ([ctypes.POINTER(_Cache), P, I, I, P, I, P, I, P, P, P, P, I, P, I, P, P, P, Z, S],
                                I),
        "int2kv_set_decode_events": ([P, P], I),
    }
    for name, (args, res) in sig.items():
        fn = getattr(lib, name)
        fn.argtypes = args
        fn.restype = res
    _lib = lib
    return lib


def _check(status: int, name: str) -> None:
    if status != INT2KV_OK:
        msg = load_library().int2kv_last_error().decode()
        raise RuntimeError(f"{name} failed with status {status}: {msg}")


def _stream() -> int:
    return torch.cuda.current_stream().cuda_stream


def _ptr(t: Optional[torch.Tensor], dtypes, name: str):
    if t is None:
        return None
    if not isinstance(t, torch.Tensor) or not t.is_cuda:
        raise TypeError(f"{name} must be a CUDA (HIP) tensor")
    if t.dtype not in dtypes:
        raise TypeError(f"{name} has dtype {t.dtype}, expected one of {dtypes}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    return t.data_ptr()


_BF16 = (torch.bfloat16, torch.int16, torch.uint16)
_F32 = (torch.float32,)
_I32 = (torch.int32,)


class Int2KVCache:
    """The paged INT2 pool (uint8 [num_blocks, num_kv_heads, record bytes]) and its C descriptor;
    group_size 32 (1536-byte records) or 128 (1152-byte records)."""

    def __init__(self, num_blocks: int, num_kv_heads: int, device="cuda", pool: Optional[torch.Tensor] = None,
                 group_size: int = GROUP_SIZE):
        rec = RECORD_BYTES_BY_GROUP.get(group_size)
        if rec is None:
            raise ValueError("group_size must be 32 or 128")
        if pool is None:
            pool = torch.zeros((num_blocks, num_kv_heads, rec), dtype=torch.uint8, device=device)
        if pool.shape != (num_blocks, num_kv_heads, rec) or pool.dtype != torch.uint8:
            raise ValueError(f"pool must be uint8 [num_blocks, num_kv_heads, {rec}]")
        self.pool = pool
        self.num_blocks = num_blocks
        self.num_kv_heads = num_kv_heads
        self.group_size = group_size
        self._desc = _Cache(pool.data_ptr(), num_blocks, num_kv_heads, BLOCK_SIZE, HEAD_DIM, group_size)

    @property
    def desc(self):
        return ctypes.byref(self._desc)


def int2kv_record_bytes(group_size: int) -> int:
    return load_library().int2kv_record_bytes(group_size)


def int2kv_version() -> str:
    return load_library().int2kv_version().decode()


def int2kv_pool_bytes(num_blocks: int, num_kv_heads: int, group_size: int = GROUP_SIZE) -> int:
    return load_library().int2kv_pool_bytes(num_blocks, num_kv_heads, group_size)


def int2kv_prepare_mu_rot(R_k: torch.Tensor, mu: torch.Tensor, mu_rk: Optional[torch.Tensor] = None) -> torch.Tensor:
    H = R_k.shape[0]
    if mu_rk is None:
        mu_rk = torch.empty((H, HEAD_DIM), dtype=torch.float32, device=R_k.device)
    st = load_library().int2kv_prepare_mu_rot(_ptr(R_k, _F32, "R_k"), _ptr(mu, _F32, "mu"),
                                              _ptr(mu_rk, _F32, "mu_rk"), H, _stream())
    _check(st, "int2kv_prepare_mu_rot")
    return mu_rk


def int2kv_fold_wo(W_o: torch.Tensor, R_v: torch.Tensor, num_q_heads: int,
                   out: Optional[torch.Tensor] = None) -> torch.Tensor:
    d_model = W_o.shape[0]
    if out is None:
        out = torch.empty_like(W_o)
    st = load_library().int2kv_fold_wo(_ptr(W_o, _BF16, "W_o"), _ptr(R_v, _F32, "R_v"), _ptr(out, _BF16, "out"),
                                       d_model, num_q_heads, R_v.shape[0], _stream())
    _check(st, "int2kv_fold_wo")
    return out


def int2kv_prepared_wo_bytes(d_model: int, num_q_heads: int) -> int:
    return load_library().int2kv_prepared_wo_bytes(d_model, num_q_heads)


def int2kv_prepare_wo(W_o: torch.Tensor, R_v: Optional[torch.Tensor], num_q_heads: int,
                      num_kv_heads: Optional[int] = None, out: Optional[torch.Tensor] = None) -> torch.Tensor:
    """Prepared (fp16, tiled) output-projection weights; R_v folds the value rotation in (None: no
    fold, then num_kv_heads must be given). Returns a flat float16 tensor."""
    d_model = W_o.shape[0]
    H = R_v.shape[0] if R_v is not None else num_kv_heads
    if H is None:
        raise ValueError("num_kv_heads is required without R_v")
    n = int2kv_prepared_wo_bytes(d_model, num_q_heads) // 2
    if out is None:
        out = torch.empty(n, dtype=torch.float16, device=W_o.device)
    if out.numel() < n:
        raise ValueError("out is smaller than int2kv_prepared_wo_bytes()")
    st = load_library().int2kv_prepare_wo(_ptr(W_o, _BF16, "W_o"), _ptr(R_v, _F32, "R_v"),
                                          _ptr(out, (torch.float16, torch.int16, torch.uint16), "out"), d_model,
                                          num_q_heads, H, _stream())
    _check(st, "int2kv_prepare_wo")
    return out


def int2kv_quantize_pack_rotated(cache: Int2KVCache, k_rot: torch.Tensor, v_rot: torch.Tensor,
                                 slot_mapping: torch.Tensor, clip_k: float = 1.0, clip_v: float = 1.0) -> None:
    n = slot_mapping.shape[0]
    if k_rot.numel() != n * cache.num_kv_heads * HEAD_DIM or v_rot.numel() != k_rot.numel():
        raise ValueError("k_rot / v_rot must be [n, num_kv_heads, 128]")
    st = load_library().int2kv_quantize_pack_rotated(cache.desc, _ptr(k_rot, _F32, "k_rot"), _ptr(v_rot, _F32, "v_rot"),
                                                     _ptr(slot_mapping, _I32, "slot_mapping"), n, clip_k, clip_v,
                                                     _stream())
    _check(st, "int2kv_quantize_pack_rotated")


def int2kv_quantize_append(cache: Int2KVCache, k: torch.Tensor, v: torch.Tensor, slot_mapping: torch.Tensor,
                           R_k: torch.Tensor, R_v: torch.Tensor, mu_rk: torch.Tensor, clip_k: float = 1.0,
                           clip_v: float = 1.0) -> None:
    n = slot_mapping.shape[0]
    if k.numel() != n * cache.num_kv_heads * HEAD_DIM or v.numel() != k.numel():
        raise ValueError("k / v must be [n, num_kv_heads, 128]")
    st = load_library().int2kv_quantize_append(cache.desc, _ptr(k, _BF16, "k"), _ptr(v, _BF16, "v"),
                                               _ptr(slot_mapping, _I32, "slot_mapping"), n, _ptr(R_k, _F32, "R_k"),
                                               _ptr(R_v, _F32, "R_v"), _ptr(mu_rk, _F32, "mu_rk"), clip_k, clip_v,
                                               _stream())
    _check(st, "int2kv_quantize_append")


def int2kv_decode_workspace_bytes(batch: int, num_q_heads: int, num_kv_heads: int, max_ctx: int,
                                  d_model: int = 0) -> int:
    return load_library().int2kv_decode_workspace_bytes(batch, num_q_heads, num_kv_heads, max_ctx, d_model)


def int2kv_set_decode_tuning(chunk_tokens: int = 0, variant: int = 0) -> None:
    _check(load_library().int2kv_set_decode_tuning(chunk_tokens, variant), "int2kv_set_decode_tuning")


def int2kv_set_decode_events(before_scan: Optional[int], after_scan: Optional[int]) -> None:
    """Record two raw hipEvent_t handles around the split-context scan kernel of later decodes
    (None, None disables)."""
    _check(load_library().int2kv_set_decode_events(before_scan, after_scan), "int2kv_set_decode_events")


def int2kv_decode(cache: Int2KVCache, q: torch.Tensor, block_table: torch.Tensor, ctx_lens: torch.Tensor,
                  max_ctx: int, R_k: torch.Tensor, R_v: Optional[torch.Tensor], W_o: Optional[torch.Tensor] = None,
                  wo_is_folded: bool = False, out: Optional[torch.Tensor] = None,
                  workspace: Optional[torch.Tensor] = None, wo_format: Optional[int] = None,
                  d_model: Optional[int] = None) -> torch.Tensor:
    """wo_format (INT2KV_WO_*) overrides wo_is_folded; prepared weights (flat) need d_model."""
    B, Hq = q.shape[0], q.shape[1]
    if wo_format is None:
        wo_format = INT2KV_WO_FOLDED if wo_is_folded else INT2KV_WO_PLAIN
    if W_o is None:
        d_model = 0
    elif wo_format >= INT2KV_WO_PREPARED:
        if d_model is None:
            raise ValueError("d_model is required with prepared W_o")
    else:
        d_model = W_o.shape[0]
    if out is None:
        shape = (B, d_model) if W_o is not None else (B, Hq, HEAD_DIM)
        out = torch.empty(shape, dtype=torch.float32, device=q.device)
    need = int2kv_decode_workspace_bytes(B, Hq, cache.num_kv_heads, max_ctx, d_model)
    if workspace is None:
        workspace = torch.empty(max(need, 256), dtype=torch.uint8, device=q.device)
    st = load_library().int2kv_decode(
        cache.desc, _ptr(q, _BF16, "q"), B, Hq, _ptr(block_table, _I32, "block_table"), block_table.shape[1],
        _ptr(ctx_lens, _I32, "ctx_lens"), max_ctx, _ptr(R_k, _F32, "R_k"), _ptr(R_v, _F32, "R_v"),
        _ptr(W_o, _BF16 + (torch.float16,), "W_o"), d_model, wo_format, _ptr(out, _F32, "out"),
        _ptr(workspace, (torch.uint8,), "workspace"), workspace.numel(), _stream())
    _check(st, "int2kv_decode")
    return out


def int2kv_append_decode(cache: Int2KVCache, k: torch.Tensor, v: torch.Tensor, slot_mapping: torch.Tensor,
                         mu_rk: torch.Tensor, q: torch.Tensor, block_table: torch.Tensor, ctx_lens: torch.Tensor,
                         max_ctx: int, R_k: torch.Tensor, R_v: torch.Tensor, W_o: Optional[torch.Tensor] = None,
                         wo_format: int = INT2KV_WO_PLAIN, d_model: Optional[int] = None, clip_k: float = 1.0,
                         clip_v: float = 1.0, out: Optional[torch.Tensor] = None,
                         workspace: Optional[torch.Tensor] = None) -> torch.Tensor:
    """int2kv_quantize_append(k, v, slot_mapping) then int2kv_decode, with the cache write beside the
    query preparation. Prepared W_o (flat) needs d_model."""
    n = slot_mapping.shape[0]
    if k.numel() != n * cache.num_kv_heads * HEAD_DIM or v.numel() != k.numel():
        raise ValueError("k / v must be [n, num_kv_heads, 128]")
    B, Hq = q.shape[0], q.shape[1]
    if W_o is None:
        d_model = 0
    elif wo_format < INT2KV_WO_PREPARED:
        d_model = W_o.shape[0]
    elif d_model is None:
        raise ValueError("d_model is required with prepared W_o")
    if out is None:
        shape = (B, d_model) if W_o is not None else (B, Hq, HEAD_DIM)
        out = torch.empty(shape, dtype=torch.float32, device=q.device)
    need = int2kv_decode_workspace_bytes(B, Hq, cache.num_kv_heads, max_ctx, d_model)
    if workspace is None:
        workspace = torch.empty(max(need, 256), dtype=torch.uint8, device=q.device)
    st = load_library().int2kv_append_decode(
        cache.desc, _ptr(k, _BF16, "k"), _ptr(v, _BF16, "v"), _ptr(slot_mapping, _I32, "slot_mapping"), n,
        _ptr(mu_rk, _F32, "mu_rk"), clip_k, clip_v, _ptr(q, _BF16, "q"), B, Hq,
        _ptr(block_table, _I32, "block_table"), block_table.shape[1], _ptr(ctx_lens, _I32, "ctx_lens"), max_ctx,
        _ptr(R_k, _F32, "R_k"), _ptr(R_v, _F32, "R_v"), _ptr(W_o, _BF16 + (torch.float16,), "W_o"), d_model,
        wo_format, _ptr(out, _F32, "out"), _ptr(workspace, (torch.uint8,), "workspace"), workspace.numel(),
        _stream())
    _check(st, "int2kv_append_decode")
    return out


def int2kv_append_decode_noalloc(cache: Int2KVCache, k: torch.Tensor, v: torch.Tensor, slot_mapping: torch.Tensor,
                                 mu_rk: torch.Tensor, q: torch.Tensor, block_table: torch.Tensor,
                                 ctx_lens: torch.Tensor, max_ctx: int, R_k: torch.Tensor, R_v: torch.Tensor,
                                 W_o: Optional[torch.Tensor] = None, wo_format: int = INT2KV_WO_PLAIN,
                                 d_model: Optional[int] = None, clip_k: float = 1.0, clip_v: float = 1.0,
                                 out: Optional[torch.Tensor] = None) -> torch.Tensor:
    """int2kv_append_decode with the library's static scratch as its workspace (no workspace
    argument; the library allocates nothing). Prepared W_o (flat) needs d_model."""
    n = slot_mapping.shape[0]
    if k.numel() != n * cache.num_kv_heads * HEAD_DIM or v.numel() != k.numel():
        raise ValueError("k / v must be [n, num_kv_heads, 128]")
    B, Hq = q.shape[0], q.shape[1]
    if W_o is None:
        d_model = 0
    elif wo_format < INT2KV_WO_PREPARED:
        d_model = W_o.shape[0]
    elif d_model is None:
        raise ValueError("d_model is required with prepared W_o")
    if out is None:
        shape = (B, d_model) if W_o is not None else (B, Hq, HEAD_DIM)
        out = torch.empty(shape, dtype=torch.float32, device=q.device)
    st = load_library().int2kv_append_decode_noalloc(
        cache.desc, _ptr(k, _BF16, "k"), _ptr(v, _BF16, "v"), _ptr(slot_mapping, _I32, "slot_mapping"), n,
        _ptr(mu_rk, _F32, "mu_rk"), clip_k, clip_v, _ptr(q, _BF16, "q"), B, Hq,
        _ptr(block_table, _I32, "block_table"), block_table.shape[1], _ptr(ctx_lens, _I32, "ctx_lens"), max_ctx,
        _ptr(R_k, _F32, "R_k"), _ptr(R_v, _F32, "R_v"), _ptr(W_o, _BF16 + (torch.float16,), "W_o"), d_model,
        wo_format, _ptr(out, _F32, "out"), _stream())
    _check(st, "int2kv_append_decode_noalloc")
    return out


def int2kv_window_write(k: torch.Tensor, v: torch.Tensor, rows: torch.Tensor, mu: torch.Tensor,
                        win_k: torch.Tensor, win_v: torch.Tensor) -> None:
    """Store tokens into a BF16 window: win_k[rows] = bf16(k - mu), win_v[rows] = v.
    k, v: bf16 [n, H, 128]; rows: int32 [n]; mu: fp32 [H, 128]; win_k, win_v: bf16 [num_rows, H, 128]."""
    n, H = rows.shape[0], mu.shape[0]
    if k.numel() != n * H * HEAD_DIM or v.numel() != k.numel():
        raise ValueError("k / v must be [n, num_kv_heads, 128]")
    if win_k.shape != win_v.shape or win_k.numel() % (H * HEAD_DIM):
        raise ValueError("win_k / win_v must be [num_rows, num_kv_heads, 128]")
    st = load_library().int2kv_window_write(
        _ptr(k, _BF16, "k"), _ptr(v, _BF16, "v"), _ptr(rows, _I32, "rows"), n, H, _ptr(mu, _F32, "mu"),
        _ptr(win_k, _BF16, "win_k"), _ptr(win_v, _BF16, "win_v"), win_k.numel() // (H * HEAD_DIM), _stream())
    _check(st, "int2kv_window_write")


def int2kv_decode_window(cache: Int2KVCache, q: torch.Tensor, block_table: torch.Tensor, ctx_lens: torch.Tensor,
                         max_ctx: int, R_k: torch.Tensor, R_v: torch.Tensor, win_k: torch.Tensor,
                         win_v: torch.Tensor, win_lens: torch.Tensor, win_cap: int,
                         W_o: Optional[torch.Tensor] = None, wo_format: int = INT2KV_WO_PLAIN,
                         d_model: Optional[int] = None, out: Optional[torch.Tensor] = None,
                         workspace: Optional[torch.Tensor] = None) -> torch.Tensor:
    """int2kv_decode over the INT2 tokens and each sequence's BF16 window tokens (rows
    b * win_cap + t of win_k / win_v, win_lens[b] of them). Prepared W_o (flat) needs d_model."""
    B, Hq = q.shape[0], q.shape[1]
    if win_k.numel() < B * win_cap * cache.num_kv_heads * HEAD_DIM or win_v.shape != win_k.shape:
        raise ValueError("win_k / win_v must hold batch * win_cap rows of [num_kv_heads, 128]")
    if W_o is None:
        d_model = 0
    elif wo_format < INT2KV_WO_PREPARED:
        d_model = W_o.shape[0]
    elif d_model is None:
        raise ValueError("d_model is required with prepared W_o")
    if out is None:
        shape = (B, d_model) if W_o is not None else (B, Hq, HEAD_DIM)
        out = torch.empty(shape, dtype=torch.float32, device=q.device)
    need = int2kv_decode_workspace_bytes(B, Hq, cache.num_kv_heads, max_ctx, d_model)
    if workspace is None:
        workspace = torch.empty(max(need, 256), dtype=torch.uint8, device=q.device)
    st = load_library().int2kv_decode_window(
        cache.desc, _ptr(q, _BF16, "q"), B, Hq, _ptr(block_table, _I32, "block_table"), block_table.shape[1],
        _ptr(ctx_lens, _I32, "ctx_lens"), max_ctx, _ptr(R_k, _F32, "R_k"), _ptr(R_v, _F32, "R_v"),
        _ptr(W_o, _BF16 + (torch.float16,), "W_o"), d_model, wo_format, _ptr(win_k, _BF16, "win_k"),
        _ptr(win_v, _BF16, "win_v"), _ptr(win_lens, _I32, "win_lens"), win_cap, _ptr(out, _F32, "out"),
        _ptr(workspace, (torch.uint8,), "workspace"), workspace.numel(), _stream())
    _check(st, "int2kv_decode_window")
    return out


def int2kv_quantize_append_error(cache: Int2KVCache, k: torch.Tensor, v: torch.Tensor, slot_mapping: torch.Tensor,
                                 R_k: torch.Tensor, R_v: torch.Tensor, mu_rk: torch.Tensor, clip_k: float = 1.0,
                                 clip_v: float = 1.0, err: Optional[torch.Tensor] = None) -> torch.Tensor:
    """int2kv_quantize_append plus each token's squared reconstruction error: fp32 [n, H, 2] (key, value)."""
    n = slot_mapping.shape[0]
    if k.numel() != n * cache.num_kv_heads * HEAD_DIM or v.numel() != k.numel():
        raise ValueError("k / v must be [n, num_kv_heads, 128]")
    if err is None:
        err = torch.empty((n, cache.num_kv_heads, 2), dtype=torch.float32, device=k.device)
    st = load_library().int2kv_quantize_append_error(
        cache.desc, _ptr(k, _BF16, "k"), _ptr(v, _BF16, "v"), _ptr(slot_mapping, _I32, "slot_mapping"), n,
        _ptr(R_k, _F32, "R_k"), _ptr(R_v, _F32, "R_v"), _ptr(mu_rk, _F32, "mu_rk"), clip_k, clip_v,
        _ptr(err, _F32, "err"), _stream())
    _check(st, "int2kv_quantize_append_error")
    return err


def int2kv_output_error_workspace_bytes(batch: int, num_q_heads: int, num_kv_heads: int, max_ctx: int,
                                        d_model: int) -> int:
    return load_library().int2kv_output_error_workspace_bytes(batch, num_q_heads, num_kv_heads, max_ctx, d_model)


def int2kv_output_error(cache: Int2KVCache, q: torch.Tensor, block_table: torch.Tensor, ctx_lens: torch.Tensor,
                        max_ctx: int, R_k: torch.Tensor, R_v: torch.Tensor, k_rows: torch.Tensor,
                        v_rows: torch.Tensor, row_cap: int, W_o: torch.Tensor, want_dy: bool = False,
                        workspace: Optional[torch.Tensor] = None, stats: Optional[torch.Tensor] = None):
    """Output-error diagnostics: returns stats fp32 [B, H_q, 4] (||dy||^2, ||dy_K||^2, ||dy_V||^2,
    <dy_K, dy_V>) and, with want_dy, dy fp32 [B, H_q, 2, d_model] (dy_K, dy_V)."""
    B, Hq = q.shape[0], q.shape[1]
    d_model = W_o.shape[0]
    if stats is None:
        stats = torch.empty((B, Hq, 4), dtype=torch.float32, device=q.device)
    elif stats.numel() != B * Hq * 4:
        raise ValueError("stats must hold [B, H_q, 4] floats")
    dy = torch.empty((B, Hq, 2, d_model), dtype=torch.float32, device=q.device) if want_dy else None
    need = int2kv_output_error_workspace_bytes(B, Hq, cache.num_kv_heads, max_ctx, d_model)
    if workspace is None:
        workspace = torch.empty(max(need, 256), dtype=torch.uint8, device=q.device)
    st = load_library().int2kv_output_error(
        cache.desc, _ptr(q, _BF16, "q"), B, Hq, _ptr(block_table, _I32, "block_table"), block_table.shape[1],
        _ptr(ctx_lens, _I32, "ctx_lens"), max_ctx, _ptr(R_k, _F32, "R_k"), _ptr(R_v, _F32, "R_v"),
        _ptr(k_rows, _BF16, "k_rows"), _ptr(v_rows, _BF16, "v_rows"), row_cap, _ptr(W_o, _BF16, "W_o"), d_model,
        _ptr(stats, _F32, "stats"), _ptr(dy, _F32, "dy"), _ptr(workspace, (torch.uint8,), "workspace"),
        workspace.numel(), _stream())
    _check(st, "int2kv_output_error")
    return (stats, dy) if want_dy else stats


INT2KV_HADAMARD_K = 1
INT2KV_HADAMARD_V = 2


def int2kv_quantize_append_rope(cache: Int2KVCache, k: torch.Tensor, v: torch.Tensor, slot_mapping: torch.Tensor,
                                positions: Optional[torch.Tensor], cos_sin: Optional[torch.Tensor],
                                R_k: Optional[torch.Tensor], R_v: Optional[torch.Tensor], mu_rk: torch.Tensor,
                                clip_k: float = 1.0, clip_v: float = 1.0, flags: int = 0,
                                k_rope_out: Optional[torch.Tensor] = None) -> None:
    """Cache write of pre-RoPE keys (positions and an fp32 [max_pos, 128] cos/sin table), with the
    Hadamard rotation in place of R_K / R_V under INT2KV_HADAMARD_K / _V."""
    n = slot_mapping.shape[0]
    if k.numel() != n * cache.num_kv_heads * HEAD_DIM or v.numel() != k.numel():
        raise ValueError("k / v must be [n, num_kv_heads, 128]")
    if positions is not None and positions.numel() != n:
        raise ValueError("positions must hold one position per token")
    max_pos = cos_sin.shape[0] if cos_sin is not None else 0
    st = load_library().int2kv_quantize_append_rope(
        cache.desc, _ptr(k, _BF16, "k"), _ptr(v, _BF16, "v"), _ptr(slot_mapping, _I32, "slot_mapping"),
        _ptr(positions, _I32, "positions"), n, _ptr(cos_sin, _F32, "cos_sin"), max_pos, _ptr(R_k, _F32, "R_k"),
        _ptr(R_v, _F32, "R_v"), _ptr(mu_rk, _F32, "mu_rk"), clip_k, clip_v, flags,
        _ptr(k_rope_out, _BF16, "k_rope_out"), _stream())
    _check(st, "int2kv_quantize_append_rope")


def hadamard_rotation(num_heads: int, device="cuda") -> torch.Tensor:
    """The dense fp32 form of the library's Hadamard rotation, [num_heads, 128, 128]: entries
    (-1)^popcount(i & c) * RN(1 / sqrt(128)), as the decode and the other readers take it."""
    i = torch.arange(HEAD_DIM)
    x = i[:, None] & i[None, :]
    par = torch.zeros_like(x)
    for b in range(7):
        par ^= (x >> b) & 1
    scale = torch.tensor(1.0 / math.sqrt(HEAD_DIM), dtype=torch.float32)
    H = torch.where(par == 1, -scale, scale)
    return H[None].expand(num_heads, HEAD_DIM, HEAD_DIM).contiguous().to(device)


# ---------------------------------------------------------------------------------------------
# OptR offline calibration
_F64 = (torch.float64,)


class OptrTraces:
    """Calibration traces on the device: k, v bf16 [T, H_kv, 128], q bf16 [T, H_q, 128], and the
    sequences' token offsets (host int32 [N + 1], starting at 0)."""

    def __init__(self, k: torch.Tensor, v: torch.Tensor, q: torch.Tensor, seq_starts):
        import numpy as np
        self.k, self.v, self.q = k, v, q
        self._starts = np.ascontiguousarray(np.asarray(seq_starts, dtype=np.int32))
        if self._starts[-1] != k.shape[0] or v.shape != k.shape or q.shape[0] != k.shape[0]:
            raise ValueError("k, v, q must hold seq_starts[-1] tokens")
        self.desc = _OptrTraces(_ptr(k, _BF16, "k"), _ptr(v, _BF16, "v"), _ptr(q, _BF16, "q"),
                                self._starts.ctypes.data_as(ctypes.POINTER(ctypes.c_int32)), len(self._starts) - 1)


def optr_config(num_kv_heads: int, num_q_heads: int, d_model: int, group_size: int = 128, clip_k: float = 0.96,
                clip_v: float = 0.92, lambda_k: float = 1.0, n_last: int = 64, sink: int = 64, recent: int = 256,
                steps: int = 80, eval_every: int = 20, lr: float = 0.02):
    """Calibration settings (defaults: the paper's)."""
    return _OptrConfig(num_kv_heads, num_q_heads, d_model, group_size, clip_k, clip_v, lambda_k, n_last, sink,
                       recent, steps, eval_every, lr)


def int2kv_optr_workspace_bytes(cfg, calib: OptrTraces, heldout: Optional[OptrTraces] = None) -> int:
    n = load_library().int2kv_optr_workspace_bytes(ctypes.byref(cfg), ctypes.byref(calib.desc),
                                                   ctypes.byref(heldout.desc) if heldout else None)
    if n == 0:
        raise ValueError("int2kv_optr_workspace_bytes: " + (load_library().int2kv_last_error() or b"").decode())
    return n


def _workspace(n, device):
    return torch.empty(n, dtype=torch.uint8, device=device)


def int2kv_optr_key_mean(k: torch.Tensor) -> torch.Tensor:
    T, H = k.shape[0], k.shape[1]
    mu = torch.empty((H, HEAD_DIM), dtype=torch.float32, device=k.device)
    _check(load_library().int2kv_optr_key_mean(_ptr(k, _BF16, "k"), T, H, _ptr(mu, _F32, "mu"), _stream()),
           "int2kv_optr_key_mean")
    return mu


def int2kv_optr_key_loss(cfg, traces: OptrTraces, R0_k, mu, W_o, A, want_grad: bool = True):
    """(loss [H] fp64, grad [H, 128, 128] fp64 or None) of the key objective at generators A."""
    H = cfg.num_kv_heads
    loss = torch.empty(H, dtype=torch.float64, device=A.device)
    grad = torch.empty((H, HEAD_DIM, HEAD_DIM), dtype=torch.float64, device=A.device) if want_grad else None
    n = int2kv_optr_workspace_bytes(cfg, traces)
    ws = _workspace(n, A.device)
    _check(load_library().int2kv_optr_key_loss(
        ctypes.byref(cfg), ctypes.byref(traces.desc), _ptr(R0_k, _F32, "R0_k"), _ptr(mu, _F32, "mu"),
        _ptr(W_o, _BF16, "W_o"), _ptr(A, _F64, "A"), _ptr(loss, _F64, "loss"), _ptr(grad, _F64, "grad"),
        _ptr(ws, (torch.uint8,), "ws"), n, _stream()), "int2kv_optr_key_loss")
    return loss, grad


def int2kv_optr_value_loss(cfg, traces: OptrTraces, R0_k, A_k, mu, R0_v, W_o, A_v, want_grad: bool = True):
    H = cfg.num_kv_heads
    loss = torch.empty(H, dtype=torch.float64, device=A_v.device)
    grad = torch.empty((H, HEAD_DIM, HEAD_DIM), dtype=torch.float64, device=A_v.device) if want_grad else None
    n = int2kv_optr_workspace_bytes(cfg, traces)
    ws = _workspace(n, A_v.device)
    _check(load_library().int2kv_optr_value_loss(
        ctypes.byref(cfg), ctypes.byref(traces.desc), _ptr(R0_k, _F32, "R0_k"), _ptr(A_k, _F64, "A_k"),
        _ptr(mu, _F32, "mu"), _ptr(R0_v, _F32, "R0_v"), _ptr(W_o, _BF16, "W_o"), _ptr(A_v, _F64, "A_v"),
        _ptr(loss, _F64, "loss"), _ptr(grad, _F64, "grad"), _ptr(ws, (torch.uint8,), "ws"), n, _stream()),
        "int2kv_optr_value_loss")
    return loss, grad


def int2kv_optr_calibrate(cfg, calib: OptrTraces, heldout: OptrTraces, R0_k, R0_v, mu, W_o,
                          workspace: Optional[torch.Tensor] = None):
    """Algorithm 1 for every KV head: returns dict(R_k, R_v (fp32), A_k, A_v (fp64), history (fp64
    [2, H, steps + 1 + steps // eval_every]))."""
    H = cfg.num_kv_heads
    dev = R0_k.device
    R_k = torch.empty((H, HEAD_DIM, HEAD_DIM), dtype=torch.float32, device=dev)
    R_v = torch.empty_like(R_k)
    A_k = torch.empty((H, HEAD_DIM, HEAD_DIM), dtype=torch.float64, device=dev)
    A_v = torch.empty_like(A_k)
    hist = torch.empty((2, H, cfg.steps + 1 + cfg.steps // cfg.eval_every), dtype=torch.float64, device=dev)
    n = int2kv_optr_workspace_bytes(cfg, calib, heldout)
    ws = workspace if workspace is not None else _workspace(n, dev)
    _check(load_library().int2kv_optr_calibrate(
        ctypes.byref(cfg), ctypes.byref(calib.desc), ctypes.byref(heldout.desc), _ptr(R0_k, _F32, "R0_k"),
        _ptr(R0_v, _F32, "R0_v"), _ptr(mu, _F32, "mu"), _ptr(W_o, _BF16, "W_o"), _ptr(R_k, _F32, "R_k"),
        _ptr(R_v, _F32, "R_v"), _ptr(A_k, _F64, "A_k"), _ptr(A_v, _F64, "A_v"), _ptr(hist, _F64, "history"),
        _ptr(ws, (torch.uint8,), "ws"), ws.numel(), _stream()), "int2kv_optr_calibrate")
    return dict(R_k=R_k, R_v=R_v, A_k=A_k, A_v=A_v, history=hist)
