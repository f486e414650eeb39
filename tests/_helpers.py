"""Shared helpers of the GPU parity tests: move seeded inputs to the device, build oracle pools,
and compare results to the oracle at the tolerances the tests state."""
from __future__ import annotations

import numpy as np
import torch

from oracle import int2kv_oracle as O
from paper_2608_02691_amd import int2kv as K

# Attention outputs: max |gpu - ref| over a row <= 2e-3 * ||ref row||_2, with a row being one
# (sequence, query head) 128-vector without W_O, or one sequence's d_model vector with W_O.
ROW_REL_TOL = 2e-3
# End-to-end cache writes: at most this fraction of codes may differ from the oracle's.
CODE_MISMATCH_MAX = 1e-4
# A differing code must sit this close to a rounding tie of the oracle's t = (x - z) / s. The
# library's rotation is an fp32 accumulation of exact products (R in three bf16 terms), so its
# rotated value differs from the oracle's correctly rounded one by at most about 2^-24 times the
# sum of the 384 product magnitudes plus the fp32 rounding, i.e. below 2^-17 ||x|| for rows of
# N(0, 1)-like size; divided by s (about a third of the group's range) that is below 1e-4 in t.
TIE_WINDOW = 1e-4


def dev(a: np.ndarray) -> torch.Tensor:
    if a.dtype == np.uint16:
        return torch.from_numpy(a.view(np.int16).copy()).cuda()
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def gpu_cache(pool: np.ndarray) -> K.Int2KVCache:
    nb, H, rec = pool.shape
    G = {1536: 32, 1152: 128}[rec]
    return K.Int2KVCache(nb, H, pool=torch.from_numpy(pool).cuda(), group_size=G)


def oracle_pool(w, seqs=None, clip_k=1.0, clip_v=1.0, group=32):
    """Oracle cache holding the given sequences of workload w (all by default)."""
    pool = O.new_pool(w.num_blocks, w.num_kv_heads, group)
    for b in (range(w.batch) if seqs is None else seqs):
        if int(w.ctx_lens[b]) == 0:
            continue
        k, v = w.kv(b)
        O.quantize_append(pool, k, v, w.slot_mapping(b), w.R_k, w.R_v, w.mu, clip_k, clip_v)
    return pool


def assert_rows_close(got: np.ndarray, ref: np.ndarray, rel: float = ROW_REL_TOL, what: str = ""):
    got = np.asarray(got, dtype=np.float64).reshape(-1, ref.shape[-1])
    ref = np.asarray(ref, dtype=np.float64).reshape(-1, ref.shape[-1])
    assert np.all(np.isfinite(got)), what
    err = np.abs(got - ref).max(axis=1)
    norm = np.linalg.norm(ref, axis=1)
    zero = norm == 0
    assert np.all(got[zero] == 0), f"{what}: rows with an empty context must be zero"
    ratio = err[~zero] / norm[~zero]
    worst = float(ratio.max()) if ratio.size else 0.0
    assert worst <= rel, f"{what}: worst row error {worst:.3e} > {rel:.1e}"
    return worst


def unpack_slots(pool: np.ndarray, slots: np.ndarray):
    """codes/scales/zeros of the given slots for every KV head: arrays [n, H, ...]."""
    nb, H, _ = pool.shape
    out = [[] for _ in range(6)]
    for h in range(H):
        r = O.read_tokens(pool, np.arange(nb), nb * 16, h)
        for i in range(6):
            out[i].append(r[i][slots])
    return [np.stack(x, axis=1) for x in out]


def compare_cache_writes(pool_gpu, pool_ref, slots, k_rot, v_rot):
    """End-to-end cache-write parity. Codes may differ from the oracle's only at rounding ties:
    either the group's fp16 scale or zero is one ulp away (its fp32 value sat at an fp16 rounding
    boundary), or the oracle's t = (x - z)/s lies within TIE_WINDOW of a half-integer. Returns
    stats, including the largest tie distance |t - floor(t) - 1/2| among the differing codes."""
    g = unpack_slots(pool_gpu, slots)
    r = unpack_slots(pool_ref, slots)
    stats = {}
    total_codes = 0
    total_bad = 0
    for name, (ci, si, zi), x in (("K", (0, 1, 2), k_rot), ("V", (3, 4, 5), v_rot)):
        cg, sg, zg = g[ci], g[si], g[zi]
        cr, sr, zr = r[ci], r[si], r[zi]
        meta_diff = (sg != sr) | (zg != zr)                       # [n, H, groups]
        G = 128 // meta_diff.shape[-1]
        ulp = lambda a, b: np.abs(a.view(np.int16).astype(np.int32) - b.view(np.int16).astype(np.int32))
        assert np.all(ulp(sg, sr)[meta_diff] <= 1) and np.all(ulp(zg, zr)[meta_diff] <= 1), \
            f"{name}: scale/zero differ by more than one fp16 ulp"
        bad = cg != cr                                             # [n, H, 128]
        grp_meta = np.repeat(meta_diff, G, axis=-1)
        s = np.repeat(sr.astype(np.float64), G, axis=-1)
        z = np.repeat(zr.astype(np.float64), G, axis=-1)
        t = np.where(s > 0, (x.astype(np.float64) - z) / np.where(s > 0, s, 1), 0)
        dist = np.abs(t - np.floor(t) - 0.5)
        near_tie = dist < TIE_WINDOW
        unexplained = bad & ~grp_meta & ~near_tie
        assert not unexplained.any(), \
            f"{name}: {int(unexplained.sum())} code mismatches away from ties (closest {dist[unexplained].min():.2e})"
        total_codes += bad.size
        total_bad += int(bad.sum())
        tie_flips = bad & ~grp_meta
        stats[name] = dict(code_mismatch=int(bad.sum()), meta_mismatch_groups=int(meta_diff.sum()),
                           max_tie_distance=float(dist[tie_flips].max()) if tie_flips.any() else 0.0)
    frac = total_bad / max(total_codes, 1)
    assert frac <= CODE_MISMATCH_MAX, f"code mismatch fraction {frac:.2e}"
    stats["fraction"] = frac
    return stats
