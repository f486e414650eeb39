"""Seeded synthetic workloads for the rotated, key-centered INT2 KV cache.

This module only draws inputs. It holds none of the method's arithmetic: no
rotation is applied here, nothing is quantized, nothing is packed. The same
arrays are handed to the HIP path and to the CPU oracle, which is how the two
stay comparable while sharing no code.

The shapes stand in for the Qwen3-class decoder layers the paper evaluates
(Sec. 5 "Models and Benchmarks"; efficiency runs in the appendix "Experimental
settings"). The paper's calibration traces and models are not available, so
every tensor is drawn from a seeded distribution:

* keys   : N(0, 1) per channel (torch CPU generator, per-sequence seed) plus a constant per-channel offset on a few
           seeded channels per KV head (the channel-wise key offsets that
           motivate key centering, Sec. 4.1 and Fig. 2), rounded to bf16 (RNE);
* values : N(0, 1), rounded to bf16;
* queries: N(0, 1), rounded to bf16;
* R_k/R_v: Haar-random orthogonal 128x128 per KV head (QR of a Gaussian with
           the sign of diag(R) folded in), computed in fp64, stored fp32;
* mu     : per-channel mean of a separate seeded calibration draw of keys
           (the paper estimates mu from calibration traces and keeps it fixed
           at inference, appendix "Key-mean estimation and application");
* W_O    : N(0, 1/d_model), bf16, row-major [d_model, H_q * head_dim];
* paging : block size 16, physical blocks assigned through a seeded
           permutation of one shared pool.

Every sequence's keys and values come from their own spawned stream, so any
single sequence can be regenerated without drawing the others (the large
configurations are checked on sampled sequences).
"""
from __future__ import annotations

from dataclasses import dataclass, field
from typing import Optional

import numpy as np
import torch

HEAD_DIM = 128
BLOCK_SIZE = 16
GROUP_SIZE = 32
SEED_BASE = 20262608
N_CALIB_TOKENS = 4096

# stream indices of the per-config SeedSequence spawn
_S_ROT, _S_OFFSET, _S_QUERY, _S_PERM, _S_LEN, _S_WO, _S_CALIB, _S_SEQ = range(8)


def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round fp32 to bf16 (round-to-nearest-even, as torch's CPU cast does); uint16 bit pattern."""
    t = torch.from_numpy(np.ascontiguousarray(x, dtype=np.float32))
    return t.to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    return (np.ascontiguousarray(b, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)


def rope_cos_sin(max_pos: int, theta: float = 1.0e6, head_dim: int = HEAD_DIM) -> np.ndarray:
    """RoPE table fp32 [max_pos, head_dim]: cos of the angles p * theta^(-2 i / head_dim) in the
    first half, their sines in the second (i < head_dim / 2; angles formed and evaluated in fp64,
    then rounded to fp32). theta = 1e6 is the Qwen3 base."""
    inv = theta ** (-np.arange(0, head_dim, 2, dtype=np.float64) / head_dim)
    ang = np.arange(max_pos, dtype=np.float64)[:, None] * inv[None, :]
    return np.concatenate([np.cos(ang), np.sin(ang)], axis=1).astype(np.float32)


def haar_orthogonal(rng: np.random.Generator, n: int = HEAD_DIM) -> np.ndarray:
    """Haar-distributed orthogonal matrix (fp64): QR of a Gaussian, signs of diag(R) folded into Q."""
    g = rng.standard_normal((n, n))
    q, r = np.linalg.qr(g)
    return q * np.sign(np.diag(r))[None, :]


@dataclass
class Config:
    cfg_id: int
    name: str
    batch: int
    num_q_heads: int
    num_kv_heads: int
    ctx: Optional[int]                 # uniform context, or None for ragged
    ctx_range: Optional[tuple] = None  # (lo, hi) inclusive for ragged lengths
    d_model: Optional[int] = None      # W_O applied when set
    n_offset_channels: int = 3
    offset_range: tuple = (10.0, 30.0)
    fixed_offset: Optional[float] = None
    permute_blocks: bool = True
    append_then_decode: bool = False
    spare_blocks: int = 0


CONFIGS = {
    0: Config(0, "tiny: B1, 1/1 heads, ctx 256", 1, 1, 1, 256, n_offset_channels=4,
              fixed_offset=20.0, permute_blocks=False),
    1: Config(1, "qwen3-8b layer: B16, 32/8 heads, ctx 4096, W_O 4096^2", 16, 32, 8, 4096,
              d_model=4096),
    2: Config(2, "long context: B1, 32/8 heads, ctx 131072", 1, 32, 8, 131072),
    3: Config(3, "append 4x8192 tokens, 8 KV heads, then decode 32/8 heads", 4, 32, 8, 8192,
              append_then_decode=True),
    4: Config(4, "ragged serving: 64 seqs, ctx U[512,32768], 40/8 heads, W_O 5120^2", 64, 40, 8,
              None, ctx_range=(512, 32768), d_model=5120),
}


@dataclass
class Workload:
    cfg: Config
    ctx_lens: np.ndarray          # int32 [B]
    block_table: np.ndarray       # int32 [B, max_blocks]
    num_blocks: int
    R_k: np.ndarray               # fp32 [H_kv, 128, 128]
    R_v: np.ndarray               # fp32 [H_kv, 128, 128]
    mu: np.ndarray                # fp32 [H_kv, 128]
    q: np.ndarray                 # bf16 bits uint16 [B, H_q, 128]
    W_o: Optional[np.ndarray]     # bf16 bits uint16 [d_model, H_q*128] or None
    key_offsets: np.ndarray       # fp32 [H_kv, 128] (the constant channel offsets)
    _seq_ss: list = field(repr=False, default_factory=list)

    @property
    def batch(self) -> int:
        return self.cfg.batch

    @property
    def num_q_heads(self) -> int:
        return self.cfg.num_q_heads

    @property
    def num_kv_heads(self) -> int:
        return self.cfg.num_kv_heads

    @property
    def max_blocks(self) -> int:
        return self.block_table.shape[1]

    def kv(self, b: int, as_torch: bool = False):
        """Keys and values of sequence b: bf16 [L_b, H_kv, 128] each.

        Returned as uint16 bit patterns (numpy), or as torch.bfloat16 CPU tensors when
        as_torch is set. Drawn with torch's CPU normal generator (fast and independent of the
        thread count) seeded from this sequence's own SeedSequence."""
        L = int(self.ctx_lens[b])
        H = self.num_kv_heads
        seed_k, seed_v = (int(s) & 0x7FFFFFFFFFFFFFFF for s in self._seq_ss[b].generate_state(2, np.uint64))
        k = torch.randn((L, H, HEAD_DIM), generator=torch.Generator().manual_seed(seed_k), dtype=torch.float32)
        k += torch.from_numpy(self.key_offsets)[None]
        v = torch.randn((L, H, HEAD_DIM), generator=torch.Generator().manual_seed(seed_v), dtype=torch.float32)
        k, v = k.to(torch.bfloat16), v.to(torch.bfloat16)
        if as_torch:
            return k, v
        return (k.view(torch.int16).numpy().view(np.uint16), v.view(torch.int16).numpy().view(np.uint16))

    def slot_mapping(self, b: int, start: int = 0, stop: Optional[int] = None) -> np.ndarray:
        """Cache slot of every token position in [start, stop) of sequence b (int32)."""
        stop = int(self.ctx_lens[b]) if stop is None else stop
        pos = np.arange(start, stop, dtype=np.int64)
        return (self.block_table[b, pos // BLOCK_SIZE].astype(np.int64) * BLOCK_SIZE
                + pos % BLOCK_SIZE).astype(np.int32)


def make_workload(cfg_id: int, *, batch: Optional[int] = None, ctx: Optional[int] = None,
                  ctx_lens: Optional[np.ndarray] = None, num_q_heads: Optional[int] = None,
                  num_kv_heads: Optional[int] = None, d_model: Optional[int] = -1) -> Workload:
    """Build the seeded workload of a configuration, optionally resized (for fast tests).

    Overrides keep the distribution recipe of the configuration and only change sizes.
    """
    base = CONFIGS[cfg_id]
    cfg = Config(**{**base.__dict__})
    if batch is not None:
        cfg.batch = batch
    if num_q_heads is not None:
        cfg.num_q_heads = num_q_heads
    if num_kv_heads is not None:
        cfg.num_kv_heads = num_kv_heads
    if d_model != -1:
        cfg.d_model = d_model
    if ctx is not None:
        cfg.ctx = ctx
        cfg.ctx_range = None
    if cfg.num_q_heads % cfg.num_kv_heads:
        raise ValueError("num_q_heads must be a multiple of num_kv_heads")

    ss = np.random.SeedSequence(SEED_BASE + cfg_id)
    streams = ss.spawn(8)
    H, Hq, B = cfg.num_kv_heads, cfg.num_q_heads, cfg.batch

    if ctx_lens is not None:
        lens = np.asarray(ctx_lens, dtype=np.int32)
        if lens.shape != (B,):
            raise ValueError("ctx_lens must have shape [batch]")
    elif cfg.ctx is not None:
        lens = np.full(B, cfg.ctx, dtype=np.int32)
    else:
        lo, hi = cfg.ctx_range
        lens = np.random.default_rng(streams[_S_LEN]).integers(lo, hi, size=B, endpoint=True).astype(np.int32)

    nblk = (lens.astype(np.int64) + BLOCK_SIZE - 1) // BLOCK_SIZE
    num_blocks = int(nblk.sum()) + cfg.spare_blocks
    if cfg.permute_blocks:
        phys = np.random.default_rng(streams[_S_PERM]).permutation(num_blocks).astype(np.int32)
    else:
        phys = np.arange(num_blocks, dtype=np.int32)
    max_blocks = int(max(1, nblk.max()))
    table = np.zeros((B, max_blocks), dtype=np.int32)
    cur = 0
    for b in range(B):
        table[b, :nblk[b]] = phys[cur:cur + nblk[b]]
        cur += nblk[b]

    rng_rot = np.random.default_rng(streams[_S_ROT])
    R_k = np.stack([haar_orthogonal(rng_rot) for _ in range(H)]).astype(np.float32)
    R_v = np.stack([haar_orthogonal(rng_rot) for _ in range(H)]).astype(np.float32)

    rng_off = np.random.default_rng(streams[_S_OFFSET])
    offsets = np.zeros((H, HEAD_DIM), dtype=np.float32)
    for h in range(H):
        ch = rng_off.choice(HEAD_DIM, size=cfg.n_offset_channels, replace=False)
        if cfg.fixed_offset is not None:
            offsets[h, ch] = cfg.fixed_offset
        else:
            offsets[h, ch] = rng_off.uniform(*cfg.offset_range, size=cfg.n_offset_channels)

    rng_cal = np.random.default_rng(streams[_S_CALIB])
    calib = rng_cal.standard_normal((N_CALIB_TOKENS, H, HEAD_DIM), dtype=np.float32) + offsets[None]
    calib = bf16_bits_to_f32(f32_to_bf16_bits(calib)).astype(np.float64)
    mu = calib.mean(axis=0).astype(np.float32)

    q = f32_to_bf16_bits(np.random.default_rng(streams[_S_QUERY]).standard_normal(
        (B, Hq, HEAD_DIM), dtype=np.float32))

    W_o = None
    if cfg.d_model is not None:
        rng_wo = np.random.default_rng(streams[_S_WO])
        w = rng_wo.standard_normal((cfg.d_model, Hq * HEAD_DIM), dtype=np.float32)
        w *= np.float32(1.0 / np.sqrt(cfg.d_model))
        W_o = f32_to_bf16_bits(w)

    seq_ss = streams[_S_SEQ].spawn(B)
    return Workload(cfg=cfg, ctx_lens=lens, block_table=table, num_blocks=num_blocks, R_k=R_k, R_v=R_v,
                    mu=mu, q=q, W_o=W_o, key_offsets=offsets, _seq_ss=seq_ss)


def calibration_traces(num_seqs: int, len_range: tuple, num_kv_heads: int, num_q_heads: int, seed: int,
                       n_offset_channels: int = 3, offset_range: tuple = (10.0, 30.0)):
    """Seeded stand-in for the paper's calibration and held-out trace sets (appendix, calibration
    details: a few prompts of at least 328 tokens each, their Q/K/V of every layer). Lengths are
    uniform in len_range; keys are N(0, 1) plus constant offsets on n_offset_channels seeded
    channels per KV head (as in the decode workloads), values and queries N(0, 1); all bf16.
    Returns (k [T, H, 128], v [T, H, 128], q [T, H_q, 128]) as torch bf16 CPU tensors and the
    token offsets seq_starts (int32 [num_seqs + 1])."""
    rng = np.random.default_rng(SEED_BASE + 1000 + seed)
    lens = rng.integers(len_range[0], len_range[1], size=num_seqs, endpoint=True)
    starts = np.concatenate([[0], np.cumsum(lens)]).astype(np.int32)
    T = int(starts[-1])
    offsets = torch.zeros((num_kv_heads, HEAD_DIM))
    for h in range(num_kv_heads):
        ch = rng.choice(HEAD_DIM, size=n_offset_channels, replace=False)
        offsets[h, ch] = torch.from_numpy(rng.uniform(*offset_range, size=n_offset_channels)).float()
    g = torch.Generator().manual_seed(int(rng.integers(0, 2**62)))
    k = (torch.randn((T, num_kv_heads, HEAD_DIM), generator=g) + offsets[None]).to(torch.bfloat16)
    v = torch.randn((T, num_kv_heads, HEAD_DIM), generator=g).to(torch.bfloat16)
    q = torch.randn((T, num_q_heads, HEAD_DIM), generator=g).to(torch.bfloat16)
    return k, v, q, starts


def haar_rotations(num_heads: int, seed: int) -> np.ndarray:
    """Seeded Haar-random rotations fp32 [num_heads, 128, 128] (base rotations R^0)."""
    rng = np.random.default_rng(SEED_BASE + 2000 + seed)
    return np.stack([haar_orthogonal(rng) for _ in range(num_heads)]).astype(np.float32)
