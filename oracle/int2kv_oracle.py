"""CPU oracle for the rotated, key-centered INT2 KV cache and its decode attention.

TEST INFRASTRUCTURE ONLY. Nothing in the product path imports, calls or links
this module: only the tests, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of ``bench.py`` use it. It shares no code with the HIP
library; the only common inputs are the seeded arrays drawn by
``paper_2608_02691_amd.workloads`` (which holds none of the method's arithmetic).

It is the paper's definitions written out plainly, in fp64 numpy, except for the
quantizer, whose fp32/fp16 rounding sequence is fixed below so that its codes,
scales and zeros are reproducible bit for bit:

* attention, eq:fp_attention / eq:head_output (Sec. 3):
    a_s = <q, k_s>/sqrt(d),  p = softmax_s(a),  o = sum_s p_s v_s,
  with query head j reading KV head h(j) = floor(j / G_q) under GQA;
* the output projection, eq:residual_readout: y = concat_j(o_j) W_O^T;
* the rotated INT2 map, eq:rotated_int2_map: D_{R,c}(z) = Q_2(z R; c, G) R^T;
* key centering, Sec. 4.1: keys enter as D_{R_K,c_K}(k - mu), values as D_{R_V,c_V}(v);
* the INT2 attention of eq:int2_attention / eq:int2_residual_readout evaluated on
  those effective keys and values (the main-text, inverse-rotation form);
* the output-error diagnostics of Sec. 3.2 (dy_K, dy_V, E_out, E_rec) and the appendix's RMS
  output error relative to plain INT2;
* the cache write fed with pre-RoPE keys (appendix, key-mean estimation: the mean is subtracted
  from post-RoPE keys before rotation), and the normalized Sylvester Hadamard matrix, the QuaRot
  base rotation (Sec. 2, Sec. 5 baselines).

RoPE is the model's, not the paper's; the reading used here (and by the library): rotate-half
pairing, channel i with channel i + 64 (i < 64), at the token's position p with a caller-given
fp32 table cs[p] = (cos theta_{p,0..63}, sin theta_{p,0..63}):
    y_i = x_i cos - x_{i+64} sin,   y_{i+64} = x_{i+64} cos + x_i sin,
each evaluated in fp64 (both products exact: 8 by 24 significant bits) and rounded once to bf16
(nearest even): the post-RoPE key is a bf16 tensor, as the serving engine hands it to the cache.

Q_2 is "group-wise affine INT2" (Sec. 5 implementation details, Table A). The
paper gives no arithmetic for it; the reading used here (and by the library):
per token and per group of G consecutive rotated channels (G = 32, or the paper's
G = 128), over fp32 inputs,
    mn = min x, mx = max x;  if c != 1: mn = fp32(c*mn), mx = fp32(c*mx)
    s  = fp16_rne(fp32(fp32(mx - mn) / 3)),   z = fp16_rne(mn)
    inv = fp32(1 / s) if s > 0 else 0
    code = clamp(rne(fp32(fp32(x - z) * inv)), 0, 3)
    dequant = code * s + z            (exact in fp64)
The rotated tensor fed to Q_2 is the fp64 product rounded once to fp32.

Packed cache layout (one record per physical block and KV head, the format the
library writes; NG = 128 / G groups per token; record address =
pool + (block * H_kv + h) * R with R = 1024 + 128 * NG: 1536 bytes at G = 32, 1152 at G = 128):
    [   0,  512) K codes,  token-major: the 16-bit half m of token t at byte 32*t + 2*m
    [ 512, 1024) V codes,  half-major : the 16-bit half m of token t at byte 512 + 32*m + 2*t
    [1024, 1024 + 64 NG)       K meta,   token t, group g at 1024 + 4*NG*t + 4*g: fp16 scale, fp16 zero
    [1024 + 64 NG, + 32 NG)    V scales, group g, token t at 1024 + 64*NG + 32*g + 2*t (fp16)
    [1024 + 96 NG, + 32 NG)    V zeros,  group g, token t at 1024 + 96*NG + 32*g + 2*t (fp16)
Inside a 16-bit half m, channel c = 16*p + m occupies bits 2p..2p+1 (little endian).

Every function below is a plain definition; none is blocked, fused or reordered.
Parity pins (tests/test_oracle_pins.py) tie it to what the paper and the
mathematics fix; the packed layout is this library's own format and is pinned
by hand-derived byte fixtures.
"""
from __future__ import annotations

import numpy as np

HEAD_DIM = 128
GROUP = 32                      # default group size
N_GROUPS = HEAD_DIM // GROUP
BLOCK = 16
RECORD_BYTES = 1536             # record bytes at the default group size
OFF_KC, OFF_VC, OFF_KM, OFF_VS, OFF_VZ = 0, 512, 1024, 1280, 1408
GROUP_SIZES = (32, 128)


def record_bytes(group: int = GROUP) -> int:
    """Bytes of one (block, KV head) record: 1024 of codes and 128 of metadata per group and 16 tokens."""
    if group not in GROUP_SIZES:
        raise ValueError("group size must be 32 or 128")
    return 1024 + 128 * (HEAD_DIM // group)


def _layout(record: int):
    """(groups per token, K meta, V scale and V zero offsets) of a record size."""
    ng = (record - 1024) // 128
    if record != 1024 + 128 * ng or ng not in (1, 4):
        raise ValueError("unknown record size")
    return ng, 1024, 1024 + 64 * ng, 1024 + 96 * ng


# --------------------------------------------------------------------------- inputs
def bf16_to_f64(bits: np.ndarray) -> np.ndarray:
    """bf16 bit patterns (uint16) to fp64 values (exact)."""
    u = np.ascontiguousarray(bits, dtype=np.uint16).astype(np.uint32) << 16
    return u.view(np.float32).astype(np.float64)


# --------------------------------------------------------------------------- rotation
def mu_rot(R_k: np.ndarray, mu: np.ndarray) -> np.ndarray:
    """Rotated key mean mu_h R_{K,h} per KV head (fp64), the constant subtracted after rotation
    in the cache-write formulation (Sec. 6 efficiency analysis; appendix key-mean application)."""
    return np.einsum("hi,hic->hc", mu.astype(np.float64), R_k.astype(np.float64))


def center_rotate(k_bits: np.ndarray, mu: np.ndarray, R_k: np.ndarray) -> np.ndarray:
    """(k - mu) R_K per token and KV head, fp64 (Sec. 4.1 reparameterization). k: [n, H, 128]."""
    k = bf16_to_f64(k_bits) - mu.astype(np.float64)[None]
    return np.stack([k[:, h] @ R_k[h].astype(np.float64) for h in range(k.shape[1])], axis=1)


def rotate(v_bits: np.ndarray, R_v: np.ndarray) -> np.ndarray:
    """v R_V per token and KV head, fp64. v: [n, H, 128]."""
    v = bf16_to_f64(v_bits)
    return np.stack([v[:, h] @ R_v[h].astype(np.float64) for h in range(v.shape[1])], axis=1)


# --------------------------------------------------------------------------- quantizer
def quantize(x: np.ndarray, clip: float = 1.0, group: int = GROUP):
    """Group-wise affine INT2 quantization of fp32 rows (last axis 128, groups of `group`).

    Returns (codes uint8 [..., 128], s float16 [..., 128/group], z float16 [..., 128/group])."""
    x = np.asarray(x, dtype=np.float32)
    if x.shape[-1] != HEAD_DIM:
        raise ValueError("last axis must be 128")
    if group not in GROUP_SIZES:
        raise ValueError("group size must be 32 or 128")
    xg = x.reshape(x.shape[:-1] + (HEAD_DIM // group, group))
    mn = xg.min(axis=-1)
    mx = xg.max(axis=-1)
    if clip != 1.0:
        c = np.float32(clip)
        mn = (c * mn).astype(np.float32)
        mx = (c * mx).astype(np.float32)
    s32 = (mx - mn).astype(np.float32) / np.float32(3.0)
    s = s32.astype(np.float16)
    z = mn.astype(np.float16)
    if not (np.all(np.isfinite(s)) and np.all(np.isfinite(z))):
        raise OverflowError("group range exceeds fp16 metadata")
    sf = s.astype(np.float32)
    inv = np.where(sf > 0, np.float32(1.0) / np.where(sf > 0, sf, np.float32(1.0)), np.float32(0.0))
    inv = inv.astype(np.float32)
    d = (xg - z.astype(np.float32)[..., None]).astype(np.float32)
    t = (d * inv[..., None]).astype(np.float32)
    codes = np.clip(np.rint(t), 0, 3).astype(np.uint8)
    return codes.reshape(x.shape), s, z


def dequantize(codes: np.ndarray, s: np.ndarray, z: np.ndarray) -> np.ndarray:
    """code * s + z per group, fp64 (exact); the group size follows from s (128 / s.shape[-1])."""
    ng = s.shape[-1]
    c = codes.astype(np.float64).reshape(codes.shape[:-1] + (ng, HEAD_DIM // ng))
    out = c * s.astype(np.float64)[..., None] + z.astype(np.float64)[..., None]
    return out.reshape(codes.shape)


# --------------------------------------------------------------------------- packing
def _halves_from_codes(codes: np.ndarray) -> np.ndarray:
    """[..., 128] codes -> [..., 16] uint16 halves: channel 16p+m at bits 2p of half m."""
    c = codes.astype(np.uint16).reshape(codes.shape[:-1] + (8, 16))  # (p, m)
    shifts = (2 * np.arange(8, dtype=np.uint16))[:, None]
    return np.bitwise_or.reduce(c << shifts, axis=-2).astype(np.uint16)


def _codes_from_halves(halves: np.ndarray) -> np.ndarray:
    """Inverse of _halves_from_codes."""
    h = halves.astype(np.uint16)[..., None, :]                        # (1, m)
    shifts = (2 * np.arange(8, dtype=np.uint16))[:, None]             # (p, 1)
    c = (h >> shifts) & 3
    return c.reshape(halves.shape[:-1] + (HEAD_DIM,)).astype(np.uint8)


def write_records(pool: np.ndarray, slots: np.ndarray, kc, ks, kz, vc, vs, vz) -> None:
    """Store quantized tokens into the paged pool at the byte offsets of the layout above.

    pool: uint8 [num_blocks, H, record]; slots: [n] distinct cache slots (block * 16 + row);
    kc/vc: uint8 [n, H, 128]; ks/kz/vs/vz: float16 [n, H, NG] with the pool's NG groups per token."""
    ng, off_km, off_vs, off_vz = _layout(pool.shape[-1])
    if ks.shape[-1] != ng:
        raise ValueError("metadata groups do not match the pool's record")
    slots = np.asarray(slots, dtype=np.int64)
    if np.unique(slots).size != slots.size:
        raise ValueError("slots must be distinct")
    n, H = slots.shape[0], pool.shape[1]
    blk, t = slots // BLOCK, slots % BLOCK
    B_ = blk[:, None, None]
    H_ = np.arange(H)[None, :, None]
    # K codes: 16 halves of token t at 32*t + 2*m
    kh = _halves_from_codes(kc).astype("<u2").view(np.uint8).reshape(n, H, 32)
    pool[B_, H_, (OFF_KC + 32 * t)[:, None, None] + np.arange(32)[None, None, :]] = kh
    # V codes: half m of token t at 512 + 32*m + 2*t
    vh = _halves_from_codes(vc).astype("<u2").view(np.uint8).reshape(n, H, 32)
    vidx = (OFF_VC + 2 * t)[:, None] + (32 * np.arange(16)[:, None] + np.arange(2)[None, :]).reshape(1, 32)
    pool[B_, H_, vidx[:, None, :]] = vh
    # K meta: (s, z) of group g at 1024 + 4*NG*t + 4*g
    km = np.stack([ks, kz], axis=-1).astype("<f2").view(np.uint8).reshape(n, H, 4 * ng)
    pool[B_, H_, (off_km + 4 * ng * t)[:, None, None] + np.arange(4 * ng)[None, None, :]] = km
    # V scales / zeros: group g of token t at base + 32*g + 2*t
    gidx = (32 * np.arange(ng)[:, None] + np.arange(2)[None, :]).reshape(1, 2 * ng)
    pool[B_, H_, ((off_vs + 2 * t)[:, None] + gidx)[:, None, :]] = \
        np.ascontiguousarray(vs, dtype="<f2").view(np.uint8).reshape(n, H, 2 * ng)
    pool[B_, H_, ((off_vz + 2 * t)[:, None] + gidx)[:, None, :]] = \
        np.ascontiguousarray(vz, dtype="<f2").view(np.uint8).reshape(n, H, 2 * ng)


def read_tokens(pool: np.ndarray, block_row: np.ndarray, length: int, h: int):
    """Unpack the first `length` tokens of one sequence and KV head.

    Returns (kc, ks, kz, vc, vs, vz): codes uint8 [L, 128], metadata float16 [L, NG]."""
    ng, off_km, off_vs, off_vz = _layout(pool.shape[-1])
    nblk = (length + BLOCK - 1) // BLOCK
    recs = pool[np.asarray(block_row[:nblk], dtype=np.int64), h]          # [nb, record]
    kh = recs[:, OFF_KC:OFF_VC].copy().view("<u2").reshape(nblk, BLOCK, 16)          # [nb, t, m]
    vh = recs[:, OFF_VC:off_km].copy().view("<u2").reshape(nblk, 16, BLOCK).transpose(0, 2, 1)
    km = recs[:, off_km:off_vs].copy().view("<f2").reshape(nblk, BLOCK, ng, 2)
    vs = recs[:, off_vs:off_vz].copy().view("<f2").reshape(nblk, ng, BLOCK).transpose(0, 2, 1)
    vz = recs[:, off_vz:off_vz + 32 * ng].copy().view("<f2").reshape(nblk, ng, BLOCK).transpose(0, 2, 1)
    flat = lambda a: a.reshape((nblk * BLOCK,) + a.shape[2:])[:length]
    return (flat(_codes_from_halves(kh)), flat(km[..., 0]).astype(np.float16), flat(km[..., 1]).astype(np.float16),
            flat(_codes_from_halves(vh)), flat(vs).astype(np.float16), flat(vz).astype(np.float16))


def new_pool(num_blocks: int, num_kv_heads: int, group: int = GROUP) -> np.ndarray:
    return np.zeros((num_blocks, num_kv_heads, record_bytes(group)), dtype=np.uint8)


def pool_group(pool: np.ndarray) -> int:
    """Group size of a pool, from its record size."""
    return HEAD_DIM // _layout(pool.shape[-1])[0]


# --------------------------------------------------------------------------- cache write
def quantize_pack_rotated(pool, k_rot, v_rot, slots, clip_k=1.0, clip_v=1.0):
    """Quantize already rotated (and, for keys, centered) fp32 rows and store them (groups of the
    pool's group size)."""
    G = pool_group(pool)
    kc, ks, kz = quantize(k_rot, clip_k, G)
    vc, vs, vz = quantize(v_rot, clip_v, G)
    write_records(pool, slots, kc, ks, kz, vc, vs, vz)
    return kc, ks, kz, vc, vs, vz


def quantize_append(pool, k_bits, v_bits, slots, R_k, R_v, mu, clip_k=1.0, clip_v=1.0):
    """Cache write of Sec. 4.1 / Sec. 6: (k - mu) R_K and v R_V, each rounded once to fp32,
    group-quantized to INT2 and stored at the given slots. Returns the fp32 rotated rows too."""
    k_rot = center_rotate(k_bits, mu, R_k).astype(np.float32)
    v_rot = rotate(v_bits, R_v).astype(np.float32)
    q = quantize_pack_rotated(pool, k_rot, v_rot, slots, clip_k, clip_v)
    return k_rot, v_rot, q


# --------------------------------------------------------------------------- attention
def softmax_attention(q: np.ndarray, K: np.ndarray, V: np.ndarray) -> np.ndarray:
    """eq:fp_attention and eq:head_output for a set of query rows against one KV head.

    q: [G, d], K, V: [L, d] (fp64). Returns o: [G, d]."""
    a = (q @ K.T) / np.sqrt(q.shape[-1])
    a = a - a.max(axis=-1, keepdims=True)
    p = np.exp(a)
    p /= p.sum(axis=-1, keepdims=True)
    return p @ V


def attention_probs(q: np.ndarray, K: np.ndarray) -> np.ndarray:
    """softmax_s(<q, k_s>/sqrt(d)) (fp64), eq:fp_attention."""
    a = (q @ K.T) / np.sqrt(q.shape[-1])
    a = a - a.max(axis=-1, keepdims=True)
    p = np.exp(a)
    return p / p.sum(axis=-1, keepdims=True)


def effective_kv(pool, block_row, length, h, R_k, R_v):
    """Effective INT2 keys and values of eq:rotated_int2_map: k~ = Q2((k-mu)R_K) R_K^T and
    v~ = Q2(v R_V) R_V^T, read back from the packed cache (fp64, [L, 128] each)."""
    kc, ks, kz, vc, vs, vz = read_tokens(pool, block_row, length, h)
    k_hat = dequantize(kc, ks, kz)
    v_hat = dequantize(vc, vs, vz)
    return k_hat @ R_k[h].astype(np.float64).T, v_hat @ R_v[h].astype(np.float64).T


def decode(pool, q_bits, block_table, ctx_lens, R_k, R_v, W_o_bits=None, heads_out=False):
    """INT2 decode attention of eq:int2_attention and eq:int2_residual_readout.

    q_bits: bf16 [B, H_q, 128]; block_table: [B, max_blocks]; ctx_lens: [B];
    W_o_bits: bf16 [d_model, H_q*128] or None.
    Returns fp64 o [B, H_q, 128] when W_o_bits is None, else y [B, d_model]
    (and o as well when heads_out is set)."""
    q = bf16_to_f64(q_bits)
    B, Hq, d = q.shape
    H = R_k.shape[0]
    gq = Hq // H
    o = np.zeros((B, Hq, d), dtype=np.float64)
    for b in range(B):
        L = int(ctx_lens[b])
        if L == 0:
            continue
        for h in range(H):
            Kt, Vt = effective_kv(pool, block_table[b], L, h, R_k, R_v)
            js = slice(h * gq, (h + 1) * gq)
            o[b, js] = softmax_attention(q[b, js], Kt, Vt)
    if W_o_bits is None:
        return o
    y = o.reshape(B, Hq * d) @ bf16_to_f64(W_o_bits).T
    return (y, o) if heads_out else y


def fold_wo(W_o_bits: np.ndarray, R_v: np.ndarray, num_q_heads: int) -> np.ndarray:
    """W-bar_{O,j} = W_{O,j} R_{V,h(j)} per query head (appendix, equivalent inference
    implementation). Returns fp64 [d_model, H_q*128]."""
    W = bf16_to_f64(W_o_bits)
    H = R_v.shape[0]
    gq = num_q_heads // H
    out = np.empty_like(W)
    for j in range(num_q_heads):
        cols = slice(j * HEAD_DIM, (j + 1) * HEAD_DIM)
        out[:, cols] = W[:, cols] @ R_v[j // gq].astype(np.float64)
    return out


# --------------------------------------------------------------------------- BF16 windows
# Sec. 4.1 and the implementation details of Sec. 5 keep the sink tokens (the first 64) and the
# recent tokens (the last 256) out of INT2: their keys keep the centering and are stored in BF16,
# their values are stored unchanged. Decode attends to the union of those window tokens and the
# INT2 tokens; the softmax runs over all of them (the order of tokens does not matter). Readings
# used here and by the library: the window row of a key is bf16_rne(fp32(k - mu)) in the model's
# basis (R_K is orthogonal, so scores in either basis agree), the value row is v's bf16 bits.
def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """fp32 values to bf16 bit patterns, round to nearest even (NaN not expected)."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32).astype(np.uint64)
    r = (u + 0x7FFF + ((u >> 16) & 1)) >> 16
    return r.astype(np.uint16)


def f64_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """fp64 values to bf16 bit patterns, rounded once to nearest even (NaN and overflow not
    expected). The value is scaled by a power of two onto its bf16 quantum (8 significant bits for
    normal values, 2^-133 below 2^-126), rounded to an integer with np.rint (ties to even, exact in
    fp64), and scaled back; the result is an fp32 value whose upper 16 bits are the bf16 pattern."""
    x = np.asarray(x, dtype=np.float64)
    _, e = np.frexp(x)                        # |x| in [2^(e-1), 2^e)
    q = np.ldexp(1.0, np.maximum(e, -125) - 8)  # bf16 quantum at x's binade
    r = np.rint(x / q) * q
    u = r.astype(np.float32).view(np.uint32)
    return (u >> 16).astype(np.uint16)


def rope_values(k_bits: np.ndarray, positions: np.ndarray, cos_sin: np.ndarray) -> np.ndarray:
    """RoPE of bf16 rows at their positions, fp64 and unrounded (rotate-half pairing of the
    reading above). k_bits: [n, H, 128]; positions: int [n]; cos_sin: fp32 [max_pos, 128]."""
    x = bf16_to_f64(k_bits)
    cs = np.asarray(cos_sin, dtype=np.float64)[np.asarray(positions, dtype=np.int64)]  # [n, 128]
    c, s = cs[:, None, :HEAD_DIM // 2], cs[:, None, HEAD_DIM // 2:]
    x1, x2 = x[..., :HEAD_DIM // 2], x[..., HEAD_DIM // 2:]
    return np.concatenate([x1 * c - x2 * s, x2 * c + x1 * s], axis=-1)


def rope(k_bits: np.ndarray, positions: np.ndarray, cos_sin: np.ndarray) -> np.ndarray:
    """Post-RoPE keys as bf16 bit patterns: rope_values rounded once to bf16."""
    return f64_to_bf16_bits(rope_values(k_bits, positions, cos_sin))


def hadamard(n: int = HEAD_DIM) -> np.ndarray:
    """The normalized Sylvester Hadamard matrix H_n / sqrt(n) (fp64): entry (i, j) is
    (-1)^popcount(i & j) / sqrt(n). Orthogonal and symmetric; the QuaRot base rotation."""
    i = np.arange(n)
    bits = np.bitwise_and(i[:, None], i[None, :])
    parity = np.zeros_like(bits)
    while np.any(bits):
        parity ^= bits & 1
        bits >>= 1
    return np.where(parity == 1, -1.0, 1.0) / np.sqrt(n)


def quantize_append_rope(pool, k_bits, v_bits, slots, positions, cos_sin, R_k, R_v, mu, clip_k=1.0, clip_v=1.0):
    """Cache write fed with pre-RoPE keys: the keys are first turned into their post-RoPE bf16
    rows (rope above), then written as quantize_append writes them ((k - mu) R_K, v R_V)."""
    quantize_append(pool, rope(k_bits, positions, cos_sin), v_bits, slots, R_k, R_v, mu, clip_k, clip_v)


def window_write(win_k: np.ndarray, win_v: np.ndarray, k_bits: np.ndarray, v_bits: np.ndarray,
                 mu: np.ndarray, rows: np.ndarray) -> None:
    """Store tokens into the BF16 window. win_k, win_v: uint16 [n_rows, H, 128]; k_bits, v_bits:
    bf16 [n, H, 128]; mu: fp32 [H, 128] key mean (model basis); rows[i] < 0 skips token i."""
    k32 = bf16_to_f64(k_bits).astype(np.float32) - np.asarray(mu, dtype=np.float32)[None]
    kc = f32_to_bf16_bits(k32)
    for i, r in enumerate(np.asarray(rows)):
        if r < 0:
            continue
        win_k[r] = kc[i]
        win_v[r] = v_bits[i]


def decode_window(pool, q_bits, block_table, ctx_lens, R_k, R_v, win_k, win_v, win_lens,
                  W_o_bits=None):
    """Decode over the INT2 tokens of each sequence (as `decode`) together with its window tokens.

    win_k, win_v: uint16 [B, cap, H, 128] (window row b * cap + t holds token t of sequence b, as
    written by window_write); win_lens: [B] tokens in each sequence's window, clamped to [0, cap] (a
    count outside that range means an empty or a full window). Returns fp64 o [B, H_q, 128], or
    y [B, d_model] with W_o_bits."""
    q = bf16_to_f64(q_bits)
    B, Hq, d = q.shape
    H = R_k.shape[0]
    gq = Hq // H
    o = np.zeros((B, Hq, d), dtype=np.float64)
    for b in range(B):
        L, W = int(ctx_lens[b]), min(max(int(win_lens[b]), 0), win_k.shape[1])
        for h in range(H):
            Ks = [bf16_to_f64(win_k[b, :W, h])]
            Vs = [bf16_to_f64(win_v[b, :W, h])]
            if L > 0:
                Kt, Vt = effective_kv(pool, block_table[b], L, h, R_k, R_v)
                Ks.append(Kt)
                Vs.append(Vt)
            K, V = np.concatenate(Ks), np.concatenate(Vs)
            if K.shape[0] == 0:
                continue
            js = slice(h * gq, (h + 1) * gq)
            o[b, js] = softmax_attention(q[b, js], K, V)
    if W_o_bits is None:
        return o
    return o.reshape(B, Hq * d) @ bf16_to_f64(W_o_bits).T


# --------------------------------------------------------------------------- output-error diagnostics
# Sec. 3.2 traces the INT2 cache through attention and W_O: with full-precision keys and values
# (k, v) the head output is y_j = (p_j^T V) W_{O,j}^T; with the cache's effective INT2 keys and
# values it is y~_j = (p~_j^T V~) W_{O,j}^T, and the difference splits exactly into a key-induced
# term (through the attention distribution) and a value-induced term:
#     dy_K = ((p~ - p)^T V) W_{O,j}^T,   dy_V = (p~^T (V~ - V)) W_{O,j}^T,   y~ - y = dy_K + dy_V.
# E_out = ||y~ - y||^2 (eq:output_error_objective) and E_rec = ||K - K~||_F^2 + ||V - V~||_F^2
# (eq:raw_reconstruction_objective); the appendix reports the RMS output error of a method as a
# percentage of plain INT2 (no rotation, no centering, no clipping): 100 sqrt(err / err_plain).
def output_error(pool, k_list, v_list, q_bits, ctx_lens, block_table, R_k, R_v, mu, W_o_bits):
    """Per (sequence b, query head j) output errors of the INT2 cache `pool` against the
    full-precision keys and values it was written from (k_list[b], v_list[b]: bf16 [L_b, H, 128]).

    Returns (dyK, dyV, stats): dyK, dyV fp64 [B, H_q, d_model]; stats fp64 [B, H_q, 4] =
    (||dy_K + dy_V||^2, ||dy_K||^2, ||dy_V||^2, <dy_K, dy_V>). Sequences with no token give zeros."""
    q = bf16_to_f64(q_bits)
    B, Hq, d = q.shape
    H = R_k.shape[0]
    gq = Hq // H
    W = bf16_to_f64(W_o_bits)
    dm = W.shape[0]
    dyK = np.zeros((B, Hq, dm))
    dyV = np.zeros((B, Hq, dm))
    for b in range(B):
        L = int(ctx_lens[b])
        if L == 0:
            continue
        K_all = bf16_to_f64(k_list[b])[:L]
        V_all = bf16_to_f64(v_list[b])[:L]
        for h in range(H):
            Kc, Vt = effective_kv(pool, block_table[b], L, h, R_k, R_v)
            Kt = Kc + mu[h].astype(np.float64)          # k~ = k^ R_K^T + mu
            K, V = K_all[:, h], V_all[:, h]
            for j in range(h * gq, (h + 1) * gq):
                p = attention_probs(q[b, j][None], K)[0]
                pt = attention_probs(q[b, j][None], Kt)[0]
                Wj = W[:, j * HEAD_DIM:(j + 1) * HEAD_DIM]
                dyK[b, j] = ((pt - p) @ V) @ Wj.T
                dyV[b, j] = (pt @ (Vt - V)) @ Wj.T
    dy = dyK + dyV
    stats = np.stack([(dy * dy).sum(-1), (dyK * dyK).sum(-1), (dyV * dyV).sum(-1), (dyK * dyV).sum(-1)], axis=-1)
    return dyK, dyV, stats


def reconstruction_error(pool, k_bits, v_bits, slots, R_k, R_v, mu):
    """Per token and KV head: (||k - k~||^2, ||v - v~||^2) of tokens stored at `slots`, with
    k~ = k^ R_K^T + mu and v~ = v^ R_V^T read back from the pool (fp64, [n, H, 2])."""
    k = bf16_to_f64(k_bits)
    v = bf16_to_f64(v_bits)
    n, H = k.shape[0], k.shape[1]
    blocks = np.asarray(slots, dtype=np.int64) // BLOCK
    rows = np.asarray(slots, dtype=np.int64) % BLOCK
    out = np.zeros((n, H, 2))
    for h in range(H):
        for i in range(n):
            kc, ks, kz, vc, vs, vz = read_tokens(pool, np.array([blocks[i]]), BLOCK, h)
            kt = dequantize(kc, ks, kz)[rows[i]] @ R_k[h].astype(np.float64).T + mu[h].astype(np.float64)
            vt = dequantize(vc, vs, vz)[rows[i]] @ R_v[h].astype(np.float64).T
            out[i, h, 0] = ((k[i, h] - kt) ** 2).sum()
            out[i, h, 1] = ((v[i, h] - vt) ** 2).sum()
    return out


def rms_percent(err, err_plain):
    """RMS output error of a method as a percentage of plain INT2's (appendix per-head metric)."""
    return 100.0 * np.sqrt(np.asarray(err, dtype=np.float64) / np.asarray(err_plain, dtype=np.float64))
