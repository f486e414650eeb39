"""Bit-exact GPU parity of the quantizer inside the product cache writes (int2kv_quantize_append and
the cache write fused into int2kv_append_decode) against the oracle.

The quantizer's contract is bit-exactness when it is fed the same rotated tensor. The product
writes rotate on the matrix cores (R split into three bf16 terms, fp32 accumulation from -mu R_K),
so to feed both sides the same fp32 rotated rows, R_K and R_V here are signed permutation matrices:
every product is an exact signed copy of an input, the fp32 accumulation adds one non-zero term
to -mu R_K, and the oracle's fp64 (k - mu) R rounded once to fp32 is the same number. The rotated
rows are built first, group by group, from patterns that reach the quantizer's corner cases:
exact rounding ties of the code, fp16 rounding ties of the scale, grid-exact groups, degenerate
groups, huge ranges, fp16-subnormal scales and zeros; the inputs are those rows rotated back.
With mu = 0 the rotated rows are the patterns exactly; with a key mean whose subtraction is exact
in fp32 the key centering is checked bit for bit too. Pool bytes must equal the oracle's pool
bytes everywhere (Sec. 5 implementation details: group-wise affine INT2; Sec. 4.1 key
reparameterization; the packed layout of include/int2kv.h). With an arbitrary fp32 key mean the
rotated rows may differ in the last bit (the matrix cores' fp32 accumulation is not the oracle's
single rounding), and the cache write is checked up to rounding ties like every other one."""
import numpy as np
import pytest
import torch

from oracle import int2kv_oracle as O
from paper_2608_02691_amd import int2kv as K

from _helpers import compare_cache_writes, dev

pytestmark = pytest.mark.gpu


@pytest.fixture(autouse=True)
def _default_tuning():
    K.int2kv_set_decode_tuning(0, 0)
    yield
    K.int2kv_set_decode_tuning(0, 0)


def signed_permutations(rng, H):
    """R[h] with one +-1 per row and column (z R is a signed permutation of z's channels)."""
    R = np.zeros((H, 128, 128), np.float32)
    for h in range(H):
        R[h, np.arange(128), rng.permutation(128)] = rng.choice(np.float32([-1.0, 1.0]), 128)
    return R


def bf16_round(x):
    return O.bf16_to_f64(O.f32_to_bf16_bits(np.asarray(x, np.float32))).astype(np.float32)


N_PATTERNS = 10


def group_pattern(rng, kind, G):
    """G bf16-exact fp32 values of one rotated group (never an exact zero minimum, so the sign of a
    zero cannot differ between an fp32 sum and the oracle's fp64 product)."""
    if kind == 0:    # generic, scale spread over four decades
        return bf16_round(rng.standard_normal(G) * 10.0 ** rng.uniform(-2, 2))
    if kind == 1:    # grid-exact: z = -1.25, s = 0.5, every code present
        c = rng.integers(0, 4, G)
        c[:4] = [0, 3, 1, 2]
        return (-1.25 + 0.5 * c).astype(np.float32)
    if kind == 2:    # exact code ties: mn = 1, mx = 4 (s = 1, z = 1); t = 0.5, 1.5, 2.5 round to even
        x = rng.choice(np.float32([1.0, 1.5, 2.0, 2.5, 3.0, 3.5, 4.0]), G)
        x[:2] = [1.0, 4.0]
        return x
    if kind == 3:    # fp16 tie of the scale: (mx - mn) / 3 = 1 + 2^-11 exactly (rounds to 1.0)
        x = bf16_round(rng.uniform(0.0, 3.0, G))
        x[:2] = [3.0, -3.0 * 2.0 ** -11]
        return x
    if kind == 4:    # fp16-subnormal scale: range 3 * 2^-20 above 2^-18
        x = (2.0 ** -18 + rng.integers(0, 7, G) * 2.0 ** -21).astype(np.float32)
        x[:2] = [2.0 ** -18, 2.0 ** -18 + 3 * 2.0 ** -20]
        return x
    if kind == 5:    # huge range (s ~ 2e4, still an fp16 number)
        return bf16_round(rng.uniform(-30000, 30000, G))
    if kind == 6:    # degenerate group: s = 0, all codes 0
        return np.full(G, 0.75, np.float32)
    if kind == 7:    # tiny values: zero and scale rounded in fp16's subnormal range
        return bf16_round(rng.uniform(3 * 2.0 ** -26, 1e-5, G))
    if kind == 8:    # far from zero: a large offset with a small spread
        return bf16_round(200.0 + rng.standard_normal(G))
    # kind 9: two values only (codes 0 and 3), negative
    return rng.choice(np.float32([-7.5, -2.25]), G)


def make_inputs(seed, n, H, G, mu_kind):
    """(k, v, R_k, R_v, mu) for n tokens: rotated rows from the patterns, rotated back.

    mu_kind "zero": mu = 0, the rotated rows are the patterns exactly. "exact": mu holds multiples
    of 2^-4 in [-16, 16) and k = bf16(rows R^T + mu), with every key element whose k - mu is not an
    fp32 number replaced by 2 mu: the centering subtraction is then exact on both sides (the matrix
    cores' fp32 accumulation need not round like the oracle's single fp64 -> fp32 rounding, so only
    exact sums can be compared bit for bit). "float": mu is an arbitrary fp32 vector."""
    rng = np.random.default_rng(seed)
    R_k, R_v = signed_permutations(rng, H), signed_permutations(rng, H)
    ng = 128 // G
    rows = np.empty((2, n, H, 128), np.float32)
    for kv in range(2):
        for t in range(n):
            for h in range(H):
                for g in range(ng):
                    kind = (kv + 3 * t + 5 * h + 7 * g) % N_PATTERNS
                    rows[kv, t, h, g * G:(g + 1) * G] = group_pattern(rng, kind, G)
    # x R = rows  <=>  x = rows R^T (exact: a signed permutation of bf16 values)
    k = np.einsum("thc,hic->thi", rows[0], R_k).astype(np.float32)
    v = np.einsum("thc,hic->thi", rows[1], R_v).astype(np.float32)
    if mu_kind == "zero":
        mu = np.zeros((H, 128), np.float32)
    elif mu_kind == "exact":
        mu = (rng.integers(-256, 256, (H, 128)) / 16.0).astype(np.float32)
        k = bf16_round(k + mu[None])
        d = k.astype(np.float64) - mu[None].astype(np.float64)
        inexact = d.astype(np.float32).astype(np.float64) != d
        k = np.where(inexact, 2 * mu[None], k).astype(np.float32)
    else:
        mu = (rng.standard_normal((H, 128)) * 3.0).astype(np.float32)
        k = k + mu[None]
    return O.f32_to_bf16_bits(k), O.f32_to_bf16_bits(v), R_k, R_v, mu


def oracle_bytes(num_blocks, H, G, k, v, slots, R_k, R_v, mu, clip):
    pool = O.new_pool(num_blocks, H, G)
    keep = slots >= 0
    O.quantize_append(pool, k[keep], v[keep], slots[keep], R_k, R_v, mu, *clip)
    return pool


CLIPS = [(1.0, 1.0), (0.96, 0.92)]


@pytest.mark.parametrize("mu_kind", ["zero", "exact"])
@pytest.mark.parametrize("clip", CLIPS, ids=lambda c: f"clip{c[0]}-{c[1]}")
@pytest.mark.parametrize("G", [32, 128])
@pytest.mark.parametrize("n,H", [(37, 2), (1000, 2), (2500, 8)], ids=["short", "medium", "long2tile"])
def test_quantize_append_is_bit_exact(n, H, G, clip, mu_kind):
    """Standalone cache write: one tile per wave step (short and medium appends) and two tiles per
    step (long appends at 8 KV heads), tokens stored to scattered slots, one skipped."""
    print(f"\n[append exact] n={n} H={H} G={G} clip={clip} mu={mu_kind}", flush=True)
    k, v, R_k, R_v, mu = make_inputs(100 + n + G, n, H, G, mu_kind)
    num_blocks = (n + 15) // 16 + 3
    rng = np.random.default_rng(5)
    slots = rng.permutation(num_blocks * 16)[:n].astype(np.int32)
    slots[n // 3] = -1
    ref = oracle_bytes(num_blocks, H, G, k, v, slots, R_k, R_v, mu, clip)
    cache = K.Int2KVCache(num_blocks, H, group_size=G)
    Rk, Rv = dev(R_k), dev(R_v)
    mu_rk = K.int2kv_prepare_mu_rot(Rk, dev(mu))
    K.int2kv_quantize_append(cache, dev(k), dev(v), dev(slots), Rk, Rv, mu_rk, *clip)
    got = cache.pool.cpu().numpy()
    diff = np.argwhere(got != ref)
    assert diff.size == 0, f"{len(diff)} pool bytes differ, first (block, head, byte) {diff[:4].tolist()}"


@pytest.mark.parametrize("mu_kind", ["zero", "exact"])
@pytest.mark.parametrize("clip", CLIPS, ids=lambda c: f"clip{c[0]}-{c[1]}")
@pytest.mark.parametrize("G", [32, 128])
def test_append_decode_cache_write_is_bit_exact(G, clip, mu_kind):
    """The cache write inside int2kv_append_decode's preparation launch (<= 256 tokens): 200 current
    tokens of 5 sequences at 8 KV heads, 40 query heads, then a decode over them."""
    print(f"\n[append_decode exact] G={G} clip={clip} mu={mu_kind}", flush=True)
    H, Hq, n = 8, 40, 200
    k, v, R_k, R_v, mu = make_inputs(300 + G, n, H, G, mu_kind)
    lens = np.array([40, 40, 40, 40, 40], np.int32)
    B = lens.size
    num_blocks = 20
    rng = np.random.default_rng(9)
    table = rng.permutation(num_blocks)[:B * 3].reshape(B, 3).astype(np.int32)
    slots = np.concatenate([table[b, np.arange(40) // 16] * 16 + np.arange(40) % 16 for b in range(B)])
    slots = slots.astype(np.int32)
    ref = oracle_bytes(num_blocks, H, G, k, v, slots, R_k, R_v, mu, clip)
    cache = K.Int2KVCache(num_blocks, H, group_size=G)
    Rk, Rv = dev(R_k), dev(R_v)
    mu_rk = K.int2kv_prepare_mu_rot(Rk, dev(mu))
    q = O.f32_to_bf16_bits(rng.standard_normal((B, Hq, 128)).astype(np.float32))
    out = K.int2kv_append_decode(cache, dev(k), dev(v), dev(slots), mu_rk, dev(q), dev(table), dev(lens), 48,
                                 Rk, Rv, clip_k=clip[0], clip_v=clip[1])
    torch.cuda.synchronize()
    got = cache.pool.cpu().numpy()
    diff = np.argwhere(got != ref)
    assert diff.size == 0, f"{len(diff)} pool bytes differ, first (block, head, byte) {diff[:4].tolist()}"
    assert torch.isfinite(out).all()


@pytest.mark.parametrize("clip", CLIPS, ids=lambda c: f"clip{c[0]}-{c[1]}")
@pytest.mark.parametrize("G", [32, 128])
def test_quantize_append_with_fp32_key_mean_up_to_ties(G, clip):
    """An arbitrary fp32 key mean: the library's fp32 accumulation of -mu R_K + k R_K may differ from
    the oracle's correctly rounded (k - mu) R_K in the last bit, so codes may differ only at
    rounding ties (and scales or zeros by one fp16 ulp), at most 1e-4 of them."""
    n, H = 2500, 8
    k, v, R_k, R_v, mu = make_inputs(700 + G, n, H, G, "float")
    num_blocks = (n + 15) // 16 + 3
    slots = np.random.default_rng(5).permutation(num_blocks * 16)[:n].astype(np.int32)
    ref = oracle_bytes(num_blocks, H, G, k, v, slots, R_k, R_v, mu, clip)
    cache = K.Int2KVCache(num_blocks, H, group_size=G)
    Rk, Rv = dev(R_k), dev(R_v)
    mu_rk = K.int2kv_prepare_mu_rot(Rk, dev(mu))
    K.int2kv_quantize_append(cache, dev(k), dev(v), dev(slots), Rk, Rv, mu_rk, *clip)
    k_rot = O.center_rotate(k, mu, R_k).astype(np.float32)
    v_rot = O.rotate(v, R_v).astype(np.float32)
    stats = compare_cache_writes(cache.pool.cpu().numpy(), ref, slots, k_rot, v_rot)
    print(stats, flush=True)
