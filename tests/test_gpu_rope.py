"""GPU parity of the fused RoPE cache write and the Hadamard base rotation against the CPU
oracle: post-RoPE keys bit for bit, cache bytes up to rounding ties, the identities that tie the
new entry point to the plain cache write, and a decode over a Hadamard-written cache."""
import numpy as np
import pytest
import torch

from oracle import int2kv_oracle as O
from paper_2608_02691_amd import int2kv as K
from paper_2608_02691_amd import workloads as W

from _helpers import assert_rows_close, compare_cache_writes, dev, gpu_cache

pytestmark = pytest.mark.gpu

MAX_POS = 40000


def _tokens(w):
    ks, vs, slots = [], [], []
    for b in range(w.batch):
        k, v = w.kv(b)
        ks.append(k)
        vs.append(v)
        slots.append(w.slot_mapping(b))
    return np.concatenate(ks), np.concatenate(vs), np.concatenate(slots)


def _hadamard_np(H):
    return np.broadcast_to(O.hadamard(128), (H, 128, 128)).copy()


@pytest.mark.parametrize("G", [32, 128])
@pytest.mark.parametrize("clip", [(1.0, 1.0), (0.96, 0.92)])
@pytest.mark.parametrize("had", [0, 3])
def test_rope_write_matches_oracle(had, clip, G):
    print(f"\n[rope write] hadamard={had} clip={clip} G={G}", flush=True)
    w = W.make_workload(1, batch=3, ctx=None, ctx_lens=np.array([150, 1, 77]), num_q_heads=8, num_kv_heads=4)
    k, v, slots = _tokens(w)
    n = len(slots)
    rng = np.random.default_rng(123 + had + G)
    pos = rng.integers(0, MAX_POS, n).astype(np.int32)
    pos[0], pos[1] = 0, MAX_POS - 1
    pos[5], pos[9] = -1, MAX_POS  # outside the table: skipped
    cs = W.rope_cos_sin(MAX_POS)
    if had:
        R_k = R_v = _hadamard_np(w.num_kv_heads)
        Rd = K.hadamard_rotation(w.num_kv_heads)
        mu_rk = K.int2kv_prepare_mu_rot(Rd, dev(w.mu))
        gk = gv = None
    else:
        R_k, R_v = w.R_k, w.R_v
        mu_rk = K.int2kv_prepare_mu_rot(dev(w.R_k), dev(w.mu))
        gk, gv = dev(w.R_k), dev(w.R_v)
    cache = gpu_cache(O.new_pool(w.num_blocks, w.num_kv_heads, G))
    k_out = torch.full((n, w.num_kv_heads, 128), 0x1234, dtype=torch.int16, device="cuda")
    K.int2kv_quantize_append_rope(cache, dev(k), dev(v), dev(slots), dev(pos), dev(cs), gk, gv, mu_rk, *clip,
                                  flags=had, k_rope_out=k_out)
    got_k = k_out.cpu().numpy().view(np.uint16)
    keep = (pos >= 0) & (pos < MAX_POS)
    ref_k = O.rope(k[keep], pos[keep], cs)
    assert np.array_equal(got_k[keep], ref_k), "post-RoPE keys must be bit-exact"
    assert np.all(got_k[~keep] == 0x1234), "skipped tokens leave k_rope_out untouched"
    ref = O.new_pool(w.num_blocks, w.num_kv_heads, G)
    k_rot, v_rot, _ = O.quantize_append(ref, ref_k, v[keep], slots[keep], R_k, R_v, w.mu, *clip)
    pool = cache.pool.cpu().numpy()
    stats = compare_cache_writes(pool, ref, slots[keep], k_rot, v_rot)
    print(f"cache write vs oracle: {stats}", flush=True)
    # skipped tokens' slots hold nothing
    blk, row = slots[~keep] // 16, slots[~keep] % 16
    for b_, r_ in zip(blk, row):
        rec = pool[b_]
        assert not rec[:, 32 * r_:32 * r_ + 32].any()


@pytest.mark.parametrize("G", [32, 128])
def test_rope_write_reduces_to_plain_write(G):
    """At position 0 (cos 1, sin 0), and without positions, the fused write stores exactly the bytes
    of int2kv_quantize_append."""
    print(f"\n[rope write] identities G={G}", flush=True)
    w = W.make_workload(1, batch=2, ctx=None, ctx_lens=np.array([200, 33]), num_q_heads=8, num_kv_heads=8)
    k, v, slots = _tokens(w)
    mu_rk = K.int2kv_prepare_mu_rot(dev(w.R_k), dev(w.mu))
    args = (dev(k), dev(v), dev(slots))
    plain = gpu_cache(O.new_pool(w.num_blocks, w.num_kv_heads, G))
    K.int2kv_quantize_append(plain, *args, dev(w.R_k), dev(w.R_v), mu_rk, 0.96, 0.92)
    for positions in (dev(np.zeros(len(slots), np.int32)), None):
        c = gpu_cache(O.new_pool(w.num_blocks, w.num_kv_heads, G))
        K.int2kv_quantize_append_rope(c, *args, positions, dev(W.rope_cos_sin(8)) if positions is not None else None,
                                      dev(w.R_k), dev(w.R_v), mu_rk, 0.96, 0.92)
        assert torch.equal(c.pool, plain.pool)


def test_hadamard_write_then_decode_matches_oracle():
    """A cache written with the in-kernel Hadamard rotation, decoded with the dense Hadamard matrix
    (with and without W_O): the decode's parity against the oracle over that cache."""
    print("\n[hadamard] write + decode", flush=True)
    w = W.make_workload(1, batch=3, ctx=None, ctx_lens=np.array([700, 64, 129]), num_q_heads=16, num_kv_heads=4,
                        d_model=256)
    k, v, slots = _tokens(w)
    Rd = K.hadamard_rotation(w.num_kv_heads)
    mu_rk = K.int2kv_prepare_mu_rot(Rd, dev(w.mu))
    cache = gpu_cache(O.new_pool(w.num_blocks, w.num_kv_heads))
    K.int2kv_quantize_append_rope(cache, dev(k), dev(v), dev(slots), None, None, None, None, mu_rk,
                                  flags=K.INT2KV_HADAMARD_K | K.INT2KV_HADAMARD_V)
    ref = O.new_pool(w.num_blocks, w.num_kv_heads)
    Hn = _hadamard_np(w.num_kv_heads)
    k_rot, v_rot, _ = O.quantize_append(ref, k, v, slots, Hn, Hn, w.mu)
    pool = cache.pool.cpu().numpy()
    print(compare_cache_writes(pool, ref, slots, k_rot, v_rot), flush=True)
    H32 = Rd.cpu().numpy()
    for dm in (0, 256):
        out_ref = O.decode(pool, w.q, w.block_table, w.ctx_lens, H32, H32, w.W_o if dm else None)
        out = K.int2kv_decode(cache, dev(w.q), dev(w.block_table), dev(w.ctx_lens), int(w.ctx_lens.max()), Rd, Rd,
                              W_o=dev(w.W_o) if dm else None)
        assert_rows_close(out.cpu().numpy(), out_ref, what=f"decode over the Hadamard cache (d_model={dm})")
