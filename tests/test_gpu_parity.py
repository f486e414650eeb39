"""GPU parity of the HIP library (through the C ABI) against the CPU oracle, at sizes the oracle
finishes in seconds: several tiles, ragged tails, GQA ratios 1/4/5, empty and one-token
contexts, clipping, degenerate groups."""
import numpy as np
import pytest
import torch

from oracle import int2kv_oracle as O
from paper_2608_02691_amd import int2kv as K
from paper_2608_02691_amd import workloads as W

from _helpers import (assert_rows_close, compare_cache_writes, dev, gpu_cache, oracle_pool)

pytestmark = pytest.mark.gpu


@pytest.fixture(autouse=True)
def _default_tuning():
    K.int2kv_set_decode_tuning(0, 0)
    yield
    K.int2kv_set_decode_tuning(0, 0)


def _rotated_rows(w):
    ks, vs, slots = [], [], []
    for b in range(w.batch):
        k, v = w.kv(b)
        ks.append(O.center_rotate(k, w.mu, w.R_k).astype(np.float32))
        vs.append(O.rotate(v, w.R_v).astype(np.float32))
        slots.append(w.slot_mapping(b))
    return np.concatenate(ks), np.concatenate(vs), np.concatenate(slots)


# ----------------------------------------------------------------------------- cache write
@pytest.mark.parametrize("G", [32, 128])
@pytest.mark.parametrize("clip", [(1.0, 1.0), (0.96, 0.92)])
def test_pack_rotated_is_bit_exact(clip, G):
    print(f"\n[pack_rotated] clip={clip} G={G}", flush=True)
    w = W.make_workload(1, batch=3, ctx=None, ctx_lens=np.array([100, 1, 47]), num_q_heads=8, num_kv_heads=8)
    k_rot, v_rot, slots = _rotated_rows(w)
    # special rows: a degenerate group, a huge-range group, exact grid values
    k_rot[0, 0, 32:64] = 0.75
    v_rot[1, 3, :32] = np.linspace(-500, 500, 32, dtype=np.float32)
    k_rot[2, 1, 64:96] = (np.arange(32) % 4).astype(np.float32) * 0.5 - 1.0
    slots_in = slots.copy()
    slots_in[5] = -1  # skipped token
    ref = O.new_pool(w.num_blocks, w.num_kv_heads, G)
    keep = slots_in >= 0
    O.quantize_pack_rotated(ref, k_rot[keep], v_rot[keep], slots_in[keep], *clip)
    cache = gpu_cache(np.zeros_like(ref))
    K.int2kv_quantize_pack_rotated(cache, dev(k_rot), dev(v_rot), dev(slots_in), *clip)
    got = cache.pool.cpu().numpy()
    assert np.array_equal(got, ref)


def test_prepare_mu_rot_matches_oracle():
    w = W.make_workload(1, batch=1, ctx=16)
    mu_rk = K.int2kv_prepare_mu_rot(dev(w.R_k), dev(w.mu)).cpu().numpy()
    ref = O.mu_rot(w.R_k, w.mu)
    assert np.abs(mu_rk - ref).max() <= 1e-5 * np.abs(ref).max()


@pytest.mark.parametrize("G", [32, 128])
@pytest.mark.parametrize("clip", [(1.0, 1.0), (0.96, 0.92)])
def test_append_matches_oracle_up_to_ties(clip, G):
    print(f"\n[append] clip={clip} G={G}", flush=True)
    w = W.make_workload(4, batch=6, ctx_lens=np.array([700, 33, 1, 16, 250, 401]))
    k_rot, v_rot, slots = _rotated_rows(w)
    ref = oracle_pool(w, clip_k=clip[0], clip_v=clip[1], group=G)
    cache = K.Int2KVCache(w.num_blocks, w.num_kv_heads, group_size=G)
    mu_rk = K.int2kv_prepare_mu_rot(dev(w.R_k), dev(w.mu))
    Rk, Rv = dev(w.R_k), dev(w.R_v)
    for b in range(w.batch):
        k, v = w.kv(b)
        K.int2kv_quantize_append(cache, dev(k), dev(v), dev(w.slot_mapping(b)), Rk, Rv, mu_rk, *clip)
    stats = compare_cache_writes(cache.pool.cpu().numpy(), ref, slots, k_rot, v_rot)
    print(stats, flush=True)


@pytest.mark.parametrize("G", [32, 128])
def test_append_one_call_many_tokens_matches_oracle(G):
    """All sequences in one call (the prefill-sized path), tokens in a shuffled order."""
    w = W.make_workload(3, batch=2, ctx=1200)
    k_rot, v_rot, slots = _rotated_rows(w)
    ref = oracle_pool(w, group=G)
    kk, vv = zip(*[w.kv(b) for b in range(w.batch)])
    k, v = np.concatenate(kk), np.concatenate(vv)
    perm = np.random.default_rng(0).permutation(slots.size)
    cache = K.Int2KVCache(w.num_blocks, w.num_kv_heads, group_size=G)
    mu_rk = K.int2kv_prepare_mu_rot(dev(w.R_k), dev(w.mu))
    K.int2kv_quantize_append(cache, dev(k[perm]), dev(v[perm]), dev(slots[perm]), dev(w.R_k), dev(w.R_v), mu_rk)
    stats = compare_cache_writes(cache.pool.cpu().numpy(), ref, slots, k_rot, v_rot)
    print(stats, flush=True)


# ----------------------------------------------------------------------------- decode
DECODE_CASES = [
    # (cfg, batch, q heads, kv heads, lens, d_model)
    (0, 1, 1, 1, [256], None),
    (1, 3, 8, 2, [1, 17, 300], None),
    (4, 2, 5, 1, [700, 64], None),
    (1, 4, 32, 8, [1000, 33, 16, 0], None),
    (4, 3, 10, 2, [1500, 2, 129], 256),
    # two batch blocks and four K slices of the output projection (K = 40 * 128)
    (4, 66, 40, 8, [17 + 5 * i for i in range(66)], 1024),
    # every head-group width of the matrix-core scan (G_q 2, 3, 6, 7, 8), two work-group rows of
    # KV heads (H_kv 16), G_q 12 (vector-ALU scan only), an output width that is no multiple of 4
    (1, 2, 16, 8, [300, 45], None),
    (1, 2, 24, 8, [77, 500], None),
    (1, 2, 48, 8, [129, 31], None),
    (1, 1, 56, 8, [400], None),
    (1, 2, 64, 8, [257, 1], None),
    (1, 2, 32, 16, [200, 64], None),
    # 12 KV heads: the second row of scan work-groups has 4 waves without a head
    (1, 2, 24, 12, [300, 45], None),
    (1, 2, 96, 8, [150, 20], None),
    (4, 2, 10, 2, [300, 17], 100),
    # 256 row blocks of the output projection: one K slice, no arrival counting
    (4, 1, 2, 1, [100], 32768),
]


@pytest.mark.parametrize("variant", [1, 2])
@pytest.mark.parametrize("chunk", [0, 64])
@pytest.mark.parametrize("case", DECODE_CASES, ids=lambda c: f"cfg{c[0]}-B{c[1]}-{c[2]}x{c[3]}-dm{c[5]}-L{max(c[4])}")
def test_decode_matches_oracle(case, chunk, variant):
    cfg, B, Hq, H, lens, dm = case
    print(f"\n[decode] case={case} chunk={chunk} variant={variant}", flush=True)
    if variant == 2 and Hq // H > 8:
        pytest.skip("the matrix-core scan serves at most 8 query heads per KV head")
    st = K.load_library().int2kv_set_decode_tuning(chunk, variant)
    if st == K.INT2KV_EUNSUPPORTED:
        pytest.skip("variant not built")
    w = W.make_workload(cfg, batch=B, ctx_lens=np.array(lens), num_q_heads=Hq, num_kv_heads=H, d_model=dm)
    pool = oracle_pool(w)
    out_ref = O.decode(pool, w.q, w.block_table, w.ctx_lens, w.R_k, w.R_v, w.W_o)
    cache = gpu_cache(pool)
    max_ctx = int(max(lens))
    args = (cache, dev(w.q), dev(w.block_table), dev(w.ctx_lens), max_ctx, dev(w.R_k), dev(w.R_v))
    out = K.int2kv_decode(*args, W_o=dev(w.W_o) if dm else None)
    worst = assert_rows_close(out.cpu().numpy(), out_ref, what="decode")
    out2 = K.int2kv_decode(*args, W_o=dev(w.W_o) if dm else None)
    assert torch.equal(out, out2), "decode must be deterministic"
    print(f"worst row error {worst:.2e}", flush=True)
    if dm:
        Wf = K.int2kv_fold_wo(dev(w.W_o), dev(w.R_v), Hq)
        out_f = K.int2kv_decode(*args, W_o=Wf, wo_is_folded=True)
        assert_rows_close(out_f.cpu().numpy(), out_ref, what="decode with folded W_O")
        for fold in (False, True):
            Wp = K.int2kv_prepare_wo(dev(w.W_o), dev(w.R_v) if fold else None, Hq, num_kv_heads=H)
            fmt = K.INT2KV_WO_PREPARED_FOLDED if fold else K.INT2KV_WO_PREPARED
            out_p = K.int2kv_decode(*args, W_o=Wp, wo_format=fmt, d_model=dm)
            assert_rows_close(out_p.cpu().numpy(), out_ref, what=f"decode with prepared W_O (fold={fold})")
            assert torch.equal(out_p, K.int2kv_decode(*args, W_o=Wp, wo_format=fmt, d_model=dm))


def test_fold_wo_matches_oracle():
    w = W.make_workload(1, batch=1, ctx=16, num_q_heads=8, num_kv_heads=2, d_model=96)
    got = K.int2kv_fold_wo(dev(w.W_o), dev(w.R_v), 8).cpu().view(torch.int16).numpy().view(np.uint16)
    ref = O.fold_wo(w.W_o, w.R_v, 8)
    g = O.bf16_to_f64(got)
    # one bf16 rounding (half an ulp: 2^-8 relative) of an fp32 accumulation of 128 products
    # (absolute error ~1e-6 of the row scale, which matters only for entries near zero)
    assert np.all(np.abs(g - ref) <= 2.0 ** -8 * np.abs(ref) + 1e-6 * np.abs(ref).max())


def _untile_prepared(flat, n_rows, k):
    """Row-major [n_rows padded to 128, k] view of prepared weights: tile (row block, k step) holds
    eight 16 x 32 sub-tiles; in sub-tile a, lane r + 16 q carries row 16 a + r, columns 8 q .. 8 q + 7."""
    npad = (n_rows + 127) // 128 * 128
    t = flat.reshape(npad // 128, k // 32, 8, 4, 16, 8)  # row block, k step, a, q, r, e
    return t.transpose(0, 2, 4, 1, 3, 5).reshape(npad, k)


@pytest.mark.parametrize("fold", [False, True])
def test_prepare_wo_layout_and_values(fold):
    Hq, H, dm = 4, 2, 200
    w = W.make_workload(1, batch=1, ctx=16, num_q_heads=Hq, num_kv_heads=H, d_model=dm)
    got = K.int2kv_prepare_wo(dev(w.W_o), dev(w.R_v) if fold else None, Hq, num_kv_heads=H).cpu().numpy()
    assert got.size == K.int2kv_prepared_wo_bytes(dm, Hq) // 2
    Wr = _untile_prepared(got, dm, Hq * 128)
    assert not np.any(Wr[dm:]), "padding rows must be zero"
    if not fold:
        # bf16 -> fp16 is exact in the normal range and rounds to nearest even below it
        assert np.array_equal(Wr[:dm], O.bf16_to_f64(w.W_o).astype(np.float16))
    else:
        ref = O.fold_wo(w.W_o, w.R_v, Hq)
        g = Wr[:dm].astype(np.float64)
        # one fp16 rounding (2^-11 relative, 2^-25 absolute below 2^-14) of an fp32 accumulation
        assert np.all(np.abs(g - ref) <= 2.0 ** -11 * np.abs(ref) + 2.0 ** -25 + 1e-6 * np.abs(ref).max())


def test_out_of_range_blocks_and_lengths_are_clamped():
    """Block ids outside the pool are skipped and ctx_lens beyond max_ctx are clamped."""
    w = W.make_workload(1, batch=2, ctx_lens=np.array([64, 40]), num_q_heads=4, num_kv_heads=1)
    pool = oracle_pool(w)
    table = w.block_table.copy()
    table[0, 1] = 10 ** 6          # tokens 16..31 of sequence 0 are unreachable
    lens = w.ctx_lens.copy()
    lens[1] = 10 ** 6              # clamped to max_ctx = 64 (= 16 * max_blocks)
    cache = gpu_cache(pool)
    out = K.int2kv_decode(cache, dev(w.q), dev(table), dev(lens), 64, dev(w.R_k), dev(w.R_v)).cpu().numpy()
    # sequence 1 then reads 64 tokens through its (zero-padded) table row: never-written slots
    # decode to zero keys and values, and padding entry 0 points at a real block
    ref = O.decode(pool, w.q[1:], w.block_table[1:], np.array([64]), w.R_k, w.R_v)
    assert_rows_close(out[1], ref[0], what="clamped length")
    # sequence 0 without block 1: attend over tokens 0..15 and 32..63 only
    kc, ks, kz, vc, vs, vz = O.read_tokens(pool, w.block_table[0], 64, 0)
    keep = np.r_[0:16, 32:64]
    Kt = O.dequantize(kc, ks, kz)[keep] @ w.R_k[0].astype(np.float64).T
    Vt = O.dequantize(vc, vs, vz)[keep] @ w.R_v[0].astype(np.float64).T
    ref0 = O.softmax_attention(O.bf16_to_f64(w.q)[0], Kt, Vt)
    assert_rows_close(out[0], ref0, what="skipped block")


@pytest.mark.parametrize("variant", [1, 2])
def test_append_decode_matches_separate_calls_and_oracle(variant):
    """int2kv_append_decode (cache write on the side stream beside the query preparation) leaves the
    same pool bytes and outputs as int2kv_quantize_append followed by int2kv_decode, and its output
    matches the oracle's decode of the pool it wrote."""
    print(f"\n[append_decode] variant={variant}", flush=True)
    K.int2kv_set_decode_tuning(0, variant)
    lens = np.array([300, 17, 1, 129, 64])
    Hq, H, dm = 40, 8, 256
    w = W.make_workload(4, batch=lens.size, ctx_lens=lens, num_q_heads=Hq, num_kv_heads=H, d_model=dm)
    Rk, Rv = dev(w.R_k), dev(w.R_v)
    mu_rk = K.int2kv_prepare_mu_rot(Rk, dev(w.mu))
    caches = [K.Int2KVCache(w.num_blocks, H) for _ in range(2)]
    k_last, v_last, s_last = [], [], []
    for b in range(w.batch):
        k, v = w.kv(b, as_torch=True)
        L = int(lens[b])
        slots = w.slot_mapping(b)
        if L > 1:
            for c in caches:
                K.int2kv_quantize_append(c, k[:L - 1].cuda(), v[:L - 1].cuda(), dev(slots[:L - 1]), Rk, Rv, mu_rk)
        k_last.append(k[L - 1])
        v_last.append(v[L - 1])
        s_last.append(slots[L - 1])
    kl, vl = torch.stack(k_last).cuda(), torch.stack(v_last).cuda()
    sl = dev(np.array(s_last, np.int32))
    Wp = K.int2kv_prepare_wo(dev(w.W_o), Rv, Hq)
    dargs = (dev(w.q), dev(w.block_table), dev(w.ctx_lens), int(lens.max()), Rk, Rv)
    K.int2kv_quantize_append(caches[0], kl, vl, sl, Rk, Rv, mu_rk)
    y0 = K.int2kv_decode(caches[0], *dargs, W_o=Wp, wo_format=K.INT2KV_WO_PREPARED_FOLDED, d_model=dm)
    y1 = K.int2kv_append_decode(caches[1], kl, vl, sl, mu_rk, *dargs, W_o=Wp,
                                wo_format=K.INT2KV_WO_PREPARED_FOLDED, d_model=dm)
    torch.cuda.synchronize()
    assert torch.equal(caches[0].pool, caches[1].pool)
    assert torch.equal(y0, y1)
    ref = O.decode(caches[1].pool.cpu().numpy(), w.q, w.block_table, w.ctx_lens, w.R_k, w.R_v, w.W_o)
    worst = assert_rows_close(y1.cpu().numpy(), ref, what="append_decode")
    # no new tokens: the plain decode
    y2 = K.int2kv_append_decode(caches[1], kl[:0], vl[:0], sl[:0], mu_rk, *dargs, W_o=Wp,
                                wo_format=K.INT2KV_WO_PREPARED_FOLDED, d_model=dm)
    assert torch.equal(y2, y1)
    print(f"worst row error {worst:.2e}", flush=True)


# 128-channel groups (the paper's setting): both scans, with and without W_O and through
# int2kv_append_decode
G128_CASES = [
    (1, 3, 8, 2, [1, 17, 300], None),
    (4, 2, 5, 1, [700, 64], None),
    (4, 3, 10, 2, [1500, 2, 129], 256),
    (1, 4, 32, 8, [1000, 33, 16, 0], 96),
]


@pytest.mark.parametrize("variant", [1, 2])
@pytest.mark.parametrize("case", G128_CASES, ids=lambda c: f"cfg{c[0]}-B{c[1]}-{c[2]}x{c[3]}-dm{c[5]}")
def test_decode_group128_matches_oracle(case, variant):
    cfg, B, Hq, H, lens, dm = case
    print(f"\n[decode G=128] case={case} variant={variant}", flush=True)
    K.int2kv_set_decode_tuning(0, variant)
    w = W.make_workload(cfg, batch=B, ctx_lens=np.array(lens), num_q_heads=Hq, num_kv_heads=H, d_model=dm)
    pool = oracle_pool(w, group=128)
    ref = O.decode(pool, w.q, w.block_table, w.ctx_lens, w.R_k, w.R_v, w.W_o)
    cache = gpu_cache(pool)
    args = (cache, dev(w.q), dev(w.block_table), dev(w.ctx_lens), int(max(lens)), dev(w.R_k), dev(w.R_v))
    out = K.int2kv_decode(*args, W_o=dev(w.W_o) if dm else None)
    worst = assert_rows_close(out.cpu().numpy(), ref, what="decode G=128")
    assert torch.equal(out, K.int2kv_decode(*args, W_o=dev(w.W_o) if dm else None))
    if dm:
        Wp = K.int2kv_prepare_wo(dev(w.W_o), dev(w.R_v), Hq)
        out_p = K.int2kv_decode(*args, W_o=Wp, wo_format=K.INT2KV_WO_PREPARED_FOLDED, d_model=dm)
        assert_rows_close(out_p.cpu().numpy(), ref, what="decode G=128, prepared W_O")
    print(f"worst row error {worst:.2e}", flush=True)


@pytest.mark.parametrize("variant", [1, 2])
def test_append_decode_group128(variant):
    """int2kv_append_decode at G = 128 (inside the preparation launch of the matrix-core decode, or
    its own launch before the vector-ALU decode) leaves the pool and outputs of the two calls."""
    K.int2kv_set_decode_tuning(0, variant)
    lens = np.array([300, 17, 1, 129])
    Hq, H = 16, 4
    w = W.make_workload(1, batch=lens.size, ctx_lens=lens, num_q_heads=Hq, num_kv_heads=H)
    Rk, Rv = dev(w.R_k), dev(w.R_v)
    mu_rk = K.int2kv_prepare_mu_rot(Rk, dev(w.mu))
    caches = [K.Int2KVCache(w.num_blocks, H, group_size=128) for _ in range(2)]
    k_last, v_last, s_last = [], [], []
    for b in range(w.batch):
        k, v = w.kv(b, as_torch=True)
        L = int(lens[b])
        slots = w.slot_mapping(b)
        if L > 1:
            for c in caches:
                K.int2kv_quantize_append(c, k[:L - 1].cuda(), v[:L - 1].cuda(), dev(slots[:L - 1]), Rk, Rv, mu_rk)
        k_last.append(k[L - 1])
        v_last.append(v[L - 1])
        s_last.append(slots[L - 1])
    kl, vl = torch.stack(k_last).cuda(), torch.stack(v_last).cuda()
    sl = dev(np.array(s_last, np.int32))
    dargs = (dev(w.q), dev(w.block_table), dev(w.ctx_lens), int(lens.max()), Rk, Rv)
    K.int2kv_quantize_append(caches[0], kl, vl, sl, Rk, Rv, mu_rk)
    y0 = K.int2kv_decode(caches[0], *dargs)
    y1 = K.int2kv_append_decode(caches[1], kl, vl, sl, mu_rk, *dargs)
    torch.cuda.synchronize()
    assert torch.equal(caches[0].pool, caches[1].pool) and torch.equal(y0, y1)
    ref = O.decode(caches[1].pool.cpu().numpy(), w.q, w.block_table, w.ctx_lens, w.R_k, w.R_v)
    assert_rows_close(y1.cpu().numpy(), ref, what="append_decode G=128")


@pytest.mark.parametrize("G", [32, 128])
@pytest.mark.parametrize("variant", [1, 2])
def test_decode_large_value_and_key_ranges(G, variant):
    """Value groups whose fp16 scale is far above 256 (rotated value ranges up to ~1e5) beside
    ordinary tokens of the same pages, and key groups with wider ranges: the matrix-core scan's fp16
    value weights p * s must not overflow (its scaled form takes such pairs). The keys of one token
    in ten are scaled by 4 (logits of a few units: the matrix-core scan holds q' as an fp16 operand,
    so its score error grows with the logit magnitude, about 2^-12 of it)."""
    print(f"\n[decode large ranges] G={G} variant={variant}", flush=True)
    K.int2kv_set_decode_tuning(0, variant)
    w = W.make_workload(4, batch=3, ctx_lens=np.array([300, 47, 129]), num_q_heads=10, num_kv_heads=2)
    pool = O.new_pool(w.num_blocks, w.num_kv_heads, G)
    rng = np.random.default_rng(17)
    big_scales = []
    for b in range(w.batch):
        k, v = w.kv(b)
        k_rot = O.center_rotate(k, w.mu, w.R_k).astype(np.float32)
        v_rot = O.rotate(v, w.R_v).astype(np.float32)
        L = k.shape[0]
        v_rot *= np.where(rng.random(L) < 0.3, 10.0 ** rng.uniform(2.0, 4.0, L), 1.0)[:, None, None].astype(np.float32)
        k_rot *= np.where(rng.random(L) < 0.1, 4.0, 1.0)[:, None, None].astype(np.float32)
        _, _, _, _, vs, _ = O.quantize_pack_rotated(pool, k_rot, v_rot, w.slot_mapping(b))
        big_scales.append(vs.astype(np.float64).max())
    assert max(big_scales) > 1000.0  # the case exercises the large-scale pairs
    ref = O.decode(pool, w.q, w.block_table, w.ctx_lens, w.R_k, w.R_v)
    out = K.int2kv_decode(gpu_cache(pool), dev(w.q), dev(w.block_table), dev(w.ctx_lens), int(w.ctx_lens.max()),
                          dev(w.R_k), dev(w.R_v))
    worst = assert_rows_close(out.cpu().numpy(), ref, what="decode, large ranges")
    print(f"largest V scale {max(big_scales):.0f}; worst row error {worst:.2e}", flush=True)


@pytest.mark.parametrize("G", [32, 128])
@pytest.mark.parametrize("variant", [1, 2])
def test_decode_queries_on_one_rotated_channel_and_extreme_norms(G, variant):
    """Queries whose rotated form q R_K lies on a single channel (there the largest |q'_c| equals
    |q|_2, the bound from which the matrix-core scan takes its fp16 operand scale), and queries of
    tiny and of four times the usual norm, against the oracle."""
    print(f"\n[decode extreme queries] G={G} variant={variant}", flush=True)
    K.int2kv_set_decode_tuning(0, variant)
    w = W.make_workload(4, batch=3, ctx_lens=np.array([300, 47, 129]), num_q_heads=10, num_kv_heads=2)
    gq = w.num_q_heads // w.num_kv_heads
    qf = W.bf16_bits_to_f32(w.q).astype(np.float64)
    for j in range(w.num_q_heads):
        h = j // gq
        qf[0, j] = 8.0 * w.R_k[h][:, (37 * j + 5) % 128]  # q R_K = 8 e_c (up to the rotation's rounding)
    qf[1] *= 1e-3  # near-uniform softmax
    qf[2] *= 4.0   # logits of several units (the fp16 query operand's score error is about 2^-12 of them)
    q = W.f32_to_bf16_bits(qf.astype(np.float32))
    pool = oracle_pool(w, group=G)
    ref = O.decode(pool, q, w.block_table, w.ctx_lens, w.R_k, w.R_v)
    out = K.int2kv_decode(gpu_cache(pool), dev(q), dev(w.block_table), dev(w.ctx_lens), int(w.ctx_lens.max()),
                          dev(w.R_k), dev(w.R_v))
    got = out.cpu().numpy()
    assert np.isfinite(got).all()
    worst = assert_rows_close(got, ref, what="decode, extreme queries")
    print(f"worst row error {worst:.2e}", flush=True)
