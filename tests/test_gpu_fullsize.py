"""GPU parity at the full sizes of the benchmark configurations, in the launch configuration that
bench.py times (default decode plan, W_O folded once). The GPU builds its cache with
int2kv_quantize_append from the seeded keys and values, the oracle builds its own from the same
inputs (end-to-end parity). Compared: every output of configurations 1, 2 and 3, and eight sampled
sequences of configuration 4 (the oracle cache holds only those sequences, with their pages
renumbered), both in the default setting and in the paper's serving setting (groups of 128, clip
ratios, BF16 sink and recent windows)."""
import numpy as np
import pytest
import torch

from oracle import int2kv_oracle as O
from paper_2608_02691_amd import int2kv as K
from paper_2608_02691_amd import workloads as W

from _helpers import assert_rows_close, compare_cache_writes, dev, gpu_cache, oracle_pool

pytestmark = pytest.mark.gpu


@pytest.fixture(autouse=True)
def _default_tuning():
    K.int2kv_set_decode_tuning(0, 0)
    yield


def gpu_build(w, seqs=None, hold_last=False):
    """Cache written by the library, one append call per sequence (the prefill-sized path). With
    hold_last, every sequence's last token is left out and returned as the current tokens of a
    decode step: (k, v, slots) for all sequences, plus mu R_K."""
    cache = K.Int2KVCache(w.num_blocks, w.num_kv_heads)
    Rk, Rv = dev(w.R_k), dev(w.R_v)
    mu_rk = K.int2kv_prepare_mu_rot(Rk, dev(w.mu))
    last = ([], [], [])
    for b in (range(w.batch) if seqs is None else seqs):
        L = int(w.ctx_lens[b])
        if L == 0:
            continue
        k, v = w.kv(b, as_torch=True)
        slots = w.slot_mapping(b)
        n = L - 1 if hold_last else L
        if n > 0:
            K.int2kv_quantize_append(cache, k[:n].cuda(), v[:n].cuda(), dev(slots[:n]), Rk, Rv, mu_rk)
        if hold_last:
            last[0].append(k[L - 1])
            last[1].append(v[L - 1])
            last[2].append(slots[L - 1])
    torch.cuda.synchronize()
    if hold_last:
        cur = (torch.stack(last[0]).cuda(), torch.stack(last[1]).cuda(), dev(np.array(last[2], np.int32)))
        return cache, Rk, Rv, cur, mu_rk
    return cache, Rk, Rv


def test_config1_full_decode_with_wo():
    """16 x 4096 tokens, 32/8 heads, W_O 4096^2: every output, W_O plain and folded."""
    print("\n[full] config 1", flush=True)
    w = W.make_workload(1)
    ref = O.decode(oracle_pool(w), w.q, w.block_table, w.ctx_lens, w.R_k, w.R_v, w.W_o)
    cache, Rk, Rv = gpu_build(w)
    args = (cache, dev(w.q), dev(w.block_table), dev(w.ctx_lens), int(w.ctx_lens.max()), Rk, Rv)
    Wo = dev(w.W_o)
    worst = assert_rows_close(K.int2kv_decode(*args, W_o=Wo).cpu().numpy(), ref, what="config 1, W_O")
    Wf = K.int2kv_fold_wo(Wo, Rv, w.num_q_heads)
    worst_f = assert_rows_close(K.int2kv_decode(*args, W_o=Wf, wo_is_folded=True).cpu().numpy(), ref,
                                what="config 1, folded W_O")
    Wp = K.int2kv_prepare_wo(Wo, Rv, w.num_q_heads)
    worst_p = assert_rows_close(K.int2kv_decode(*args, W_o=Wp, wo_format=K.INT2KV_WO_PREPARED_FOLDED,
                                                d_model=w.W_o.shape[0]).cpu().numpy(), ref,
                                what="config 1, prepared folded W_O")
    print(f"worst row error {worst:.2e} (plain W_O), {worst_f:.2e} (folded), {worst_p:.2e} (prepared)", flush=True)


def test_config2_long_context_all_heads():
    """1 x 131072 tokens, 32/8 heads (8192 pages, split over every CU): every query head of every
    KV head against the oracle's cache of the same inputs."""
    print("\n[full] config 2", flush=True)
    w = W.make_workload(2)
    cache, Rk, Rv = gpu_build(w)
    L = int(w.ctx_lens[0])
    out = K.int2kv_decode(cache, dev(w.q), dev(w.block_table), dev(w.ctx_lens), L, Rk, Rv).cpu().numpy()
    ref = O.decode(oracle_pool(w), w.q, w.block_table, w.ctx_lens, w.R_k, w.R_v)
    worst = assert_rows_close(out, ref, what="config 2")
    print(f"worst row error {worst:.2e}", flush=True)


def test_config3_prefill_append_then_decode():
    """4 x 8192 new tokens written in one append call (32768 tokens x 8 KV heads), checked end to
    end against the oracle's cache (codes may differ only at rounding ties, at most 1e-4 of them);
    then the decode with 32 query heads at full size:

    * over the oracle's cache, against the oracle's decode (the attention bar);
    * over the library-written cache, against the oracle's decode of that same cache (the bar);
    * end to end against the oracle's decode of its own cache, within the bar plus the effect of the
      allowed tie flips, which the oracle computes exactly: |decode(gpu cache) - decode(oracle
      cache)| per row."""
    print("\n[full] config 3", flush=True)
    w = W.make_workload(3)
    kk, vv, ss, kr, vr = [], [], [], [], []
    for b in range(w.batch):
        k, v = w.kv(b)
        kk.append(k)
        vv.append(v)
        ss.append(w.slot_mapping(b))
        kr.append(O.center_rotate(k, w.mu, w.R_k).astype(np.float32))
        vr.append(O.rotate(v, w.R_v).astype(np.float32))
    k, v, slots = np.concatenate(kk), np.concatenate(vv), np.concatenate(ss)
    cache = K.Int2KVCache(w.num_blocks, w.num_kv_heads)
    Rk, Rv = dev(w.R_k), dev(w.R_v)
    mu_rk = K.int2kv_prepare_mu_rot(Rk, dev(w.mu))
    K.int2kv_quantize_append(cache, dev(k), dev(v), dev(slots), Rk, Rv, mu_rk)
    ref_pool = oracle_pool(w)
    gpu_pool = cache.pool.cpu().numpy()
    stats = compare_cache_writes(gpu_pool, ref_pool, slots, np.concatenate(kr), np.concatenate(vr))
    print(stats, flush=True)
    assert stats["fraction"] <= 1e-4
    ref = O.decode(ref_pool, w.q, w.block_table, w.ctx_lens, w.R_k, w.R_v)
    dargs = (dev(w.q), dev(w.block_table), dev(w.ctx_lens), int(w.ctx_lens.max()), Rk, Rv)
    out = K.int2kv_decode(gpu_cache(ref_pool), *dargs)
    worst = assert_rows_close(out.cpu().numpy(), ref, what="config 3 decode (oracle cache)")
    e2e = K.int2kv_decode(cache, *dargs).cpu().numpy()
    ref_gp = O.decode(gpu_pool, w.q, w.block_table, w.ctx_lens, w.R_k, w.R_v)
    worst_gp = assert_rows_close(e2e, ref_gp, what="config 3 decode (library-written cache)")
    norm = np.linalg.norm(ref, axis=-1)
    flips = np.abs(ref_gp - ref).max(axis=-1)
    err = np.abs(e2e - ref).max(axis=-1)
    assert np.all(err <= flips + 2e-3 * norm), "end-to-end error beyond the bar plus the tie flips' effect"
    print(f"worst row error {worst:.2e} (oracle cache), {worst_gp:.2e} (library cache); end to end "
          f"{(err / norm).max():.2e}, of which tie flips {(flips / norm).max():.2e}", flush=True)


def test_config4_sampled_sequences():
    """The benchmark workload (64 ragged sequences, 40/8 heads, W_O 5120^2 prepared with R_V folded
    in) run as the benchmark runs it: every sequence but its last token prefilled, then
    int2kv_append_decode (also a row-major folded W_O decode of the same cache); the shortest, the
    longest and six seeded other sequences are checked, each against an oracle cache holding that
    sequence alone."""
    print("\n[full] config 4", flush=True)
    w = W.make_workload(4)
    cache, Rk, Rv, (kc, vc, sc), mu_rk = gpu_build(w, hold_last=True)
    dargs = (cache, dev(w.q), dev(w.block_table), dev(w.ctx_lens), int(w.ctx_lens.max()), Rk, Rv)
    Wp = K.int2kv_prepare_wo(dev(w.W_o), Rv, w.num_q_heads)
    # the benchmark's step: the current tokens' cache write inside the decode's first launch
    y = K.int2kv_append_decode(cache, kc, vc, sc, mu_rk, *dargs[1:], W_o=Wp, wo_format=K.INT2KV_WO_PREPARED_FOLDED,
                               d_model=w.W_o.shape[0]).cpu().numpy()
    Wf = K.int2kv_fold_wo(dev(w.W_o), Rv, w.num_q_heads)
    y_f = K.int2kv_decode(*dargs, W_o=Wf, wo_is_folded=True).cpu().numpy()
    lens = w.ctx_lens
    rng = np.random.default_rng(4)
    picks = sorted({int(np.argmin(lens)), int(np.argmax(lens)), *rng.choice(w.batch, 6, replace=False).tolist()})
    for b in picks:
        L = int(lens[b])
        nblk = (L + 15) // 16
        pool = O.new_pool(nblk, w.num_kv_heads)
        k, v = w.kv(b)
        O.quantize_append(pool, k, v, np.arange(L, dtype=np.int32), w.R_k, w.R_v, w.mu)
        ref = O.decode(pool, w.q[b:b + 1], np.arange(nblk, dtype=np.int32)[None], np.array([L], np.int32),
                       w.R_k, w.R_v, w.W_o)
        worst = assert_rows_close(y[b:b + 1], ref, what=f"config 4 sequence {b} (L={L})")
        worst_f = assert_rows_close(y_f[b:b + 1], ref, what=f"config 4 sequence {b} (L={L}), row-major W_O")
        print(f"sequence {b} (L={L}): worst row error {worst:.2e} (prepared), {worst_f:.2e} (row-major)", flush=True)


def test_config4_serving_setting_sampled_sequences():
    """The paper's serving setting on the benchmark workload (Sec. 5 implementation details): groups
    of 128 channels, clip ratios c_K = 0.96 and c_V = 0.92, the first 64 and last 256 tokens of
    every sequence in the BF16 window and the rest in INT2, W_O 5120^2 prepared with R_V folded in;
    run as bench.py --group 128 --window 64,256 runs it. Eight sequences (the shortest, the longest
    and six seeded others) are checked against the oracle's decode_window of that sequence alone."""
    print("\n[full] config 4, G = 128, windows 64 + 256, clip 0.96 / 0.92", flush=True)
    w = W.make_workload(4)
    G, sink, recent, clip = 128, 64, 256, (0.96, 0.92)
    cap = sink + recent
    H, B = w.num_kv_heads, w.batch
    lens = w.ctx_lens.astype(np.int64)
    n2 = np.maximum(lens - cap, 0)
    cache = K.Int2KVCache(w.num_blocks, H, group_size=G)
    Rk, Rv, mu = dev(w.R_k), dev(w.R_v), dev(w.mu)
    mu_rk = K.int2kv_prepare_mu_rot(Rk, mu)
    win_k = torch.zeros((B * cap, H, 128), dtype=torch.int16, device="cuda")
    win_v = torch.zeros_like(win_k)
    wl = np.minimum(lens, cap).astype(np.int32)

    def split(L):
        wi = np.r_[0:min(sink, L), max(L - recent, min(sink, L)):L]
        return wi, np.arange(min(sink, L), min(sink, L) + max(L - cap, 0))

    for b in range(B):
        k, v = w.kv(b, as_torch=True)
        L = int(lens[b])
        wi, ii = split(L)
        kd, vd = k.cuda(), v.cuda()
        K.int2kv_window_write(kd[wi], vd[wi], dev(np.arange(b * cap, b * cap + wi.size, dtype=np.int32)), mu,
                              win_k, win_v)
        if ii.size:
            K.int2kv_quantize_append(cache, kd[ii], vd[ii], dev(w.slot_mapping(b, 0, ii.size)), Rk, Rv, mu_rk, *clip)
    torch.cuda.synchronize()
    Wp = K.int2kv_prepare_wo(dev(w.W_o), Rv, w.num_q_heads)
    dm = w.W_o.shape[0]
    y = K.int2kv_decode_window(cache, dev(w.q), dev(w.block_table), dev(n2.astype(np.int32)), int(n2.max()), Rk, Rv,
                               win_k, win_v, dev(wl), cap, W_o=Wp, wo_format=K.INT2KV_WO_PREPARED_FOLDED,
                               d_model=dm).cpu().numpy()
    rng = np.random.default_rng(44)
    picks = sorted({int(np.argmin(lens)), int(np.argmax(lens)), *rng.choice(B, 6, replace=False).tolist()})
    for b in picks:
        L = int(lens[b])
        wi, ii = split(L)
        k, v = w.kv(b)
        nblk = max(1, (ii.size + 15) // 16)
        pool = O.new_pool(nblk, H, G)
        if ii.size:
            O.quantize_append(pool, k[ii], v[ii], np.arange(ii.size, dtype=np.int32), w.R_k, w.R_v, w.mu, *clip)
        wk = np.zeros((cap, H, 128), np.uint16)
        wv = np.zeros_like(wk)
        O.window_write(wk, wv, k[wi], v[wi], w.mu, np.arange(wi.size))
        ref = O.decode_window(pool, w.q[b:b + 1], np.arange(nblk, dtype=np.int32)[None],
                              np.array([ii.size], np.int32), w.R_k, w.R_v, wk[None], wv[None],
                              np.array([wi.size]), w.W_o)
        worst = assert_rows_close(y[b:b + 1], ref, what=f"serving setting, sequence {b} (L={L})")
        print(f"sequence {b} (L={L}, {ii.size} INT2 tokens): worst row error {worst:.2e}", flush=True)
