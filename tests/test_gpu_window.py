"""GPU parity of the BF16 sink/recent window path (int2kv_window_write, int2kv_decode_window)
through the C ABI against the CPU oracle: the window store bit for bit, and decode over window
plus INT2 tokens for both scans, both group sizes, GQA 4, 5 and 12, empty windows, empty INT2
contexts, full windows, with and without W_O."""
import numpy as np
import pytest
import torch

from oracle import int2kv_oracle as O
from paper_2608_02691_amd import int2kv as K
from paper_2608_02691_amd import workloads as W

from _helpers import assert_rows_close, dev, gpu_cache, oracle_pool

pytestmark = pytest.mark.gpu


@pytest.fixture(autouse=True)
def _default_tuning():
    K.int2kv_set_decode_tuning(0, 0)
    yield
    K.int2kv_set_decode_tuning(0, 0)


def _window(w, cap, wl):
    """Window rows of each sequence: its first wl[b] tokens (sink-like), written by the oracle and
    by the library from the same bf16 inputs."""
    H = w.num_kv_heads
    ks, vs, rows = [], [], []
    for b in range(w.batch):
        k, v = w.kv(b)
        n = int(wl[b])
        ks.append(k[:n])
        vs.append(v[:n])
        rows.append(b * cap + np.arange(n))
    k = np.concatenate(ks).reshape(-1, H, 128)
    v = np.concatenate(vs).reshape(-1, H, 128)
    rows = np.concatenate(rows).astype(np.int32)
    win_k = np.zeros((w.batch * cap, H, 128), np.uint16)
    win_v = np.zeros_like(win_k)
    O.window_write(win_k, win_v, k, v, w.mu, rows)
    return k, v, rows, win_k, win_v


def test_window_write_bit_exact():
    w = W.make_workload(1, batch=3, ctx_lens=np.array([70, 300, 5]), num_q_heads=8, num_kv_heads=2)
    cap = 64
    wl = np.array([64, 40, 5])
    k, v, rows, wk_ref, wv_ref = _window(w, cap, wl)
    rows = rows.copy()
    rows[3] = -1  # skipped token
    rows[7] = w.batch * cap + 5  # past the store: skipped
    wk_ref = np.zeros_like(wk_ref)
    wv_ref = np.zeros_like(wv_ref)
    O.window_write(wk_ref, wv_ref, k, v, w.mu, np.where(rows < w.batch * cap, rows, -1))
    wk = torch.zeros(wk_ref.shape, dtype=torch.int16, device="cuda")
    wv = torch.zeros_like(wk)
    K.int2kv_window_write(dev(k.view(np.int16)), dev(v.view(np.int16)), dev(rows), dev(w.mu), wk, wv)
    torch.cuda.synchronize()
    assert np.array_equal(wk.cpu().numpy().view(np.uint16), wk_ref)
    assert np.array_equal(wv.cpu().numpy().view(np.uint16), wv_ref)


CASES = [
    # (Hq, H, ctx lens, window lens, cap, d_model); a sequence with neither window nor INT2 tokens,
    # and window counts below 0 and above cap (clamped to an empty and a full window)
    (8, 2, [300, 0, 17, 1, 129, 0], [64, 5, 0, 320, 1, 0], 320, 0),
    (10, 2, [700, 0, 33, 40], [100, 7, 0, -3], 128, 96),
    (24, 2, [250, 64, 10], [30, 64, 1000], 64, 0),
    # the largest window (512 tokens: every slice of the window attention, the last one partial)
    (8, 2, [40, 600, 3], [512, 200, 511], 512, 0),
]


@pytest.mark.parametrize("G", [32, 128])
@pytest.mark.parametrize("variant", [1, 2])
@pytest.mark.parametrize("case", CASES, ids=["gqa4", "gqa5_wo", "gqa12", "gqa4_cap512"])
def test_decode_window_matches_oracle(case, variant, G):
    Hq, H, lens, wls, cap, dm = case
    print(f"\n[decode window] case={case} variant={variant} G={G}", flush=True)
    K.int2kv_set_decode_tuning(0, variant)
    lens, wl = np.array(lens), np.array(wls, np.int32)
    wl_rows = np.clip(wl, 0, cap)  # tokens actually stored in each window
    w = W.make_workload(1, batch=lens.size, ctx_lens=np.maximum(lens, wl_rows), num_q_heads=Hq, num_kv_heads=H,
                        d_model=dm or None)
    k, v, rows, wk_ref, wv_ref = _window(w, cap, wl_rows)
    w.ctx_lens = lens.astype(np.int32)  # the INT2 part: the first lens[b] tokens
    pool = oracle_pool(w, group=G)
    win_k = wk_ref.reshape(w.batch, cap, H, 128)
    win_v = wv_ref.reshape(w.batch, cap, H, 128)
    ref = O.decode_window(pool, w.q, w.block_table, w.ctx_lens, w.R_k, w.R_v, win_k, win_v, wl, w.W_o)
    cache = gpu_cache(pool)
    wk = torch.zeros(wk_ref.shape, dtype=torch.int16, device="cuda")
    wv = torch.zeros_like(wk)
    K.int2kv_window_write(dev(k.view(np.int16)), dev(v.view(np.int16)), dev(rows), dev(w.mu), wk, wv)
    args = (cache, dev(w.q), dev(w.block_table), dev(w.ctx_lens), int(max(lens.max(), 1)), dev(w.R_k), dev(w.R_v),
            wk, wv, dev(wl), cap)
    out = K.int2kv_decode_window(*args, W_o=dev(w.W_o) if dm else None)
    worst = assert_rows_close(out.cpu().numpy(), ref, what="decode window")
    assert torch.equal(out, K.int2kv_decode_window(*args, W_o=dev(w.W_o) if dm else None))
    if dm:
        Wp = K.int2kv_prepare_wo(dev(w.W_o), dev(w.R_v), Hq)
        out_p = K.int2kv_decode_window(*args, W_o=Wp, wo_format=K.INT2KV_WO_PREPARED_FOLDED, d_model=dm)
        assert_rows_close(out_p.cpu().numpy(), ref, what="decode window, prepared W_O")
    print(f"worst row error {worst:.2e}", flush=True)


def test_decode_window_empty_windows_equal_decode():
    """win_lens all zero: the result is int2kv_decode's, bit for bit (the empty window partial is
    dropped by the merge)."""
    lens = np.array([300, 17, 1, 129])
    w = W.make_workload(1, batch=lens.size, ctx_lens=lens, num_q_heads=16, num_kv_heads=4)
    cache = gpu_cache(oracle_pool(w))
    dargs = (cache, dev(w.q), dev(w.block_table), dev(w.ctx_lens), int(lens.max()), dev(w.R_k), dev(w.R_v))
    wk = torch.zeros((w.batch * 8, 4, 128), dtype=torch.int16, device="cuda")
    y0 = K.int2kv_decode(*dargs)
    y1 = K.int2kv_decode_window(*dargs, wk, wk.clone(), dev(np.zeros(w.batch, np.int32)), 8)
    assert torch.equal(y0, y1)
