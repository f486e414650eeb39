"""Pins of the calibration oracle (Sec. 4.2 - 4.5, Algorithm 1) to what the paper and the
mathematics fix (CPU only): orthogonality of the corrected rotations, the matrix exponential
against scipy, the objectives against the independently pinned output-error diagnostics, the
straight-through gradient against finite differences of its smooth surrogate, windows that
remove every quantized token, and the calibration's selection and descent."""
import numpy as np
import pytest
import torch

from oracle import int2kv_oracle as O
from oracle import optr_oracle as P
from paper_2608_02691_amd import workloads as W


def _traces(lens, Hq=8, H=2, dm=64, seed=0):
    w = W.make_workload(1, batch=len(lens), ctx_lens=np.array(lens), num_q_heads=Hq, num_kv_heads=H, d_model=dm)
    ks, vs = zip(*[w.kv(b) for b in range(len(lens))])
    k, v = np.concatenate(ks), np.concatenate(vs)
    rng = np.random.default_rng(seed)
    q = W.f32_to_bf16_bits(rng.standard_normal((len(k), Hq, 128)).astype(np.float32) * 2.0)
    st = np.concatenate([[0], np.cumsum(lens)]).astype(np.int64)
    return w, k, v, q, st


def test_corrected_rotation_is_orthogonal():
    """eq:OptR_skew: exp of a skew-symmetric generator is orthogonal, so R^0 exp(A - A^T) is."""
    w, *_ = _traces([20])
    rng = np.random.default_rng(1)
    R0 = w.R_k[0].astype(np.float64)  # an fp32 rotation: orthogonal to about 1e-7 itself
    base = np.abs(R0 @ R0.T - np.eye(128)).max()
    for scale in (0.01, 0.3, 2.0):
        A = torch.from_numpy(rng.standard_normal((128, 128)) * scale)
        R = P.rotation(R0, A).numpy()
        assert np.abs(R @ R.T - np.eye(128)).max() <= base + 1e-12
    R0 = O.hadamard(128)[None]
    A = torch.from_numpy(rng.standard_normal((128, 128)) * 0.5)
    R = P.rotation(R0[0], A).numpy()
    assert np.abs(R @ R.T - np.eye(128)).max() <= 1e-12


def test_matrix_exponential_matches_scipy():
    from scipy.linalg import expm
    rng = np.random.default_rng(2)
    A = rng.standard_normal((128, 128)) * 0.4
    S = A - A.T
    E = torch.linalg.matrix_exp(torch.from_numpy(S)).numpy()
    assert np.abs(E - expm(S)).max() <= 1e-12


def test_key_objective_matches_output_error_diagnostics():
    """With one query row per sequence (its last position), lambda_K = 1 and no window, the key
    objective's output term is the key-induced error dy_K of the output-error diagnostics over the
    cache written with the same rotation, and its KL term is KL(p || p~) of the attention
    probabilities over the raw and the effective keys."""
    lens = [70, 33]
    w, k, v, q, st = _traces(lens)
    mu = P.key_mean(k)
    A = torch.zeros((128, 128), dtype=torch.float64)
    for h in range(2):
        L = float(P.key_loss(A, w.R_k, k, v, q, st, mu, w.W_o, h, 4, lam=1.0, group=32, n_last=1))
        # the same rotation in the cache: R = R^0 exactly (A = 0)
        pool = O.new_pool(w.num_blocks, 2)
        for b in range(2):
            O.quantize_append(pool, k[st[b]:st[b + 1]], v[st[b]:st[b + 1]], w.slot_mapping(b), w.R_k, w.R_v, mu)
        q_last = np.stack([q[st[b + 1] - 1] for b in range(2)])
        dyK, dyV, stats = O.output_error(pool, [k[st[b]:st[b + 1]] for b in range(2)],
                                         [v[st[b]:st[b + 1]] for b in range(2)], q_last, np.array(lens),
                                         w.block_table, w.R_k, w.R_v, mu, w.W_o)
        kl = []
        for b in range(2):
            Kc, _ = O.effective_kv(pool, w.block_table[b], lens[b], h, w.R_k, w.R_v)
            Kraw = O.bf16_to_f64(k[st[b]:st[b + 1], h])
            for j in range(4 * h, 4 * h + 4):
                qq = O.bf16_to_f64(q_last[b, j])[None]
                p = O.attention_probs(qq, Kraw)[0]
                pt = O.attention_probs(qq, Kc)[0]
                kl.append(float((p * (np.log(p) - np.log(pt))).sum()))
        ref = np.mean(np.array(kl) + stats[:, 4 * h:4 * h + 4, 1].ravel() / 64.0)  # rows (b, j)
        assert abs(L - ref) <= 1e-10 * abs(ref)


def test_value_objective_matches_output_error_diagnostics():
    """The value objective under the key distribution of the same rotation is the value-induced
    error dy_V of the diagnostics (one query row per sequence, no window)."""
    lens = [64, 40]
    w, k, v, q, st = _traces(lens, seed=3)
    mu = P.key_mean(k)
    A0 = np.zeros((128, 128))
    pool = O.new_pool(w.num_blocks, 2)
    for b in range(2):
        O.quantize_append(pool, k[st[b]:st[b + 1]], v[st[b]:st[b + 1]], w.slot_mapping(b), w.R_k, w.R_v, mu)
    q_last = np.stack([q[st[b + 1] - 1] for b in range(2)])
    _, _, stats = O.output_error(pool, [k[st[b]:st[b + 1]] for b in range(2)], [v[st[b]:st[b + 1]] for b in range(2)],
                                 q_last, np.array(lens), w.block_table, w.R_k, w.R_v, mu, w.W_o)
    for h in range(2):
        probs = P.key_probs(w.R_k, A0, k, q, st, mu, h, 4, group=32, n_last=1)
        L = float(P.value_loss(torch.zeros((128, 128), dtype=torch.float64), w.R_v, v, st, probs, w.W_o, h, 4,
                               group=32, n_last=1))
        # rows visited per sequence, then query head: stats[b, j]
        ref = np.mean([stats[b, j, 2] / 64.0 for b in range(2) for j in range(4 * h, 4 * h + 4)])
        assert abs(L - ref) <= 1e-10 * abs(ref)


def test_windows_covering_everything_give_zero_objectives():
    """With sink + recent windows covering every token no key or value is quantized: p^K = p and
    V~ = V, so both objectives vanish (Algorithm 1: window tokens skip INT2)."""
    w, k, v, q, st = _traces([50, 30])
    mu = P.key_mean(k)
    A = torch.from_numpy(np.random.default_rng(4).standard_normal((128, 128)) * 0.1)
    Lk = float(P.key_loss(A, w.R_k, k, v, q, st, mu, w.W_o, 1, 4, group=32, n_last=8, sink=16, recent=64))
    assert abs(Lk) <= 1e-14
    probs = P.key_probs(w.R_k, A.numpy(), k, q, st, mu, 1, 4, group=32, n_last=8, sink=16, recent=64)
    Lv = float(P.value_loss(A, w.R_v, v, st, probs, w.W_o, 1, 4, group=32, n_last=8, sink=16, recent=64))
    assert Lv == 0.0


@pytest.mark.parametrize("which", ["key", "value"])
def test_straight_through_gradient_matches_finite_differences(which):
    """eq:OptR_ste: the gradient at A0 equals the derivative of the surrogate that keeps the codes,
    scales and zeros of A0 and lets in-range elements move with the rotation; checked by central
    differences along random directions (clip 0.9, so some elements are blocked)."""
    w, k, v, q, st = _traces([60, 45], seed=5)
    mu = P.key_mean(k)
    rng = np.random.default_rng(6)
    A0 = rng.standard_normal((128, 128)) * 0.05
    h, gq, clip = 1, 4, 0.9
    if which == "key":
        frozen = P.frozen_point(w.R_k, A0, k, h, clip, 32, mu=mu)
        f = lambda A, fr: P.key_loss(A, w.R_k, k, v, q, st, mu, w.W_o, h, gq, lam=1.0, clip=clip, group=32,
                                     n_last=10, frozen=fr)
    else:
        probs = P.key_probs(w.R_k, A0 * 0.5, k, q, st, mu, h, gq, group=32, n_last=10)
        frozen = P.frozen_point(w.R_v, A0, v, h, clip, 32)
        f = lambda A, fr: P.value_loss(A, w.R_v, v, st, probs, w.W_o, h, gq, clip=clip, group=32, n_last=10,
                                       frozen=fr)
    assert float(frozen[1].min()) == 0.0 and float(frozen[1].max()) == 1.0
    A = torch.from_numpy(A0.copy()).requires_grad_(True)
    L = f(A, None)
    L.backward()
    g = A.grad.numpy()
    # the surrogate equals the real loss at A0
    assert abs(float(f(torch.from_numpy(A0), frozen)) - float(L)) <= 1e-12 * abs(float(L))
    eps = 1e-5
    for _ in range(3):
        dA = rng.standard_normal((128, 128))
        fd = (float(f(torch.from_numpy(A0 + eps * dA), frozen)) - float(f(torch.from_numpy(A0 - eps * dA), frozen))) / (2 * eps)
        an = float((g * dA).sum())
        assert abs(fd - an) <= 1e-6 * abs(an) + 1e-12


def _structured(lens, seed, H=2, Hq=8):
    """Traces with four high-variance channels (std 8) in keys, values and queries: the raw-channel
    INT2 groups that hold them quantize badly, which a rotation can spread out."""
    rng = np.random.default_rng(seed)
    T = sum(lens)
    scale = np.ones(128)
    scale[[3, 50, 77, 100]] = 8.0
    f = lambda x: W.f32_to_bf16_bits(x.astype(np.float32))
    k = f(rng.standard_normal((T, H, 128)) * scale)
    v = f(rng.standard_normal((T, H, 128)) * scale[::-1])
    q = f(rng.standard_normal((T, Hq, 128)) * scale * 0.3)
    return k, v, q, np.concatenate([[0], np.cumsum(lens)]).astype(np.int64)


def test_calibration_selects_and_descends():
    """Algorithm 1 from the identity as R^0 (group 32, clips 0.96 / 0.92, a small window, the
    paper's lr 0.02): the selected rotations are orthogonal, their held-out objectives are no worse
    than the start's, and the value calibration lowers both its training and held-out objectives."""
    w = W.make_workload(1, batch=1, ctx=16, num_q_heads=8, num_kv_heads=2, d_model=64)
    R0 = np.broadcast_to(np.eye(128), (2, 128, 128)).copy()
    calib, held = _structured([150, 120], 7), _structured([140, 130], 8)
    mu = P.key_mean(calib[0])
    out = P.calibrate_head(R0, R0, calib, held, mu, w.W_o, 0, 4, lam=1.0, clip_k=0.96, clip_v=0.92, group=32,
                           n_last=16, sink=4, recent=16, steps=20, lr=0.02, eval_every=5)
    for R in (out["R_k"], out["R_v"]):
        assert np.abs(R @ R.T - np.eye(128)).max() <= 1e-12
    assert min(out["heldout_k"]) <= out["heldout_k"][0]
    assert min(out["heldout_v"]) < 0.6 * out["heldout_v"][0]
    assert out["value_curve"][-1] < 0.6 * out["value_curve"][0]
