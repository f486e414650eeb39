"""CPU oracle of OptR's offline calibration (Sec. 4.2 - 4.5, Algorithm 1 of the appendix).

TEST INFRASTRUCTURE ONLY, like int2kv_oracle: nothing in the product path imports or calls it; it
shares no code with the HIP library. It is written in fp64 with plain PyTorch CPU ops, and its
gradients come from torch's automatic differentiation (the library derives its own by hand), so
the two agree only if both derivations are right.

What it computes, per KV head h with query heads j in its group G_h:

* corrected rotations (eq:OptR_skew): R(A) = R^0 exp(A - A^T);
* effective INT2 keys (Sec. 4.1): k~_s = Q2((k_s - mu) R_K) R_K^T, in the centered basis (the
  constant mu leaves every softmax unchanged); effective values v~_s = Q2(v_s R_V) R_V^T;
* Q2 is the cache's quantizer (int2kv_oracle.quantize: group-wise affine INT2 with clip ratio c,
  fp16 scale and zero) applied to the fp32 rounding of the fp64 rotated row, so that calibration
  sees exactly the codes the cache write would store;
* the straight-through estimator of eq:OptR_ste. Reading: the quantizer passes the gradient of an
  element unchanged when it lies inside its group's clipped range [c mn, c mx] (the range the
  affine grid covers) and blocks it outside; scale and zero carry no gradient;
* BF16 sink and recent windows (appendix, Algorithm 1): for a query at position t, tokens
  s < sink and s > t - recent keep their full-precision (centered) keys and exact values;
* the key objective (eq:OptR_key_attention, eq:key_output_error, eq:OptR_key_loss): over rows
  (t, j), t among the final n_last positions of each sequence, attention over s <= t,
      L_K = mean_rows [ KL(p_t || p^K_t) + lambda_K ||((p^K_t - p_t)^T V) W_{O,j}^T||^2 / d_model ];
* the value objective (eq:value_output_error, eq:OptR_value_loss) under the selected key
  rotation's distribution p^K-hat:
      L_V = mean_rows ||(p^K-hat_t^T (V~ - V)) W_{O,j}^T||^2 / d_model;
* Algorithm 1: A = 0, T Adam steps (torch.optim.Adam, the paper's lr 0.02) on L_K, the iterate
  with the lowest held-out L_K among A = 0 and every eval_every-th step is selected; then the same
  for A_V on L_V. Reading: the start A = 0 is a candidate of the selection too.
"""
from __future__ import annotations

import numpy as np
import torch

from oracle import int2kv_oracle as O

D = 128
_NEG = -1.0e300  # masked logits: exp gives exactly 0, and logs stay finite (no 0 * inf)


def key_mean(k_bits: np.ndarray) -> np.ndarray:
    """Per-channel mean of the calibration keys per KV head (appendix, key-mean estimation):
    fp64 mean over tokens, rounded to fp32. k_bits: bf16 [T, H, 128] -> [H, 128]."""
    return O.bf16_to_f64(k_bits).mean(axis=0).astype(np.float32)


def rotation(R0: np.ndarray, A: torch.Tensor) -> torch.Tensor:
    """R^0 exp(A - A^T) (fp64), eq:OptR_skew."""
    return torch.as_tensor(R0, dtype=torch.float64) @ torch.linalg.matrix_exp(A - A.T)


def _fake_quant(Z: torch.Tensor, clip: float, group: int, frozen=None) -> torch.Tensor:
    """Q2 of the fp32 rounding of Z with the straight-through gradient of the reading above.
    With frozen = (deq0, inside0, Z0) from an earlier point, returns the straight-through
    surrogate deq0 + inside0 (Z - Z0) instead: smooth in Z, with the same gradient at Z0."""
    if frozen is not None:
        deq0, inside0, Z0 = frozen
        return deq0 + inside0 * (Z - Z0)
    z32 = Z.detach().numpy().astype(np.float32)
    codes, s, z = O.quantize(z32, clip, group)
    deq = torch.from_numpy(O.dequantize(codes, s, z))
    g = z32.reshape(z32.shape[:-1] + (D // group, group))
    lo = g.min(axis=-1, keepdims=True)
    hi = g.max(axis=-1, keepdims=True)
    if clip != 1.0:
        lo = (np.float32(clip) * lo).astype(np.float32)
        hi = (np.float32(clip) * hi).astype(np.float32)
    inside = torch.from_numpy(((g >= lo) & (g <= hi)).reshape(z32.shape).astype(np.float64))
    return deq + inside * (Z - Z.detach())


def _rows(seq_starts, n_last):
    """(sequence, start, length, first query position) of each calibration sequence."""
    out = []
    for n in range(len(seq_starts) - 1):
        a, b = int(seq_starts[n]), int(seq_starts[n + 1])
        L = b - a
        if L > 0:
            out.append((n, a, L, max(0, L - n_last)))
    return out


def _int2_mask(L, t0, sink, recent):
    """[rows t = t0 .. L-1, tokens s = 0 .. L-1]: 1 where token s is read from the INT2 cache by
    the query at t, 0 where it is a window token or in the future (s > t)."""
    t = np.arange(t0, L)[:, None]
    s = np.arange(L)[None, :]
    return (s <= t) & (s >= sink) & (s <= t - recent)


def _causal(L, t0):
    t = np.arange(t0, L)[:, None]
    s = np.arange(L)[None, :]
    return s <= t


def _softmax_rows(logits: torch.Tensor, valid: np.ndarray) -> torch.Tensor:
    x = logits.masked_fill(torch.from_numpy(~valid), _NEG)
    return torch.softmax(x, dim=-1)


def _log_softmax_rows(logits: torch.Tensor, valid: np.ndarray) -> torch.Tensor:
    x = logits.masked_fill(torch.from_numpy(~valid), _NEG)
    return torch.log_softmax(x, dim=-1)


def key_loss(A, R0, k_bits, v_bits, q_bits, seq_starts, mu, W_o_bits, h, gq, lam=1.0, clip=1.0, group=128,
             n_last=64, sink=0, recent=0, frozen=None):
    """L_K of KV head h at generator A (a torch fp64 [128, 128] tensor, possibly requiring grad).
    k_bits, v_bits: bf16 [T, H, 128]; q_bits: bf16 [T, H_q, 128]; seq_starts: [N + 1] token
    offsets; mu: fp32 [H, 128]; W_o_bits: bf16 [d_model, H_q * 128]."""
    R = rotation(R0[h], A)
    Kc = torch.from_numpy(O.bf16_to_f64(k_bits[:, h]) - mu[h].astype(np.float64))
    V = torch.from_numpy(O.bf16_to_f64(v_bits[:, h]))
    Q = torch.from_numpy(O.bf16_to_f64(q_bits))
    W = torch.from_numpy(O.bf16_to_f64(W_o_bits))
    dm = W.shape[0]
    Kq = _fake_quant(Kc @ R, clip, group, frozen) @ R.T
    scale = 1.0 / np.sqrt(D)
    total, count = 0.0, 0
    for n, a, L, t0 in _rows(seq_starts, n_last):
        causal = _causal(L, t0)
        use_q = torch.from_numpy(_int2_mask(L, t0, sink, recent))
        for j in range(h * gq, (h + 1) * gq):
            q = Q[a + t0:a + L, j]                                   # [rows, 128]
            full = (q @ Kc[a:a + L].T) * scale
            quant = (q @ Kq[a:a + L].T) * scale
            logits_k = torch.where(use_q, quant, full)
            p = _softmax_rows(full, causal)
            lp = _log_softmax_rows(full, causal)
            lpk = _log_softmax_rows(logits_k, causal)
            pk = torch.exp(lpk)
            kl = torch.where(torch.from_numpy(causal), p * (lp - lpk), torch.zeros_like(p)).sum(-1)
            e = ((pk - p) @ V[a:a + L]) @ W[:, j * D:(j + 1) * D].T
            total = total + (kl + lam * (e * e).sum(-1) / dm).sum()
            count += L - t0
    return total / count


def key_probs(R0, A, k_bits, q_bits, seq_starts, mu, h, gq, clip=1.0, group=128, n_last=64, sink=0, recent=0):
    """p^K-hat of every row under the key rotation R^0 exp(A - A^T) (no gradient): a list of
    [rows, L] arrays, one per (sequence, query head) in the order the losses visit them."""
    with torch.no_grad():
        R = rotation(R0[h], torch.as_tensor(A, dtype=torch.float64))
        Kc = torch.from_numpy(O.bf16_to_f64(k_bits[:, h]) - mu[h].astype(np.float64))
        Q = torch.from_numpy(O.bf16_to_f64(q_bits))
        Kq = _fake_quant(Kc @ R, clip, group) @ R.T
        out = []
        for n, a, L, t0 in _rows(seq_starts, n_last):
            causal = _causal(L, t0)
            use_q = torch.from_numpy(_int2_mask(L, t0, sink, recent))
            for j in range(h * gq, (h + 1) * gq):
                q = Q[a + t0:a + L, j]
                logits = torch.where(use_q, q @ Kq[a:a + L].T, q @ Kc[a:a + L].T) / np.sqrt(D)
                out.append(_softmax_rows(logits, causal).numpy())
        return out


def value_loss(A, R0, v_bits, seq_starts, probs, W_o_bits, h, gq, clip=1.0, group=128, n_last=64, sink=0,
               recent=0, frozen=None):
    """L_V of KV head h at generator A under the fixed distributions `probs` (key_probs)."""
    R = rotation(R0[h], A)
    V = torch.from_numpy(O.bf16_to_f64(v_bits[:, h]))
    W = torch.from_numpy(O.bf16_to_f64(W_o_bits))
    dm = W.shape[0]
    Vq = _fake_quant(V @ R, clip, group, frozen) @ R.T
    total, count, i = 0.0, 0, 0
    for n, a, L, t0 in _rows(seq_starts, n_last):
        use_q = torch.from_numpy(_int2_mask(L, t0, sink, recent).astype(np.float64))
        for j in range(h * gq, (h + 1) * gq):
            p = torch.from_numpy(probs[i]) * use_q                  # window tokens add nothing
            i += 1
            e = (p @ (Vq[a:a + L] - V[a:a + L])) @ W[:, j * D:(j + 1) * D].T
            total = total + ((e * e).sum(-1) / dm).sum()
            count += L - t0
    return total / count


def calibrate_head(R0_k, R0_v, calib, heldout, mu, W_o_bits, h, gq, lam=1.0, clip_k=1.0, clip_v=1.0, group=128,
                   n_last=64, sink=0, recent=0, steps=80, lr=0.02, eval_every=20):
    """Algorithm 1 for one KV head. calib / heldout: (k_bits, v_bits, q_bits, seq_starts).
    Returns dict(A_k, A_v, R_k, R_v (fp64), key_curve, value_curve, heldout_k, heldout_v): the
    training losses before each step and the held-out losses of the candidates."""
    kw = dict(group=group, n_last=n_last, sink=sink, recent=recent)

    def lk(A, data):
        k, v, q, st = data
        return key_loss(A, R0_k, k, v, q, st, mu, W_o_bits, h, gq, lam, clip_k, **kw)

    A = torch.zeros((D, D), dtype=torch.float64, requires_grad=True)
    opt = torch.optim.Adam([A], lr=lr)
    best = (float(lk(A.detach(), heldout)), A.detach().clone())
    held_k, curve_k = [best[0]], []
    for i in range(1, steps + 1):
        opt.zero_grad()
        loss = lk(A, calib)
        curve_k.append(float(loss.detach()))
        loss.backward()
        opt.step()
        if i % eval_every == 0:
            hl = float(lk(A.detach(), heldout))
            held_k.append(hl)
            if hl < best[0]:
                best = (hl, A.detach().clone())
    A_k = best[1]

    probs_c = key_probs(R0_k, A_k, calib[0], calib[2], calib[3], mu, h, gq, clip_k, **kw)
    probs_h = key_probs(R0_k, A_k, heldout[0], heldout[2], heldout[3], mu, h, gq, clip_k, **kw)

    def lv(A, data, probs):
        return value_loss(A, R0_v, data[1], data[3], probs, W_o_bits, h, gq, clip_v, **kw)

    B = torch.zeros((D, D), dtype=torch.float64, requires_grad=True)
    opt = torch.optim.Adam([B], lr=lr)
    best = (float(lv(B.detach(), heldout, probs_h)), B.detach().clone())
    held_v, curve_v = [best[0]], []
    for i in range(1, steps + 1):
        opt.zero_grad()
        loss = lv(B, calib, probs_c)
        curve_v.append(float(loss.detach()))
        loss.backward()
        opt.step()
        if i % eval_every == 0:
            hl = float(lv(B.detach(), heldout, probs_h))
            held_v.append(hl)
            if hl < best[0]:
                best = (hl, B.detach().clone())
    A_v = best[1]
    with torch.no_grad():
        R_k = rotation(R0_k[h], A_k).numpy()
        R_v = rotation(R0_v[h], A_v).numpy()
    return dict(A_k=A_k.numpy(), A_v=A_v.numpy(), R_k=R_k, R_v=R_v, key_curve=curve_k, value_curve=curve_v,
                heldout_k=held_k, heldout_v=held_v)


def frozen_point(R0, A, x_bits, h, clip, group, mu=None):
    """(deq0, inside0, Z0) of the rows x (keys centered by mu when given) at generator A: the
    point a straight-through surrogate expands around (see _fake_quant)."""
    with torch.no_grad():
        R = rotation(R0[h], torch.as_tensor(A, dtype=torch.float64))
        X = O.bf16_to_f64(x_bits[:, h])
        if mu is not None:
            X = X - mu[h].astype(np.float64)
        Z = torch.from_numpy(X) @ R
    Zr = Z.clone().requires_grad_(True)
    out = _fake_quant(Zr, clip, group)
    inside0 = torch.autograd.grad(out.sum(), Zr)[0]
    return out.detach(), inside0, Z
