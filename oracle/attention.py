"""fp64 decode attention over the dequantized D-Quant cache (oracle).

TEST INFRASTRUCTURE ONLY -- see the package header.

What the paper fixes
--------------------
* App. A: a key channel is reconstructed as k_hat_tj = s_t v_{m_tj} + o_t + mu_j
  (mu: windowed channel mean), a value channel as s_t v_{m_tj} + o_t, where the
  reconstruction level v_m of symbol m is m itself on the affine grid of
  Eq. (affine_token).
* Eq. (fold-key): q . k_hat_t = s_t sum_j q_j v_{m_tj} + o_t sum_j q_j
  + sum_j q_j mu_j.
* Eq. (fold-value): sum_t a_t v_hat_tj = sum_t (a_t s_t) v_{m_tj} + sum_t a_t o_t.

Readings
--------
* A1 the reconstruction lives in the rotated basis; with the unnormalized
  Sylvester H (H H^T = d I) the original-basis key is H k_hat / d, so the logit
  is (H q) . k_hat / d and the output is H (sum_t a_t v_hat_t) / d.
* A2 a query head i reads KV head floor(i / G) (GQA); the logit is
  softmax_scale * q . k (softmax_scale = 1/sqrt(d) by default) and the softmax
  runs over the first seq_len[b] tokens of sequence b.
* A3 residual window: Sec. 5.1 keeps the most recent tokens in BF16.  A
  sequence is then seq_len[b] compressed tokens followed by res_len[b] raw
  tokens (original basis, no rotation, no mean removal), and the softmax runs
  over all of them; a sequence with no tokens at all gives 0.
* A4 prerotated tensors (reading V0 of kv): keys coded without rotation are
  in the caller's basis, and so is the query (logit q . k_hat, no 1/d);
  values coded without rotation give the output in their own basis
  (sum_t a_t v_hat_t, no inverse rotation), which the caller's output
  projection absorbs.  Raw residual tokens are taken in the same bases.
"""

from __future__ import annotations

import numpy as np

from . import hadamard


def dequantize(sym, s16, o16, mean_hat=None, window=128):
    """Rotated-basis reconstruction [..., T, d] in fp64."""
    x = s16.astype(np.float64)[..., None] * sym.astype(np.float64) + o16.astype(np.float64)[..., None]
    if mean_hat is not None:
        x = x + np.repeat(mean_hat, window, axis=-2)[..., : x.shape[-2], :]
    return x


def attention_direct(q, k_rot, v_rot, seq_lens, gqa, softmax_scale, rotate_k=True, rotate_v=True):
    """Textbook softmax(q K^T * scale) V in the original basis, fp64.

    q [B, Hq, d] fp64; k_rot, v_rot [B, Hkv, T, d] rotated reconstructions
    (in the caller's basis when rotate_k / rotate_v is False, reading A4).
    """
    B, Hq, d = q.shape
    H = hadamard.sylvester(d).astype(np.float64)
    k = k_rot @ H / d if rotate_k else k_rot
    v = v_rot @ H / d if rotate_v else v_rot
    out = np.zeros((B, Hq, d), dtype=np.float64)
    for b in range(B):
        T = int(seq_lens[b])
        if T == 0:
            continue            # no tokens: the output stays 0 (reading A3)
        for i in range(Hq):
            h = i // gqa
            s = (k[b, h, :T] @ q[b, i]) * softmax_scale
            s = s - s.max()
            a = np.exp(s)
            a = a / a.sum()
            out[b, i] = a @ v[b, h, :T]
    return out


def attention_folded(q, k_sym, k_s, k_o, k_mean_hat, v_sym, v_s, v_o, seq_lens,
                     gqa, softmax_scale, window=128, rotate_k=True, rotate_v=True):
    """Eq. (fold-key) / Eq. (fold-value) evaluated directly on the symbols, fp64.

    k_mean_hat [B, Hkv, T/W, d] or None.  rotate_k / rotate_v False: the
    keys / values were coded without rotation (reading A4).
    """
    B, Hq, d = q.shape
    q_rot = hadamard.fwht(q) if rotate_k else q
    scale = softmax_scale / d if rotate_k else softmax_scale
    out = np.zeros((B, Hq, d), dtype=np.float64)
    for b in range(B):
        T = int(seq_lens[b])
        if T == 0:
            continue            # no tokens: the output stays 0 (reading A3)
        for i in range(Hq):
            h = i // gqa
            qr = q_rot[b, i]
            dot = k_sym[b, h, :T].astype(np.float64) @ qr
            logit = k_s[b, h, :T].astype(np.float64) * dot + k_o[b, h, :T].astype(np.float64) * qr.sum()
            if k_mean_hat is not None:
                logit = logit + np.repeat(k_mean_hat[b, h] @ qr, window)[:T]
            s = logit * scale
            s = s - s.max()
            a = np.exp(s)
            a = a / a.sum()
            acc = (a * v_s[b, h, :T].astype(np.float64)) @ v_sym[b, h, :T].astype(np.float64)
            acc = acc + (a * v_o[b, h, :T].astype(np.float64)).sum()
            out[b, i] = hadamard.fwht(acc) / d if rotate_v else acc
    return out


def attention_with_residual(q, k_rot, v_rot, seq_lens, res_k, res_v, res_lens, gqa, softmax_scale,
                            rotate_k=True, rotate_v=True):
    """Decode attention over compressed tokens and a raw residual window, fp64.

    q [B, Hq, d]; k_rot, v_rot [B, Hkv, T, d] rotated reconstructions of the
    compressed tokens; res_k, res_v [B, Hkv, R, d] raw residual tokens, of
    which the first res_lens[b] are in use.  Textbook softmax over the union
    of the two sets in the original basis (reading A3; the caller's basis
    for tensors coded without rotation, reading A4).
    """
    B, Hq, d = q.shape
    H = hadamard.sylvester(d).astype(np.float64)
    k = k_rot @ H / d if rotate_k else k_rot
    v = v_rot @ H / d if rotate_v else v_rot
    out = np.zeros((B, Hq, d), dtype=np.float64)
    for b in range(B):
        T, R = int(seq_lens[b]), int(res_lens[b])
        for i in range(Hq):
            h = i // gqa
            keys = np.concatenate([k[b, h, :T], res_k[b, h, :R]], axis=0)
            vals = np.concatenate([v[b, h, :T], res_v[b, h, :R]], axis=0)
            if keys.shape[0] == 0:
                continue
            s = (keys @ q[b, i]) * softmax_scale
            s = s - s.max()
            a = np.exp(s)
            a = a / a.sum()
            out[b, i] = a @ vals
    return out
