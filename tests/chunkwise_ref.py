"""Chunkwise (tile-parallel) form of the gated delta rule in fp64 numpy.

Test-only.  This is an independent formulation used to pin the token-by-token
oracle; it is not the oracle and the product library never sees it.

Derivation (from Eq. 1 / Eq. 2 of Section 3.2).  Inside a tile of n tokens
with entry state S0 (d_v x d_k), let gamma_r = sum_{j<=r} g_j,
Gamma_r = exp(gamma_r) and D_ri = exp(gamma_r - gamma_i).  Unrolling Eq. 2,
the decayed state seen by token r is Gamma_r S0 + sum_{i<r} D_ri e_i k_i^T,
so the writes e_r satisfy the unit lower-triangular system

    e_r + beta_r sum_{i<r} D_ri (k_r . k_i) e_i = beta_r (v_r - Gamma_r S0 k_r)

i.e. (I + A) E = diag(beta) (V - diag(Gamma) K S0^T) with
A_ri = beta_r D_ri (k_r . k_i) for i < r.  Then

    O   = diag(Gamma) Q S0^T + (D (.) Q K^T)_{i<=r} E
    S_n = Gamma_last S0 + E^T diag(D_last,.) K
"""
from __future__ import annotations

import numpy as np

from synth import bf16_bits_to_f64


def _tile(Q, K, V, g, beta, S0):
    n = Q.shape[0]
    gam = np.cumsum(g)
    Gam = np.exp(gam)
    Dm = np.exp(gam[:, None] - gam[None, :])
    low = np.tril(np.ones((n, n)), -1)
    low_incl = np.tril(np.ones((n, n)), 0)
    A = beta[:, None] * Dm * (K @ K.T) * low
    T = np.linalg.inv(np.eye(n) + A)
    R = V - Gam[:, None] * (K @ S0.T)
    E = T @ (beta[:, None] * R)
    O = Gam[:, None] * (Q @ S0.T) + ((Dm * low_incl) * (Q @ K.T)) @ E
    d_last = np.exp(gam[-1] - gam)
    S = Gam[-1] * S0 + E.T @ (d_last[:, None] * K)
    return O, S


def chunkwise_forward(q, k, v, g, beta, cu_seqlens, frame_len, C=64, S0=None, scale=1.0):
    """Same outputs as the oracle's gdn_forward (o, S, partials), tile by tile.

    Tiles of C tokens restart at every frame boundary, so every frame end is
    a tile end.
    """
    q = bf16_bits_to_f64(q)
    k = bf16_bits_to_f64(k)
    v = bf16_bits_to_f64(v)
    g = np.asarray(g, np.float64)
    beta = np.asarray(beta, np.float64)
    T, H_k, d_k = q.shape
    H_v, d_v = v.shape[1:]
    grp = H_v // H_k
    B = len(cu_seqlens) - 1
    o = np.zeros((T, H_v, d_v))
    S_out = np.zeros((B, H_v, d_v, d_k))
    parts = []
    for b in range(B):
        t0, t1 = int(cu_seqlens[b]), int(cu_seqlens[b + 1])
        n = t1 - t0
        if n <= 0:
            if S0 is not None:
                S_out[b] = S0[b]
            continue
        fl = frame_len if frame_len > 0 else n
        frames = [(s, min(s + fl, n)) for s in range(0, n, fl)]
        fparts = np.zeros((len(frames), H_v, 2))
        for j in range(H_v):
            h = j // grp
            S = np.zeros((d_v, d_k)) if S0 is None else np.array(S0[b, j], np.float64)
            for fi, (fs, fe) in enumerate(frames):
                S_start = S.copy()
                for ts in range(fs, fe, C):
                    te = min(ts + C, fe)
                    sl = slice(t0 + ts, t0 + te)
                    O, S = _tile(q[sl, h], k[sl, h], v[sl, j], g[sl, j], beta[sl, j], S)
                    o[sl, j] = scale * O
                fparts[fi, j, 0] = np.sum((S - S_start) ** 2)
                fparts[fi, j, 1] = np.sum(S_start ** 2)
            S_out[b, j] = S
        parts.append(fparts)
    partials = np.concatenate(parts, axis=0) if parts else np.zeros((0, H_v, 2))
    return dict(o=o, S=S_out, partials=partials)


def eq1_forward(q, k, v, g, beta, T_len, H_k, H_v, S0=None):
    """Eq. 1 literally: S_t = S_{t-1} (alpha_t (I - beta_t k_t k_t^T)) + beta_t v_t k_t^T,
    with the d_k x d_k product formed explicitly; one stream; returns (o, S)."""
    q = bf16_bits_to_f64(q)
    k = bf16_bits_to_f64(k)
    v = bf16_bits_to_f64(v)
    d_k = q.shape[2]
    d_v = v.shape[2]
    grp = H_v // H_k
    o = np.zeros((T_len, H_v, d_v))
    S_all = np.zeros((H_v, d_v, d_k))
    I = np.eye(d_k)
    for j in range(H_v):
        h = j // grp
        S = np.zeros((d_v, d_k)) if S0 is None else np.array(S0[j], np.float64)
        for t in range(T_len):
            a = np.exp(float(g[t, j]))
            bt = float(beta[t, j])
            kt = k[t, h]
            S = S @ (a * (I - bt * np.outer(kt, kt))) + bt * np.outer(v[t, j], kt)
            o[t, j] = S @ q[t, h]
        S_all[j] = S
    return o, S_all
