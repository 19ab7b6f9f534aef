"""Bifurcated attention as two segment statistics and their merge -- TEST INFRASTRUCTURE ONLY.

numpy fp64, an evaluation of Section 4.2 written from Eq. 3-4 (not from the
listing the paper prints). For one sample ``i`` and KV group ``gam`` the
query rows are the ``p`` heads of the group times the ``n`` new tokens
(``n = 1`` for incremental decoding; ``n_g`` draft tokens in the appendix on
speculative decoding). Eq. 3 splits their logits along the key axis into

* a context part against the group's one shared context cache (no sample
  index: every sample reads the same ``K_c``), and
* a decode part against the sample's own decode cache, of which token ``r``
  sees the first ``max(0, len_i - n + r + 1)`` rows,

and Eq. 4 splits the weighted sum of values the same way; one softmax spans
both parts. Here each part is reduced on its own to three statistics per
query row -- its largest logit ``mu``, the sum ``z`` of ``exp(logit - mu)``
over its keys and the sum ``a`` of those weights times the value rows -- and
the row's output is their merge

    M = max(mu_c, mu_d),   out = (e^(mu_c-M) a_c + e^(mu_d-M) a_d)
                                 / (e^(mu_c-M) z_c + e^(mu_d-M) z_d),

which equals the softmax over the concatenated logits applied to the
concatenated values (an empty part has ``mu = -inf`` and drops out). Rows a
token does not see are excluded before any arithmetic, so whatever they hold
(NaN included) cannot reach the result. Scale: ``1/sqrt(k)`` by default.

With 8-bit or 4-bit caches (the FAQ on attention quantization) every cache is first
widened to its values: code value times the per-group scale of keys or
values (``widen_codes``, a numpy decoder of its own).

This module shares no code with ``oracle.c``; the two agree only because the
bifurcated method is exact (Appendix E.1).
"""
from __future__ import annotations

import numpy as np

from . import default_scale, widen_bf16, widen_codes


def _segment(logits, values):
    """(mu, z, a) of one key segment for every row of ``logits`` [rows, m]
    (entries -inf where a row does not see a key) against ``values`` [m, k]."""
    rows = logits.shape[0]
    if logits.shape[1] == 0:
        return (np.full(rows, -np.inf), np.zeros(rows), np.zeros((rows, values.shape[1])))
    mu = logits.max(axis=1)
    seen = np.isfinite(mu)
    w = np.zeros_like(logits)
    w[seen] = np.exp(logits[seen] - mu[seen, None])
    return mu, w.sum(axis=1), w @ values


def _merge(parts):
    """Merge segment statistics of the same rows into the normalised output."""
    M = np.max([mu for mu, _, _ in parts], axis=0)
    num = 0.0
    den = 0.0
    for mu, z, a in parts:
        f = np.where(np.isfinite(mu), np.exp(np.where(np.isfinite(mu), mu - M, 0.0)), 0.0)
        num = num + f[:, None] * a
        den = den + f * z
    return num / den[:, None]


def bifurcated_attention(q, Kc, Vc, Kd, Vd, lens, scale=None, kv="bf16", k_scale=None,
                         v_scale=None):
    """q [b, h, k] or [b, h, n, k]; the output has q's shape."""
    qf = widen_bf16(q)
    single = qf.ndim == 3
    if single:
        qf = qf[:, :, None, :]
    b, h, n, k = qf.shape
    g, m_c, _ = np.asarray(Kc).shape
    p = h // g
    ks = np.ones(g) if k_scale is None else np.asarray(k_scale, np.float32).astype(np.float64)
    vs = np.ones(g) if v_scale is None else np.asarray(v_scale, np.float32).astype(np.float64)
    Kcf = widen_codes(Kc, kv)
    Vcf = widen_codes(Vc, kv)
    lens = np.asarray(lens, dtype=np.int64)
    if scale is None:
        scale = default_scale(k)
    out = np.empty((b, h, n, k))
    tok = np.arange(n)
    for i in range(b):
        # decode rows the sample's tokens see, at most len_i of them
        vis = np.maximum(0, lens[i] - n + tok + 1)            # [n]
        L = int(vis.max()) if n else 0
        for gam in range(g):
            Q = qf[i, gam * p:(gam + 1) * p].reshape(p * n, k)  # rows head-major, then token
            Kg, Vg = Kcf[gam] * ks[gam], Vcf[gam] * vs[gam]
            ctx = _segment(scale * (Q @ Kg.T), Vg)              # Eq. 3 / Eq. 4, context part
            Kdi = widen_codes(np.asarray(Kd)[i, gam, :L], kv) * ks[gam]
            Vdi = widen_codes(np.asarray(Vd)[i, gam, :L], kv) * vs[gam]
            s_d = scale * (Q @ Kdi.T) if L else np.zeros((p * n, 0))
            row_vis = np.tile(vis, p)                            # row r = head * n + token
            s_d = np.where(np.arange(L)[None, :] < row_vis[:, None], s_d, -np.inf)
            dec = _segment(s_d, Vdi)                             # Eq. 3 / Eq. 4, decode part
            out[i, gam * p:(gam + 1) * p] = _merge([ctx, dec]).reshape(p, n, k)
    return out[:, :, 0, :] if single else out
