"""Bifurcated attention evaluated as the paper writes it -- TEST INFRASTRUCTURE ONLY.

numpy fp64, following Section 4.2 step by step (notation ``b g p n k``,
``n`` new tokens per sample -- 1 for incremental decoding, ``n_g`` draft
tokens for the speculative decoding of the appendix -- and ``k`` = head
dimension):

1. Eq. 3, context logits: einsum(bgpnk, g m_c k -> bgpn m_c); the context
   cache has no ``b`` axis because it is shared by all samples.
2. Eq. 3, decode logits: einsum(bgpnk, b g m_d k -> bgpn m_d).
3. Concatenate along the key axis and take one softmax over both parts
   (the paper leaves the softmax out of its listing; the scaled,
   max-subtracted softmax is the standard one). Decode positions at or beyond
   a sample's valid length get weight 0.
4. Eq. 4: split the weights at ``m_c`` and sum
   einsum(bgpn m_c, g m_c k -> bgpnk) + einsum(bgpn m_d, b g m_d k -> bgpnk).

With 8-bit caches (the FAQ on attention quantization) every cache is first
widened to its values: code value times the per-group scale of keys or
values (``widen_codes``, a numpy decoder of its own).

This module shares no code with ``oracle.c``; the two agree only because the
bifurcated method is exact (Appendix E.1).
"""
from __future__ import annotations

import numpy as np

from . import default_scale, widen_bf16, widen_codes


def bifurcated_attention(q, Kc, Vc, Kd, Vd, lens, scale=None, kv="bf16", k_scale=None,
                         v_scale=None):
    """q [b, h, k] or [b, h, n, k]; the output has q's shape."""
    qf = widen_bf16(q)
    g = np.asarray(Kc).shape[0]
    ks = np.ones(g) if k_scale is None else np.asarray(k_scale, np.float32).astype(np.float64)
    vs = np.ones(g) if v_scale is None else np.asarray(v_scale, np.float32).astype(np.float64)
    Kcf = widen_codes(Kc, kv) * ks[:, None, None]
    Vcf = widen_codes(Vc, kv) * vs[:, None, None]
    Kdf = widen_codes(Kd, kv) * ks[None, :, None, None]
    Vdf = widen_codes(Vd, kv) * vs[None, :, None, None]
    lens = np.asarray(lens, dtype=np.int64)
    if qf.ndim == 3:
        b, h, k = qf.shape
        n = 1
    else:
        b, h, n, k = qf.shape
    g, m_c, _ = Kcf.shape
    m_d = Kdf.shape[2]
    p = h // g
    if scale is None:
        scale = default_scale(k)
    valid = np.arange(m_d)[None, :] < lens[:, None]                   # [b, m_d]
    # Rows past a sample's length take no part: zero them so that whatever
    # they hold (NaN included) cannot reach the sums.
    Kdf = np.where(valid[:, None, :, None], Kdf, 0.0)
    Vdf = np.where(valid[:, None, :, None], Vdf, 0.0)
    # Token r of n sees decode positions < len_i - n + r + 1.
    seen = (np.arange(m_d)[None, None, :]
            < (lens[:, None, None] - n + np.arange(n)[None, :, None] + 1))  # [b, n, m_d]
    q5 = qf.reshape(b, g, p, n, k)                                    # bgpnk
    logits_c = np.einsum("bgpnk,gmk->bgpnm", q5, Kcf)                 # Eq. 3, context part
    logits_d = np.einsum("bgpnk,bgmk->bgpnm", q5, Kdf)                # Eq. 3, decode part
    logits = np.concatenate([logits_c, logits_d], axis=-1) * scale
    logits[..., m_c:] = np.where(seen[:, None, None, :, :], logits[..., m_c:], -np.inf)
    mu = logits.max(axis=-1, keepdims=True)
    w = np.exp(logits - mu)
    w /= w.sum(axis=-1, keepdims=True)
    o = np.einsum("bgpnm,gmk->bgpnk", w[..., :m_c], Vcf) \
        + np.einsum("bgpnm,bgmk->bgpnk", w[..., m_c:], Vdf)           # Eq. 4
    return o.reshape(qf.shape)
