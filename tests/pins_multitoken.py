"""Pins for evaluators of n > 1 new tokens per sample (draft tokens verified in
one step; the appendix on speculative decoding, where n_g replaces the query
length n of Eq. 3-4).

Reading: the n new tokens are the last n of a sample's len_i valid decode
rows, and token r sees the context and the decode rows before and including
itself, i.e. the first max(0, len_i - n + r + 1) of them. ``attn`` takes q as
[b, h, n, d] (the paper's b g p n k order) and returns fp64 [b, h, n, d].

The reference for every pin is the single-token oracle (n = 1), which the
pins in tests/pins.py fix independently, or a property that any correct
evaluator has. A pin raises AssertionError when the evaluator breaks it.
"""
from __future__ import annotations

import numpy as np

import oracle
import workloads


def _close(a, b, tol, what):
    a = np.asarray(a, np.float64)
    b = np.asarray(b, np.float64)
    assert np.all(np.isfinite(a)), f"{what}: non-finite output"
    err = float(np.max(np.abs(a - b))) if a.size else 0.0
    assert err <= tol, f"{what}: max abs diff {err:.3e} > {tol:.1e}"


# (b, h, g, d, m_c, m_d, n, lens) -- lens below n, equal to n, zero, full.
_CASES = [
    (3, 4, 2, 16, 5, 9, 3, [9, 2, 4]),
    (2, 6, 3, 8, 1, 6, 4, [0, 6]),
    (4, 2, 1, 32, 7, 12, 2, [2, 12, 7, 1]),
]


def _inst(case, seed):
    b, h, g, d, m_c, m_d, n, lens = case
    return workloads.make_inputs(b, h, g, d, m_c, m_d, seed=seed, n=n, lens=lens)


def pin_mt_token_decomposition(attn):
    """Token r of an n-token step equals a one-token step of length
    max(0, len_i - n + r + 1) with that token's query."""
    for k, case in enumerate(_CASES):
        x = _inst(case, 300 + k)
        n = case[6]
        out = attn(**x)
        for r in range(n):
            one = dict(x, q=np.ascontiguousarray(x["q"][:, :, r, :]),
                       lens=np.maximum(x["lens"] - n + r + 1, 0).astype(np.int32))
            _close(out[:, :, r, :], oracle.attention(**one), 1e-13, f"{case} token {r}")


def pin_mt_causal(attn):
    """Changing the keys and values of draft token r changes no earlier
    token's output and changes token r's."""
    case = (2, 4, 2, 16, 6, 10, 4, [10, 7])
    x = _inst(case, 310)
    n = case[6]
    base = attn(**x)
    for i, L in enumerate(case[7]):
        for r in range(n):
            row = L - n + r  # the decode row holding draft token r of sample i
            y = {k: v.copy() for k, v in x.items()}
            y["Kd"][i, :, row, :] = workloads.f32_to_bf16_bits(
                np.full(case[3], 3.0, np.float32))
            y["Vd"][i, :, row, :] = workloads.f32_to_bf16_bits(
                np.full(case[3], -2.0, np.float32))
            out = attn(**y)
            assert np.array_equal(out[i, :, :r, :], base[i, :, :r, :]), \
                f"sample {i}: draft token {r} leaks into earlier tokens"
            assert not np.allclose(out[i, :, r, :], base[i, :, r, :]), \
                f"sample {i}: token {r} does not see its own row"


def pin_mt_single_token_reduces(attn):
    """n = 1 given as [b, h, 1, d] is the one-token step."""
    x = workloads.make_inputs(3, 4, 2, 16, 5, 7, seed=320, ragged=True)
    one = dict(x, q=np.ascontiguousarray(x["q"][:, :, None, :]))
    _close(attn(**one)[:, :, 0, :], oracle.attention(**x), 1e-13, "n = 1")


MT_PINS = [pin_mt_token_decomposition, pin_mt_causal, pin_mt_single_token_reduces]
