"""Pins for any attention evaluator with the oracle's interface.

Each pin checks one fact that the paper and the mathematics fix, independently
of how the evaluator is written: closed forms, invariants and brute force on
tiny inputs. ``attn(q, Kc, Vc, Kd, Vd, lens, scale)`` takes bf16 bit patterns
(uint16) and returns fp64 ``[b, h, d]``. A pin raises AssertionError when the
evaluator breaks it.

The oracle must pass all of them (tests/test_oracle_pins.py); planted mistakes
must each fail at least one (tests/test_pin_power.py).
"""
from __future__ import annotations

import math
from fractions import Fraction

import numpy as np

import workloads
from oracle import widen_bf16


def _bits(x):
    return workloads.f32_to_bf16_bits(np.asarray(x, dtype=np.float32))


def _inst(b, h, g, d, m_c, m_d, seed, ragged=True, lens=None, poison=False):
    return workloads.make_inputs(b, h, g, d, m_c, m_d, seed=seed, ragged=ragged,
                                 lens=lens, poison_tail=poison)


def _close(a, b, tol, what):
    a = np.asarray(a, np.float64)
    b = np.asarray(b, np.float64)
    err = float(np.max(np.abs(a - b))) if a.size else 0.0
    assert np.all(np.isfinite(a)), f"{what}: non-finite output"
    assert err <= tol, f"{what}: max abs diff {err:.3e} > {tol:.1e}"


def pin_zero_query_is_mean(attn):
    """q = 0 makes every logit 0, so the weights are uniform and the output is
    the plain mean of the sample's m_c + len_i value rows (Section 3.3)."""
    x = _inst(3, 4, 2, 8, 5, 4, seed=11)
    x["q"][:] = 0
    out = attn(**x, scale=0.3)
    Vc, Vd = widen_bf16(x["Vc"]), widen_bf16(x["Vd"])
    for i in range(3):
        for j in range(4):
            gam = j // 2
            rows = list(Vc[gam]) + list(Vd[i, gam, :x["lens"][i]])
            exp = [math.fsum(r[u] for r in rows) / len(rows) for u in range(8)]
            _close(out[i, j], exp, 1e-14, "zero query")


def pin_single_key(attn):
    """m_c = 1 and len_i = 0: the softmax has one entry, the output is that
    context value row, whatever the query."""
    x = _inst(2, 6, 3, 16, 1, 3, seed=12, lens=[0, 0])
    out = attn(**x, scale=0.25)
    Vc = widen_bf16(x["Vc"])
    for j in range(6):
        _close(out[:, j], np.stack([Vc[j // 2, 0]] * 2), 0.0, "single key")


def _exact_logit(qrow, krow, scale):
    s = sum((Fraction(float(a)) * Fraction(float(c)) for a, c in zip(qrow, krow)), Fraction(0))
    return float(s) * scale


def pin_two_keys_sigmoid(attn):
    """One context row and one decode row: the weights are the logistic
    sigmoid of the logit difference, out = sig(s1-s2) v1 + sig(s2-s1) v2."""
    x = _inst(3, 2, 1, 8, 1, 2, seed=13, lens=[1, 1, 1])
    sc = 0.7
    out = attn(**x, scale=sc)
    q, Kc, Vc = widen_bf16(x["q"]), widen_bf16(x["Kc"]), widen_bf16(x["Vc"])
    Kd, Vd = widen_bf16(x["Kd"]), widen_bf16(x["Vd"])
    for i in range(3):
        for j in range(2):
            s1 = _exact_logit(q[i, j], Kc[0, 0], sc)
            s2 = _exact_logit(q[i, j], Kd[i, 0, 0], sc)
            w1 = 1.0 / (1.0 + math.exp(s2 - s1))
            w2 = 1.0 / (1.0 + math.exp(s1 - s2))
            _close(out[i, j], w1 * Vc[0, 0] + w2 * Vd[i, 0, 0], 1e-14, "two keys")


def pin_constant_values(attn):
    """All value rows equal c: the weights sum to one, so the output is c."""
    x = _inst(4, 8, 4, 16, 9, 6, seed=14)
    c = _bits(np.linspace(-2, 2, 16))
    x["Vc"][:] = c
    x["Vd"][:] = c
    out = attn(**x, scale=0.5)
    _close(out, np.broadcast_to(widen_bf16(c), out.shape), 1e-14, "constant values")


def pin_dominant_key(attn):
    """One key whose logit exceeds every other by >= 60: the output is that
    key's value row to within e^-60 (exercises the max-subtracted softmax at
    logits far beyond exp's range)."""
    d = 8
    x = _inst(2, 2, 2, d, 6, 3, seed=15, lens=[3, 3])
    x["q"][:] = _bits(np.full(d, 8.0))
    x["Kc"][:] = _bits(np.zeros(d))
    x["Kd"][:] = _bits(np.zeros(d))
    # decode row 1 of sample 1, group 1 dominates: logit 8*8*8*scale
    x["Kd"][1, 1, 1] = _bits(np.full(d, 8.0))
    x["Kc"][0, 2] = _bits(np.full(d, 8.0))   # context row 2 of group 0 dominates there
    sc = 1.0
    out = attn(**x, scale=sc)
    Vc, Vd = widen_bf16(x["Vc"]), widen_bf16(x["Vd"])
    _close(out[1, 1], Vd[1, 1, 1], 1e-20, "dominant decode key")
    _close(out[0, 0], Vc[0, 2], 1e-20, "dominant context key")
    _close(out[1, 0], Vc[0, 2], 1e-20, "dominant context key")


def pin_brute_force(attn):
    """Tiny shapes: exact rational dot products, fsum-accumulated weights."""
    for (b, h, g, d, m_c, m_d, seed) in [(2, 4, 2, 4, 3, 2, 16), (3, 3, 1, 5, 2, 3, 17),
                                          (1, 2, 2, 8, 6, 1, 18), (3, 4, 4, 3, 1, 4, 19)]:
        x = _inst(b, h, g, d, m_c, m_d, seed=seed)
        sc = 1.0 / math.sqrt(d)
        out = attn(**x, scale=sc)
        q, Kc, Vc = widen_bf16(x["q"]), widen_bf16(x["Kc"]), widen_bf16(x["Vc"])
        Kd, Vd = widen_bf16(x["Kd"]), widen_bf16(x["Vd"])
        p = h // g
        for i in range(b):
            for j in range(h):
                gam = j // p
                keys = list(Kc[gam]) + list(Kd[i, gam, :x["lens"][i]])
                vals = list(Vc[gam]) + list(Vd[i, gam, :x["lens"][i]])
                s = [_exact_logit(q[i, j], kr, sc) for kr in keys]
                mu = max(s)
                w = [math.exp(t - mu) for t in s]
                Z = math.fsum(w)
                exp = [math.fsum(wt * vr[u] for wt, vr in zip(w, vals)) / Z for u in range(d)]
                _close(out[i, j], exp, 1e-14, f"brute force {(b, h, g, d, m_c, m_d)}")


def pin_b1_equivalence(attn):
    """Batch rows are independent: row i of a b-sample call equals a b = 1
    call on (q_i, Kd_i, Vd_i, len_i) (Section 3.2: batch size 1 reduces to
    single-context inference)."""
    x = _inst(4, 4, 2, 16, 10, 7, seed=20)
    out = attn(**x, scale=0.25)
    for i in range(4):
        one = attn(q=x["q"][i:i + 1], Kc=x["Kc"], Vc=x["Vc"], Kd=x["Kd"][i:i + 1],
                   Vd=x["Vd"][i:i + 1], lens=x["lens"][i:i + 1], scale=0.25)
        _close(out[i], one[0], 1e-15, "b=1 equivalence")


def pin_group_repeat(attn):
    """Multi-group with g groups equals multi-head with every KV group
    repeated p times, group-major (head j reads group j // p, Section 3.3);
    g = 1 is multi-query."""
    for g in (1, 2):
        x = _inst(3, 4, g, 8, 7, 5, seed=21 + g)
        p = 4 // g
        out = attn(**x, scale=0.4)
        rep = dict(x)
        rep["Kc"] = np.repeat(x["Kc"], p, axis=0)
        rep["Vc"] = np.repeat(x["Vc"], p, axis=0)
        rep["Kd"] = np.repeat(x["Kd"], p, axis=1)
        rep["Vd"] = np.repeat(x["Vd"], p, axis=1)
        mha = attn(**rep, scale=0.4)
        _close(out, mha, 1e-15, f"g={g} vs repeated multi-head")


def pin_split_point(attn):
    """Moving decode rows that every sample shares into the context leaves the
    output unchanged (Eq. 3-4 split the key axis at an arbitrary m_c)."""
    b, g, d, m_c, m_d, t = 3, 2, 8, 5, 6, 2
    x = _inst(b, 4, g, d, m_c, m_d, seed=24, lens=[4, 6, 3])
    for i in range(1, b):
        x["Kd"][i, :, :t] = x["Kd"][0, :, :t]
        x["Vd"][i, :, :t] = x["Vd"][0, :, :t]
    out = attn(**x, scale=0.35)
    y = dict(x)
    y["Kc"] = np.concatenate([x["Kc"], x["Kd"][0, :, :t]], axis=1)
    y["Vc"] = np.concatenate([x["Vc"], x["Vd"][0, :, :t]], axis=1)
    y["Kd"] = np.ascontiguousarray(x["Kd"][:, :, t:])
    y["Vd"] = np.ascontiguousarray(x["Vd"][:, :, t:])
    y["lens"] = x["lens"] - t
    moved = attn(**y, scale=0.35)
    _close(out, moved, 1e-14, "split point")


def pin_permutation(attn):
    """Permuting the samples permutes the outputs."""
    x = _inst(5, 4, 2, 8, 6, 5, seed=25)
    out = attn(**x, scale=0.3)
    perm = np.array([3, 0, 4, 1, 2])
    y = dict(x)
    for key in ("q", "Kd", "Vd", "lens"):
        y[key] = np.ascontiguousarray(x[key][perm])
    _close(attn(**y, scale=0.3), out[perm], 0.0, "sample permutation")


def pin_masked_tail(attn):
    """Decode rows at or beyond len_i never reach the output: NaN there
    changes nothing (n = 1, so the only mask is the valid length)."""
    x = _inst(4, 4, 2, 8, 6, 7, seed=26)
    y = _inst(4, 4, 2, 8, 6, 7, seed=26, poison=True)
    _close(attn(**y, scale=0.3), attn(**x, scale=0.3), 0.0, "masked tail")


def pin_context_only(attn):
    """len_i = 0 for every sample: plain attention over the context alone,
    identical for every sample that has the same query."""
    x = _inst(3, 2, 2, 8, 6, 4, seed=27, lens=[0, 0, 0])
    x["q"][1] = x["q"][0]
    out = attn(**x, scale=0.3)
    _close(out[1], out[0], 0.0, "context only, same query")
    y = _inst(3, 2, 2, 8, 6, 4, seed=27, lens=[0, 0, 0])
    y["q"][1] = y["q"][0]
    y["Kd"][:] = _bits(np.full(8, 50.0))  # never read: lens are 0
    _close(attn(**y, scale=0.3), out, 0.0, "context only ignores decode cache")


ALL_PINS = [pin_zero_query_is_mean, pin_single_key, pin_two_keys_sigmoid, pin_constant_values,
            pin_dominant_key, pin_brute_force, pin_b1_equivalence, pin_group_repeat,
            pin_split_point, pin_permutation, pin_masked_tail, pin_context_only]
