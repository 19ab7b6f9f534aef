"""Pins for evaluators of attention over 8-bit KV caches (the FAQ on attention
quantization: int8 codes halve the KV bytes of bf16 and leave the method
unchanged).

Reading: a cache holds 8-bit codes (OCP fp8 E4M3 or two's complement int8)
with one fp32 scale per KV group for keys (``k_scale[g]``) and one for values
(``v_scale[g]``), shared by the context and decode caches; a key is
``k_scale[gam]`` times its code's value. ``attn(**x)`` takes the inputs of
``workloads.make_inputs(..., kv=...)`` (codes as uint8) and returns fp64.

The code values every pin expects come from library routines that do not
share the evaluators' decoders: torch's ``float8_e4m3fn`` cast and numpy's
int8 view. The attention itself is compared with the bf16 oracle, which the
pins of tests/pins.py fix independently.
"""
from __future__ import annotations

import numpy as np

import oracle
import workloads

KVS = ("fp8_e4m3", "int8")


def code_table(kv: str) -> np.ndarray:
    """Value of each of the 256 codes from a library routine (NaN for the
    two fp8 NaN codes)."""
    codes = np.arange(256, dtype=np.uint8)
    if kv == "int8":
        return codes.view(np.int8).astype(np.float64)
    import torch
    return torch.from_numpy(codes).view(torch.float8_e4m3fn).to(torch.float64).numpy()


def _finite_codes(kv):
    """The codes with finite values (all but 0x7F and 0xFF in fp8)."""
    t = code_table(kv)
    return np.nonzero(np.isfinite(t))[0].astype(np.uint8)


def _close(a, b, tol, what):
    a = np.asarray(a, np.float64)
    b = np.asarray(b, np.float64)
    assert np.all(np.isfinite(a)), f"{what}: non-finite output"
    err = float(np.max(np.abs(a - b))) if a.size else 0.0
    assert err <= tol, f"{what}: max abs diff {err:.3e} > {tol:.1e}"


def _one(kv):
    return np.uint8(0x38) if kv == "fp8_e4m3" else np.uint8(1)  # the code of 1.0


def pin_kvq_value_table(attn):
    """One context key and no decode rows: the weight is 1, so every output
    is v_scale[gam] times the value of the context value code under it. The
    value rows hold every finite code."""
    for kv in KVS:
        codes = _finite_codes(kv)
        d = 128
        g = -(-codes.size // d)
        x = workloads.make_inputs(2, 2 * g, g, d, 1, 2, seed=400, kv=kv, lens=[0, 0])
        vc = np.zeros(g * d, np.uint8)
        vc[:codes.size] = codes
        x["Vc"] = vc.reshape(g, 1, d)
        x["v_scale"] = np.array([0.75, 3.0, 0.1][:g], np.float32)
        out = attn(**x)
        table = code_table(kv)
        for j in range(2 * g):
            gam = j // 2
            exp = float(x["v_scale"][gam]) * table[x["Vc"][gam, 0]]
            _close(out[:, j], np.broadcast_to(exp, out[:, j].shape), 0.0, f"{kv} value table")


def pin_kvq_key_table(attn):
    """Two keys: a context key of code value 0 and one decode key whose code
    is under test. With q one-hot at dimension u the decode key's weight is
    sigmoid(scale * k_scale * value(code)), so the output (value rows 0 and 1)
    is v_scale times that. Head j of sample i tests code 64 i + j at u = j."""
    for kv in KVS:
        table = code_table(kv)
        b, h, d = 4, 64, 64
        x = workloads.make_inputs(b, h, 1, d, 1, 1, seed=401, kv=kv, lens=[1] * b)
        x["q"] = workloads.f32_to_bf16_bits(np.broadcast_to(np.eye(h, d, dtype=np.float32),
                                                            (b, h, d)).copy())
        x["Kc"][:] = 0
        x["Vc"][:] = 0
        x["Vd"][:] = _one(kv)
        kd = np.arange(256, dtype=np.uint8).reshape(b, d)
        if kv == "fp8_e4m3":
            kd = np.where(np.isfinite(table[kd]), kd, np.uint8(0))  # NaN codes -> 0
        x["Kd"] = kd.reshape(b, 1, 1, d).astype(np.uint8)
        ks, vs, sc = 2.0 ** -9 * 1.3, 0.7, 0.5
        x["k_scale"] = np.array([ks], np.float32)
        x["v_scale"] = np.array([vs], np.float32)
        out = attn(**x, scale=sc)
        for i in range(b):
            for j in range(h):
                z = sc * float(np.float32(ks)) * table[x["Kd"][i, 0, 0, j]]
                w = 1.0 / (1.0 + np.exp(-z))
                _close(out[i, j], np.full(d, float(np.float32(vs)) * w), 1e-15,
                       f"{kv} key table code {x['Kd'][i, 0, 0, j]}")


def _dequantized_bf16(x):
    """The same problem with bf16 caches holding the dequantized values
    (exact when the scales are powers of two)."""
    kv = x["kv"]
    table = code_table(kv)
    y = {k: v for k, v in x.items() if k not in ("kv", "k_scale", "v_scale")}
    for name, sc, grp in (("Kc", x["k_scale"], 0), ("Vc", x["v_scale"], 0),
                          ("Kd", x["k_scale"], 1), ("Vd", x["v_scale"], 1)):
        shape = [1] * x[name].ndim
        shape[grp] = -1
        vals = (table[x[name]] * sc.astype(np.float64).reshape(shape)).astype(np.float32)
        bits = workloads.f32_to_bf16_bits(vals)
        assert np.array_equal(oracle.widen_bf16(bits)[np.isfinite(vals)],
                              vals[np.isfinite(vals)].astype(np.float64))
        y[name] = bits
    return y


def pin_kvq_equals_bf16_of_values(attn):
    """With power-of-two scales every dequantized value is a bf16 value, so
    the 8-bit problem is the bf16 problem on those values (up to fp64
    rounding order): several tokens, ragged lengths, per-group scales, a
    poisoned tail."""
    for kv in KVS:
        for k, (b, h, g, d, m_c, m_d, n) in enumerate([(3, 8, 2, 32, 40, 12, 2),
                                                       (2, 4, 4, 16, 9, 6, 1)]):
            x = workloads.make_inputs(b, h, g, d, m_c, m_d, seed=410 + k, ragged=True, n=n,
                                      kv=kv)
            x["k_scale"] = np.exp2(np.arange(g) - 3.0).astype(np.float32)
            x["v_scale"] = np.exp2(2.0 - np.arange(g)).astype(np.float32)
            ref = oracle.attention(**_dequantized_bf16(x))
            for i in range(b):  # poison after building the reference
                x["Kd"][i, :, x["lens"][i]:] = workloads.KV_POISON[kv]
                x["Vd"][i, :, x["lens"][i]:] = workloads.KV_POISON[kv]
            _close(attn(**x), ref, 1e-13 * max(1.0, float(np.max(np.abs(ref)))),
                   f"{kv} vs bf16 of the dequantized values")


def pin_kvq_scale_identities(attn):
    """Per group: multiplying k_scale by s equals multiplying the softmax
    scale by s, and multiplying v_scale by t multiplies the output by t."""
    for kv in KVS:
        x = workloads.make_inputs(3, 6, 3, 16, 11, 7, seed=420, ragged=True, kv=kv)
        base = attn(**dict(x, k_scale=np.ones(3, np.float32), v_scale=np.ones(3, np.float32)),
                    scale=0.25)
        s = np.array([0.37, 1.9, 0.061], np.float32)
        t = np.array([2.3, 0.41, 1.0], np.float32)
        out = attn(**dict(x, k_scale=s, v_scale=t), scale=0.25)
        for gam in range(3):
            heads = slice(2 * gam, 2 * gam + 2)
            y = dict(x, k_scale=np.ones(3, np.float32), v_scale=np.ones(3, np.float32))
            folded = attn(**y, scale=0.25 * float(s[gam]))
            _close(out[:, heads], float(t[gam]) * folded[:, heads], 1e-12,
                   f"{kv} group {gam} scale identities")
        assert not np.allclose(out, base), "scales ignored"


QUANT_PINS = [pin_kvq_value_table, pin_kvq_key_table, pin_kvq_equals_bf16_of_values,
              pin_kvq_scale_identities]
