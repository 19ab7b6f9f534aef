"""Pins for evaluators of attention over quantized KV caches (the FAQ on
attention quantization: int8 codes halve the KV bytes of bf16, int4 codes
quarter them, and the method is unchanged).

Reading: a cache holds 8-bit codes (OCP fp8 E4M3 or two's complement int8)
or 4-bit codes (two's complement int4, two per byte, element 2u in the low
nibble of byte u of the row) with one fp32 scale per KV group for keys
(``k_scale[g]``) and one for values (``v_scale[g]``), shared by the context
and decode caches; a key is ``k_scale[gam]`` times its code's value.
``attn(**x)`` takes the inputs of ``workloads.make_inputs(..., kv=...)``
(codes as uint8) and returns fp64.

The code values every pin expects come from library routines that do not
share the evaluators' decoders: torch's ``float8_e4m3fn`` cast, numpy's int8
view, and for int4 numpy's ``unpackbits`` with the two's complement bit
weights (1, 2, 4, -8). The attention itself is compared with the bf16
oracle, which the pins of tests/pins.py fix independently, and the int4
attention with the int8 attention on 16 times the codes.
"""
from __future__ import annotations

import numpy as np

import oracle
import workloads

KVS = ("fp8_e4m3", "int8", "int4")

_NIBBLE_WEIGHTS = np.array([1, 2, 4, 8])


def code_table(kv: str) -> np.ndarray:
    """Value of each code from a library routine: the 256 8-bit codes (NaN
    for the two fp8 NaN codes), or the 16 int4 codes."""
    if kv == "int4":
        bits = np.unpackbits(np.arange(16, dtype=np.uint8)[:, None], axis=1, bitorder="little")
        return (bits[:, :4] @ np.array([1, 2, 4, -8])).astype(np.float64)
    codes = np.arange(256, dtype=np.uint8)
    if kv == "int8":
        return codes.view(np.int8).astype(np.float64)
    import torch
    return torch.from_numpy(codes).view(torch.float8_e4m3fn).to(torch.float64).numpy()


def elements(stored, kv: str) -> np.ndarray:
    """The code (an index into code_table(kv)) of every element of a cache
    array: the bytes themselves, or for int4 the two nibbles of each byte
    in element order, low nibble first (bits from numpy's unpackbits)."""
    a = np.asarray(stored).astype(np.uint8)
    if kv != "int4":
        return a.astype(np.int64)
    bits = np.unpackbits(a[..., None], axis=-1, bitorder="little")  # [..., d/2, 8]
    pair = np.stack([bits[..., :4] @ _NIBBLE_WEIGHTS, bits[..., 4:] @ _NIBBLE_WEIGHTS], axis=-1)
    return pair.reshape(a.shape[:-1] + (2 * a.shape[-1],))


def stored(codes, kv: str) -> np.ndarray:
    """Element codes (indices into code_table(kv)) -> the cache array: the
    codes as bytes, or for int4 two per byte, element 2u in the low nibble
    of byte u and element 2u+1 in the high nibble."""
    c = np.asarray(codes).astype(np.uint8)
    if kv != "int4":
        return c
    return (c[..., 0::2] | (c[..., 1::2] << 4)).astype(np.uint8)


def fill_code(kv: str, code: int) -> np.uint8:
    """The byte that sets every element it covers to `code`."""
    return np.uint8(code | (code << 4)) if kv == "int4" else np.uint8(code)


def _finite_codes(kv):
    """The codes with finite values (all but 0x7F and 0xFF in fp8; all 16
    int4 codes)."""
    t = code_table(kv)
    return np.nonzero(np.isfinite(t))[0].astype(np.uint8)


def _close(a, b, tol, what):
    a = np.asarray(a, np.float64)
    b = np.asarray(b, np.float64)
    assert np.all(np.isfinite(a)), f"{what}: non-finite output"
    err = float(np.max(np.abs(a - b))) if a.size else 0.0
    assert err <= tol, f"{what}: max abs diff {err:.3e} > {tol:.1e}"


def _one(kv):
    return 0x38 if kv == "fp8_e4m3" else 1  # the code of 1.0


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
        x["Vc"] = stored(vc.reshape(g, 1, d), kv)
        x["v_scale"] = np.array([0.75, 3.0, 0.1][:g], np.float32)
        out = attn(**x)
        table = code_table(kv)
        for j in range(2 * g):
            gam = j // 2
            exp = float(x["v_scale"][gam]) * table[elements(x["Vc"], kv)[gam, 0]]
            _close(out[:, j], np.broadcast_to(exp, out[:, j].shape), 0.0, f"{kv} value table")


def pin_kvq_key_table(attn):
    """Two keys: a context key of code value 0 and one decode key whose code
    is under test. With q one-hot at dimension u the decode key's weight is
    sigmoid(scale * k_scale * value(code)), so the output (value rows 0 and 1)
    is v_scale times that. Head j of sample i tests code (64 i + j) mod the
    number of codes at u = j."""
    for kv in KVS:
        table = code_table(kv)
        b, h, d = 4, 64, 64
        x = workloads.make_inputs(b, h, 1, d, 1, 1, seed=401, kv=kv, lens=[1] * b)
        x["q"] = workloads.f32_to_bf16_bits(np.broadcast_to(np.eye(h, d, dtype=np.float32),
                                                            (b, h, d)).copy())
        x["Kc"][:] = 0
        x["Vc"][:] = 0
        x["Vd"][:] = fill_code(kv, _one(kv))
        kd = (np.arange(b * d) % table.size).reshape(b, d)
        if kv == "fp8_e4m3":
            kd = np.where(np.isfinite(table[kd]), kd, 0)  # NaN codes -> 0
        x["Kd"] = stored(kd.reshape(b, 1, 1, d), kv)
        ks, vs, sc = 2.0 ** -9 * 1.3, 0.7, 0.5
        x["k_scale"] = np.array([ks], np.float32)
        x["v_scale"] = np.array([vs], np.float32)
        out = attn(**x, scale=sc)
        for i in range(b):
            for j in range(h):
                code = elements(x["Kd"], kv)[i, 0, 0, j]
                z = sc * float(np.float32(ks)) * table[code]
                w = 1.0 / (1.0 + np.exp(-z))
                _close(out[i, j], np.full(d, float(np.float32(vs)) * w), 1e-15,
                       f"{kv} key table code {code}")


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
        vals = table[elements(x[name], kv)] * sc.astype(np.float64).reshape(shape)
        vals = vals.astype(np.float32)
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


def pin_kvq_int4_is_int8_of_sixteen_times(attn):
    """An int4 problem is the int8 problem whose codes are 16 times the int4
    codes' values and whose scales are 1/16 of the int4 scales: every
    dequantized key and value is the same number (exactly: the scales are
    fp32 and 1/16 is a power of two), so the outputs agree to fp64 rounding.
    Ties the int4 decoding, nibble order included, to the pinned int8 one."""
    for k, (b, h, g, d, m_c, m_d, n) in enumerate([(3, 8, 2, 32, 40, 12, 2),
                                                   (2, 6, 3, 16, 9, 7, 1)]):
        x = workloads.make_inputs(b, h, g, d, m_c, m_d, seed=470 + k, ragged=True, n=n,
                                  kv="int4")
        rng = np.random.default_rng(470 + k)
        for name in ("Kc", "Vc", "Kd", "Vd"):  # every code, -8 included
            x[name] = rng.integers(0, 256, x[name].shape, dtype=np.uint8)
        t4 = code_table("int4")
        y = dict(x, kv="int8", k_scale=(x["k_scale"] / 16).astype(np.float32),
                 v_scale=(x["v_scale"] / 16).astype(np.float32))
        for name in ("Kc", "Vc", "Kd", "Vd"):
            y[name] = (16 * t4[elements(x[name], "int4")]).astype(np.int8).view(np.uint8)
        ref = attn(**y)
        _close(attn(**x), ref, 1e-13 * max(1.0, float(np.max(np.abs(ref)))),
               "int4 vs int8 of sixteen times the codes")


QUANT_PINS = [pin_kvq_value_table, pin_kvq_key_table, pin_kvq_equals_bf16_of_values,
              pin_kvq_scale_identities, pin_kvq_int4_is_int8_of_sixteen_times]
