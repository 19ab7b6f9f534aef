"""Oracle over 8-bit and 4-bit KV caches against its pins (CPU only); planted
mistakes in the decoding or the scales each fail a pin."""
import numpy as np
import pytest

import oracle
import workloads
from oracle import widen_bf16
from oracle.bifurcated import bifurcated_attention

from .pins_kvquant import KVS, QUANT_PINS, code_table, elements, stored


def test_code_tables_match_library():
    """Both decoders against torch's float8_e4m3fn cast and numpy's int8
    view over all 256 codes (NaN where the library gives NaN), and against
    the int4 table from numpy's unpackbits over all 16 codes."""
    for kv in KVS:
        ref = code_table(kv)
        codes = np.arange(ref.size, dtype=np.uint8)
        c_side = np.array([oracle.code_value(kv, int(c)) for c in codes])
        np_side = oracle.widen_codes(stored(codes, kv), kv)
        for got in (c_side, np_side):
            assert np.array_equal(np.isnan(got), np.isnan(ref))
            assert np.array_equal(got[~np.isnan(ref)], ref[~np.isnan(ref)])


def test_int4_every_byte_unpacks_low_nibble_first():
    """All 256 bytes: the numpy decoder yields (value of the low nibble,
    value of the high nibble) per byte, as the unpackbits table says."""
    b = np.arange(256, dtype=np.uint8).reshape(16, 16)
    got = oracle.widen_codes(b, "int4")
    assert got.shape == (16, 32)
    assert np.array_equal(got, code_table("int4")[elements(b, "int4")])
    assert np.array_equal(got[:, 0::2], code_table("int4")[np.arange(256).reshape(16, 16) & 15])


def test_int4_anchors():
    """Two's complement 4-bit values: 0..7 as they are, 8 -> -8, 15 -> -1."""
    for c, v in {0: 0.0, 1: 1.0, 7: 7.0, 8: -8.0, 9: -7.0, 14: -2.0, 15: -1.0}.items():
        assert oracle.code_value("int4", c) == v


def test_fp8_spec_anchors():
    """Values the OCP E4M3 definition fixes: bias 7, subnormals m/8 * 2^-6,
    largest finite 448, S.1111.111 NaN, signed zero."""
    anchors = {0x00: 0.0, 0x01: 2.0 ** -9, 0x07: 7 * 2.0 ** -9, 0x08: 2.0 ** -6, 0x38: 1.0,
               0x39: 1.125, 0x40: 2.0, 0x7E: 448.0, 0xB8: -1.0, 0xFE: -448.0}
    for c, v in anchors.items():
        assert oracle.code_value("fp8_e4m3", c) == v
    assert np.isnan(oracle.code_value("fp8_e4m3", 0x7F))
    assert np.isnan(oracle.code_value("fp8_e4m3", 0xFF))
    assert np.signbit(oracle.code_value("fp8_e4m3", 0x80))


@pytest.mark.parametrize("pin", QUANT_PINS, ids=lambda p: p.__name__)
def test_c_oracle_passes(pin):
    pin(oracle.attention)


@pytest.mark.parametrize("pin", QUANT_PINS, ids=lambda p: p.__name__)
def test_numpy_bifurcated_passes(pin):
    pin(bifurcated_attention)


@pytest.mark.parametrize("kv", KVS)
@pytest.mark.parametrize("case", [(3, 8, 2, 32, 40, 30, 1, True), (2, 4, 4, 16, 9, 5, 3, True),
                                  (5, 6, 1, 64, 17, 11, 2, False)])
def test_bifurcated_equals_replicated(kv, case):
    """Exactness over 8-bit caches (Appendix E.1): the numpy Eq. 3-4 and the
    replicated C evaluation agree."""
    b, h, g, d, m_c, m_d, n, ragged = case
    x = workloads.make_inputs(b, h, g, d, m_c, m_d, seed=430, n=n, ragged=ragged, kv=kv,
                              poison_tail=True)
    assert float(np.max(np.abs(bifurcated_attention(**x) - oracle.attention(**x)))) <= 1e-12


@pytest.mark.parametrize("kv", KVS)
def test_rows_match_full(kv):
    x = workloads.make_inputs(4, 8, 2, 32, 30, 20, seed=440, n=2, ragged=True, kv=kv)
    full = oracle.attention(**x)
    rng = np.random.default_rng(2)
    ri, rj, rt = rng.integers(0, 4, 25), rng.integers(0, 8, 25), rng.integers(0, 2, 25)
    rows = oracle.attention_rows(**x, rows_i=ri, rows_j=rj, rows_t=rt)
    assert np.array_equal(rows, full[ri, rj, rt])


def test_generator_recipe():
    """Codes are the saturated RNE encodings of the draws times qmax / 4.5;
    the scales undo that factor up to the per-group factors in [1/2, 2]."""
    for kv in KVS:
        x = workloads.make_inputs(2, 4, 2, 16, 64, 8, seed=450, kv=kv)
        vals = oracle.widen_codes(x["Kc"], kv)
        assert np.all(np.abs(vals) <= workloads.KV_QMAX[kv])
        base = workloads.KV_CLIP_SIGMA / workloads.KV_QMAX[kv]
        for sc in (x["k_scale"], x["v_scale"]):
            assert sc.dtype == np.float32 and sc.shape == (2,)
            assert np.all(sc >= base / 2 * (1 - 1e-6)) and np.all(sc <= base * 2 * (1 + 1e-6))
        # the unscaled code values have roughly unit spread in units of base
        assert 0.8 < float(np.std(vals * base)) < 1.2


def test_bad_arguments():
    x = workloads.make_inputs(2, 4, 2, 8, 4, 3, seed=460, kv="int8")
    with pytest.raises(ValueError):
        oracle.attention(**dict(x, kv="int2"))
    with pytest.raises(ValueError):  # 8-bit arrays (d bytes a row) handed over as int4 (d/2)
        oracle.attention(**dict(x, kv="int4"))
    with pytest.raises(ValueError):
        workloads.make_inputs(2, 4, 2, 7, 4, 3, seed=460, kv="int4")  # odd d
    with pytest.raises(ValueError):
        oracle.attention(**dict(x, k_scale=np.ones(3, np.float32)))
    with pytest.raises(ValueError):  # 8-bit codes handed over as bf16 bit patterns
        oracle.attention(**dict(x, kv="bf16"))


def _mutant(kind):
    """A plain numpy evaluator over the replicated cache with one planted
    mistake in the decoding or the scales."""
    def decode(codes, kv):
        c = np.asarray(codes).astype(np.int64)
        if kv == "int4":
            lo, hi = c & 15, c >> 4
            if kind == "int4_nibbles_swapped":
                lo, hi = hi, lo
            nib = np.stack([lo, hi], axis=-1).reshape(c.shape[:-1] + (2 * c.shape[-1],))
            return (nib if kind == "int4_unsigned" else nib - 16 * (nib >= 8)).astype(np.float64)
        if kv == "int8":
            return (c if kind == "int8_unsigned" else c - 256 * (c >= 128)).astype(np.float64)
        e, m = (c >> 3) & 15, (c & 7).astype(np.float64)
        bias = 8 if kind == "fp8_bias8" else 7
        if kind == "fp8_no_subnormals":
            mag = (1 + m / 8) * np.exp2(e - bias)
        else:
            mag = np.where(e == 0, m / 8 * np.exp2(1.0 - bias), (1 + m / 8) * np.exp2(e - bias))
        mag = np.where((e == 15) & (m == 7), np.nan, mag)
        return np.where(c >= 128, -mag, mag)

    def attn(q, Kc, Vc, Kd, Vd, lens, scale=None, kv="bf16", k_scale=None, v_scale=None):
        qf = widen_bf16(q)
        if qf.ndim == 3:
            qf = qf[:, :, None, :]
        b, h, n, d = qf.shape
        g, m_c, _ = Kc.shape
        p = h // g
        ks = np.asarray(k_scale, np.float64)
        vs = np.asarray(v_scale, np.float64)
        if kind == "swap_kv_scales":
            ks, vs = vs, ks
        sc = 1.0 / np.sqrt(d) if scale is None else scale
        out = np.zeros((b, h, n, d))
        for i in range(b):
            L = int(lens[i])
            for j in range(h):
                gam = j // p
                kd_s = 1.0 if kind == "no_scale_on_decode" else ks[gam]
                vg = (j % g) if kind == "head_major_scale_index" else gam
                for r in range(n):
                    vis = max(L - n + r + 1, 0)
                    K = np.concatenate([decode(Kc[gam], kv) * ks[gam],
                                        decode(Kd[i, gam, :vis], kv) * kd_s])
                    V = np.concatenate([decode(Vc[gam], kv), decode(Vd[i, gam, :vis], kv)])
                    s = (K @ qf[i, j, r]) * sc
                    w = np.exp(s - s.max())
                    out[i, j, r] = vs[vg] * (w @ V) / w.sum()
        return out if np.asarray(q).ndim == 4 else out[:, :, 0, :]
    return attn


def test_unmutated_evaluator_passes():
    for pin in QUANT_PINS:
        pin(_mutant(None))


@pytest.mark.parametrize("kind", ["fp8_bias8", "fp8_no_subnormals", "int8_unsigned",
                                  "int4_unsigned", "int4_nibbles_swapped",
                                  "swap_kv_scales", "no_scale_on_decode",
                                  "head_major_scale_index"])
def test_mutation_fails_some_pin(kind):
    caught = []
    for pin in QUANT_PINS:
        try:
            pin(_mutant(kind))
        except (AssertionError, ValueError, FloatingPointError):
            caught.append(pin.__name__)
    assert caught, f"no pin catches {kind}"
