"""The oracle against what the paper and the mathematics fix (CPU only)."""
import numpy as np
import pytest

import oracle
import workloads
from oracle import bifurcated

from . import pins


@pytest.mark.parametrize("pin", pins.ALL_PINS, ids=lambda f: f.__name__)
def test_oracle_pin(pin):
    pin(oracle.attention)


@pytest.mark.parametrize("pin", pins.ALL_PINS, ids=lambda f: f.__name__)
def test_bifurcated_formulation_pin(pin):
    # The numpy evaluation of Eq. 3-4 is held to the same pins.
    pin(bifurcated.bifurcated_attention)


@pytest.mark.parametrize("shape", [
    (4, 4, 4, 64, 128, 16, False),     # the tiny multi-head layer
    (3, 8, 2, 32, 50, 20, True),       # GQA, ragged
    (5, 6, 1, 16, 33, 9, True),        # MQA, ragged
    (2, 2, 2, 8, 1, 0, False),         # no decode rows at all
])
def test_exactness_bifurcated_equals_replicated(shape):
    """Section 4.2 / Appendix E.1: the bifurcated computation (Eq. 3-4 with one
    joint softmax) equals standard attention over the replicated cache."""
    b, h, g, d, m_c, m_d, ragged = shape
    x = workloads.make_inputs(b, h, g, d, m_c, m_d, seed=31, ragged=ragged)
    ref = oracle.attention(**x)
    bif = bifurcated.bifurcated_attention(**x)
    assert np.max(np.abs(ref - bif)) <= 1e-12


def test_rows_variant_matches_full():
    x = workloads.make_inputs(4, 8, 2, 32, 40, 12, seed=32, ragged=True)
    full = oracle.attention(**x)
    ri = np.array([0, 3, 2, 1, 3])
    rj = np.array([7, 0, 4, 5, 3])
    rows = oracle.attention_rows(**x, rows_i=ri, rows_j=rj)
    assert np.array_equal(rows, full[ri, rj])


def test_thread_count_does_not_change_result():
    x = workloads.make_inputs(6, 8, 4, 32, 64, 16, seed=33, ragged=True)
    assert np.array_equal(oracle.attention(**x, nthreads=1), oracle.attention(**x, nthreads=4))


def test_oracle_rejects_bad_input():
    x = workloads.make_inputs(2, 4, 2, 8, 4, 3, seed=34)
    bad = dict(x)
    bad["lens"] = np.array([1, 4], np.int32)
    with pytest.raises(ValueError):
        oracle.attention(**bad)
    bad["lens"] = np.array([-1, 0], np.int32)
    with pytest.raises(ValueError):
        oracle.attention(**bad)
    with pytest.raises(ValueError):
        oracle.attention(q=x["q"][:, :3], Kc=x["Kc"], Vc=x["Vc"], Kd=x["Kd"], Vd=x["Vd"],
                         lens=x["lens"])


def test_generator_is_deterministic_and_rounds_to_nearest_even():
    a = workloads.make_inputs(2, 2, 1, 8, 4, 4, seed=5, ragged=True)
    b = workloads.make_inputs(2, 2, 1, 8, 4, 4, seed=5, ragged=True)
    for k in a:
        assert np.array_equal(a[k], b[k])
    # 1 + 2^-8 is exactly halfway between bf16 1.0 and 1+2^-7: ties to even (1.0)
    x = np.array([1.0 + 2.0 ** -8, 1.0 + 3 * 2.0 ** -8, -2.5, 0.0], dtype=np.float32)
    bits = workloads.f32_to_bf16_bits(x)
    assert list(oracle.widen_bf16(bits)) == [1.0, 1.0 + 2 ** -6, -2.5, 0.0]


def test_io_model_matches_section_4_3():
    """Section 4.3: KV IO g*k*(m_c + b*m_d) bifurcated vs g*k*b*(m_c + m_d);
    K and V, 2 bytes each."""
    w = workloads.WORKLOADS[workloads.HEADLINE]
    lens = np.full(w.b, w.m_d_max)
    assert workloads.kv_bytes(w.g, w.d, w.m_c, lens) == 2 * 2 * w.g * w.d * (w.m_c + w.b * w.m_d_max)
    assert workloads.kv_bytes(w.g, w.d, w.m_c, lens) == 402_653_184
    assert workloads.replicated_kv_bytes(w.b, w.g, w.d, w.m_c, lens) == \
        2 * 2 * w.g * w.d * w.b * (w.m_c + w.m_d_max)


def test_io_model_golden_values():
    import json
    import os
    path = os.path.join(os.path.dirname(__file__), "golden", "io_model.json")
    for c in json.load(open(path))["cases"]:
        lens = np.full(c["b"], c["m_d"])
        assert workloads.kv_bytes(c["g"], c["d"], c["m_c"], lens) == c["bifurcated_bytes"]
        assert workloads.replicated_kv_bytes(c["b"], c["g"], c["d"], c["m_c"], lens) == \
            c["replicated_bytes"]
