"""Each plausible mistake in an oracle must fail at least one pin (CPU only).

The mutants below are small numpy evaluators of the replicated definition
(Section 3.3, Eq. 1-2) with exactly one planted mistake each. The pins in
tests/pins.py must reject every one of them, and the un-mutated evaluator must
pass them all, so the pins are strong enough to trust the oracle.
Also checks that the GPU parity gate is strong enough to reject the same
mistakes at a realistic shape, where the 1e-2 contract alone would not.
"""
import numpy as np
import pytest

import oracle
import workloads
from oracle import widen_bf16

from . import pins
from .parity import gate_errors, GATE_MAX_ABS, GATE_REL_L2


def _evaluator(mutation=None):
    def attn(q, Kc, Vc, Kd, Vd, lens, scale=None):
        qf, Kcf, Vcf, Kdf, Vdf = (widen_bf16(a) for a in (q, Kc, Vc, Kd, Vd))
        b, h, d = qf.shape
        g, m_c, _ = Kcf.shape
        m_d = Kdf.shape[2]
        if mutation == "decode_layout_transposed":
            # reads the decode cache as if it were [b, m_d, g, d]
            Kdf = Kdf.reshape(b, m_d, g, d).transpose(0, 2, 1, 3)
            Vdf = Vdf.reshape(b, m_d, g, d).transpose(0, 2, 1, 3)
        p = h // g
        sc = 1.0 / np.sqrt(d) if scale is None else scale
        out = np.zeros((b, h, d))
        with np.errstate(over="ignore", invalid="ignore"):
            for i in range(b):
                n = int(lens[i])
                if mutation == "len_plus_one":
                    n = min(n + 1, m_d)
                if mutation == "len_minus_one":
                    n = max(n - 1, 0)
                for j in range(h):
                    gam = j % g if mutation == "interleaved_groups" else j // p
                    di = (i + 1) % b if mutation == "wrong_sample_decode" else i
                    Kx = [Kcf[gam]] if mutation != "drop_context" else []
                    Vx = [Vcf[gam]] if mutation != "drop_context" else []
                    if mutation != "drop_decode":
                        Kx.append(Kdf[di, gam, :n])
                        Vx.append(Vdf[di, gam, :n])
                    K = np.concatenate(Kx)
                    V = np.concatenate(Vx)
                    if mutation == "values_from_keys":
                        V = K
                    qv = qf[i, j]
                    if mutation == "half_head_dim":
                        qv = qv.copy()
                        qv[d // 2:] = 0
                    s = K @ qv
                    if mutation == "no_scale":
                        pass
                    elif mutation == "scale_twice":
                        s = s * sc * sc
                    else:
                        s = s * sc
                    if mutation == "negated_logits":
                        s = -s
                    if mutation == "no_max_subtraction":
                        w = np.exp(s)
                    else:
                        w = np.exp(s - s.max())
                    Z = w[:m_c].sum() if mutation == "context_only_normaliser" else w.sum()
                    out[i, j] = (w @ V) / Z
        return out
    return attn


MUTATIONS = ["drop_decode", "drop_context", "interleaved_groups", "len_plus_one",
             "len_minus_one", "no_scale", "scale_twice", "negated_logits",
             "values_from_keys", "context_only_normaliser", "wrong_sample_decode",
             "no_max_subtraction", "decode_layout_transposed", "half_head_dim"]


def test_unmutated_evaluator_passes_every_pin():
    for pin in pins.ALL_PINS:
        pin(_evaluator())


@pytest.mark.parametrize("mutation", MUTATIONS)
def test_mutation_fails_some_pin(mutation):
    attn = _evaluator(mutation)
    caught = []
    for pin in pins.ALL_PINS:
        try:
            pin(attn)
        except (AssertionError, ValueError, FloatingPointError):
            # an evaluator that fails outright on a pin's input is caught too
            caught.append(pin.__name__)
    assert caught, f"no pin catches {mutation}"


@pytest.mark.parametrize("mutation", ["drop_decode", "drop_context", "interleaved_groups",
                                      "len_plus_one", "wrong_sample_decode"])
def test_parity_gate_rejects_mistake_at_realistic_shape(mutation):
    """At a GQA shape with a long context and ragged decode, a kernel making
    one of these mistakes must fail the GPU parity gate."""
    x = workloads.make_inputs(3, 8, 2, 128, 4096, 512, seed=41, ragged=True)
    ref = oracle.attention(**x)
    bad = _evaluator(mutation)(**x)
    max_abs, rel_l2 = gate_errors(bad, ref)
    assert max_abs > GATE_MAX_ABS or rel_l2 > GATE_REL_L2
