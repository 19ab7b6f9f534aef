"""Oracle for n > 1 new tokens per sample against its pins (CPU only); planted
mistakes in the causal rule each fail a pin."""
import numpy as np
import pytest

import oracle
import workloads
from oracle import widen_bf16
from oracle.bifurcated import bifurcated_attention

from .pins_multitoken import MT_PINS


@pytest.mark.parametrize("pin", MT_PINS, ids=lambda p: p.__name__)
def test_c_oracle_passes(pin):
    pin(oracle.attention)


@pytest.mark.parametrize("pin", MT_PINS, ids=lambda p: p.__name__)
def test_numpy_bifurcated_passes(pin):
    pin(bifurcated_attention)


@pytest.mark.parametrize("case", [(3, 8, 2, 32, 40, 30, 4, True), (2, 4, 4, 16, 9, 5, 5, False),
                                  (5, 6, 1, 64, 17, 11, 3, True)])
def test_bifurcated_equals_replicated(case):
    """Exactness with n tokens: Eq. 3-4 with the causal rule equals the
    replicated evaluation (Appendix E.1)."""
    b, h, g, d, m_c, m_d, n, ragged = case
    x = workloads.make_inputs(b, h, g, d, m_c, m_d, seed=330, n=n, ragged=ragged)
    assert float(np.max(np.abs(bifurcated_attention(**x) - oracle.attention(**x)))) <= 1e-12


def test_rows_match_full():
    x = workloads.make_inputs(4, 8, 2, 32, 30, 20, seed=340, n=3, ragged=True)
    full = oracle.attention(**x)
    rng = np.random.default_rng(1)
    ri, rj, rt = rng.integers(0, 4, 25), rng.integers(0, 8, 25), rng.integers(0, 3, 25)
    rows = oracle.attention_rows(**x, rows_i=ri, rows_j=rj, rows_t=rt)
    assert np.array_equal(rows, full[ri, rj, rt])


def test_shapes_and_errors():
    x = workloads.make_inputs(2, 4, 2, 8, 0, 5, seed=350, n=3, lens=[1, 5])
    with pytest.raises(ValueError):  # sample 0's first token sees no key at all
        oracle.attention(**x)


def _mutant(kind):
    def attn(q, Kc, Vc, Kd, Vd, lens, scale=None):
        qf, Kcf, Vcf, Kdf, Vdf = (widen_bf16(a) for a in (q, Kc, Vc, Kd, Vd))
        b, h, n, d = qf.shape
        g, m_c, _ = Kcf.shape
        p = h // g
        if kind == "token_major_layout":
            qf = qf.reshape(b, n, h, d).transpose(0, 2, 1, 3)
        sc = 1.0 / np.sqrt(d) if scale is None else scale
        out = np.zeros((b, h, n, d))
        for i in range(b):
            L = int(lens[i])
            for j in range(h):
                gam = j // p
                for r in range(n):
                    vis = {"causal_off_by_one": L - n + r, "no_causal_mask": L,
                           "reversed_tokens": L - r}.get(kind, L - n + r + 1)
                    vis = min(max(vis, 0), L)
                    K = np.concatenate([Kcf[gam], Kdf[i, gam, :vis]])
                    V = np.concatenate([Vcf[gam], Vdf[i, gam, :vis]])
                    qv = qf[i, j, 0 if kind == "tokens_share_query" else r]
                    s = (K @ qv) * sc
                    w = np.exp(s - s.max())
                    out[i, j, r] = (w @ V) / w.sum()
        return out
    return attn


def test_unmutated_numpy_evaluator_passes():
    for pin in MT_PINS:
        pin(_mutant(None))


@pytest.mark.parametrize("kind", ["causal_off_by_one", "no_causal_mask", "reversed_tokens",
                                  "tokens_share_query", "token_major_layout"])
def test_mutation_fails_some_pin(kind):
    caught = []
    for pin in MT_PINS:
        try:
            pin(_mutant(kind))
        except (AssertionError, ValueError, FloatingPointError):
            caught.append(pin.__name__)
    assert caught, f"no pin catches {kind}"
