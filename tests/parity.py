"""Parity gate used by every GPU test.

The contract is max |gpu - oracle| <= 1e-2 for bf16 inputs with fp32
accumulation. That bound alone would accept a kernel that silently drops the
decode part on long contexts (output entries there are only ~0.005-0.02 in
size), so every GPU comparison also applies a relative-L2 gate derived from
the kernel's arithmetic.

Error model: logits, softmax statistics and accumulators are fp32; the
softmax weights enter the weighted sum over values rounded to bf16 (relative
error <= 2^-9 each, independent across keys). The output is a weighted mean
of value rows with random signs, so those roundings perturb it by about
2^-9/sqrt(3) ~ 1.1e-3 of its own norm (measured: 1.1e-3 to 1.7e-3 relative
L2 on every workload); fp32 summation adds orders of magnitude less. The
gate allows 5e-3 relative L2. Per entry the same rounding is bounded by
2^-9 * max_t |v_t| (~1e-2 for N(0,1) values), but few-key rows with O(1)
outputs reach ~2e-3 in practice, so the max-abs gate is 5e-3.
"""
import numpy as np

CONTRACT_MAX_ABS = 1e-2
GATE_MAX_ABS = 5e-3
GATE_REL_L2 = 5e-3


def gate_errors(out, ref):
    out = np.asarray(out, np.float64)
    ref = np.asarray(ref, np.float64)
    max_abs = float(np.max(np.abs(out - ref))) if out.size else 0.0
    denom = float(np.linalg.norm(ref))
    rel_l2 = float(np.linalg.norm(out - ref)) / denom if denom > 0 else 0.0
    return max_abs, rel_l2


def assert_parity(out, ref, what="", gate_max_abs=GATE_MAX_ABS):
    """gate_max_abs: a test whose softmax is much sharper than the workloads'
    (a few bf16-rounded weights then make up an output entry) may raise the
    max-abs gate up to the contract, never the relative-L2 gate."""
    assert gate_max_abs <= CONTRACT_MAX_ABS
    out = np.asarray(out, np.float64)
    assert np.all(np.isfinite(out)), f"{what}: non-finite GPU output"
    max_abs, rel_l2 = gate_errors(out, ref)
    assert max_abs <= CONTRACT_MAX_ABS, f"{what}: max abs {max_abs:.3e} breaks the 1e-2 contract"
    assert max_abs <= gate_max_abs and rel_l2 <= GATE_REL_L2, \
        f"{what}: max abs {max_abs:.3e} / rel L2 {rel_l2:.3e} outside the gate " \
        f"({gate_max_abs:.0e} / {GATE_REL_L2:.0e})"
    return max_abs, rel_l2
