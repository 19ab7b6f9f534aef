"""Parity gate used by every GPU test.

The contract is max |gpu - oracle| <= 1e-2 for bf16 inputs with fp32
accumulation. That bound alone would accept a kernel that silently drops the
decode part on long contexts (output entries there are only ~0.005-0.02 in
size), so every GPU comparison also applies a tighter gate derived from the
kernel's arithmetic: fp32 logits, softmax statistics and accumulators, with
the softmax weights rounded to bf16 (relative error <= 2^-9) before the
weighted sum over values. Summed over m independent keys that rounding gives
an output error of order 2^-9 * |o| / sqrt(m) per entry, well under 1e-4 for
these workloads; 2e-3 max-abs and 5e-3 relative L2 leave a wide margin.
"""
import numpy as np

CONTRACT_MAX_ABS = 1e-2
GATE_MAX_ABS = 2e-3
GATE_REL_L2 = 5e-3


def gate_errors(out, ref):
    out = np.asarray(out, np.float64)
    ref = np.asarray(ref, np.float64)
    max_abs = float(np.max(np.abs(out - ref))) if out.size else 0.0
    denom = float(np.linalg.norm(ref))
    rel_l2 = float(np.linalg.norm(out - ref)) / denom if denom > 0 else 0.0
    return max_abs, rel_l2


def assert_parity(out, ref, what=""):
    out = np.asarray(out, np.float64)
    assert np.all(np.isfinite(out)), f"{what}: non-finite GPU output"
    max_abs, rel_l2 = gate_errors(out, ref)
    assert max_abs <= CONTRACT_MAX_ABS, f"{what}: max abs {max_abs:.3e} breaks the 1e-2 contract"
    assert max_abs <= GATE_MAX_ABS and rel_l2 <= GATE_REL_L2, \
        f"{what}: max abs {max_abs:.3e} / rel L2 {rel_l2:.3e} outside the gate " \
        f"({GATE_MAX_ABS:.0e} / {GATE_REL_L2:.0e})"
    return max_abs, rel_l2
