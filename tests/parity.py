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
gate allows 5e-3 relative L2.

Max-abs gate, split by how many keys a row sees. Per entry the same rounding
is bounded by 2^-9 * max_t |v_t| (~1e-2 for N(0,1) values), reached only when
one weight carries the entry. Rows over long sequences average thousands of
independently rounded weights (measured max-abs on the five workloads:
0.8e-4 to 7.6e-4), so the gate there is 2e-3. Two kinds of rows come closer
to the per-entry bound and get 5e-3 (measured up to 3.6e-3):
  * few keys: some row sees fewer than FEW_KEYS keys (a single context key,
    short contexts with several tokens), so single weights are O(0.1-1);
  * sharpened softmax: 8-bit caches, whose per-group key scales make some
    groups' logits up to 2x larger than the bf16 workloads'.
Tests that sharpen the softmax further on purpose (key scales up to 8x) may
pass the contract bound itself; the relative-L2 gate is never raised.

The gates are stated for values of unit spread, as the bf16 workloads draw
them. 8-bit caches carry per-group value scales that spread the groups'
values by up to 2x either way, and the rounding error of an output entry
scales with its group's values; so for a full output of an 8-bit problem
both sides are first divided, per head, by the spread of its group's values
(value_units).
"""
import numpy as np

CONTRACT_MAX_ABS = 1e-2
GATE_MAX_ABS = 2e-3
GATE_MAX_ABS_FEW_KEYS = 5e-3
GATE_REL_L2 = 5e-3
FEW_KEYS = 256


def gate_max_abs_for(x):
    """The max-abs gate for the rows of problem x (a make_inputs dict)."""
    q = np.asarray(x["q"])
    n = 1 if q.ndim == 3 else q.shape[2]
    m_c = np.asarray(x["Kc"]).shape[1]
    lens = np.asarray(x["lens"])
    min_keys = m_c + max(0, int(lens.min()) - n + 1) if lens.size else m_c
    if min_keys < FEW_KEYS or x.get("kv", "bf16") != "bf16":
        return GATE_MAX_ABS_FEW_KEYS
    return GATE_MAX_ABS


def gate_errors(out, ref):
    out = np.asarray(out, np.float64)
    ref = np.asarray(ref, np.float64)
    max_abs = float(np.max(np.abs(out - ref))) if out.size else 0.0
    denom = float(np.linalg.norm(ref))
    rel_l2 = float(np.linalg.norm(out - ref)) / denom if denom > 0 else 0.0
    return max_abs, rel_l2


def value_units(x):
    """Per query head: the value scale of its group times the standard
    deviation of the group's value codes (context and valid decode rows)."""
    from .pins_kvquant import code_table, elements
    b, h = x["q"].shape[:2]
    g = x["Vc"].shape[0]
    kv = x["kv"]
    table = code_table(kv)
    units = np.empty(g)
    for gam in range(g):
        vals = [table[elements(x["Vc"][gam], kv)].ravel()]
        vals += [table[elements(x["Vd"][i, gam, :x["lens"][i]], kv)].ravel() for i in range(b)]
        units[gam] = float(x["v_scale"][gam]) * float(np.std(np.concatenate(vals)))
    return np.repeat(units, h // g)


def assert_parity(out, ref, what="", gate_max_abs=None, x=None):
    """The gate is gate_max_abs_for(x) when the problem x is given, else
    GATE_MAX_ABS; gate_max_abs overrides it (a test whose softmax is much
    sharper than the workloads' may raise it up to the contract, never the
    relative-L2 gate)."""
    if gate_max_abs is None:
        gate_max_abs = GATE_MAX_ABS if x is None else gate_max_abs_for(x)
    assert gate_max_abs <= CONTRACT_MAX_ABS
    out = np.asarray(out, np.float64)
    ref = np.asarray(ref, np.float64)
    if (x is not None and x.get("kv", "bf16") != "bf16" and x.get("v_scale") is not None
            and out.shape == np.asarray(x["q"]).shape):
        u = value_units(x).reshape((1, -1) + (1,) * (out.ndim - 2))
        out, ref = out / u, ref / u
    assert np.all(np.isfinite(out)), f"{what}: non-finite GPU output"
    max_abs, rel_l2 = gate_errors(out, ref)
    print(f"[gate] {what}: max_abs={max_abs:.3e} rel_l2={rel_l2:.3e}", flush=True)
    assert max_abs <= CONTRACT_MAX_ABS, f"{what}: max abs {max_abs:.3e} breaks the 1e-2 contract"
    assert max_abs <= gate_max_abs and rel_l2 <= GATE_REL_L2, \
        f"{what}: max abs {max_abs:.3e} / rel L2 {rel_l2:.3e} outside the gate " \
        f"({gate_max_abs:.0e} / {GATE_REL_L2:.0e})"
    return max_abs, rel_l2
