"""The workload-based switch (FAQ on caveats: bifurcation for high workloads,
standard attention otherwise): the standard path against the oracle on the
same seeded inputs, and the plan's automatic choice (MI355X only)."""
import numpy as np
import pytest

import oracle
import paper_2403_08845_amd as bif
import workloads

from .gpu_util import dims_of, kv_of, to_device, tokens_of
from .parity import assert_parity

pytestmark = pytest.mark.gpu


def _report(name, max_abs, rel):
    print(f"[parity] {name}: max_abs={max_abs:.3e} rel_l2={rel:.3e}", flush=True)


def run_path(x, path, scale=0.0, expect=bif.OK):
    import torch
    b, h, g, d, m_c, m_d_max = dims_of(x)
    with bif.Plan(b, h, g, d, m_c, m_d_max, scale, n=tokens_of(x), kv=kv_of(x), path=path) as plan:
        if path != "auto":
            assert plan.info()["path"] == bif.PATHS[path]
        dev = to_device(x)
        out = torch.full(tuple(x["q"].shape), float("nan"), dtype=torch.float32, device="cuda")
        bif.bifattn_decode_scaled(plan, dev["q"], dev["Kc"], dev["Vc"], dev["Kd"], dev["Vd"],
                                  dev["lens"], dev["k_scale"], dev["v_scale"], out)
        assert bif.bifattn_plan_status(plan) == expect
        return out.cpu().double().numpy()


# b, h, g, d, m_c, m_d_max, n, kv: every tile count (p*n = 1..64 rows), both
# head dims, ragged tails, context-only samples, several tokens, 8-/4-bit caches.
STD_CASES = [
    (4, 4, 4, 64, 128, 16, 1, "bf16"),
    (3, 8, 8, 128, 1000, 77, 1, "bf16"),
    (7, 32, 8, 128, 700, 129, 1, "bf16"),     # p = 4
    (5, 16, 1, 64, 517, 45, 1, "bf16"),       # MQA, p = 16
    (6, 32, 1, 128, 300, 40, 1, "bf16"),      # MQA, p = 32: two query tiles
    (9, 64, 1, 128, 257, 33, 1, "bf16"),      # p = 64: four query tiles
    (4, 8, 2, 128, 600, 90, 3, "bf16"),       # three tokens
    (3, 6, 3, 64, 1, 3, 1, "bf16"),           # a single context key
    (2, 4, 2, 128, 96, 0, 1, "bf16"),         # no decode cache
    (4, 16, 4, 128, 400, 60, 2, "fp8_e4m3"),
    (5, 32, 1, 64, 333, 50, 1, "int8"),
    (6, 32, 1, 128, 300, 40, 1, "int4"),      # two query tiles
    (4, 8, 2, 64, 600, 90, 3, "int4"),
]


@pytest.mark.parametrize("case", STD_CASES, ids=lambda c: "b%d_h%d_g%d_d%d_mc%d_md%d_n%d_%s" % c)
def test_standard_path_full_output(case):
    b, h, g, d, m_c, m_d, n, kv = case
    x = workloads.make_inputs(b, h, g, d, m_c, m_d, seed=1100 + m_c, ragged=True, n=n, kv=kv)
    if b >= 3 and m_d > 0:
        x["lens"][1] = 0 if n == 1 else n   # a context-only sample / shortest lengths
        x["lens"][-1] = m_d
    print(f"[case] standard {case} lens={x['lens'].tolist()[:8]}", flush=True)
    out = run_path(x, "standard")
    ref = oracle.attention(**x)
    _report(f"standard {case}", *assert_parity(out, ref, f"standard {case}", x=x))


def test_standard_path_poisoned_tail_and_flags():
    """Rows past each length are never read; an out-of-range length is
    clamped and flagged; a bad scale is flagged, on the standard path too."""
    args = (6, 16, 4, 128, 300, 150)
    x = workloads.make_inputs(*args, seed=1110, ragged=True)
    y = workloads.make_inputs(*args, seed=1110, ragged=True, poison_tail=True)
    assert np.array_equal(run_path(x, "standard"), run_path(y, "standard"))
    z = dict(x, lens=x["lens"].copy())
    z["lens"][2] = 10 ** 6
    out = run_path(z, "standard", expect=bif.ELENS)
    z["lens"][2] = 150
    assert_parity(out, oracle.attention(**z), "clamped length", x=z)
    w8 = workloads.make_inputs(*args, seed=1111, ragged=True, kv="fp8_e4m3")
    w8["v_scale"] = w8["v_scale"].copy()
    w8["v_scale"][3] = -1.0
    run_path(w8, "standard", expect=bif.ESCALE)


@pytest.mark.parametrize("shape,expect", [
    ((4, 4, 4, 64, 128, 16), "standard"),       # the tiny layer
    ((16, 32, 1, 128, 512, 64), "standard"),    # small MQA
    ((32, 32, 32, 128, 8192, 512), "bifurcated"),
    ((128, 32, 1, 128, 16384, 512), "bifurcated"),
    ((9, 64, 1, 128, 257, 33), "bifurcated"),   # 64 query rows per unit
    ((16, 32, 32, 128, 1024, 64), "bifurcated"),  # 512 units of 1088 keys
    ((64, 32, 8, 128, 2048, 64), "standard"),   # 256 rows per group
    ((4, 32, 8, 128, 2048, 64), "bifurcated"),  # 16 rows per group
])
def test_automatic_choice(shape, expect):
    with bif.Plan(*shape) as plan:
        assert plan.info()["path"] == bif.PATHS[expect]


def test_paths_agree_on_the_workloads():
    """Both paths on the tiny layer and a small multi-query layer."""
    for name, shape in (("tiny", (4, 4, 4, 64, 128, 16)), ("mqa", (16, 32, 1, 128, 512, 64))):
        x = workloads.make_inputs(*shape, seed=1120, ragged=True)
        ref = oracle.attention(**x)
        for path in ("bifurcated", "standard", "auto"):
            _report(f"{name} {path}", *assert_parity(run_path(x, path), ref, f"{name} {path}", x=x))
