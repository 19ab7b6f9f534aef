"""GPU parity over quantized KV caches (OCP fp8 E4M3, int8 and int4 codes
with per-group scales): bifattn_decode_scaled through the C ABI against the
fp64 oracle on the same seeded codes (MI355X only)."""
import numpy as np
import pytest

import oracle
import paper_2403_08845_amd as bif
import workloads

from .gpu_util import run_decode, run_replicated, to_device
from .parity import assert_parity, value_units
from .pins_kvquant import KVS, code_table, elements, fill_code, stored

pytestmark = pytest.mark.gpu


def _report(name, max_abs, rel):
    print(f"[parity] {name}: max_abs={max_abs:.3e} rel_l2={rel:.3e}", flush=True)


def _value_units(x):
    """Per output head, broadcast over samples and head dims."""
    return value_units(x)[None, :, None]


@pytest.mark.parametrize("kv", KVS)
@pytest.mark.parametrize("d", [64, 128])
def test_every_code_widens_exactly(kv, d):
    """One context key, no decode rows and q = 0 (so the logit is exactly 0
    and the weight exactly 1): the output is v_scale times the code's value,
    rounded once to fp32. Every code with a finite value passes through the
    value path of the kernel."""
    table = code_table(kv)
    codes = np.nonzero(np.isfinite(table))[0].astype(np.uint8)
    g = -(-codes.size // d)
    b, h = 2, 2 * g
    x = workloads.make_inputs(b, h, g, d, 1, 4, seed=900, kv=kv, lens=[0, 0])
    vc = np.zeros(g * d, np.uint8)
    vc[:codes.size] = codes
    x["Vc"] = stored(vc.reshape(g, 1, d), kv)
    x["q"][:] = 0
    x["v_scale"] = np.linspace(0.5, 3.0, g).astype(np.float32)
    print(f"[case] {kv} d={d} value table", flush=True)
    out = run_decode(x)
    for j in range(h):
        gam = j // (h // g)
        vals = table[elements(x["Vc"], kv)[gam, 0]]
        exp = (vals.astype(np.float32) * x["v_scale"][gam]).astype(np.float64)
        assert np.array_equal(out[:, j], np.broadcast_to(exp, out[:, j].shape)), (kv, j)


@pytest.mark.parametrize("kv", KVS)
def test_every_key_code(kv):
    """Two keys, one of them a decode key holding the code under test, q
    one-hot: the weight of the decode key is a sigmoid of the code's value,
    for every code (fp8 NaN codes replaced by 0)."""
    table = code_table(kv)
    b, h, d = 4, 64, 64
    x = workloads.make_inputs(b, h, 1, d, 1, 1, seed=901, kv=kv, lens=[1] * b)
    x["q"] = workloads.f32_to_bf16_bits(np.broadcast_to(np.eye(h, d, dtype=np.float32),
                                                        (b, h, d)).copy())
    x["Kc"][:] = 0
    x["Vc"][:] = 0
    x["Vd"][:] = fill_code(kv, 0x38 if kv == "fp8_e4m3" else 1)
    kd = (np.arange(b * d) % table.size).reshape(b, d)
    kd = np.where(np.isfinite(table[kd]), kd, 0)
    x["Kd"] = stored(kd.reshape(b, 1, 1, d), kv)
    x["k_scale"] = np.array([2.0 ** -7], np.float32)
    x["v_scale"] = np.array([0.7], np.float32)
    print(f"[case] {kv} key table", flush=True)
    out = run_decode(x, scale=0.5)
    ref = oracle.attention(**x, scale=0.5)
    _report(f"{kv} key table", *assert_parity(out, ref, f"{kv} key table", x=x))


# (b, h, g, d, m_c, m_d_max, n, ragged): few-row and many-row context paths,
# both head dims, ragged tails, several tokens.
KVQ_CASES = [
    (4, 4, 4, 64, 128, 16, 1, False),
    (3, 8, 8, 128, 1000, 77, 1, True),
    (7, 32, 8, 128, 700, 129, 1, True),      # GQA p = 4, M = 28
    (5, 16, 1, 64, 517, 45, 1, True),        # MQA, M = 80: many-row context path
    (40, 32, 1, 128, 2000, 64, 1, True),     # M = 1280, 5 row blocks
    (9, 64, 1, 128, 257, 33, 1, True),       # p = 64: four query tiles per decode wave
    (4, 8, 2, 128, 600, 90, 3, True),        # three tokens per sample
    (2, 4, 2, 128, 96, 0, 1, False),         # no decode cache
]


@pytest.mark.parametrize("kv", KVS)
@pytest.mark.parametrize("case", KVQ_CASES, ids=lambda c: "b%d_h%d_g%d_d%d_mc%d_md%d_n%d" % c[:7])
def test_small_shapes_full_output(kv, case):
    b, h, g, d, m_c, m_d, n, ragged = case
    x = workloads.make_inputs(b, h, g, d, m_c, m_d, seed=910 + m_c, ragged=ragged, n=n, kv=kv)
    print(f"[case] {kv} {case} lens={x['lens'].tolist()[:8]}", flush=True)
    out = run_decode(x)
    ref = oracle.attention(**x)
    _report(f"{kv} {case}", *assert_parity(out, ref, f"{kv} {case}", x=x))


@pytest.mark.parametrize("kv", KVS)
def test_masked_tail_is_never_read(kv):
    """Poison codes (NaN in fp8) past each sample's length change no bit."""
    args = (6, 16, 4, 128, 300, 150)
    x = workloads.make_inputs(*args, seed=920, ragged=True, kv=kv)
    y = workloads.make_inputs(*args, seed=920, ragged=True, kv=kv, poison_tail=True)
    assert np.array_equal(run_decode(x), run_decode(y))


@pytest.mark.parametrize("kv", KVS)
def test_unit_scales_equal_no_scales(kv):
    """NULL scales mean 1: bifattn_decode equals bifattn_decode_scaled with
    all-ones scales, bit for bit."""
    x = workloads.make_inputs(3, 8, 2, 128, 400, 50, seed=930, ragged=True, kv=kv)
    ones = dict(x, k_scale=np.ones(2, np.float32), v_scale=np.ones(2, np.float32))
    bare = {k: v for k, v in x.items() if k not in ("k_scale", "v_scale")}
    assert np.array_equal(run_decode(ones), run_decode(bare))


@pytest.mark.parametrize("kv", KVS)
def test_strongly_different_group_scales(kv):
    """Scales spread over a factor 64 between groups, on both paths."""
    for case in [(3, 16, 4, 128, 500, 60), (6, 32, 2, 128, 700, 40)]:
        b, h, g, d, m_c, m_d = case
        x = workloads.make_inputs(b, h, g, d, m_c, m_d, seed=940, ragged=True, kv=kv)
        x["k_scale"] = (x["k_scale"] * np.exp2(np.linspace(-3, 3, g))).astype(np.float32)
        x["v_scale"] = (x["v_scale"] * np.exp2(np.linspace(3, -3, g))).astype(np.float32)
        out = run_decode(x)
        ref = oracle.attention(**x)
        u = _value_units(x)
        # key scales up to 8x make the first groups' softmax ~8x sharper than
        # the workloads': one bf16-rounded weight can carry an output entry,
        # bounded by 2^-9 * max|v| (~9e-3 in value units): the contract bound
        _report(f"{kv} {case} spread",
                *assert_parity(out / u, ref / u, f"{kv} {case}", gate_max_abs=1e-2))


@pytest.mark.parametrize("kv", KVS)
def test_replicated_ablation(kv):
    x = workloads.make_inputs(3, 16, 4, 128, 700, 90, seed=950, ragged=True, kv=kv)
    out = run_replicated(x)
    ref = oracle.attention(**x)
    _report(f"{kv} replicated", *assert_parity(out, ref, f"{kv} replicated", x=x))


@pytest.mark.parametrize("bad", [0.0, -1.0, float("nan"), float("inf"), 1e-40])
def test_bad_scale_is_flagged(bad):
    """A scale that is not a positive normal float raises the plan's flag;
    the call still completes (its output is unspecified)."""
    import torch
    x = workloads.make_inputs(2, 4, 2, 64, 64, 8, seed=960, kv="fp8_e4m3")
    with bif.Plan(2, 4, 2, 64, 64, 8, kv="fp8_e4m3") as plan:
        dev = to_device(x)
        out = torch.empty(2, 4, 64, dtype=torch.float32, device="cuda")
        for which in ("k_scale", "v_scale"):
            s = dev[which].clone()
            s[1] = bad
            args = dict(k_scale=dev["k_scale"], v_scale=dev["v_scale"])
            args[which] = s
            bif.bifattn_decode_scaled(plan, dev["q"], dev["Kc"], dev["Vc"], dev["Kd"], dev["Vd"],
                                      dev["lens"], args["k_scale"], args["v_scale"], out)
            assert bif.bifattn_plan_status(plan) == bif.ESCALE
        bif.bifattn_decode_scaled(plan, dev["q"], dev["Kc"], dev["Vc"], dev["Kd"], dev["Vd"],
                                  dev["lens"], dev["k_scale"], dev["v_scale"], out)
        assert bif.bifattn_plan_status(plan) == bif.OK


@pytest.mark.parametrize("kv", KVS)
def test_generation_loop_with_codes(kv):
    """Append of 8-bit codes then decode, step after step: the append copies
    codes bit for bit and each step matches the oracle."""
    import torch
    b, h, g, d, m_c, m_d, n = 4, 8, 2, 128, 300, 12, 2
    x = workloads.make_inputs(b, h, g, d, m_c, m_d, seed=970, n=n, kv=kv, lens=[0] * b)
    dev = to_device(x)
    rng = np.random.default_rng(11)
    Kd_host, Vd_host = x["Kd"].copy(), x["Vd"].copy()
    lens_host = np.zeros(b, np.int32)
    out = torch.empty((b, h, n, d), dtype=torch.float32, device="cuda")
    from .gpu_util import cache_to_device
    with bif.Plan(b, h, g, d, m_c, m_d, n=n, kv=kv) as plan:
        for step in range(m_d // n):
            q = workloads.f32_to_bf16_bits(rng.standard_normal((b, h, n, d), dtype=np.float32))
            cols = workloads.cache_cols(d, kv)
            k_new = rng.integers(0, 256, (b, g, n, cols), dtype=np.uint8)
            v_new = rng.integers(0, 256, (b, g, n, cols), dtype=np.uint8)
            if kv == "fp8_e4m3":  # finite codes only
                k_new[(k_new & 0x7F) == 0x7F] = 0
                v_new[(v_new & 0x7F) == 0x7F] = 0
            bif.bifattn_append_kv(plan, cache_to_device(k_new, kv), cache_to_device(v_new, kv),
                                  dev["Kd"], dev["Vd"], dev["lens"])
            bif.bifattn_decode_scaled(plan, cache_to_device(q, "bf16"), dev["Kc"], dev["Vc"],
                                      dev["Kd"], dev["Vd"], dev["lens"], dev["k_scale"],
                                      dev["v_scale"], out)
            Kd_host[:, :, lens_host[0]:lens_host[0] + n] = k_new
            Vd_host[:, :, lens_host[0]:lens_host[0] + n] = v_new
            lens_host += n
            assert np.array_equal(dev["Kd"].cpu().numpy(), Kd_host)
            assert np.array_equal(dev["lens"].cpu().numpy(), lens_host)
            y = dict(x, q=q, Kd=Kd_host, Vd=Vd_host, lens=lens_host)
            ref = oracle.attention(**y)
            got = out.cpu().double().numpy()
            _report(f"{kv} loop step {step}", *assert_parity(got, ref, f"{kv} loop step {step}", x=y))
        assert bif.bifattn_plan_status(plan) == bif.OK
