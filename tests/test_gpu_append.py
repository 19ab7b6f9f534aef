"""Decode-cache append and a generation loop built on it (MI355X only):
append is byte work, checked bit for bit; each decode step of the loop is
checked against the oracle on the cache the loop has built."""
import numpy as np
import pytest

import oracle
import paper_2403_08845_amd as bif
import workloads

from .gpu_util import to_device
from .parity import assert_parity

pytestmark = pytest.mark.gpu


def _bf16(a):
    import torch
    return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).view(torch.bfloat16).cuda()


def _bits(t):
    return t.view(__import__("torch").int16).cpu().numpy().view(np.uint16)


@pytest.mark.parametrize("n", [1, 3])
def test_append_is_exact_and_flags_overflow(n):
    import torch
    b, h, g, d, m_c, m_d = 5, 8, 4, 128, 64, 20
    x = workloads.make_inputs(b, h, g, d, m_c, m_d, seed=800 + n, n=n)
    lens = np.array([0, 7, m_d - n, m_d - 1, m_d], np.int32)  # the last two run out of room
    rng = np.random.default_rng(5)
    k_new = workloads.f32_to_bf16_bits(rng.standard_normal((b, g, n, d), dtype=np.float32))
    v_new = workloads.f32_to_bf16_bits(rng.standard_normal((b, g, n, d), dtype=np.float32))
    Kd, Vd = _bf16(x["Kd"]), _bf16(x["Vd"])
    lens_t = torch.from_numpy(lens.copy()).cuda()
    with bif.Plan(b, h, g, d, m_c, m_d, n=n) as plan:
        bif.bifattn_append_kv(plan, _bf16(k_new), _bf16(v_new), Kd, Vd, lens_t)
        assert bif.bifattn_plan_status(plan) == bif.ELENS  # capacity reached for two samples
        expK, expV = x["Kd"].copy(), x["Vd"].copy()
        for i in range(b):
            room = min(n, m_d - lens[i])
            expK[i, :, lens[i]:lens[i] + room] = k_new[i, :, :room]
            expV[i, :, lens[i]:lens[i] + room] = v_new[i, :, :room]
        assert np.array_equal(_bits(Kd), expK)
        assert np.array_equal(_bits(Vd), expV)
        assert np.array_equal(lens_t.cpu().numpy(), np.minimum(lens + n, m_d))
        # within capacity: no flag
        lens_t.copy_(torch.from_numpy(np.array([0, 1, 2, 3, 4], np.int32)))
        bif.bifattn_append_kv(plan, _bf16(k_new), _bf16(v_new), Kd, Vd, lens_t)
        assert bif.bifattn_plan_status(plan) == bif.OK


@pytest.mark.parametrize("case", [(4, 8, 8, 128, 500, 40, 1), (3, 8, 2, 64, 300, 40, 2),
                                  (6, 32, 32, 128, 1024, 24, 1)],
                         ids=lambda c: "b%d_h%d_g%d_d%d_mc%d_md%d_n%d" % c)
def test_generation_loop(case):
    """Append then decode, step after step, on one plan and one device cache:
    every step matches the oracle on the cache the loop has built so far."""
    import torch
    b, h, g, d, m_c, m_d, n = case
    x = workloads.make_inputs(b, h, g, d, m_c, m_d, seed=820, n=n, lens=[0] * b)
    dev = to_device(x)
    rng = np.random.default_rng(9)
    Kd_host, Vd_host = x["Kd"].copy(), x["Vd"].copy()
    lens_host = np.zeros(b, np.int32)
    qshape = (b, h, d) if n == 1 else (b, h, n, d)
    out = torch.empty(qshape, dtype=torch.float32, device="cuda")
    with bif.Plan(b, h, g, d, m_c, m_d, n=n) as plan:
        for step in range(m_d // n):
            q = workloads.f32_to_bf16_bits(rng.standard_normal(qshape, dtype=np.float32))
            k_new = workloads.f32_to_bf16_bits(rng.standard_normal((b, g, n, d), dtype=np.float32))
            v_new = workloads.f32_to_bf16_bits(rng.standard_normal((b, g, n, d), dtype=np.float32))
            bif.bifattn_append_kv(plan, _bf16(k_new), _bf16(v_new), dev["Kd"], dev["Vd"], dev["lens"])
            bif.bifattn_decode(plan, _bf16(q), dev["Kc"], dev["Vc"], dev["Kd"], dev["Vd"],
                               dev["lens"], out)
            Kd_host[:, :, lens_host[0]:lens_host[0] + n] = k_new
            Vd_host[:, :, lens_host[0]:lens_host[0] + n] = v_new
            lens_host += n
            if step % 5 == 0 or step == m_d // n - 1:
                y = dict(q=q, Kc=x["Kc"], Vc=x["Vc"], Kd=Kd_host, Vd=Vd_host, lens=lens_host)
                ref = oracle.attention(**y)
                assert_parity(out.cpu().double().numpy(), ref, f"{case} step {step}", x=y)
        assert bif.bifattn_plan_status(plan) == bif.OK
    assert np.array_equal(dev["lens"].cpu().numpy(), lens_host)
