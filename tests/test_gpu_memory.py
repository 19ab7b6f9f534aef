"""GPU checks of memory discipline through the C ABI (MI355X only):

* nothing is written outside `out` and, for the append, outside the rows it
  owns: canary bytes around the output and the decode caches are unchanged
  after every path (few-row fused launch, many-row context with and without
  the side-stream decode launch, standard path, replicated ablation, append);
* a plan's destroy and set_timing wait for the plan's own work only, not for
  unrelated work on other streams of the device.
"""
import numpy as np
import pytest

import oracle
import paper_2403_08845_amd as bif
import workloads

from .gpu_util import cache_to_device, replicate
from .parity import assert_parity

pytestmark = pytest.mark.gpu

CANARY = 0xA5
PAD = 4096  # bytes of canary on each side


def _guarded(nbytes, dtype, shape, fill=None):
    """A tensor of `shape` inside a uint8 buffer with PAD canary bytes on each
    side; returns (buffer, view). `fill`: bytes (uint8 numpy) for the view."""
    import torch
    buf = torch.full((nbytes + 2 * PAD,), CANARY, dtype=torch.uint8, device="cuda")
    if fill is not None:
        buf[PAD:PAD + nbytes] = torch.from_numpy(np.ascontiguousarray(fill).view(np.uint8).reshape(-1)).cuda()
    view = buf[PAD:PAD + nbytes].view(dtype).view(shape)
    return buf, view


def _intact(buf, nbytes, what):
    host = buf.cpu().numpy()
    assert np.all(host[:PAD] == CANARY), f"{what}: bytes before the tensor overwritten"
    assert np.all(host[PAD + nbytes:] == CANARY), f"{what}: bytes after the tensor overwritten"


def _guarded_cache(a, kv):
    import torch
    dt = torch.bfloat16 if kv == "bf16" else torch.uint8
    return _guarded(a.nbytes, dt, a.shape, fill=a)


# (b, h, g, d, m_c, m_d, n, kv, path, fork): every launch structure of a call
CASES = [
    (6, 16, 4, 128, 700, 90, 1, "bf16", "bifurcated", None),   # few-row fused launch
    (40, 32, 1, 128, 1000, 64, 1, "bf16", "bifurcated", "0"),  # many-row, one stream
    (40, 32, 1, 128, 1000, 64, 1, "bf16", "bifurcated", "1"),  # many-row, side stream
    (8, 32, 32, 128, 600, 120, 4, "fp8_e4m3", "bifurcated", None),
    (5, 16, 4, 64, 300, 40, 1, "int8", "standard", None),      # standard path
    (40, 32, 1, 128, 1000, 64, 2, "int4", "bifurcated", "1"),  # int4 many-row, side stream
    (5, 16, 4, 64, 300, 40, 1, "int4", "standard", None),
]


@pytest.mark.parametrize("case", CASES, ids=lambda c: "b%d_h%d_g%d_d%d_mc%d_md%d_n%d_%s_%s_fork%s" % c)
def test_canaries_around_output_and_caches(case, monkeypatch):
    import torch
    b, h, g, d, m_c, m_d, n, kv, path, fork = case
    if fork is not None:
        monkeypatch.setenv("BIFATTN_FORK", fork)
    x = workloads.make_inputs(b, h, g, d, m_c, m_d, seed=1400 + m_c, ragged=True, n=n, kv=kv)
    qshape = x["q"].shape
    nout = int(np.prod(qshape)) * 4
    ob, out = _guarded(nout, torch.float32, qshape)
    kb, Kd = _guarded_cache(x["Kd"], kv)
    vb, Vd = _guarded_cache(x["Vd"], kv)
    dev = {k: cache_to_device(x[k], "bf16" if k == "q" else kv) for k in ("q", "Kc", "Vc")}
    lens = torch.from_numpy(x["lens"]).cuda()
    ks = None if x.get("k_scale") is None else torch.from_numpy(x["k_scale"]).cuda()
    vs = None if x.get("v_scale") is None else torch.from_numpy(x["v_scale"]).cuda()
    print(f"[case] canaries {case}", flush=True)
    with bif.Plan(b, h, g, d, m_c, m_d, n=n, kv=kv, path=path) as plan:
        bif.bifattn_decode_scaled(plan, dev["q"], dev["Kc"], dev["Vc"], Kd, Vd, lens, ks, vs, out)
        assert bif.bifattn_plan_status(plan) == bif.OK
        _intact(ob, nout, "out")
        _intact(kb, x["Kd"].nbytes, "Kd")
        _intact(vb, x["Vd"].nbytes, "Vd")
        assert_parity(out.cpu().double().numpy(), oracle.attention(**x), f"canaries {case}", x=x)
        # the replicated ablation into a fresh guarded output
        K, V = replicate(x)
        Kr, Vr = cache_to_device(K, kv), cache_to_device(V, kv)
        ob2, out2 = _guarded(nout, torch.float32, qshape)
        bif.bifattn_decode_replicated_scaled(plan, dev["q"], Kr, Vr, lens, ks, vs, out2)
        assert bif.bifattn_plan_status(plan) == bif.OK
        _intact(ob2, nout, "out (replicated)")
        # the append writes rows len_i .. len_i + n - 1 of the guarded caches only
        if m_d >= n:
            room = torch.from_numpy(np.minimum(x["lens"], m_d - n)).cuda()
            rng = np.random.default_rng(3)
            codes = rng.integers(0, 127, (b, g, n, workloads.cache_cols(d, kv)), dtype=np.uint8)
            new = (workloads.f32_to_bf16_bits(rng.standard_normal((b, g, n, d), dtype=np.float32))
                   if kv == "bf16" else codes)
            bif.bifattn_append_kv(plan, cache_to_device(new, kv), cache_to_device(new, kv), Kd, Vd,
                                  room)
            assert bif.bifattn_plan_status(plan) == bif.OK
            _intact(kb, x["Kd"].nbytes, "Kd after append")
            _intact(vb, x["Vd"].nbytes, "Vd after append")


def test_destroy_and_set_timing_wait_for_the_plan_only():
    """Work queued on another stream (a bounded spin kernel) is still running
    when the plan has been re-armed for timing and destroyed: both waited for
    the plan's last call only, and that call's output is complete."""
    import torch
    b, h, g, d, m_c, m_d = 4, 8, 2, 128, 500, 60
    x = workloads.make_inputs(b, h, g, d, m_c, m_d, seed=1450, ragged=True)
    dev = {k: cache_to_device(x[k], "bf16") for k in ("q", "Kc", "Vc", "Kd", "Vd")}
    lens = torch.from_numpy(x["lens"]).cuda()
    out = torch.empty((b, h, d), dtype=torch.float32, device="cuda")
    plan = bif.Plan(b, h, g, d, m_c, m_d, path="bifurcated")
    bif.bifattn_decode(plan, dev["q"], dev["Kc"], dev["Vc"], dev["Kd"], dev["Vd"], lens, out)
    torch.cuda.synchronize()  # code objects loaded, first call done
    busy = torch.cuda.Stream()
    with torch.cuda.stream(busy):
        torch.cuda._sleep(400_000_000)  # bounded spin: ~0.2 s at the shader clock
    out.fill_(float("nan"))
    bif.bifattn_decode(plan, dev["q"], dev["Kc"], dev["Vc"], dev["Kd"], dev["Vd"], lens, out)
    bif.bifattn_plan_set_timing(plan, bif.KERNEL_PARTIALS, 2)
    after_timing = not busy.query()
    plan.close()
    after_destroy = not busy.query()
    busy.synchronize()
    assert after_timing, "set_timing waited for another stream's work"
    assert after_destroy, "destroy waited for another stream's work"
    assert_parity(out.cpu().double().numpy(), oracle.attention(**x), "after destroy", x=x)
