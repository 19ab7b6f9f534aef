"""bifattn_decode captured in a HIP graph (torch.cuda.graph) and replayed: a
call enqueues only kernel launches (and, on the two-stream many-row path, an
event fork and join), no memory set or copy, so a serving loop can capture a
decode step once and replay it. Every replay, with eager work and
synchronisations in between, equals the eager call bit for bit (MI355X only)."""
import numpy as np
import pytest

import paper_2403_08845_amd as bif
import workloads

from .gpu_util import dims_of, kv_of, to_device, tokens_of

pytestmark = pytest.mark.gpu

# b, h, g, d, m_c, m_d_max, n, kv, fork: the standard path (tiny layer), the
# fused few-row launch, the many-row context kernel then the decode launch,
# the two-stream many-row path, several tokens, an 8-bit cache with scales.
CASES = [
    (4, 4, 4, 64, 128, 16, 1, "bf16", None),
    (8, 32, 32, 128, 2048, 256, 1, "bf16", None),
    (40, 32, 1, 128, 2000, 64, 1, "bf16", "0"),
    (40, 32, 1, 128, 2000, 64, 1, "bf16", "1"),
    (8, 32, 32, 128, 900, 120, 4, "bf16", "1"),
    (16, 32, 8, 128, 1500, 100, 1, "fp8_e4m3", None),
]


@pytest.mark.parametrize("case", CASES, ids=lambda c: "b%d_h%d_g%d_d%d_mc%d_md%d_n%d_%s_fork%s" % c)
def test_graph_replays_equal_the_eager_call(case, monkeypatch):
    import torch
    b, h, g, d, m_c, m_d, n, kv, fork = case
    if fork is not None:
        monkeypatch.setenv("BIFATTN_FORK", fork)
    x = workloads.make_inputs(b, h, g, d, m_c, m_d, seed=1600 + m_c, ragged=True, n=n, kv=kv)
    y = workloads.make_inputs(b, h, g, d, m_c, m_d, seed=1601 + m_c, ragged=True, n=n, kv=kv)
    with bif.Plan(*dims_of(x), n=tokens_of(x), kv=kv_of(x)) as plan:
        print(f"[case] graph {case} plan={plan.info()}", flush=True)
        dev, devy = to_device(x), to_device(y)

        def call(v, out):
            bif.bifattn_decode_scaled(plan, v["q"], v["Kc"], v["Vc"], v["Kd"], v["Vd"], v["lens"],
                                      v["k_scale"], v["v_scale"], out)

        shape = tuple(x["q"].shape)
        eager = torch.empty(shape, dtype=torch.float32, device="cuda")
        call(dev, eager)
        eager_y = torch.empty(shape, dtype=torch.float32, device="cuda")
        call(devy, eager_y)
        torch.cuda.synchronize()
        assert bif.bifattn_plan_status(plan) == bif.OK

        replay = torch.full(shape, float("nan"), dtype=torch.float32, device="cuda")
        graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(graph):
            call(dev, replay)
        for r in range(5):
            replay.fill_(float("nan"))
            graph.replay()
            torch.cuda.synchronize()
            assert torch.equal(replay, eager), f"replay {r}"
            # eager work on the same plan between replays (other inputs)
            other = torch.empty(shape, dtype=torch.float32, device="cuda")
            call(devy, other)
            torch.cuda.synchronize()
            assert torch.equal(other, eager_y), f"eager call after replay {r}"
        assert bif.bifattn_plan_status(plan) == bif.OK
        assert np.all(np.isfinite(replay.cpu().numpy()))
