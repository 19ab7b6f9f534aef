"""The allocation-free entry point (bifattn_decode_noalloc) through the C ABI:
its output against bifattn_decode_scaled's on the same inputs, on calls in
a row that share the fixed per-GPU scratch buffer (each later call smaller
than the one before it), and its host-side refusal of problems whose
workspace exceeds that buffer."""
import ctypes

import numpy as np
import pytest

import oracle
import paper_2403_08845_amd as bif
import workloads

from .gpu_util import to_device
from .parity import assert_parity


def _run_noalloc(x, dims):
    import torch
    dev = to_device(x)
    out = torch.full(tuple(x["q"].shape), float("nan"), dtype=torch.float32, device="cuda")
    bif.bifattn_decode_noalloc(dims, dev["q"], dev["Kc"], dev["Vc"], dev["Kd"], dev["Vd"],
                               dev["lens"], dev["k_scale"], dev["v_scale"], out)
    torch.cuda.synchronize()
    return out.cpu().double().numpy()


def _run_plan(x, case, path="auto"):
    import torch
    b, h, g, d, m_c, m_d, n, kv = case
    dev = to_device(x)
    out = torch.full(tuple(x["q"].shape), float("nan"), dtype=torch.float32, device="cuda")
    with bif.Plan(b, h, g, d, m_c, m_d, n=n, kv=kv, path=path) as plan:
        bif.bifattn_decode_scaled(plan, dev["q"], dev["Kc"], dev["Vc"], dev["Kd"], dev["Vd"],
                                  dev["lens"], dev["k_scale"], dev["v_scale"], out)
        assert bif.bifattn_plan_status(plan) == bif.OK
    return out.cpu().double().numpy()


# Calls in a row on one GPU, each smaller than the one before: the few-row
# path of a 7B-shaped MHA layer, the many-row path (MQA), fp8 caches with
# draft tokens, a grouped layer, int4 caches, and a tiny layer.
SEQUENCE = [
    # b, h, g, d, m_c, m_d, n, kv, path
    (16, 32, 32, 128, 4096, 256, 1, "bf16", "auto"),            # few-row, one launch
    (24, 32, 1, 128, 2000, 64, 1, "bf16", "bifurcated"),        # many-row context kernel
    (8, 32, 32, 128, 600, 120, 4, "fp8_e4m3", "bifurcated"),    # draft tokens, fp8
    (7, 32, 8, 128, 700, 129, 1, "int8", "auto"),               # standard path
    (3, 8, 2, 64, 200, 30, 1, "int4", "bifurcated"),            # int4 codes
    (4, 4, 4, 64, 128, 16, 1, "bf16", "bifurcated"),
]


@pytest.mark.gpu
def test_noalloc_matches_the_planned_call_over_calls_in_a_row():
    for k, (*case, path) in enumerate(SEQUENCE):
        b, h, g, d, m_c, m_d, n, kv = case
        x = workloads.make_inputs(b, h, g, d, m_c, m_d, seed=1500 + k, ragged=True, n=n, kv=kv)
        print(f"[case] noalloc call {k}: {case} {path}", flush=True)
        dims = bif.noalloc_dims(b, h, g, d, m_c, m_d, n=n, kv=kv, path=path)
        got = _run_noalloc(x, dims)
        planned = _run_plan(x, case, path)
        assert_parity(got, planned, f"noalloc vs plan {case}", x=x)
        # neither plan nor call uses a side stream at these sizes: same
        # splits, same kernels, so the two agree bit for bit
        assert np.array_equal(got, planned), f"{case}: differs from the planned call"
        assert_parity(got, oracle.attention(**x), f"noalloc vs oracle {case}", x=x)


@pytest.mark.gpu
def test_noalloc_twice_second_smaller_after_large():
    """A large call then a small one: the second must not see any of the
    first call's partials left in the shared scratch."""
    first = (32, 32, 32, 128, 8192, 512, 1, "bf16")
    second = (3, 8, 2, 128, 333, 77, 1, "bf16")
    for k, case in enumerate((first, second)):
        b, h, g, d, m_c, m_d, n, kv = case
        x = workloads.make_inputs(b, h, g, d, m_c, m_d, seed=1550 + k, ragged=True, n=n, kv=kv)
        print(f"[case] noalloc pair {k}: {case}", flush=True)
        got = _run_noalloc(x, bif.noalloc_dims(b, h, g, d, m_c, m_d, n=n, kv=kv,
                                               path="bifurcated"))
        planned = _run_plan(x, case, "bifurcated")
        assert np.array_equal(got, planned), f"{case}: differs from the planned call"
        assert_parity(got, oracle.attention(**x), f"noalloc pair {case}", x=x)


def test_noalloc_refuses_workspace_beyond_the_scratch():
    """Checked on the host before any HIP call (the pointers are never read):
    65536 query rows over one group need ~170 MB of partials."""
    L = bif.lib()
    dims = bif.noalloc_dims(1024, 64, 1, 128, 65536, 1024)
    fake = ctypes.c_void_p(256)
    st = L.bifattn_decode_noalloc(ctypes.byref(dims), fake, fake, fake, fake, fake, fake, None,
                                  None, fake, None)
    assert st == bif.ESCRATCH, bif.status_string(st)
    assert "scratch" in bif.status_string(bif.ESCRATCH)
