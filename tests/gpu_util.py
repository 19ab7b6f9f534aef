"""Helpers for GPU tests: seeded inputs to device, calls through the C ABI."""
import numpy as np

import paper_2403_08845_amd as bif


def kv_of(x):
    return x.get("kv", "bf16")


def cache_to_device(a, kv):
    """bf16 bit patterns -> torch bf16, 8-bit codes (int4: bytes of two
    codes) -> torch uint8, on the GPU."""
    import torch
    if kv == "bf16":
        return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).view(torch.bfloat16).cuda()
    return torch.from_numpy(np.ascontiguousarray(a).view(np.uint8)).cuda()


def to_device(x):
    import torch
    kv = kv_of(x)
    out = {"q": cache_to_device(x["q"], "bf16")}
    for k in ("Kc", "Vc", "Kd", "Vd"):
        out[k] = cache_to_device(x[k], kv)
    out["lens"] = torch.from_numpy(np.ascontiguousarray(x["lens"], dtype=np.int32)).cuda()
    for k in ("k_scale", "v_scale"):
        out[k] = (None if x.get(k) is None else
                  torch.from_numpy(np.ascontiguousarray(x[k], dtype=np.float32)).cuda())
    return out


def dims_of(x):
    """(b, h, g, d, m_c, m_d_max); q is [b, h, d] or [b, h, n, d]."""
    q = x["q"]
    b, h, d = q.shape[0], q.shape[1], q.shape[-1]
    g, m_c, _ = x["Kc"].shape
    m_d_max = x["Kd"].shape[2]
    return b, h, g, d, m_c, m_d_max


def tokens_of(x):
    return 1 if x["q"].ndim == 3 else x["q"].shape[2]


def run_decode(x, scale=0.0, plan=None, dev=None, check_status=True):
    """Bifurcated call on seeded numpy inputs; returns fp64 numpy [b,h,d]."""
    import torch
    b, h, g, d, m_c, m_d_max = dims_of(x)
    own = plan is None
    if own:
        plan = bif.Plan(b, h, g, d, m_c, m_d_max, scale, n=tokens_of(x), kv=kv_of(x))
    try:
        dev = dev or to_device(x)
        out = torch.full(tuple(x["q"].shape), float("nan"), dtype=torch.float32, device="cuda")
        if dev.get("k_scale") is None and dev.get("v_scale") is None:
            bif.bifattn_decode(plan, dev["q"], dev["Kc"], dev["Vc"], dev["Kd"], dev["Vd"],
                               dev["lens"], out)
        else:
            bif.bifattn_decode_scaled(plan, dev["q"], dev["Kc"], dev["Vc"], dev["Kd"], dev["Vd"],
                                      dev["lens"], dev["k_scale"], dev["v_scale"], out)
        st = bif.bifattn_plan_status(plan)
        if check_status:
            assert st == bif.OK, bif.status_string(st)
        return out.cpu().double().numpy()
    finally:
        if own:
            plan.close()


def replicate(x):
    """Physically replicated cache [b, g, m_c + m_d_max, d] (ablation input;
    the last axis as stored: d/2 bytes for int4)."""
    b, h, g, d, m_c, m_d_max = dims_of(x)
    cols = x["Kc"].shape[-1]
    K = np.concatenate([np.broadcast_to(x["Kc"][None], (b, g, m_c, cols)), x["Kd"]], axis=2)
    V = np.concatenate([np.broadcast_to(x["Vc"][None], (b, g, m_c, cols)), x["Vd"]], axis=2)
    return np.ascontiguousarray(K), np.ascontiguousarray(V)


def run_replicated(x, scale=0.0):
    import torch
    b, h, g, d, m_c, m_d_max = dims_of(x)
    K, V = replicate(x)
    kv = kv_of(x)
    with bif.Plan(b, h, g, d, m_c, m_d_max, scale, n=tokens_of(x), kv=kv) as plan:
        dev = to_device(x)
        Kt, Vt = cache_to_device(K, kv), cache_to_device(V, kv)
        out = torch.full(tuple(x["q"].shape), float("nan"), dtype=torch.float32, device="cuda")
        bif.bifattn_decode_replicated_scaled(plan, dev["q"], Kt, Vt, dev["lens"], dev["k_scale"],
                                             dev["v_scale"], out)
        assert bif.bifattn_plan_status(plan) == bif.OK
        return out.cpu().double().numpy()


def sample_rows(b, h, lens, n_random, seed):
    """Rows (i, j) covering every head of the first, last, longest and
    shortest sample plus seeded random rows."""
    rng = np.random.default_rng(seed)
    lens = np.asarray(lens)
    samples = sorted({0, b - 1, int(np.argmax(lens)), int(np.argmin(lens))})
    ri, rj = [], []
    for i in samples:
        for j in range(h):
            ri.append(i)
            rj.append(j)
    ri += list(rng.integers(0, b, n_random))
    rj += list(rng.integers(0, h, n_random))
    return np.array(ri, np.int32), np.array(rj, np.int32)
