"""GPU parity: bifattn_decode (through the C ABI) against the fp64 oracle on
the same seeded inputs, element by element (MI355X only)."""
import numpy as np
import pytest

import oracle
import paper_2403_08845_amd as bif
import workloads

from .gpu_util import dims_of, run_decode, run_replicated, sample_rows, to_device, tokens_of
from .parity import CONTRACT_MAX_ABS, assert_parity

pytestmark = pytest.mark.gpu


def _report(name, max_abs, rel):
    print(f"[parity] {name}: max_abs={max_abs:.3e} rel_l2={rel:.3e}", flush=True)


# Shapes the oracle finishes in seconds that span several tiles, ragged tails
# (lengths not multiples of the 32-key tile or of a work-group's key chunk),
# both head dims, multi-head / grouped / multi-query, the many-row context
# path, context-only samples and a single context key.
SMALL_CASES = [
    # b, h, g, d, m_c, m_d_max, ragged
    (4, 4, 4, 64, 128, 16, False),
    (3, 8, 8, 128, 1000, 77, True),
    (2, 8, 2, 128, 333, 200, True),
    (5, 16, 1, 64, 517, 45, True),        # MQA, p = 16, M = 80 -> many-row context path
    (1, 32, 32, 128, 4096, 300, True),    # b = 1
    (7, 32, 8, 128, 700, 129, True),      # GQA p = 4, M = 28
    (9, 64, 1, 128, 257, 33, True),       # MQA p = 64 (four query tiles per decode wave)
    (3, 6, 3, 64, 1, 3, True),            # single context key
    (2, 4, 2, 128, 96, 0, False),         # no decode cache
    (40, 32, 1, 128, 2000, 64, True),     # M = 1280 -> 5 row blocks, ragged last block
    (100, 6, 2, 64, 300, 40, True),       # p = 3, M = 300: a sample's rows straddle two row blocks
]


@pytest.mark.parametrize("case", SMALL_CASES, ids=lambda c: "b%d_h%d_g%d_d%d_mc%d_md%d" % c[:6])
def test_small_shapes_full_output(case):
    b, h, g, d, m_c, m_d, ragged = case
    x = workloads.make_inputs(b, h, g, d, m_c, m_d, seed=500 + m_c, ragged=ragged)
    if ragged and b >= 3 and m_d > 0:
        x["lens"][1] = 0          # a context-only sample
        x["lens"][-1] = m_d       # a full one
    print(f"[case] {case} lens={x['lens'].tolist()[:8]}", flush=True)
    out = run_decode(x)
    ref = oracle.attention(**x)
    _report(str(case), *assert_parity(out, ref, str(case), x=x))


@pytest.mark.parametrize("name", workloads.WORKLOAD_ORDER)
def test_workload_full_output(name):
    """Every workload at full size, in the configuration the benchmark times:
    the whole output against the fp64 oracle on all host threads."""
    w = workloads.WORKLOADS[name]
    x = workloads.make_workload_inputs(w)
    print(f"[case] {name} sum(lens)={int(x['lens'].sum())}", flush=True)
    out = run_decode(x)
    ref = oracle.attention(**x)
    assert out.shape == ref.shape
    _report(name, *assert_parity(out, ref, name, x=x))


@pytest.mark.parametrize("name", workloads.WORKLOAD_ORDER[2:5])
def test_workload_sampled_rows_match_full(name):
    """The oracle's row-by-row evaluation (used where the full output would
    be too costly) agrees with the full evaluation on sampled rows of the
    large workloads, and the GPU rows agree with both."""
    w = workloads.WORKLOADS[name]
    x = workloads.make_workload_inputs(w)
    ri, rj = sample_rows(w.b, w.h, x["lens"], 16, seed=w.seed)
    rows = oracle.attention_rows(**x, rows_i=ri, rows_j=rj)
    out = run_decode(x)
    _report(f"{name} sampled", *assert_parity(out[ri, rj], rows, name, x=x))


@pytest.mark.parametrize("case", [(2048, 8, 1, 64, 300, 20), (512, 64, 64, 128, 100, 40)],
                         ids=lambda c: "b%d_h%d_g%d_d%d_mc%d_md%d" % c)
def test_large_batches_sampled_rows(case):
    """Very many samples: 16384 query rows in 128 row blocks on one group, and
    32768 (sample, group) units of a 64-head MHA layer; every output finite,
    sampled rows (first, last, longest and shortest samples, random ones)
    against the oracle row by row."""
    b, h, g, d, m_c, m_d = case
    x = workloads.make_inputs(b, h, g, d, m_c, m_d, seed=1700 + b, ragged=True)
    print(f"[case] large batch {case}", flush=True)
    out = run_decode(x)
    assert np.all(np.isfinite(out))
    ri, rj = sample_rows(b, h, x["lens"], 64, seed=1701)
    ref = oracle.attention_rows(**x, rows_i=ri, rows_j=rj)
    _report(f"large batch {case}", *assert_parity(out[ri, rj], ref, str(case), x=x))


def test_masked_tail_is_never_read():
    """NaN in decode rows past each sample's length changes no output bit."""
    b, h, g, d, m_c, m_d = 6, 16, 4, 128, 300, 150
    x = workloads.make_inputs(b, h, g, d, m_c, m_d, seed=71, ragged=True)
    y = workloads.make_inputs(b, h, g, d, m_c, m_d, seed=71, ragged=True, poison_tail=True)
    a = run_decode(x)
    c = run_decode(y)
    assert np.array_equal(a, c)


def test_deterministic_and_plan_reuse():
    b, h, g, d, m_c, m_d = 5, 32, 32, 128, 1500, 100
    x = workloads.make_inputs(b, h, g, d, m_c, m_d, seed=72, ragged=True)
    with bif.Plan(b, h, g, d, m_c, m_d) as plan:
        dev = to_device(x)
        a = run_decode(x, plan=plan, dev=dev)
        c = run_decode(x, plan=plan, dev=dev)
    assert np.array_equal(a, c)


def test_b1_equivalence_on_gpu():
    """Row i of a batched call equals a b = 1 call on sample i."""
    b, h, g, d, m_c, m_d = 4, 8, 2, 128, 640, 90
    x = workloads.make_inputs(b, h, g, d, m_c, m_d, seed=73, ragged=True)
    full = run_decode(x)
    for i in range(b):
        one = {k: x[k] for k in ("Kc", "Vc")}
        one.update(q=x["q"][i:i + 1], Kd=x["Kd"][i:i + 1], Vd=x["Vd"][i:i + 1],
                   lens=x["lens"][i:i + 1])
        single = run_decode(one)
        assert_parity(single[0], full[i], f"b=1 sample {i}")


@pytest.mark.parametrize("scale", [0.05, -0.08])
@pytest.mark.parametrize("shape", [(3, 8, 4, 64, 200, 40), (4, 32, 1, 128, 300, 50)],
                         ids=["few_rows", "many_rows"])
def test_explicit_scale(shape, scale):
    """A caller-given scale, including a negative one (the kernels then negate
    q, exactly), on the few-row and the many-row context paths."""
    b, h, g, d, m_c, m_d = shape
    x = workloads.make_inputs(b, h, g, d, m_c, m_d, seed=74, ragged=True)
    out = run_decode(x, scale=scale)
    ref = oracle.attention(**x, scale=scale)
    assert_parity(out, ref, f"scale {scale}", x=x)


def test_out_of_range_lengths_are_clamped_and_flagged():
    import torch
    b, h, g, d, m_c, m_d = 3, 4, 2, 128, 64, 40
    x = workloads.make_inputs(b, h, g, d, m_c, m_d, seed=75)
    bad = dict(x)
    bad["lens"] = np.array([50, -3, 17], np.int32)
    with bif.Plan(b, h, g, d, m_c, m_d) as plan:
        dev = to_device(bad)
        out = torch.empty((b, h, d), dtype=torch.float32, device="cuda")
        bif.bifattn_decode(plan, dev["q"], dev["Kc"], dev["Vc"], dev["Kd"], dev["Vd"],
                           dev["lens"], out)
        assert bif.bifattn_plan_status(plan) == bif.ELENS
        assert bif.bifattn_plan_status(plan) == bif.OK  # flag cleared
        got = out.cpu().double().numpy()
    clamped = dict(x)
    clamped["lens"] = np.array([40, 0, 17], np.int32)
    assert_parity(got, oracle.attention(**clamped), "clamped lengths", x=clamped)


@pytest.mark.parametrize("case", [(4, 4, 4, 64, 128, 16, False), (3, 16, 4, 128, 700, 90, True),
                                  (6, 32, 1, 128, 300, 64, True)],
                         ids=lambda c: "b%d_h%d_g%d_d%d_mc%d_md%d" % c[:6])
def test_replicated_ablation_matches_oracle(case):
    b, h, g, d, m_c, m_d, ragged = case
    x = workloads.make_inputs(b, h, g, d, m_c, m_d, seed=76, ragged=ragged)
    out = run_replicated(x)
    assert_parity(out, oracle.attention(**x), f"replicated {case}", x=x)


@pytest.mark.parametrize("case", [(3, 8, 2, 128, 300, 70, 3, [50, 2, 0]),
                                  (4, 16, 1, 64, 100, 40, 4, [1, 0, 40, 3]),
                                  (2, 4, 4, 128, 33, 9, 8, [0, 6])],
                         ids=lambda c: "b%d_h%d_g%d_d%d_mc%d_md%d_n%d" % c[:7])
def test_replicated_short_lengths_keep_the_context(case):
    """Replicated ablation with several tokens and lengths below n - 1: a
    token's causal limit never cuts into the context rows that precede the
    decode rows in the replicated cache (every token sees all m_c of them)."""
    b, h, g, d, m_c, m_d, n, lens = case
    x = workloads.make_inputs(b, h, g, d, m_c, m_d, seed=660 + n, lens=lens, n=n)
    ref = oracle.attention(**x)
    _report(f"replicated short {case}", *assert_parity(run_replicated(x), ref, str(case), x=x))
    _report(f"bifurcated short {case}", *assert_parity(run_decode(x), ref, str(case), x=x))


def test_timing_api_counts_calls():
    import torch
    b, h, g, d, m_c, m_d = 4, 32, 32, 128, 2048, 128
    x = workloads.make_inputs(b, h, g, d, m_c, m_d, seed=77)
    with bif.Plan(b, h, g, d, m_c, m_d) as plan:
        dev = to_device(x)
        out = torch.empty((b, h, d), dtype=torch.float32, device="cuda")
        bif.bifattn_plan_set_timing(plan, bif.KERNEL_PARTIALS, 3)
        for _ in range(5):
            bif.bifattn_decode(plan, dev["q"], dev["Kc"], dev["Vc"], dev["Kd"], dev["Vd"],
                               dev["lens"], out)
        n, ms = bif.bifattn_plan_read_timing(plan)
        assert n == 3 and 0 < ms < 1000
        bif.bifattn_plan_set_timing(plan, bif.KERNEL_PARTIALS, 0)


@pytest.mark.parametrize("case", [(32, 32, 32, 128, 3000, 300, True), (12, 64, 2, 128, 900, 200, True),
                                  (8, 32, 8, 64, 1500, 90, True)],
                         ids=lambda c: "b%d_h%d_g%d_d%d_mc%d_md%d" % c[:6])
def test_workspace_reuse_over_many_calls(case):
    """One plan, inputs alternating between two problems for 40 calls: every
    output equals the first result for its input bit for bit (no partial of
    a previous call can leak into the next one)."""
    import torch
    b, h, g, d, m_c, m_d, ragged = case
    xs = [workloads.make_inputs(b, h, g, d, m_c, m_d, seed=80 + k, ragged=ragged) for k in range(2)]
    devs = [to_device(x) for x in xs]
    with bif.Plan(b, h, g, d, m_c, m_d) as plan:
        refs = []
        for dv in devs:
            out = torch.empty((b, h, d), dtype=torch.float32, device="cuda")
            bif.bifattn_decode(plan, dv["q"], dv["Kc"], dv["Vc"], dv["Kd"], dv["Vd"], dv["lens"], out)
            refs.append(out)
        torch.cuda.synchronize()
        assert_parity(refs[0].cpu().double().numpy(), oracle.attention(**xs[0]), "first call",
                      x=xs[0])
        outs = [torch.empty((b, h, d), dtype=torch.float32, device="cuda") for _ in range(2)]
        for it in range(40):
            k = it % 2
            dv = devs[k]
            bif.bifattn_decode(plan, dv["q"], dv["Kc"], dv["Vc"], dv["Kd"], dv["Vd"], dv["lens"],
                               outs[k])
            if k == 1:
                torch.cuda.synchronize()
                for kk in range(2):
                    assert torch.equal(outs[kk], refs[kk]), f"call {it}: input {kk} differs"
        assert bif.bifattn_plan_status(plan) == bif.OK


# n new tokens per sample (draft tokens verified in one step): MHA / GQA / MQA,
# both head dims, the few-row and the many-row context paths, ragged lengths
# including lengths below n and zero.
DRAFT_CASES = [
    # b, h, g, d, m_c, m_d_max, n, lens (None: drawn in [n, m_d_max])
    (4, 8, 8, 128, 700, 90, 4, None),
    (3, 8, 2, 64, 333, 70, 3, [70, 2, 0]),
    (5, 16, 1, 128, 517, 45, 2, None),       # MQA, p*n = 32
    (2, 4, 4, 128, 1000, 300, 8, [300, 5]),  # n = 8 across two 32-key tiles
    (40, 32, 32, 128, 600, 64, 4, None),     # M = 160 rows per group: many-row context path
    (6, 8, 1, 64, 200, 33, 8, None),         # MQA, p*n = 64
]


@pytest.mark.parametrize("case", DRAFT_CASES, ids=lambda c: "b%d_h%d_g%d_d%d_mc%d_md%d_n%d" % c[:7])
def test_draft_tokens_full_output(case):
    b, h, g, d, m_c, m_d, n, lens = case
    x = workloads.make_inputs(b, h, g, d, m_c, m_d, seed=600 + n, ragged=lens is None, lens=lens, n=n)
    print(f"[case] {case} lens={x['lens'].tolist()[:8]}", flush=True)
    out = run_decode(x)
    assert out.shape == (b, h, n, d)
    _report(str(case), *assert_parity(out, oracle.attention(**x), str(case), x=x))


def test_draft_tokens_masked_tail_and_replicated():
    """Rows past each sample's length stay unread with n tokens, and the
    replicated ablation applies the same causal rule."""
    b, h, g, d, m_c, m_d, n = 4, 8, 2, 128, 300, 80, 4
    x = workloads.make_inputs(b, h, g, d, m_c, m_d, seed=650, ragged=True, n=n)
    y = workloads.make_inputs(b, h, g, d, m_c, m_d, seed=650, ragged=True, n=n, poison_tail=True)
    a = run_decode(x)
    assert np.array_equal(a, run_decode(y))
    assert_parity(run_replicated(x), oracle.attention(**x), "replicated, n = 4", x=x)


@pytest.mark.parametrize("case", [(40, 32, 1, 128, 2000, 64, 1), (6, 32, 2, 128, 700, 40, 1),
                                  (8, 32, 32, 128, 900, 120, 4)],
                         ids=lambda c: "b%d_h%d_g%d_d%d_mc%d_md%d_n%d" % c)
def test_side_stream_decode(case, monkeypatch):
    """Many-row plans may run the decode launch on a side stream beside the
    context kernel (the call's stream waits for it before the combine):
    forced on and off with either context kernel, every output matches the
    oracle, and with the same kernel the two are bitwise equal when the plans
    split the context alike."""
    b, h, g, d, m_c, m_d, n = case
    x = workloads.make_inputs(b, h, g, d, m_c, m_d, seed=1200 + m_c, ragged=True, n=n)
    ref = oracle.attention(**x)
    for wide in ("0", "1"):
        monkeypatch.setenv("BIFATTN_CTX_WIDE", wide)
        runs = []
        for fork in ("0", "1"):
            monkeypatch.setenv("BIFATTN_FORK", fork)
            with bif.Plan(b, h, g, d, m_c, m_d, n=n) as plan:
                info = plan.info()
                if b * (h // g) * n > 64:  # many rows per group (else the few-row launch)
                    assert info["side_stream"] == int(fork)
                    assert info["ctx_kernel"] == (2 if wide == "1" else 1)
                out = run_decode(x, plan=plan)
            _report(f"side stream {case} wide={wide} fork={fork}",
                    *assert_parity(out, ref, f"{case} wide={wide} fork={fork}", x=x))
            runs.append((info["ctx_splits"], out))
        if runs[0][0] == runs[1][0]:
            assert np.array_equal(runs[0][1], runs[1][1])


def test_plan_rule_for_large_decode_parts(monkeypatch):
    """Without overrides, a many-row plan whose decode part is large takes the
    side stream; with 256 or more rows per group it keeps the eight-wave 32x32
    context kernel on five eighths of the CUs, with 128 to 255 rows its
    four-wave form on about one work-group per CU."""
    for var in ("BIFATTN_FORK", "BIFATTN_CTX_WIDE", "BIFATTN_CTX_WGS"):
        monkeypatch.delenv(var, raising=False)
    with bif.Plan(256, 32, 8, 128, 32768, 1024) as plan:  # 1024 rows per group
        info = plan.info()
        assert info["side_stream"] == 1 and info["ctx_kernel"] == 2
        assert info["ctx_blocks"] <= 160
    with bif.Plan(32, 32, 32, 128, 8192, 512, n=4) as plan:  # 128 rows per group
        info = plan.info()
        assert info["side_stream"] == 1 and info["ctx_kernel"] == 2
        assert info["ctx_blocks"] <= 256


def test_largest_context_rows_are_addressed():
    """A context near the per-cache limit ((m_c + m_d_max) * d * 2 bytes just
    under 2^31; prefetches past its end wrap their 32-bit offsets): every
    logit is 0 except one key at the far end of the context, whose logit is
    ~30, so each output row is that key's value row up to its softmax weight
    1 / (1 + (N - 1) e^-logit) (a property that holds at any size; the
    oracle would need gigabytes per row)."""
    import torch
    b, h, g, d, m_d = 2, 4, 1, 128, 64
    m_c = (2 ** 31 - 1) // (d * 2) - m_d - 1
    with bif.Plan(b, h, g, d, m_c, m_d) as plan:
        assert plan.info()["path"] == bif.PATHS["bifurcated"]
        print(f"[case] m_c={m_c} plan={plan.info()}", flush=True)
        bf = torch.bfloat16
        q = torch.zeros(b, h, d, dtype=bf, device="cuda")
        q[..., 0] = 1.0
        Kc = torch.zeros(g, m_c, d, dtype=bf, device="cuda")
        Vc = torch.zeros(g, m_c, d, dtype=bf, device="cuda")
        Kd = torch.zeros(b, g, m_d, d, dtype=bf, device="cuda")
        Vd = torch.zeros(b, g, m_d, d, dtype=bf, device="cuda")
        lens = torch.tensor([m_d, 17], dtype=torch.int32, device="cuda")
        far = m_c - 1
        Kc[0, far, 0] = 340.0                      # exact in bf16
        v = (torch.arange(d, dtype=torch.float32) - 64.0) / 64.0  # exact in bf16
        Vc[0, far] = v.to(bf).cuda()
        out = torch.empty(b, h, d, dtype=torch.float32, device="cuda")
        bif.bifattn_decode(plan, q, Kc, Vc, Kd, Vd, lens, out)
        assert bif.bifattn_plan_status(plan) == bif.OK
        got = out.cpu().double().numpy()
    z = 340.0 / np.sqrt(d)
    for i, L in enumerate((m_d, 17)):
        w = 1.0 / (1.0 + (m_c + L - 1) * np.exp(-z))
        exp = w * v.double().numpy()
        err = float(np.max(np.abs(got[i] - exp[None, :])))
        print(f"[parity] far key, sample {i}: max_abs={err:.3e}", flush=True)
        assert err <= 1e-5, err


@pytest.mark.parametrize("case", [(3, 8, 8, 128, 1000, 77), (7, 32, 8, 128, 700, 129),
                                  (2, 4, 2, 128, 96, 0)],
                         ids=lambda c: "b%d_h%d_g%d_d%d_mc%d_md%d" % c)
def test_split_launch_equals_fused(case, monkeypatch):
    """The few-row context work-groups and the decode work-groups in two
    launches (BIFATTN_LAUNCH=2) instead of one: the same work-groups, so the
    outputs are bitwise equal, and they match the oracle."""
    b, h, g, d, m_c, m_d = case
    x = workloads.make_inputs(b, h, g, d, m_c, m_d, seed=1300 + m_c, ragged=True)
    fused = run_decode(x)
    monkeypatch.setenv("BIFATTN_LAUNCH", "2")
    split = run_decode(x)
    assert np.array_equal(fused, split)
    _report(f"split launch {case}", *assert_parity(split, oracle.attention(**x), str(case), x=x))


# Many-row context shapes for both context kernels (the 32x32 MFMA kernel of
# 32-row waves, and the kernel of 16-row waves): 128- and 64-key stages,
# ragged last chunks, row blocks whose last waves hold no rows, several
# tokens, grouped heads, and four-wave work-groups (fewer than 256 rows).
WIDE_CASES = [
    # b, h, g, d, m_c, m_d_max, n
    (48, 32, 1, 128, 50000, 64, 1),   # 1280-key chunks: 128-key stages, ragged last chunk
    (48, 32, 1, 128, 4000, 64, 1),    # 128-key chunks: 64-key stages
    (37, 16, 2, 128, 3000, 50, 1),    # 296 rows per group: an idle wave in the last row block
    (20, 16, 1, 128, 2500, 40, 2),    # two tokens per sample
    (64, 32, 8, 128, 6000, 200, 1),   # grouped heads, 256 rows per group
    (5, 32, 1, 128, 1777, 30, 1),     # 160 rows: four-wave work-groups
]


@pytest.mark.parametrize("case", WIDE_CASES, ids=lambda c: "b%d_h%d_g%d_d%d_mc%d_md%d_n%d" % c)
def test_many_row_context_kernels(case, monkeypatch):
    b, h, g, d, m_c, m_d, n = case
    x = workloads.make_inputs(b, h, g, d, m_c, m_d, seed=1600 + m_c, ragged=True, n=n)
    ref = oracle.attention(**x)
    monkeypatch.setenv("BIFATTN_FORK", "0")
    for wide in ("1", "0"):
        monkeypatch.setenv("BIFATTN_CTX_WIDE", wide)
        with bif.Plan(b, h, g, d, m_c, m_d, n=n, path="bifurcated") as plan:
            info = plan.info()
            print(f"[case] many-row {case} wide={wide} {info}", flush=True)
            out = run_decode(x, plan=plan)
        _report(f"many-row {case} wide={wide}", *assert_parity(out, ref, f"{case} wide={wide}", x=x))



@pytest.mark.parametrize("pattern", ["growing", "needle"])
@pytest.mark.parametrize("case", [(48, 32, 1, 128, 6000, 64), (64, 32, 8, 128, 3000, 100)],
                         ids=lambda c: "b%d_h%d_g%d_d%d_mc%d_md%d" % c)
def test_many_row_context_with_rising_logits(case, pattern, monkeypatch):
    """Context keys whose logits keep rising past the running reference
    maximum: key rows whose norm grows from 1x to 4x over every 128 keys (the
    row maxima rise by more than 2^8 several times inside a key chunk), or
    one key row scaled 8x in the middle of the context (a jump far above the
    reference). Both many-row kernels take their rescale paths inside their
    chunks and still match the oracle. The softmax is sharpened on purpose,
    so single weights carry whole rows: the max-abs gate is the contract
    bound and the values are halved (exactly), which keeps a dominant
    weight's bf16 rounding (2^-9 of its value row) well inside it; the
    relative-L2 gate is unchanged."""
    b, h, g, d, m_c, m_d = case
    x = workloads.make_inputs(b, h, g, d, m_c, m_d, seed=1700 + m_c, ragged=True)
    kc = (x["Kc"].astype(np.uint32) << 16).view(np.float32)
    t = np.arange(m_c, dtype=np.float32)
    if pattern == "growing":
        factor = (1.0 + 3.0 * (t % 128) / 127.0)[None, :, None]
    else:
        factor = np.ones((1, m_c, 1), np.float32)
        # past the first 32-key block of its chunk for chunks of 96-192 keys
        needle = next(t for t in range((3 * m_c) // 5, m_c)
                      if all(t % c >= 32 for c in (96, 128, 160, 192)))
        factor[0, needle] = 8.0
    x["Kc"] = workloads.f32_to_bf16_bits(kc * factor)
    for name in ("Vc", "Vd"):
        x[name] = workloads.f32_to_bf16_bits((x[name].astype(np.uint32) << 16).view(np.float32) * 0.5)
    ref = oracle.attention(**x)
    monkeypatch.setenv("BIFATTN_FORK", "0")
    for wide in ("1", "0"):
        monkeypatch.setenv("BIFATTN_CTX_WIDE", wide)
        with bif.Plan(b, h, g, d, m_c, m_d, path="bifurcated") as plan:
            print(f"[case] rising logits {pattern} {case} wide={wide} {plan.info()}", flush=True)
            out = run_decode(x, plan=plan)
        _report(f"rising logits {pattern} {case} wide={wide}",
                *assert_parity(out, ref, f"{pattern} {case} wide={wide}", x=x,
                               gate_max_abs=CONTRACT_MAX_ABS))


@pytest.mark.parametrize("kv", ["fp8_e4m3", "int8", "int4"])
@pytest.mark.parametrize("case", WIDE_CASES, ids=lambda c: "b%d_h%d_g%d_d%d_mc%d_md%d_n%d" % c)
def test_many_row_context_kernels_code_caches(case, kv, monkeypatch):
    """Both many-row context kernels over 8-bit and int4 caches: the 32x32
    kernel stages the codes through registers and widens them into its LDS
    stages, the 16x16 kernel widens them while staging its tiles."""
    b, h, g, d, m_c, m_d, n = case
    x = workloads.make_inputs(b, h, g, d, m_c, m_d, seed=1650 + m_c, ragged=True, n=n, kv=kv)
    ref = oracle.attention(**x)
    monkeypatch.setenv("BIFATTN_FORK", "0")
    for wide in ("1", "0"):
        monkeypatch.setenv("BIFATTN_CTX_WIDE", wide)
        with bif.Plan(b, h, g, d, m_c, m_d, n=n, kv=kv, path="bifurcated") as plan:
            info = plan.info()
            assert info["ctx_kernel"] == (2 if wide == "1" else 1)
            print(f"[case] many-row {kv} {case} wide={wide} {info}", flush=True)
            out = run_decode(x, plan=plan)
        _report(f"many-row {kv} {case} wide={wide}",
                *assert_parity(out, ref, f"{kv} {case} wide={wide}", x=x))