"""Seeded synthetic inputs for bifurcated decode attention.

This module is the only code shared by the HIP path's callers (tests, bench,
smoke) and the oracle's callers. It draws random numbers and rounds them to
bf16 bit patterns; it contains none of the attention arithmetic.

Shapes follow the paper's statement of the problem (Section 3.1 notation,
Section 4.1-4.2): ``b`` samples sharing one context of length ``m_c``, ``h``
query heads in ``g`` KV groups (``p = h/g`` heads per group, group-major:
head ``j`` belongs to group ``j // p``), head dimension ``d`` (the paper's
``k``), and per-sample decode lengths ``len_i <= m_d_max``.

Layouts (row-major, bf16 stored as uint16 bit patterns):
    q       [b, h, d]
    Kc, Vc  [g, m_c, d]            one shared copy of the context cache
    Kd, Vd  [b, g, m_d_max, d]     per-sample decode cache
    lens    [b] int32              valid decode rows per sample
(int4 caches hold two codes per byte: their last axis is d/2 bytes.)

Recipe: numpy PCG64 seeded per workload, draws in the order q, Kc, Vc, Kd, Vd,
each ``standard_normal(float32)`` rounded to bf16 with round-to-nearest-even;
then ``lens`` (``integers(1, m_d_max + 1)`` when ragged, else all ``m_d_max``).

8-bit caches (``kv="fp8_e4m3"`` or ``"int8"``, stored as uint8 codes): the
same draws, multiplied by ``qmax / 4.5`` (4.5 standard deviations map to the
largest code: 448 for OCP fp8 E4M3, 127 for int8), saturated at +-qmax and
encoded with round-to-nearest-even (fp8 through torch's ``float8_e4m3fn``
cast, int8 through ``numpy.rint``). 4-bit caches (``kv="int4"``): the same
with qmax = 7, the codes then packed two per byte, element 2u in the low
nibble of byte u and element 2u+1 in the high nibble. After ``lens``, per-group factors
``c = 2**uniform(-1, 1)`` are drawn for keys, then for values, and the
scales are ``k_scale = c_k * 4.5 / qmax`` (``v_scale`` likewise), so a
group's dequantized keys are close to its draws times ``c_k``: heads of
different magnitude, as in trained models.
"""
from __future__ import annotations

import dataclasses

import numpy as np

BF16_NAN = np.uint16(0x7FC0)
KV_TYPES = ("bf16", "fp8_e4m3", "int8", "int4")
KV_BITS = {"bf16": 16, "fp8_e4m3": 8, "int8": 8, "int4": 4}
KV_QMAX = {"fp8_e4m3": 448.0, "int8": 127.0, "int4": 7.0}
KV_CLIP_SIGMA = 4.5
# A byte that poisons rows past a sample's length: NaN in fp8 E4M3, the
# largest value in int8 and (in both nibbles) in int4.
KV_POISON = {"fp8_e4m3": np.uint8(0x7F), "int8": np.uint8(0x7F), "int4": np.uint8(0x77)}


def row_bytes(d: int, kv: str) -> int:
    """Bytes of one cache row of d elements."""
    return d * KV_BITS[kv] // 8


def cache_cols(d: int, kv: str) -> int:
    """Length of a cache array's last axis: d elements, or d/2 bytes for int4."""
    return d // 2 if kv == "int4" else d


@dataclasses.dataclass(frozen=True)
class Workload:
    name: str
    b: int
    h: int
    g: int
    d: int
    m_c: int
    m_d_max: int
    ragged: bool
    seed: int
    n: int = 1  # new tokens per sample (draft tokens verified together when > 1)
    kv: str = "bf16"  # cache element type: bf16, or 8-/4-bit codes with per-group scales

    @property
    def p(self) -> int:
        return self.h // self.g


# The five synthetic layers: a tiny MHA layer; 7B-shaped MHA layers (32 heads
# of 128) at 16 and 32 samples over an 8k context; an MQA layer with 128
# samples over 16k; and a GQA layer (8 KV groups) with 256 samples over 32k
# and ragged decode lengths uniform in [1, 1024]. Then the 32-sample MHA layer
# verifying 4 draft tokens per sample in one step (speculative decoding), and
# the 32-sample MHA and the MQA layer with 8-bit KV caches, and the 32-sample
# MHA layer with int4 caches.
WORKLOADS = {
    w.name: w
    for w in (
        Workload("tiny_mha_b4_mc128", 4, 4, 4, 64, 128, 16, False, 1001),
        Workload("mha7b_b16_mc8k_md256", 16, 32, 32, 128, 8192, 256, False, 1002),
        Workload("mha7b_b32_mc8k_md512", 32, 32, 32, 128, 8192, 512, False, 1003),
        Workload("mqa_b128_mc16k_md512", 128, 32, 1, 128, 16384, 512, False, 1004),
        Workload("gqa8_b256_mc32k_ragged1024", 256, 32, 8, 128, 32768, 1024, True, 1005),
        Workload("mha7b_b32_mc8k_md512_draft4", 32, 32, 32, 128, 8192, 512, False, 1006, 4),
        Workload("mha7b_b32_mc8k_md512_fp8", 32, 32, 32, 128, 8192, 512, False, 1007, 1,
                 "fp8_e4m3"),
        Workload("mha7b_b32_mc8k_md512_int8", 32, 32, 32, 128, 8192, 512, False, 1008, 1, "int8"),
        Workload("mqa_b128_mc16k_md512_fp8", 128, 32, 1, 128, 16384, 512, False, 1009, 1,
                 "fp8_e4m3"),
        Workload("mha7b_b32_mc8k_md512_int4", 32, 32, 32, 128, 8192, 512, False, 1010, 1, "int4"),
    )
}
WORKLOAD_ORDER = list(WORKLOADS)
HEADLINE = "mha7b_b32_mc8k_md512"


def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round float32 to bf16 (nearest, ties to even); returns uint16 bits."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    u = x.view(np.uint32)
    rounded = (u + np.uint32(0x7FFF) + ((u >> np.uint32(16)) & np.uint32(1))) >> np.uint32(16)
    out = rounded.astype(np.uint16)
    nan = np.isnan(x)
    if nan.any():
        out[nan] = BF16_NAN
    return out


def _normal_bf16(rng: np.random.Generator, shape) -> np.ndarray:
    n = int(np.prod(shape))
    out = np.empty(n, dtype=np.uint16)
    step = 1 << 24  # bound the float32 temporary to 64 MiB
    for s in range(0, n, step):
        e = min(n, s + step)
        out[s:e] = f32_to_bf16_bits(rng.standard_normal(e - s, dtype=np.float32))
    return out.reshape(shape)


def pack_int4(codes: np.ndarray) -> np.ndarray:
    """Integer codes in [-8, 7] (last axis even) -> bytes, two codes each:
    element 2u in the low nibble of byte u, element 2u+1 in the high one."""
    c = np.asarray(codes).astype(np.int64) & 15
    return (c[..., 0::2] | (c[..., 1::2] << 4)).astype(np.uint8)


def _encode(y: np.ndarray, kv: str) -> np.ndarray:
    """float32 values already in code units -> saturated codes (RNE); int4
    codes come out one per element, unpacked."""
    qmax = KV_QMAX[kv]
    y = np.clip(y, -qmax, qmax)
    if kv in ("int8", "int4"):
        return np.rint(y).astype(np.int8).view(np.uint8)
    import torch
    return torch.from_numpy(np.ascontiguousarray(y)).to(torch.float8_e4m3fn) \
        .view(torch.uint8).numpy()


def _normal_codes(rng: np.random.Generator, shape, kv: str) -> np.ndarray:
    n = int(np.prod(shape))
    per = 2 if kv == "int4" else 1  # codes per stored byte
    out = np.empty(n // per, dtype=np.uint8)
    mult = np.float32(KV_QMAX[kv] / KV_CLIP_SIGMA)
    step = 1 << 24  # even, so int4 pairs never straddle two steps
    for s in range(0, n, step):
        e = min(n, s + step)
        codes = _encode(rng.standard_normal(e - s, dtype=np.float32) * mult, kv)
        out[s // per:e // per] = pack_int4(codes.view(np.int8)) if per == 2 else codes
    return out.reshape(tuple(shape[:-1]) + (shape[-1] // per,))


def make_inputs(b, h, g, d, m_c, m_d_max, *, seed, ragged=False, lens=None,
                poison_tail=False, with_decode_tail=True, n=1, kv="bf16"):
    """Draw one problem instance.

    ``lens`` overrides the drawn lengths (it is applied after all draws, so the
    tensors stay identical). ``poison_tail`` fills decode rows ``t >= len_i``
    with bf16 NaN, so any read of them shows up in the output. With ``n > 1``
    new tokens per sample, q is [b, h, n, d] and ragged lengths are drawn in
    [n, m_d_max] (the n tokens are the last n valid decode rows). With an
    8-bit ``kv`` the caches are uint8 codes, with ``"int4"`` uint8 bytes of
    two codes each (last axis d/2), and the dict also holds ``kv``,
    ``k_scale`` and ``v_scale`` (float32 [g]).
    """
    if h % g:
        raise ValueError("h must be a multiple of g")
    if kv not in KV_TYPES:
        raise ValueError(f"unknown cache type {kv!r}")
    if kv == "int4" and d % 2:
        raise ValueError("int4 caches need an even head dimension")
    rng = np.random.Generator(np.random.PCG64(seed))
    q = _normal_bf16(rng, (b, h, d) if n == 1 else (b, h, n, d))
    cache = _normal_bf16 if kv == "bf16" else (lambda r, shp: _normal_codes(r, shp, kv))
    Kc = cache(rng, (g, m_c, d))
    Vc = cache(rng, (g, m_c, d))
    Kd = cache(rng, (b, g, m_d_max, d))
    Vd = cache(rng, (b, g, m_d_max, d))
    if ragged:
        drawn = rng.integers(min(n, m_d_max) if m_d_max > 0 else 0, m_d_max + 1,
                             size=b).astype(np.int32) if m_d_max > 0 else np.zeros(b, np.int32)
    else:
        drawn = np.full(b, m_d_max, dtype=np.int32)
    if lens is not None:
        drawn = np.asarray(lens, dtype=np.int32).reshape(b).copy()
    scales = {}
    if kv != "bf16":
        base = KV_CLIP_SIGMA / KV_QMAX[kv]
        c_k = np.exp2(rng.uniform(-1.0, 1.0, size=g))
        c_v = np.exp2(rng.uniform(-1.0, 1.0, size=g))
        scales = dict(kv=kv, k_scale=(c_k * base).astype(np.float32),
                      v_scale=(c_v * base).astype(np.float32))
    if poison_tail:
        poison = BF16_NAN if kv == "bf16" else KV_POISON[kv]
        for i in range(b):
            Kd[i, :, drawn[i]:, :] = poison
            Vd[i, :, drawn[i]:, :] = poison
    return dict(q=q, Kc=Kc, Vc=Vc, Kd=Kd, Vd=Vd, lens=drawn, **scales)


def make_workload_inputs(w: Workload, *, seed=None, poison_tail=False):
    return make_inputs(w.b, w.h, w.g, w.d, w.m_c, w.m_d_max,
                       seed=w.seed if seed is None else seed, ragged=w.ragged,
                       poison_tail=poison_tail, n=w.n, kv=w.kv)


def make_workload_lens(w: Workload) -> np.ndarray:
    """The workload's decode lengths (ragged ones come after the tensors in
    the draw order, so those are drawn in full)."""
    if not w.ragged:
        return np.full(w.b, w.m_d_max, dtype=np.int32)
    return make_workload_inputs(w)["lens"]


def first_samples(x, nb):
    """The inputs of the first nb samples (the shared context unchanged)."""
    y = dict(x)
    for k in ("q", "Kd", "Vd", "lens"):
        y[k] = np.ascontiguousarray(x[k][:nb])
    return y


def kv_bytes(g, d, m_c, lens, kv="bf16") -> int:
    """Algorithmic KV bytes of one bifurcated step: one copy of context K and
    V plus every sample's valid decode K and V (Section 4.3), at the cache's
    element size (2 bytes bf16, 1 byte for 8-bit codes, 1/2 byte for int4)."""
    return 2 * g * row_bytes(d, kv) * (int(m_c) + int(np.sum(lens, dtype=np.int64)))


def replicated_kv_bytes(b, g, d, m_c, lens, kv="bf16") -> int:
    """KV bytes when the context is read once per sample (Section 4.3)."""
    return 2 * g * row_bytes(d, kv) * (b * int(m_c) + int(np.sum(lens, dtype=np.int64)))


def attention_flops(h, d, b, m_c, lens, n=1) -> int:
    """Multiply-adds of QK^T and PV counted as 2 flops each: identical for the
    bifurcated and the standard formulation (Section 4.2). With n tokens per
    sample, token r sees m_c + max(0, len_i - n + r + 1) keys."""
    lens = np.asarray(lens, dtype=np.int64)
    seen = sum(int(np.maximum(lens - n + r + 1, 0).sum()) for r in range(n))
    return 4 * h * d * (n * b * int(m_c) + seen)
