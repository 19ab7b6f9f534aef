"""The C-ABI library on the host: it loads, exports every declared entry
point, and rejects bad arguments before touching the GPU (CPU only)."""
import ctypes
import os
import re

import numpy as np
import pytest

import paper_2403_08845_amd as bif

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "bifattn.h")


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(bifattn_[a-z_]+)\s*\(", text)))


@pytest.fixture(scope="module")
def L():
    if not os.path.exists(bif.LIB_PATH):
        pytest.fail("libbifattn.so is not built: run `python -m paper_2403_08845_amd.build`")
    return bif.lib()


def test_every_declared_symbol_is_exported(L):
    names = declared_functions()
    assert len(names) >= 10
    for name in names:
        assert hasattr(L, name), name
    assert sorted(bif.EXPORTED) == names


def test_version_and_status_strings(L):
    assert bif.bifattn_version() == 4
    for code in (bif.OK, bif.EINVAL, bif.EUNSUPPORTED, bif.EALIGN, bif.ENOMEM, bif.EHIP, bif.ELENS,
                 bif.ESCALE):
        assert bif.status_string(code)
    assert bif.status_string(12345) == "unknown status"


def _create(L, *dims):
    d = bif.Dims(*dims)
    h = ctypes.c_void_p(1234)
    st = L.bifattn_plan_create(ctypes.byref(d), ctypes.byref(h))
    return st, h.value


@pytest.mark.parametrize("dims,expect", [
    ((0, 4, 4, 64, 128, 16, 0.0), bif.EINVAL),        # b < 1
    ((4, 4, 3, 64, 128, 16, 0.0), bif.EINVAL),        # h % g
    ((4, 4, 4, 64, 0, 16, 0.0), bif.EINVAL),          # m_c < 1
    ((4, 4, 4, 64, 128, -1, 0.0), bif.EINVAL),        # m_d_max < 0
    ((4, 4, 4, 64, 128, 16, float("nan")), bif.EINVAL),
    ((4, 4, 4, 96, 128, 16, 0.0), bif.EUNSUPPORTED),  # d not 64/128
    ((4, 128, 1, 128, 128, 16, 0.0), bif.EUNSUPPORTED),  # p = 128 > 64
    ((2**30, 2**30, 2**30, 128, 128, 16, 0.0), bif.EINVAL),  # overflowing sizes
    ((1, 32, 32, 128, 2**23, 0, 0.0), bif.EUNSUPPORTED),    # one cache past 2^31 bytes
    ((1, 32, 32, 128, 2**23 - 64, 64, 0.0), bif.EUNSUPPORTED),  # context + decode rows
    ((2, 4, 2, 64, 128, 16, 0.0, -1), bif.EINVAL),          # negative token count
    ((2, 32, 1, 64, 128, 16, 0.0, 3), bif.EUNSUPPORTED),    # p * n = 96 query rows per unit
    ((2, 4, 2, 64, 128, 16, 0.0, 1, 4), bif.EINVAL),        # unknown cache type
    ((2, 4, 2, 64, 128, 16, 0.0, 1, -1), bif.EINVAL),
    ((1, 32, 32, 128, 2**24, 0, 0.0, 1, 1), bif.EUNSUPPORTED),  # fp8 cache past 2^31 bytes
    ((1, 32, 32, 128, 2**24 - 64, 64, 0.0, 1, 2), bif.EUNSUPPORTED),  # int8, both parts
    ((1, 32, 32, 128, 2**25, 0, 0.0, 1, 3), bif.EUNSUPPORTED),  # int4 cache past 2^31 bytes
])
def test_plan_create_rejects_bad_dims_without_a_device(L, dims, expect):
    st, handle = _create(L, *dims)
    assert st == expect
    assert handle is None


def test_null_arguments(L):
    assert L.bifattn_plan_create(None, None) == bif.EINVAL
    assert L.bifattn_plan_destroy(None) == bif.OK
    assert L.bifattn_plan_get_info(None, None) == bif.EINVAL
    assert L.bifattn_decode(None, *([None] * 8)) == bif.EINVAL
    assert L.bifattn_decode_replicated(None, *([None] * 6)) == bif.EINVAL
    assert L.bifattn_decode_scaled(None, *([None] * 10)) == bif.EINVAL
    assert L.bifattn_decode_replicated_scaled(None, *([None] * 8)) == bif.EINVAL
    assert L.bifattn_plan_status(None, None) == bif.EINVAL
    assert L.bifattn_plan_set_timing(None, 0, 1) == bif.EINVAL


def test_binding_refuses_host_tensors_before_any_call():
    torch = pytest.importorskip("torch")

    class FakePlan:
        dims = bif.Dims(2, 4, 2, 64, 32, 8, 0.0)
        handle = ctypes.c_void_p(0)
        device = torch.device("cuda", 0)

    q = torch.zeros(2, 4, 64, dtype=torch.bfloat16)
    with pytest.raises(ValueError):
        bif.bifattn_decode(FakePlan(), q, q, q, q, q, q, q, stream=0)
    with pytest.raises(TypeError):
        bif.bifattn_decode(FakePlan(), q.float(), q, q, q, q, q, q, stream=0)
    with pytest.raises(ValueError):
        bif.bifattn_decode(FakePlan(), q[:1], q, q, q, q, q, q, stream=0)


def test_byte_bound_follows_the_cache_type(L):
    """One sample's cache rows must fit 2^31 bytes: 2^23 rows of 128 bf16 do
    not, the same rows of 8-bit codes pass the shape checks (and then need a
    device)."""
    bf16 = _create(L, 1, 32, 32, 128, 2**23, 0, 0.0, 1, 0)
    assert bf16 == (bif.EUNSUPPORTED, None)
    for kv in (1, 2):
        st, handle = _create(L, 1, 32, 32, 128, 2**23, 0, 0.0, 1, kv)
        assert st in (bif.EHIP, bif.OK, bif.ENOMEM)
        if st == bif.OK:
            assert L.bifattn_plan_destroy(ctypes.c_void_p(handle)) == bif.OK
