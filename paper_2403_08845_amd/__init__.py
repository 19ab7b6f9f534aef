"""Python binding of libbifattn (bifurcated decode attention on MI355X).

Argument marshalling only: every step of the computation runs in the HIP
kernels of ``libbifattn.so``. The functions carry the C ABI's names
(include/bifattn.h); torch tensors are checked against the plan's shape,
dtype, device and contiguity before their device pointers are handed over,
so a mismatched tensor is refused on the host instead of being read out of
bounds on the GPU. There is no fallback: without the built library every
entry point raises.
"""
from __future__ import annotations

import ctypes
import os

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libbifattn.so")

OK, EINVAL, EUNSUPPORTED, EALIGN, ENOMEM, EHIP, ELENS, ESCALE, ESCRATCH = 0, -1, -2, -3, -4, -5, -6, -7, -8
#: Size of the fixed device scratch of bifattn_decode_noalloc (BIFATTN_NOALLOC_SCRATCH_BYTES).
NOALLOC_SCRATCH_BYTES = 64 << 20
KERNEL_PARTIALS, KERNEL_COMBINE, KERNEL_CALL, KERNEL_CONTEXT, KERNEL_DECODE = 0, 1, 2, 3, 4
#: Cache element types (bifattn_kv_type_t).
KV_TYPES = {"bf16": 0, "fp8_e4m3": 1, "int8": 2, "int4": 3}
#: Paths of bifattn_decode (bifattn_path_t): "auto" lets the plan choose.
PATHS = {"auto": 0, "bifurcated": 1, "standard": 2}

EXPORTED = (
    "bifattn_plan_create", "bifattn_plan_destroy", "bifattn_plan_get_info", "bifattn_decode",
    "bifattn_decode_scaled", "bifattn_decode_replicated", "bifattn_decode_replicated_scaled",
    "bifattn_append_kv", "bifattn_plan_status", "bifattn_plan_set_timing",
    "bifattn_plan_read_timing", "bifattn_status_string", "bifattn_version",
    "bifattn_decode_noalloc",
)


class BifattnError(RuntimeError):
    def __init__(self, status: int, what: str):
        self.status = status
        super().__init__(f"{what}: {status_string(status)} ({status})")


class Dims(ctypes.Structure):
    _fields_ = [("b", ctypes.c_int32), ("h", ctypes.c_int32), ("g", ctypes.c_int32),
                ("d", ctypes.c_int32), ("m_c", ctypes.c_int32), ("m_d_max", ctypes.c_int32),
                ("scale", ctypes.c_float), ("n", ctypes.c_int32), ("kv_type", ctypes.c_int32),
                ("path", ctypes.c_int32)]


class PlanInfo(ctypes.Structure):
    _fields_ = [("ctx_keys_per_block", ctypes.c_int32), ("ctx_splits", ctypes.c_int32),
                ("ctx_row_blocks", ctypes.c_int32), ("ctx_blocks", ctypes.c_int32),
                ("dec_keys_per_block", ctypes.c_int32), ("dec_splits", ctypes.c_int32),
                ("dec_blocks", ctypes.c_int32),
                ("fused", ctypes.c_int32), ("path", ctypes.c_int32),
                ("workspace_bytes", ctypes.c_size_t), ("ctx_kernel", ctypes.c_int32),
                ("side_stream", ctypes.c_int32)]

    def as_dict(self):
        return {name: getattr(self, name) for name, _ in self._fields_}


_lib = None


def lib() -> ctypes.CDLL:
    """Load libbifattn.so (built in-tree); raises if it has not been built."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it with "
                               "`python -m paper_2403_08845_amd.build`")
        # One HIP runtime per process: torch's is loaded first, so that the
        # library's libamdhip64 dependency resolves to it (the tensors and
        # streams handed over are torch's); a second runtime loaded beside it
        # keeps the first from opening the device.
        import torch  # noqa: F401
        L = ctypes.CDLL(LIB_PATH)
        vp, i32, st = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int
        L.bifattn_plan_create.argtypes = [ctypes.POINTER(Dims), ctypes.POINTER(vp)]
        L.bifattn_plan_destroy.argtypes = [vp]
        L.bifattn_plan_get_info.argtypes = [vp, ctypes.POINTER(PlanInfo)]
        L.bifattn_decode.argtypes = [vp, vp, vp, vp, vp, vp, vp, vp, vp]
        L.bifattn_decode_scaled.argtypes = [vp, vp, vp, vp, vp, vp, vp, vp, vp, vp, vp]
        L.bifattn_decode_replicated.argtypes = [vp, vp, vp, vp, vp, vp, vp]
        L.bifattn_decode_replicated_scaled.argtypes = [vp, vp, vp, vp, vp, vp, vp, vp, vp]
        L.bifattn_append_kv.argtypes = [vp, vp, vp, vp, vp, vp, vp]
        L.bifattn_decode_noalloc.argtypes = [ctypes.POINTER(Dims), vp, vp, vp, vp, vp, vp, vp, vp,
                                             vp, vp]
        L.bifattn_plan_status.argtypes = [vp, vp]
        L.bifattn_plan_set_timing.argtypes = [vp, st, i32]
        L.bifattn_plan_read_timing.argtypes = [vp, ctypes.POINTER(i32), ctypes.POINTER(ctypes.c_double)]
        L.bifattn_status_string.argtypes = [st]
        L.bifattn_status_string.restype = ctypes.c_char_p
        L.bifattn_version.restype = i32
        for name in EXPORTED:
            if name not in ("bifattn_status_string", "bifattn_version"):
                getattr(L, name).restype = st
        _lib = L
    return _lib


def status_string(status: int) -> str:
    return lib().bifattn_status_string(int(status)).decode()


def bifattn_version() -> int:
    return int(lib().bifattn_version())


def _check(status: int, what: str):
    if status != OK:
        raise BifattnError(status, what)


class Plan:
    """A bifattn_plan_t: problem dimensions plus the workspace it owns
    (n = new tokens per sample; kv = cache element type, a KV_TYPES name;
    path = a PATHS name, "auto" for the workload-based switch)."""

    def __init__(self, b, h, g, d, m_c, m_d_max, scale=0.0, n=1, kv="bf16", path="auto"):
        if kv not in KV_TYPES:
            raise ValueError(f"kv must be one of {sorted(KV_TYPES)}")
        if path not in PATHS:
            raise ValueError(f"path must be one of {sorted(PATHS)}")
        self.kv = kv
        self.dims = Dims(b, h, g, d, m_c, m_d_max, scale, n, KV_TYPES[kv], PATHS[path])
        handle = ctypes.c_void_p()
        _check(lib().bifattn_plan_create(ctypes.byref(self.dims), ctypes.byref(handle)),
               "bifattn_plan_create")
        self.handle = handle
        import torch
        #: The device the plan's workspace lives on (current at creation):
        #: every tensor and the stream of a call must belong to it.
        self.device = torch.device("cuda", torch.cuda.current_device())

    def close(self):
        if getattr(self, "handle", None) is not None and self.handle.value:
            _check(lib().bifattn_plan_destroy(self.handle), "bifattn_plan_destroy")
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def __enter__(self):
        return self

    def __exit__(self, *exc):
        self.close()

    def info(self) -> dict:
        info = PlanInfo()
        _check(lib().bifattn_plan_get_info(self.handle, ctypes.byref(info)), "bifattn_plan_get_info")
        return info.as_dict()


def bifattn_plan_create(b, h, g, d, m_c, m_d_max, scale=0.0, n=1, kv="bf16",
                        path="auto") -> Plan:
    return Plan(b, h, g, d, m_c, m_d_max, scale, n, kv, path)


def bifattn_plan_destroy(plan: Plan):
    plan.close()


def bifattn_plan_get_info(plan: Plan) -> dict:
    return plan.info()


def _torch():
    import torch
    return torch


def _stream_ptr(stream, device=None):
    """A torch stream, a raw hipStream_t (int), or None for torch's current
    stream of `device`."""
    if stream is None:
        torch = _torch()
        raw = getattr(torch._C, "_cuda_getCurrentRawStream", None)
        if raw is not None:
            return ctypes.c_void_p(raw(device.index if device is not None
                                       else torch.cuda.current_device()))
        stream = torch.cuda.current_stream(device)
    return ctypes.c_void_p(stream.cuda_stream if hasattr(stream, "cuda_stream") else int(stream))


def _tensor(t, shape, dtype, device, name):
    """The device pointer of torch tensor t after checking it. shape: one
    shape, or a list of accepted shapes; dtype: one dtype or a tuple of
    accepted dtypes; device: the plan's device. The common case passes one
    combined test; a failing tensor gets the specific error."""
    dtypes = dtype if isinstance(dtype, tuple) else (dtype,)
    shapes = shape if isinstance(shape, list) else [shape]
    torch = _torch()
    if (isinstance(t, torch.Tensor) and t.dtype in dtypes and t.device == device
            and t.shape in shapes and t.is_contiguous()):
        return ctypes.c_void_p(t.data_ptr())
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{name} must be a torch.Tensor")
    if t.dtype not in dtypes:
        raise TypeError(f"{name} must be {' or '.join(map(str, dtypes))}, got {t.dtype}")
    shapes = [tuple(x) for x in shapes]
    if tuple(t.shape) not in shapes:
        raise ValueError(f"{name} must have shape {' or '.join(map(str, shapes))}, "
                         f"got {tuple(t.shape)}")
    if not t.is_cuda or t.device != device:
        raise ValueError(f"{name} must live on {device}")
    raise ValueError(f"{name} must be contiguous")


def _cache_dtypes(plan):
    """torch dtypes accepted for the plan's cache tensors: bf16, or any
    one-byte type holding the 8-bit codes (int4: bytes of two codes)."""
    import torch
    if plan.dims.kv_type == KV_TYPES["bf16"]:
        return torch.bfloat16
    if plan.dims.kv_type == KV_TYPES["int4"]:
        return (torch.uint8, torch.int8)
    return (torch.uint8, torch.int8, torch.float8_e4m3fn)


def _cols(D):
    """Last axis of a cache tensor: d elements, or d/2 bytes for int4."""
    return D.d // 2 if D.kv_type == KV_TYPES["int4"] else D.d


def _scales(plan, k_scale, v_scale, dev):
    import torch
    D = plan.dims
    return [ctypes.c_void_p(None) if s is None else _tensor(s, (D.g,), torch.float32, dev, name)
            for s, name in ((k_scale, "k_scale"), (v_scale, "v_scale"))]


def _query_shapes(D):
    """[b, h, n, d], or [b, h, d] too when n = 1."""
    n = max(1, D.n)
    shapes = [(D.b, D.h, n, D.d)]
    if n == 1:
        shapes.append((D.b, D.h, D.d))
    return shapes


def bifattn_decode(plan: Plan, q, Kc, Vc, Kd, Vd, decode_lens, out, stream=None):
    """Enqueue one bifurcated decode step (see include/bifattn.h).

    q bf16 [b,h,n,d] ([b,h,d] when n = 1); Kc, Vc [g,m_c,d] and Kd, Vd
    [b,g,m_d_max,d] of the plan's cache type (bf16, or one-byte codes;
    int4 caches hold two codes a byte, last axis d/2);
    decode_lens int32 [b]; out fp32 shaped like q; all on the same GPU.
    """
    bifattn_decode_scaled(plan, q, Kc, Vc, Kd, Vd, decode_lens, None, None, out, stream)


def bifattn_decode_scaled(plan: Plan, q, Kc, Vc, Kd, Vd, decode_lens, k_scale, v_scale, out,
                          stream=None):
    """bifattn_decode with per-group key / value scales (fp32 [g] tensors on
    the GPU, or None for 1)."""
    import torch
    D = plan.dims
    dev = plan.device
    cd = _cache_dtypes(plan)
    args = [
        _tensor(q, _query_shapes(D), torch.bfloat16, dev, "q"),
        _tensor(Kc, (D.g, D.m_c, _cols(D)), cd, dev, "Kc"),
        _tensor(Vc, (D.g, D.m_c, _cols(D)), cd, dev, "Vc"),
        _tensor(Kd, (D.b, D.g, D.m_d_max, _cols(D)), cd, dev, "Kd"),
        _tensor(Vd, (D.b, D.g, D.m_d_max, _cols(D)), cd, dev, "Vd"),
        _tensor(decode_lens, (D.b,), torch.int32, dev, "decode_lens"),
        *_scales(plan, k_scale, v_scale, dev),
        _tensor(out, [tuple(q.shape)], torch.float32, dev, "out"),
    ]
    _check(lib().bifattn_decode_scaled(plan.handle, *args, _stream_ptr(stream, dev)),
           "bifattn_decode_scaled")


class _Unplanned:
    """Dimensions and device of a call that has no plan (the allocation-free
    entry point): what the tensor checks compare against."""

    def __init__(self, dims, device):
        self.dims = dims
        self.device = device


def noalloc_dims(b, h, g, d, m_c, m_d_max, scale=0.0, n=1, kv="bf16", path="auto") -> Dims:
    """The bifattn_dims_t of a bifattn_decode_noalloc call."""
    if kv not in KV_TYPES:
        raise ValueError(f"kv must be one of {sorted(KV_TYPES)}")
    if path not in PATHS:
        raise ValueError(f"path must be one of {sorted(PATHS)}")
    return Dims(b, h, g, d, m_c, m_d_max, scale, n, KV_TYPES[kv], PATHS[path])


def bifattn_decode_noalloc(dims: Dims, q, Kc, Vc, Kd, Vd, decode_lens, k_scale, v_scale, out,
                           stream=None):
    """bifattn_decode_scaled without a plan and without any device
    allocation (see include/bifattn.h): the partials live in the library's
    fixed per-GPU scratch buffer, so calls on one GPU must not overlap.
    dims: from noalloc_dims(); tensors as for bifattn_decode_scaled, on the
    current device."""
    import torch
    dev = torch.device("cuda", torch.cuda.current_device())
    shape = _Unplanned(dims, dev)
    cd = _cache_dtypes(shape)
    D = dims
    args = [
        _tensor(q, _query_shapes(D), torch.bfloat16, dev, "q"),
        _tensor(Kc, (D.g, D.m_c, _cols(D)), cd, dev, "Kc"),
        _tensor(Vc, (D.g, D.m_c, _cols(D)), cd, dev, "Vc"),
        _tensor(Kd, (D.b, D.g, D.m_d_max, _cols(D)), cd, dev, "Kd"),
        _tensor(Vd, (D.b, D.g, D.m_d_max, _cols(D)), cd, dev, "Vd"),
        _tensor(decode_lens, (D.b,), torch.int32, dev, "decode_lens"),
        *_scales(shape, k_scale, v_scale, dev),
        _tensor(out, [tuple(q.shape)], torch.float32, dev, "out"),
    ]
    _check(lib().bifattn_decode_noalloc(ctypes.byref(dims), *args, _stream_ptr(stream, dev)),
           "bifattn_decode_noalloc")


def bifattn_decode_replicated(plan: Plan, q, K, V, decode_lens, out, stream=None):
    """Enqueue the ablation over a physically replicated cache
    K, V [b, g, m_c + m_d_max, d] of the plan's cache type."""
    bifattn_decode_replicated_scaled(plan, q, K, V, decode_lens, None, None, out, stream)


def bifattn_decode_replicated_scaled(plan: Plan, q, K, V, decode_lens, k_scale, v_scale, out,
                                     stream=None):
    """The replicated ablation with per-group scales."""
    import torch
    D = plan.dims
    dev = plan.device
    rows = D.m_c + D.m_d_max
    cd = _cache_dtypes(plan)
    args = [
        _tensor(q, _query_shapes(D), torch.bfloat16, dev, "q"),
        _tensor(K, (D.b, D.g, rows, _cols(D)), cd, dev, "K"),
        _tensor(V, (D.b, D.g, rows, _cols(D)), cd, dev, "V"),
        _tensor(decode_lens, (D.b,), torch.int32, dev, "decode_lens"),
        *_scales(plan, k_scale, v_scale, dev),
        _tensor(out, [tuple(q.shape)], torch.float32, dev, "out"),
    ]
    _check(lib().bifattn_decode_replicated_scaled(plan.handle, *args, _stream_ptr(stream, dev)),
           "bifattn_decode_replicated_scaled")


def bifattn_append_kv(plan: Plan, k_new, v_new, Kd, Vd, decode_lens, stream=None):
    """Enqueue the decode-cache append of one step (see include/bifattn.h):
    k_new, v_new [b,g,n,d] go to rows decode_lens[i] .. + n - 1 of
    Kd, Vd [b,g,m_d_max,d] (the plan's cache type); decode_lens int32 [b]
    advances by n."""
    import torch
    D = plan.dims
    dev = plan.device
    n = max(1, D.n)
    cd = _cache_dtypes(plan)
    args = [
        _tensor(k_new, (D.b, D.g, n, _cols(D)), cd, dev, "k_new"),
        _tensor(v_new, (D.b, D.g, n, _cols(D)), cd, dev, "v_new"),
        _tensor(Kd, (D.b, D.g, D.m_d_max, _cols(D)), cd, dev, "Kd"),
        _tensor(Vd, (D.b, D.g, D.m_d_max, _cols(D)), cd, dev, "Vd"),
        _tensor(decode_lens, (D.b,), torch.int32, dev, "decode_lens"),
    ]
    _check(lib().bifattn_append_kv(plan.handle, *args, _stream_ptr(stream, dev)),
           "bifattn_append_kv")


def bifattn_plan_status(plan: Plan, stream=None) -> int:
    """Synchronise the stream; return OK, ELENS or ESCALE (and clear the flags)."""
    st = lib().bifattn_plan_status(plan.handle, _stream_ptr(stream, plan.device))
    if st not in (OK, ELENS, ESCALE):
        raise BifattnError(st, "bifattn_plan_status")
    return st


def bifattn_plan_set_timing(plan: Plan, kernel: int, capacity: int):
    _check(lib().bifattn_plan_set_timing(plan.handle, int(kernel), int(capacity)),
           "bifattn_plan_set_timing")


def bifattn_plan_read_timing(plan: Plan):
    """(number of timed calls, total milliseconds)."""
    n = ctypes.c_int32()
    ms = ctypes.c_double()
    _check(lib().bifattn_plan_read_timing(plan.handle, ctypes.byref(n), ctypes.byref(ms)),
           "bifattn_plan_read_timing")
    return int(n.value), float(ms.value)
