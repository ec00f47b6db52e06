"""ctypes binding of ``libaq.so`` (the C ABI declared in ``include/aq.h``).

Argument marshalling only: every step of the forward runs in the library's
HIP kernels.  PyTorch supplies device memory and the current stream.  If the
library is not built, loading fails loudly; there is no fallback.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional

import numpy as np

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libaq.so")

AQ_OK, AQ_ERR_INVALID_ARGUMENT, AQ_ERR_UNSUPPORTED, AQ_ERR_OUT_OF_MEMORY, AQ_ERR_DEVICE = range(5)
AQ_F32, AQ_F16, AQ_BF16, AQ_I8 = range(4)
AQ_PATH_AUTO, AQ_PATH_LUT, AQ_PATH_DECODE = range(3)

DTYPE_CODES = {"f32": AQ_F32, "f16": AQ_F16, "bf16": AQ_BF16, "i8": AQ_I8}
PATH_CODES = {"auto": AQ_PATH_AUTO, "lut": AQ_PATH_LUT, "decode": AQ_PATH_DECODE}
PATH_NAMES = {v: k for k, v in PATH_CODES.items()}
STATUS_NAMES = {0: "AQ_OK", 1: "AQ_ERR_INVALID_ARGUMENT", 2: "AQ_ERR_UNSUPPORTED", 3: "AQ_ERR_OUT_OF_MEMORY",
                4: "AQ_ERR_DEVICE"}
# aq_option (include/aq.h)
OPTION_CODES = {"lut_max_tokens": 1, "weights": 2, "generic": 3, "record_product": 4, "fused_tile": 5,
                "dense_tile": 6, "rec_linear_tile": 7, "tile_order": 8, "stage_rows": 9, "split_k": 10,
                "grad_splits": 11, "grad_regs": 12, "grad_tile": 13, "table_one_launch": 14}
_TILE_OPTIONS = ("fused_tile", "dense_tile", "grad_tile")

EXPORTED = ("aq_layer_create", "aq_layer_forward", "aq_layer_forward_static", "aq_layer_prepare", "aq_layers_prepare",
            "aq_layer_decode",
            "aq_layer_codebook_grad",
            "aq_layer_set_path", "aq_layer_set_option", "aq_layer_get_option", "aq_layer_set_launch_events",
            "aq_layer_last_launches", "aq_layer_describe", "aq_layer_choose_path", "aq_layer_destroy",
            "aq_last_error", "aq_version")


class AQError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(f"{STATUS_NAMES.get(status, status)}: {msg}")
        self.status = status


class aq_layer_desc(ctypes.Structure):
    _fields_ = [
        ("out_features", ctypes.c_int32),
        ("in_features", ctypes.c_int32),
        ("codebook_dtype", ctypes.c_int32),
        ("x_dtype", ctypes.c_int32),
        ("y_dtype", ctypes.c_int32),
        ("tile_dtype", ctypes.c_int32),
        ("conv_kh", ctypes.c_int32),
        ("conv_kw", ctypes.c_int32),
        ("conv_cin", ctypes.c_int32),
        ("conv_stride", ctypes.c_int32),
        ("conv_pad", ctypes.c_int32),
        ("in_h", ctypes.c_int32),
        ("in_w", ctypes.c_int32),
        ("max_tokens", ctypes.c_int64),
    ]


_lib = None


def load_library(path: str = LIB_PATH) -> ctypes.CDLL:
    """Load libaq.so once; raise if it has not been built."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise RuntimeError(f"{path} is not built: run `python -m paper_2506_05960_amd.build` "
                           "(the AQ layer has no non-HIP fallback)")
    lib = ctypes.CDLL(path)
    vp, i32, i64 = ctypes.c_void_p, ctypes.c_int, ctypes.c_int64
    lib.aq_layer_create.argtypes = [ctypes.POINTER(aq_layer_desc), vp, vp, vp, i32, i32, i32, ctypes.POINTER(vp)]
    lib.aq_layer_forward.argtypes = [vp, vp, vp, vp, i64, vp]
    lib.aq_layer_forward_static.argtypes = [vp, vp, vp, vp, i64, vp]
    lib.aq_layer_prepare.argtypes = [vp, i64, vp]
    lib.aq_layers_prepare.argtypes = [ctypes.POINTER(vp), ctypes.POINTER(i64), i32, vp]
    lib.aq_layer_decode.argtypes = [vp, vp, vp]
    lib.aq_layer_codebook_grad.argtypes = [vp, vp, vp, i32, vp, i64, vp]
    lib.aq_layer_set_path.argtypes = [vp, i32]
    lib.aq_layer_set_option.argtypes = [vp, i32, i64]
    lib.aq_layer_get_option.argtypes = [vp, i32, ctypes.POINTER(ctypes.c_int64)]
    lib.aq_layer_set_launch_events.argtypes = [vp, ctypes.POINTER(vp), i32]
    lib.aq_layer_last_launches.argtypes = [vp, ctypes.POINTER(ctypes.c_int32), ctypes.c_char_p, i64]
    lib.aq_layer_describe.argtypes = [vp, i64, ctypes.c_char_p, i64]
    lib.aq_layer_choose_path.argtypes = [vp, i64, ctypes.POINTER(ctypes.c_int)]
    lib.aq_layer_destroy.argtypes = [vp]
    for f in ("aq_layer_create", "aq_layer_forward", "aq_layer_forward_static", "aq_layer_prepare",
              "aq_layers_prepare", "aq_layer_decode",
              "aq_layer_codebook_grad",
              "aq_layer_set_path", "aq_layer_set_option", "aq_layer_get_option", "aq_layer_set_launch_events",
              "aq_layer_last_launches", "aq_layer_describe", "aq_layer_choose_path", "aq_layer_destroy"):
        getattr(lib, f).restype = ctypes.c_int
    lib.aq_last_error.restype = ctypes.c_char_p
    lib.aq_last_error.argtypes = []
    lib.aq_version.restype = ctypes.c_char_p
    lib.aq_version.argtypes = []
    _lib = lib
    return lib


def _check(status: int) -> None:
    if status != AQ_OK:
        raise AQError(status, load_library().aq_last_error().decode())


def make_desc(C_out: int, K: int, codebook_dtype: str, x_dtype: str, y_dtype: str, tile_dtype: str,
              max_tokens: int, conv=None) -> aq_layer_desc:
    d = aq_layer_desc()
    d.out_features, d.in_features = C_out, K
    d.codebook_dtype = DTYPE_CODES[codebook_dtype]
    d.x_dtype = DTYPE_CODES[x_dtype]
    d.y_dtype = DTYPE_CODES[y_dtype]
    d.tile_dtype = DTYPE_CODES[tile_dtype]
    if conv is not None:
        d.conv_kh, d.conv_kw, d.conv_cin = conv.kh, conv.kw, conv.cin
        d.conv_stride, d.conv_pad, d.in_h, d.in_w = conv.stride, conv.pad, conv.H, conv.W
    d.max_tokens = max_tokens
    return d


# ---- thin wrappers with the C names ----

def aq_layer_create(desc: aq_layer_desc, codebooks: np.ndarray, codes: np.ndarray, scales: np.ndarray,
                    g: int, M: int, B: int) -> int:
    lib = load_library()
    cb = np.ascontiguousarray(codebooks)
    cd = np.ascontiguousarray(codes)
    sc = np.ascontiguousarray(scales, dtype=np.float32)
    h = ctypes.c_void_p()
    _check(lib.aq_layer_create(ctypes.byref(desc), cb.ctypes.data, cd.ctypes.data, sc.ctypes.data,
                               g, M, B, ctypes.byref(h)))
    return h.value


def aq_layer_forward(handle: int, X: int, x_scales: int, Y: int, n: int, stream: int) -> None:
    _check(load_library().aq_layer_forward(handle, X, x_scales, Y, n, stream))


def aq_layer_forward_static(handle: int, X: int, x_scales: int, Y: int, n: int, stream: int) -> None:
    _check(load_library().aq_layer_forward_static(handle, X, x_scales, Y, n, stream))


def aq_layer_prepare(handle: int, n: int, stream: int) -> None:
    _check(load_library().aq_layer_prepare(handle, n, stream))


def aq_layers_prepare(handles, ns, stream: int) -> None:
    count = len(handles)
    if len(ns) != count:
        raise ValueError("one n per layer")
    hs = (ctypes.c_void_p * max(1, count))(*handles)
    nv = (ctypes.c_int64 * max(1, count))(*ns)
    _check(load_library().aq_layers_prepare(hs, nv, count, stream))


def aq_layer_decode(handle: int, W: int, stream: int) -> None:
    _check(load_library().aq_layer_decode(handle, W, stream))


def aq_layer_codebook_grad(handle: int, X: int, dY: int, dtype: str, dC: int, n: int, stream: int) -> None:
    _check(load_library().aq_layer_codebook_grad(handle, X, dY, DTYPE_CODES[dtype], dC, n, stream))


def aq_layer_set_path(handle: int, path: str) -> None:
    _check(load_library().aq_layer_set_path(handle, PATH_CODES[path]))


def aq_layer_set_option(handle: int, option: int, value: int) -> None:
    _check(load_library().aq_layer_set_option(handle, option, value))


def aq_layer_get_option(handle: int, option: int) -> int:
    out = ctypes.c_int64()
    _check(load_library().aq_layer_get_option(handle, option, ctypes.byref(out)))
    return out.value


def aq_layer_set_launch_events(handle: int, events) -> None:
    """``events``: HIP event handles (ints), recorded around the layer's later kernel launches."""
    arr = (ctypes.c_void_p * max(1, len(events)))(*events)
    _check(load_library().aq_layer_set_launch_events(handle, arr, len(events)))


def aq_layer_last_launches(handle: int):
    """(number of kernel launches of the layer's last call, their kernel names)."""
    n = ctypes.c_int32()
    buf = ctypes.create_string_buffer(4096)
    _check(load_library().aq_layer_last_launches(handle, ctypes.byref(n), buf, len(buf)))
    names = buf.value.decode()
    return n.value, (names.split("\n") if names else [])


def aq_layer_describe(handle: int, n: int) -> dict:
    """The route a forward over ``n`` tokens (linear) or images (conv) would take, as a dict."""
    buf = ctypes.create_string_buffer(1024)
    _check(load_library().aq_layer_describe(handle, n, buf, len(buf)))
    out = {}
    for kv in buf.value.decode().split(" "):
        k, _, v = kv.partition("=")
        out[k] = v
    return out


def aq_layer_choose_path(handle: int, tokens: int) -> str:
    out = ctypes.c_int()
    _check(load_library().aq_layer_choose_path(handle, tokens, ctypes.byref(out)))
    return PATH_NAMES[out.value]


def aq_layer_destroy(handle: Optional[int]) -> None:
    _check(load_library().aq_layer_destroy(handle))


def aq_version() -> str:
    return load_library().aq_version().decode()


# ---- convenience object over the same calls ----

def _torch_dtypes(name: str):
    """torch dtypes accepted for a storage dtype (bf16 also as its int16 bit pattern)."""
    import torch
    return {"f32": (torch.float32,), "f16": (torch.float16,), "bf16": (torch.bfloat16, torch.int16),
            "i8": (torch.int8,)}[name]


def _torch_dtype(name: str):
    return _torch_dtypes(name)[0]


_NP_DTYPES = {"f32": (np.float32,), "f16": (np.float16,), "bf16": (np.uint16, np.int16)}
_DEVICE_TYPE = "cuda"   # where every tensor argument must live (host-side tests of the checks change it)


def _check_tensor(what: str, t, dtypes, shape, device) -> None:
    """ValueError unless ``t`` is a contiguous device tensor of one of ``dtypes`` and exactly ``shape``."""
    import torch
    if not isinstance(t, torch.Tensor):
        raise ValueError(f"{what} must be a torch tensor, got {type(t).__name__}")
    if t.dtype not in dtypes:
        raise ValueError(f"{what} must have dtype {' or '.join(str(d) for d in dtypes)}, got {t.dtype}")
    if tuple(t.shape) != tuple(shape):
        raise ValueError(f"{what} must have shape {tuple(shape)}, got {tuple(t.shape)}")
    if not t.is_contiguous():
        raise ValueError(f"{what} must be contiguous")
    if t.device.type != _DEVICE_TYPE or (device is not None and t.device.index != device):
        raise ValueError(f"{what} must be on {_DEVICE_TYPE}:{device}, got {t.device}")


class AQLayer:
    """A device-resident AQ layer.

    ``spec`` carries C_out, K, g, M, B, the dtypes and ``conv`` geometry (or
    None); ``inputs`` carries host numpy ``codebooks``, ``codes`` and ``scales``.
    Every tensor argument is checked (dtype, exact shape, contiguity, device)
    before the library is called: the C ABI cannot see buffer extents.
    """

    def __init__(self, spec, inputs, max_tokens: Optional[int] = None):
        self.spec = spec
        s = spec
        mt = max_tokens if max_tokens is not None else s.tokens
        cb = np.asarray(inputs["codebooks"])
        if cb.shape != (s.M, 1 << s.B, s.g):
            raise ValueError(f"codebooks must have shape {(s.M, 1 << s.B, s.g)}, got {cb.shape}")
        if cb.dtype.type not in _NP_DTYPES[s.codebook_dtype]:
            raise ValueError(f"codebooks must be {s.codebook_dtype} storage, got {cb.dtype}")
        codes = np.asarray(inputs["codes"])
        if codes.shape != (s.C_out, s.K // s.g, s.M):
            raise ValueError(f"codes must have shape {(s.C_out, s.K // s.g, s.M)}, got {codes.shape}")
        if not np.issubdtype(codes.dtype, np.integer):
            raise ValueError(f"codes must be integers, got {codes.dtype}")
        if codes.size and (int(codes.min()) < 0 or int(codes.max()) >= (1 << s.B)):
            raise ValueError(f"codes must lie in [0, 2^{s.B})")
        codes = codes.astype(np.uint8 if s.B <= 8 else np.uint16, copy=False)
        scales = np.asarray(inputs["scales"])
        if scales.shape != (s.C_out,):
            raise ValueError(f"scales must have shape {(s.C_out,)}, got {scales.shape}")
        self.desc = make_desc(s.C_out, s.K, s.codebook_dtype, s.x_dtype, s.y_dtype, s.tile_dtype, mt, s.conv)
        import torch
        self.device = torch.cuda.current_device() if torch.cuda.is_available() else None
        self.handle = aq_layer_create(self.desc, cb, codes, scales, s.g, s.M, s.B)

    def out_shape(self, n: int):
        s = self.spec
        if s.conv is None:
            return (n, s.C_out)
        return (n, s.C_out, s.conv.OH, s.conv.OW)

    def in_shape(self, n: int):
        s = self.spec
        if s.conv is None:
            return (n, s.K)
        return (n, s.conv.cin, s.conv.H, s.conv.W)

    def tokens(self, n: int) -> int:
        s = self.spec
        return n if s.conv is None else n * s.conv.OH * s.conv.OW

    def forward(self, x, x_scales=None, out=None, stream=None, static=False):
        """Y for device tensor ``x`` (token-major [n, K] or NCHW); returns ``out``.

        ``static=True`` calls the allocation-free entry point (scratch in the
        library's static device array instead of the layer's workspace)."""
        import torch
        s = self.spec
        if not isinstance(x, torch.Tensor) or x.dim() < 1 or x.shape[0] < 1:
            raise ValueError("x must be a torch tensor with at least one row or image")
        n = x.shape[0]
        _check_tensor("x", x, _torch_dtypes(s.x_dtype), self.in_shape(n), self.device)
        if s.x_dtype == "i8":
            if x_scales is None:
                raise ValueError("int8 activations need x_scales")
            _check_tensor("x_scales", x_scales, (torch.float32,), (self.tokens(n),), self.device)
        elif x_scales is not None:
            raise ValueError("x_scales apply to int8 activations only")
        if out is None:
            out = torch.empty(self.out_shape(n), dtype=_torch_dtype(s.y_dtype), device=x.device)
        _check_tensor("out", out, _torch_dtypes(s.y_dtype), self.out_shape(n), self.device)
        st = stream if stream is not None else torch.cuda.current_stream(x.device).cuda_stream
        xs = 0 if x_scales is None else x_scales.data_ptr()
        (aq_layer_forward_static if static else aq_layer_forward)(self.handle, x.data_ptr(), xs, out.data_ptr(), n, st)
        return out

    __call__ = forward

    def prepare(self, n=None, stream=None):
        """Decode the weight records of the next forward over ``n`` tokens or
        images (default: the spec's n) on ``stream`` (a raw stream handle;
        default: the current stream), ahead of that forward; see
        ``aq_layer_prepare`` for the ordering the caller owes."""
        import torch
        n = self.spec.n if n is None else n
        if not isinstance(n, int) or n < 1:
            raise ValueError("n must be a positive int")
        st = stream if stream is not None else torch.cuda.current_stream(self.device).cuda_stream
        aq_layer_prepare(self.handle, n, st)

    @staticmethod
    def prepare_all(layers, ns=None, stream=None):
        """``prepare`` for every layer of ``layers`` (each at its ``ns`` entry;
        default: its spec's n) through one ``aq_layers_prepare`` call, which
        decodes the records of layers sharing a records kernel in one launch."""
        import torch
        layers = list(layers)
        ns = [lay.spec.n for lay in layers] if ns is None else list(ns)
        if len(ns) != len(layers) or any(not isinstance(n, int) or n < 1 for n in ns):
            raise ValueError("one positive int n per layer")
        if not layers:
            return
        dev = layers[0].device
        if any(lay.device != dev for lay in layers):
            raise ValueError("layers on different devices")
        st = stream if stream is not None else torch.cuda.current_stream(dev).cuda_stream
        aq_layers_prepare([lay.handle for lay in layers], ns, st)

    def decode(self, out=None, stream=None):
        import torch
        s = self.spec
        dts = {"f32": (torch.float32,), "f16": (torch.float16,), "bf16": (torch.int16, torch.bfloat16)}[s.tile_dtype]
        if out is None:
            out = torch.empty((s.C_out, s.K), dtype=dts[0], device=f"cuda:{self.device}")
        _check_tensor("out", out, dts, (s.C_out, s.K), self.device)
        st = stream if stream is not None else torch.cuda.current_stream().cuda_stream
        aq_layer_decode(self.handle, out.data_ptr(), st)
        return out

    def codebook_grad(self, x, dy, out=None, stream=None):
        """dC [M, 2**B, g] fp32 for input ``x`` and output gradient ``dy`` (both fp16 or bf16 device tensors)."""
        import torch
        s = self.spec
        if not isinstance(x, torch.Tensor) or not isinstance(dy, torch.Tensor):
            raise ValueError("x and dy must be torch tensors")
        if x.dtype != dy.dtype or x.dtype not in (torch.float16, torch.bfloat16):
            raise ValueError("x and dy must share one dtype, float16 or bfloat16")
        if x.dim() < 1 or x.shape[0] < 1:
            raise ValueError("x must have at least one row or image")
        n = x.shape[0]
        _check_tensor("x", x, (x.dtype,), self.in_shape(n), self.device)
        _check_tensor("dy", dy, (x.dtype,), self.out_shape(n), self.device)
        if out is None:
            out = torch.empty((s.M, 1 << s.B, s.g), dtype=torch.float32, device=x.device)
        _check_tensor("out", out, (torch.float32,), (s.M, 1 << s.B, s.g), self.device)
        st = stream if stream is not None else torch.cuda.current_stream(x.device).cuda_stream
        dt = "f16" if x.dtype == torch.float16 else "bf16"
        aq_layer_codebook_grad(self.handle, x.data_ptr(), dy.data_ptr(), dt, out.data_ptr(), n, st)
        return out

    def set_path(self, path: str) -> None:
        aq_layer_set_path(self.handle, path)

    def set_option(self, name: str, value) -> None:
        """Set an ``aq_option`` by name; tile options also take ``"BMxBN"`` strings."""
        if name not in OPTION_CODES:
            raise ValueError(f"unknown option {name!r}; known: {sorted(OPTION_CODES)}")
        if name in _TILE_OPTIONS and isinstance(value, str):
            bm, bn = (int(v) for v in value.split("x"))
            value = bm * 1000 + bn
        aq_layer_set_option(self.handle, OPTION_CODES[name], int(value))

    def get_option(self, name: str) -> int:
        return aq_layer_get_option(self.handle, OPTION_CODES[name])

    def choose_path(self, tokens: int) -> str:
        return aq_layer_choose_path(self.handle, tokens)

    def set_launch_events(self, events) -> None:
        """torch.cuda.Event objects (timing enabled, recorded once so they exist) or raw handles."""
        hs = [e if isinstance(e, int) else e.cuda_event for e in events]
        if any(h == 0 for h in hs):
            raise ValueError("events must exist: record each torch.cuda.Event once first")
        aq_layer_set_launch_events(self.handle, hs)

    def last_launches(self):
        return aq_layer_last_launches(self.handle)

    def describe(self, n: int) -> dict:
        return aq_layer_describe(self.handle, n)

    def close(self) -> None:
        if getattr(self, "handle", None):
            aq_layer_destroy(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass
