"""Host-side checks of the Python binding's argument validation and of the
option entry points.

The C ABI receives bare pointers and cannot see buffer extents, so the
binding checks dtype, exact shape, contiguity and device of every tensor
before it calls the library.  Nothing here needs a GPU: invalid arguments
are rejected before any device call.
"""
import ctypes
import glob
import os

import numpy as np
import pytest
import torch

from paper_2506_05960_amd import aq as A
from workloads import ConvGeom, LayerSpec, generate

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))

LIN = LayerSpec(name="v_lin", C_out=24, K=32, g=8, M=2, B=8, n=5)
LIN_I8 = LayerSpec(name="v_i8", C_out=24, K=32, g=8, M=2, B=8, n=5, x_dtype="i8")
CONV = LayerSpec(name="v_conv", C_out=16, K=8 * 9, g=8, M=2, B=8, n=2, conv=ConvGeom(8, 3, 3, 1, 1, 6, 4))


def _shell(spec):
    """An AQLayer that never reached the library (validation runs before any call)."""
    obj = object.__new__(A.AQLayer)
    obj.spec = spec
    obj.device = None
    obj.handle = None
    return obj


@pytest.fixture
def host_tensors(monkeypatch):
    """Host tensors stand in for device tensors, so each check after the device one is reached."""
    monkeypatch.setattr(A, "_DEVICE_TYPE", "cpu")


def _good(spec):
    inp = generate(spec, 1)
    return {"codebooks": inp["codebooks"], "codes": inp["codes"], "scales": inp["scales"]}


@pytest.mark.parametrize("key, value, text", [
    ("codebooks", np.zeros((2, 256, 4), np.float16), "codebooks must have shape"),
    ("codebooks", np.zeros((2, 256, 8), np.float32), "codebooks must be f16"),
    ("codes", np.zeros((24, 4, 3), np.uint8), "codes must have shape"),
    ("codes", np.zeros((24, 4, 2), np.float32), "codes must be integers"),
    ("codes", np.full((24, 4, 2), 256, np.int32), "codes must lie in"),
    ("codes", np.full((24, 4, 2), -1, np.int32), "codes must lie in"),
    ("scales", np.ones(23, np.float32), "scales must have shape"),
])
def test_create_rejects_bad_host_arrays(key, value, text):
    inp = _good(LIN)
    inp[key] = value
    with pytest.raises(ValueError, match=text):
        A.AQLayer(LIN, inp)


def _x(spec, n, dtype=torch.float16):
    shape = (n, spec.K) if spec.conv is None else (n, spec.conv.cin, spec.conv.H, spec.conv.W)
    return torch.zeros(shape, dtype=dtype)


@pytest.mark.parametrize("spec", [LIN, CONV], ids=lambda s: s.name)
def test_forward_rejects_bad_input(spec, host_tensors):
    lay = _shell(spec)
    with pytest.raises(ValueError, match="dtype"):
        lay.forward(_x(spec, 3, torch.float32))
    bad_shape = torch.zeros((3, spec.K + 8), dtype=torch.float16) if spec.conv is None else \
        torch.zeros((3, spec.conv.cin, spec.conv.H + 1, spec.conv.W), dtype=torch.float16)
    with pytest.raises(ValueError, match="shape"):
        lay.forward(bad_shape)
    nc = _x(spec, 3)
    nc = torch.cat([nc, nc], dim=-1)[..., ::2]
    with pytest.raises(ValueError, match="contiguous"):
        lay.forward(nc)
    with pytest.raises(ValueError):
        lay.forward(torch.zeros((0,) + tuple(_x(spec, 1).shape[1:]), dtype=torch.float16))
    with pytest.raises(ValueError, match="int8"):
        lay.forward(_x(spec, 3), x_scales=torch.ones(3))
    yshape = (3, spec.C_out) if spec.conv is None else (3, spec.C_out, spec.conv.OH, spec.conv.OW)
    with pytest.raises(ValueError, match="out must have dtype"):
        lay.forward(_x(spec, 3), out=torch.zeros(yshape, dtype=torch.float32))
    with pytest.raises(ValueError, match="out must have shape"):
        lay.forward(_x(spec, 3), out=torch.zeros((4,) + yshape[1:], dtype=torch.float16))


@pytest.mark.parametrize("spec", [LIN, CONV], ids=lambda s: s.name)
def test_forward_rejects_host_tensors(spec):
    lay = _shell(spec)
    with pytest.raises(ValueError, match="must be on cuda"):
        lay.forward(_x(spec, 3))                          # right dtype and shape, on the host


def test_forward_rejects_bad_int8_scales(host_tensors):
    lay = _shell(LIN_I8)
    x = torch.zeros((5, 32), dtype=torch.int8)
    with pytest.raises(ValueError, match="need x_scales"):
        lay.forward(x)
    with pytest.raises(ValueError, match="x_scales must have shape"):
        lay.forward(x, x_scales=torch.ones(4))
    with pytest.raises(ValueError, match="x_scales must have dtype"):
        lay.forward(x, x_scales=torch.ones(5, dtype=torch.float64))


def test_codebook_grad_rejects_bad_arguments(host_tensors):
    lay = _shell(LIN)
    x = torch.zeros((5, 32), dtype=torch.float16)
    with pytest.raises(ValueError, match="share one dtype"):
        lay.codebook_grad(x, torch.zeros((5, 24), dtype=torch.bfloat16))
    with pytest.raises(ValueError, match="share one dtype"):
        lay.codebook_grad(x.float(), torch.zeros((5, 24)))
    with pytest.raises(ValueError, match="dy must have shape"):
        lay.codebook_grad(x, torch.zeros((5, 23), dtype=torch.float16))
    with pytest.raises(ValueError, match="x must have shape"):
        lay.codebook_grad(torch.zeros((5, 31), dtype=torch.float16), torch.zeros((5, 24), dtype=torch.float16))
    with pytest.raises(ValueError, match="out must have shape"):
        lay.codebook_grad(x, torch.zeros((5, 24), dtype=torch.float16), out=torch.zeros((2, 256, 4)))


def test_decode_rejects_bad_output(host_tensors):
    lay = _shell(LIN)
    with pytest.raises(ValueError, match="out must have shape"):
        lay.decode(out=torch.zeros((24, 31), dtype=torch.float16))
    with pytest.raises(ValueError, match="out must have dtype"):
        lay.decode(out=torch.zeros((24, 32), dtype=torch.float32))


def test_option_names_and_null_layer():
    lay = _shell(LIN)
    with pytest.raises(ValueError, match="unknown option"):
        lay.set_option("no_such_option", 1)
    lib = A.load_library()
    assert lib.aq_layer_set_option(None, A.OPTION_CODES["weights"], 1) == A.AQ_ERR_INVALID_ARGUMENT
    v = ctypes.c_int64()
    assert lib.aq_layer_get_option(None, A.OPTION_CODES["weights"], ctypes.byref(v)) == A.AQ_ERR_INVALID_ARGUMENT
    with pytest.raises(A.AQError):
        lay.set_option("fused_tile", "64x96")      # parsed, then rejected by the library (no layer)


def test_option_codes_match_the_header():
    src = open(os.path.join(ROOT, "include", "aq.h")).read()
    import re
    enum = dict((k.lower(), int(v)) for k, v in re.findall(r"AQ_OPT_([A-Z_]+)\s*=\s*(\d+)", src))
    assert enum == A.OPTION_CODES


def test_library_reads_no_environment():
    # route choices are per-layer options of the C ABI, never environment variables
    for f in glob.glob(os.path.join(ROOT, "paper_2506_05960_amd", "csrc", "*")):
        assert "getenv" not in open(f).read(), f
