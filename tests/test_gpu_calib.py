"""The benchmark's read-modify-write ceiling kernel (libzo_calib.so) on the GPU: in every launch
shape it XORs each 32-bit word of the buffer with the key exactly once (full row groups, a
ragged tail of edge tiles, buffers smaller than one row group), and a second call restores
the buffer. A ceiling that skipped or repeated memory would misstate the bound the sweeps are
compared with."""

import ctypes
import os

import pytest
import torch

import paper_2609_38095_amd as zo

pytestmark = pytest.mark.gpu
DEV = "cuda:0"
KEY = 0x5A5A5A5A


@pytest.fixture(scope="module")
def calib():
    zo.library()  # loads libzo.so (and fails loudly without it)
    lib = ctypes.CDLL(os.path.join(os.path.dirname(zo.LIB_PATH), "libzo_calib.so"))
    lib.zo_calib_rmw_shape.argtypes = [ctypes.c_void_p, ctypes.c_uint64, ctypes.c_uint32, ctypes.c_uint32,
                                       ctypes.c_void_p]
    return lib


@pytest.mark.parametrize("nbytes", [48, 4096 + 16, 300 * 2 ** 20 + 2048 * 7 + 48])
@pytest.mark.parametrize("shape", range(8))
def test_ceiling_xors_every_word_once(calib, nbytes, shape):
    print(f"calib shape {shape} bytes {nbytes}", flush=True)
    gen = torch.Generator(device=DEV)
    gen.manual_seed(nbytes + shape)
    src = torch.randint(-2 ** 31, 2 ** 31 - 1, (nbytes // 4,), dtype=torch.int32, device=DEV, generator=gen)
    buf = src.clone()
    stream = torch.cuda.current_stream().cuda_stream
    assert calib.zo_calib_rmw_shape(ctypes.c_void_p(buf.data_ptr()), nbytes, KEY, shape, ctypes.c_void_p(stream)) == 0
    torch.cuda.synchronize()
    assert torch.equal(buf, torch.bitwise_xor(src, KEY))
    assert calib.zo_calib_rmw_shape(ctypes.c_void_p(buf.data_ptr()), nbytes, KEY, shape, ctypes.c_void_p(stream)) == 0
    torch.cuda.synchronize()
    assert torch.equal(buf, src)
