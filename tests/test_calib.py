"""The HBM calibration kernels the benchmark's ceiling figures come from
(libema_calib.so): exported entry points and argument checks on the CPU; on
the GPU, the copy is exact and the read folds every byte it was given."""
import ctypes
import os

import numpy as np
import pytest

LIB = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))),
                   "paper_2609_27040_amd", "lib", "libema_calib.so")
pytestmark = pytest.mark.skipif(not os.path.exists(LIB), reason="calibration library not built")


def lib():
    c = ctypes.CDLL(LIB)
    c.ema_calib_read.argtypes = [ctypes.c_void_p, ctypes.c_size_t, ctypes.c_void_p, ctypes.c_void_p]
    c.ema_calib_copy.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_size_t, ctypes.c_void_p]
    return c


def test_bad_arguments_are_refused_before_any_launch():
    c = lib()
    assert c.ema_calib_read(None, 65536, None, None) == -1
    assert c.ema_calib_read(ctypes.c_void_p(16), 4096, ctypes.c_void_p(16), None) == -1
    assert c.ema_calib_copy(ctypes.c_void_p(16), None, 16384, None) == -1
    assert c.ema_calib_copy(ctypes.c_void_p(16), ctypes.c_void_p(16), 0, None) == -1


@pytest.mark.gpu
def test_copy_is_exact_and_read_folds_every_word():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    print("calibration kernels, 8 MiB", flush=True)
    c = lib()
    rng = np.random.default_rng(5)
    host = rng.integers(0, 2 ** 32, size=(8 << 20) // 4, dtype=np.uint32)
    x = torch.from_numpy(host.view(np.int32)).cuda()
    y = torch.zeros_like(x)
    sink = torch.zeros((8 << 20) // 4096, dtype=torch.int32, device="cuda")
    s = torch.cuda.current_stream().cuda_stream
    assert c.ema_calib_copy(x.data_ptr(), y.data_ptr(), 8 << 20, s) == 0
    assert c.ema_calib_read(x.data_ptr(), 8 << 20, sink.data_ptr(), s) == 0
    torch.cuda.synchronize()
    assert torch.equal(x, y)
    # word c is the XOR of the 1024 words of 4 KiB chunk c
    want = np.bitwise_xor.reduce(host.reshape(-1, 1024), axis=1)
    assert np.array_equal(sink.cpu().numpy().view(np.uint32), want)
