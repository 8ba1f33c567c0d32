"""The benchmark's streaming copies (libgrpo_bench.so): every variant copies a buffer exactly, including a tail that
fills no whole workgroup.  The row pass's copy ceiling is only meaningful if these copies move every byte."""
import ctypes

import pytest
import torch

pytestmark = pytest.mark.gpu


def _lib():
    from paper_2606_05597_amd.build import BENCH_SO
    lib = ctypes.CDLL(BENCH_SO)
    lib.stream_copy.argtypes = [ctypes.c_int, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int64, ctypes.c_void_p]
    lib.stream_copy.restype = ctypes.c_int
    lib.stream_copy_name.argtypes = [ctypes.c_int]
    lib.stream_copy_name.restype = ctypes.c_char_p
    return lib


@pytest.mark.parametrize("n_vec", [1, 1000, (1 << 22) + 12345])
def test_every_variant_copies_exactly(n_vec):
    lib = _lib()
    g = torch.Generator(device="cuda").manual_seed(n_vec)
    src = torch.randint(0, 1 << 30, (n_vec * 4,), dtype=torch.int32, device="cuda", generator=g)
    stream = torch.cuda.current_stream()
    for v in range(lib.stream_copy_variants()):
        dst = torch.full((n_vec * 4 + 4,), -7, dtype=torch.int32, device="cuda")
        rc = lib.stream_copy(v, src.data_ptr(), dst.data_ptr(), n_vec, ctypes.c_void_p(stream.cuda_stream))
        assert rc == 0, (v, rc)
        torch.cuda.synchronize()
        assert torch.equal(dst[:n_vec * 4], src), lib.stream_copy_name(v)
        assert (dst[n_vec * 4:] == -7).all(), lib.stream_copy_name(v)  # nothing written past the end


def test_bad_arguments_are_refused():
    lib = _lib()
    stream = ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
    buf = torch.empty(64, dtype=torch.int32, device="cuda")
    assert lib.stream_copy(lib.stream_copy_variants(), buf.data_ptr(), buf.data_ptr(), 1, stream) == -1
    assert lib.stream_copy(0, buf.data_ptr() + 4, buf.data_ptr(), 1, stream) == -1  # misaligned
    assert lib.stream_copy(0, buf.data_ptr(), buf.data_ptr(), -1, stream) == -1
    assert lib.stream_copy(0, buf.data_ptr(), buf.data_ptr(), 0, stream) == 0
