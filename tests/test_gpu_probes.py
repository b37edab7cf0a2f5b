"""The ceiling probes (libdlfp_probe.so) read what they claim: every wavefront's
per-lane XOR fold of its pieces equals the same fold computed with NumPy from
the buffer, with default caching and with non-temporal loads, at each depth of
pieces in flight; the MFMA probe is deterministic and finite.  Argument
errors are refused before any launch."""
import ctypes
import os

import numpy as np
import pytest
import torch

pytestmark = pytest.mark.gpu

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.fixture(scope="module")
def probe():
    assert torch.cuda.is_available(), "GPU tests need a HIP device"
    path = os.path.join(ROOT, "paper_2609_38386_amd", "libdlfp_probe.so")
    L = ctypes.CDLL(path)
    vp, i32, i64 = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64
    L.dlfp_probe_hbm_read.argtypes = [vp, i64, vp, i32, i32, i32, i32, i32, vp, vp]
    L.dlfp_probe_mfma.argtypes = [i32, i32, vp, vp]
    return L


def _fold(buf_u32, pieces, waves, per_wave, piece_bytes):
    """Lane l of wavefront w: XOR of the four words at byte r * 1024 + 16 l of
    every round r of every piece the wavefront reads."""
    rounds = piece_bytes // 1024
    p = buf_u32.reshape(-1, rounds, 64, 4)[pieces.reshape(waves, per_wave)]
    return np.bitwise_xor.reduce(p.reshape(waves, per_wave * rounds, 64, 4), axis=(1, 3))


@pytest.mark.parametrize("nt", [0, 1])
@pytest.mark.parametrize("inflight", [1, 2, 4])
@pytest.mark.parametrize("piece_bytes", [1024, 8192])
def test_hbm_probe_folds_exactly_the_pieces_it_reads(probe, nt, inflight, piece_bytes):
    dev = torch.device("cuda:0")
    rng = np.random.default_rng(7 + inflight + nt)
    buf_bytes = 4 << 20
    host = rng.integers(0, 2**32, size=buf_bytes // 4, dtype=np.uint64).astype(np.uint32)
    n_pieces = buf_bytes // piece_bytes
    waves, per_wave = 16, 7   # not a multiple of the depth: the last group is partial
    pieces = rng.integers(0, n_pieces, size=waves * per_wave).astype(np.int32)
    d_buf = torch.from_numpy(host.view(np.int32)).to(dev)
    d_pieces = torch.from_numpy(pieces).to(dev)
    sink = torch.zeros(waves * 64, dtype=torch.int32, device=dev)
    stream = ctypes.c_void_p(int(torch.cuda.current_stream().cuda_stream))
    st = probe.dlfp_probe_hbm_read(ctypes.c_void_p(d_buf.data_ptr()), buf_bytes,
                                   ctypes.c_void_p(d_pieces.data_ptr()), waves, per_wave,
                                   piece_bytes, inflight, nt, ctypes.c_void_p(sink.data_ptr()),
                                   stream)
    assert st == 0
    torch.cuda.synchronize()
    got = sink.cpu().numpy().view(np.uint32).reshape(waves, 64)
    assert np.array_equal(got, _fold(host, pieces, waves, per_wave, piece_bytes))


def test_hbm_probe_refuses_bad_arguments(probe):
    vp = ctypes.c_void_p
    dummy = vp(16)  # never dereferenced: every call below is refused first
    stream = vp(0)
    assert probe.dlfp_probe_hbm_read(dummy, 1 << 20, dummy, 6, 4, 8192, 1, 0, dummy, stream) == -1
    assert probe.dlfp_probe_hbm_read(dummy, 1 << 20, dummy, 8, 4, 8192, 3, 0, dummy, stream) == -1
    assert probe.dlfp_probe_hbm_read(dummy, 1 << 20, dummy, 8, 4, 8192, 1, 2, dummy, stream) == -1
    assert probe.dlfp_probe_hbm_read(dummy, 1 << 20, dummy, 8, 4, 1000, 1, 0, dummy, stream) == -1
    assert probe.dlfp_probe_hbm_read(None, 1 << 20, dummy, 8, 4, 8192, 1, 0, dummy, stream) == -1
    assert probe.dlfp_probe_mfma(0, 4, dummy, stream) == -1


def test_mfma_probe_is_deterministic_and_finite(probe):
    dev = torch.device("cuda:0")
    stream = ctypes.c_void_p(int(torch.cuda.current_stream().cuda_stream))
    outs = []
    for _ in range(2):
        sink = torch.full((8 * 256,), float("nan"), dtype=torch.float32, device=dev)
        assert probe.dlfp_probe_mfma(8, 64, ctypes.c_void_p(sink.data_ptr()), stream) == 0
        torch.cuda.synchronize()
        outs.append(sink.cpu())
    assert bool(torch.isfinite(outs[0]).all())
    assert torch.equal(outs[0], outs[1])
