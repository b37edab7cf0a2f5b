"""GPU: dlfp_linear_bf16 (the projections of the full-iteration proxy) against the oracle.

Shapes are the projections of a Qwen3-0.6B layer (hidden 1024, 16 x 128 query
and 8 x 128 key/value features, MLP 3072) at token counts from 1 to a
2048-token chunk beside 32 decoders, including counts that leave a ragged last
tile, a strided input (the MLP's down projection reads the first half of the
gate/up output rows) and a strided output.  Inputs N(0,1) bf16, weights
N(0,1)/sqrt(k) bf16.  Bars: fp32 output max |err| <= 5e-4 (fp32 accumulation
over k <= 3072 terms of O(1) partial sums); bf16 output within half a bf16
step of the exact value plus 5e-4.
"""
import math

import numpy as np
import pytest
import torch

from oracle import attention as oa
from oracle import linear as ol
from paper_2609_38386_amd import dlfp as D

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def dev():
    assert torch.cuda.is_available()
    D.lib()
    return torch.device("cuda:0")


def _bits64(t):
    return oa.bf16_bits_to_float64_tensor(t.view(torch.int16).cpu()).numpy()


SHAPES = [(2048, 1024), (1024, 1024), (1024, 2048), (6144, 1024)]


@pytest.mark.parametrize("m", [1, 37, 128, 300, 2080])
@pytest.mark.parametrize("n,k", SHAPES)
def test_linear_parity(dev, m, n, k):
    g = torch.Generator(device=dev)
    g.manual_seed(m * 7 + n + k)
    x = torch.empty((m, k), dtype=torch.bfloat16, device=dev).normal_(generator=g)
    w = (torch.empty((n, k), dtype=torch.float32, device=dev).normal_(generator=g)
         / math.sqrt(k)).to(torch.bfloat16)
    want = ol.linear(_bits64(x), _bits64(w))
    out32 = torch.full((m, n), float("nan"), dtype=torch.float32, device=dev)
    D.dlfp_linear_bf16(x, w, out32)
    out16 = torch.full((m, n), float("nan"), dtype=torch.bfloat16, device=dev)
    D.dlfp_linear_bf16(x, w, out16)
    torch.cuda.synchronize()
    got32 = out32.cpu().numpy().astype(np.float64)
    assert np.isfinite(got32).all()
    assert np.abs(got32 - want).max() <= 5e-4, np.abs(got32 - want).max()
    got16 = _bits64(out16)
    assert np.all(np.abs(got16 - want) <= np.abs(want) * 2.0 ** -8 + 5e-4)


def test_linear_strided_input_and_output(dev):
    """The down projection reads the first 3072 of 6144 features per row and
    writes into rows of a wider buffer."""
    g = torch.Generator(device=dev)
    g.manual_seed(9)
    m, k, n = 261, 3072, 1024
    gu = torch.empty((m, 6144), dtype=torch.bfloat16, device=dev).normal_(generator=g)
    w = (torch.empty((n, k), dtype=torch.float32, device=dev).normal_(generator=g)
         / math.sqrt(k)).to(torch.bfloat16)
    big = torch.full((m, 1536), float("nan"), dtype=torch.float32, device=dev)
    D.dlfp_linear_bf16(gu[:, :k], w, big[:, 256:256 + n])
    torch.cuda.synchronize()
    want = ol.linear(_bits64(gu[:, :k].contiguous()), _bits64(w))
    got = big.cpu().numpy().astype(np.float64)
    assert np.abs(got[:, 256:256 + n] - want).max() <= 5e-4
    assert np.isnan(got[:, :256]).all() and np.isnan(got[:, 256 + n:]).all()


def test_linear_rejects_unsupported_shapes(dev):
    x = torch.zeros((4, 64), dtype=torch.bfloat16, device=dev)
    with pytest.raises(D.DlfpError) as e:
        D.dlfp_linear_bf16(x, torch.zeros((100, 64), dtype=torch.bfloat16, device=dev),
                           torch.zeros((4, 100), dtype=torch.float32, device=dev))
    assert e.value.status == -5
    empty = torch.zeros((0, 64), dtype=torch.bfloat16, device=dev)
    D.dlfp_linear_bf16(empty, torch.zeros((128, 64), dtype=torch.bfloat16, device=dev),
                       torch.zeros((0, 128), dtype=torch.float32, device=dev))
