"""GPU parity: min-max quantization sender and receiver (Sec. 2.2) against the
CPU oracle: packed code bytes and (lo, scale) bit for bit, reconstruction bit
for bit, for every bit width 1..8 and 32, group lengths with ragged words and
tails, groups spread over several workgroups, and constant groups.  Both
receiver forms run: 16-byte output pieces (b = 2, 4, 8, 32 and groups of
whole pieces) and per-thread runs (everything else)."""
import numpy as np
import pytest
import torch

from gpu_helpers import DTN, TORCH, assert_bits_equal, raw
from paper_2401_07788_amd import workloads as W

pytestmark = pytest.mark.gpu


def run_case(tc, orc, x, n_grp, G, b):
    dt = DTN[x.dtype]
    xd = x.cuda()
    codes, meta = tc.quant_pack(xd, b, n_grp)
    y = tc.quant_unpack(codes, meta, G, b, out_dtype=x.dtype)
    torch.cuda.synchronize()
    assert tc.device_errors() == 0
    oc, om = orc.quant_pack(raw(x), dt, n_grp, G, b)
    assert_bits_equal(raw(codes), oc, "codes")
    assert_bits_equal(raw(meta), om, "meta")
    oy = orc.quant_unpack(oc, om, n_grp, G, b, dt)
    assert_bits_equal(raw(y), oy, "dense")


@pytest.mark.parametrize("b", [1, 2, 3, 4, 5, 6, 7, 8, 32])
@pytest.mark.parametrize("G", [1, 31, 768, 1000, 2048, 2049, 40000])
def test_quant_parity_f32(tc, orc, b, G):
    n_grp = 3
    x = (W.randn((n_grp, G), seed=G, tensor_id=b) * torch.tensor([[1e-3], [1.0], [30.0]])).contiguous()
    run_case(tc, orc, x, n_grp, G, b)


@pytest.mark.parametrize("dt", ["bf16", "f16"])
@pytest.mark.parametrize("b", [2, 4, 6, 8, 32])
@pytest.mark.parametrize("G", [36, 768, 1000, 32768])
def test_quant_parity_half(tc, orc, dt, b, G):
    n_grp = 4
    x = W.randn((n_grp, G), seed=3, tensor_id=b).to(TORCH[dt])
    run_case(tc, orc, x, n_grp, G, b)


def test_quant_constant_and_relu_groups(tc, orc):
    x = torch.relu(W.randn((4, 32768), seed=1, tensor_id=2))
    x[1] = 2.5
    x[2] = -0.0
    run_case(tc, orc, x.contiguous(), 4, 32768, 4)


@pytest.mark.parametrize("b", [2, 8])
def test_quant_receiver_grid_stride(tc, orc, b):
    # more 16-byte pieces than the receiver's grid holds threads: each thread
    # takes several pieces
    n_grp, G = 40, 131072
    x = W.randn((n_grp, G), seed=9, tensor_id=b)
    run_case(tc, orc, x, n_grp, G, b)


@pytest.mark.parametrize("b", [2, 4, 8])
@pytest.mark.parametrize("R", [1.0, 1.7, 3.0e-3, 6.5e4])
def test_quant_codes_at_rounding_ties(tc, orc, b, R):
    # values whose scaled position (v - lo) / (hi - lo) * (2^b - 1) lies on,
    # or a few ulps either side of, a half-integer: the code there depends on
    # every rounding of the quotient
    LV = (1 << b) - 1
    G = 8192
    half = (np.arange(G, dtype=np.float64) % LV + 0.5) * (np.float32(R) / LV)
    v = half.astype(np.float32)
    steps = (np.arange(G) % 7) - 3
    for _ in range(3):
        up, dn = steps > 0, steps < 0
        v[up] = np.nextafter(v[up], np.float32(np.inf))
        v[dn] = np.nextafter(v[dn], np.float32(-np.inf))
        steps = steps - np.sign(steps)
    v[0], v[1] = 0.0, np.float32(R)
    x = torch.from_numpy(np.stack([v, v[::-1].copy()]))
    run_case(tc, orc, x, 2, G, b)
