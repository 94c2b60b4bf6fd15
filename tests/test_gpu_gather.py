"""GPU parity: TopK at given indices (Sec. 3.2: gradients compressed at the
indices the activations' TopK kept), alone and inside error feedback
(Sec. 2.4), against the CPU oracle bit for bit: sent values, the residual
over several steps, the receiver's dense tensor; with and without the
forward payload's block table; ragged sizes, k edges and out-of-range
indices (flagged, no fault)."""
import numpy as np
import pytest
import torch

from gpu_helpers import DTN, assert_bits_equal, raw
from paper_2401_07788_amd import workloads as W

pytestmark = pytest.mark.gpu


def fwd_payload(tc, n_seg, L, k, dt, seed):
    a = W.randn((n_seg, L), seed, 1).to(dt).cuda()
    return tc.topk_compress(a, k, n_seg)


@pytest.mark.parametrize("dt", [torch.float32, torch.bfloat16, torch.float16])
@pytest.mark.parametrize("n_seg,L", [(4096, 768), (3, 50001), (5, 999)])
def test_gather_parity(tc, orc, dt, n_seg, L):
    k = tc.topk_count(L, 1, 10)
    pl = fwd_payload(tc, n_seg, L, k, dt, L)
    g = (1e-4 * W.randn((n_seg, L), L, 2)).to(dt)
    val = tc.topk_gather(pl, g.cuda())
    y = tc.topk_decompress(pl._replace(val=val), L)
    torch.cuda.synchronize()
    assert tc.device_errors() == 0
    idx = raw(pl.idx)
    ov = orc.topk_gather(raw(g), DTN[dt], idx, n_seg, L, k)
    assert_bits_equal(raw(val), ov, "val")
    assert_bits_equal(raw(y), orc.topk_decompress(idx, ov, DTN[dt], n_seg, L, k), "received")


@pytest.mark.parametrize("dt", [torch.float32, torch.bfloat16])
@pytest.mark.parametrize("n_seg,L", [(4096, 768), (5, 999), (9000, 37), (3, 50001), (2, 4096 * 3)])
@pytest.mark.parametrize("use_blk", [True, False])
def test_gather_ef_parity(tc, orc, dt, n_seg, L, use_blk):
    k = tc.topk_count(L, 1, 10)
    e_gpu = torch.zeros(n_seg * L, dtype=torch.float32, device="cuda")
    e_orc = np.zeros((n_seg, L), np.float32)
    for t in range(3):
        pl = fwd_payload(tc, n_seg, L, k, dt, 10 * t + L)
        g = (1e-4 * W.randn((n_seg, L), L, 3 + t)).to(dt)
        val = tc.topk_gather(pl, g.cuda(), e=e_gpu, use_blk=use_blk)
        torch.cuda.synchronize()
        assert tc.device_errors() == 0
        ov, e_orc = orc.topk_gather(raw(g), DTN[dt], raw(pl.idx), n_seg, L, k, e=e_orc)
        assert_bits_equal(raw(val), ov, f"val step {t}")
        assert_bits_equal(raw(e_gpu).reshape(n_seg, L), e_orc, f"e step {t}")


@pytest.mark.parametrize("n_seg,L", [(3, 5000), (70, 768)])
def test_gather_k_edges(tc, orc, n_seg, L):
    # the chunk kernel (5000) and the one-wavefront-per-row kernel (768)
    x = W.randn((n_seg, L), 9, 1)
    for k in (0, L):
        pl = fwd_payload(tc, n_seg, L, k, torch.float32, 9)
        e0 = W.randn((n_seg, L), 9, 2)
        e = e0.clone().cuda().reshape(-1)
        val = tc.topk_gather(pl, x.cuda(), e=e)
        torch.cuda.synchronize()
        assert tc.device_errors() == 0
        ov, oe = orc.topk_gather(raw(x), "f32", raw(pl.idx), n_seg, L, k, e=raw(e0))
        assert_bits_equal(raw(val), ov, f"val k={k}")
        assert_bits_equal(raw(e).reshape(n_seg, L), oe, f"e k={k}")


def test_gather_flags_bad_index_without_fault(tc):
    x = torch.arange(100, dtype=torch.float32, device="cuda").reshape(1, 100)
    idx = torch.tensor([[1, 5, 1 << 20]], dtype=torch.int32, device="cuda")
    pl = tc.TopkPayload(idx, None, None)
    tc.device_errors(clear=True)
    val = tc.topk_gather(pl, x)
    torch.cuda.synchronize()
    assert tc.device_errors(clear=True) & tc.TC_KERR_BAD_INDEX
    assert val.cpu().tolist() == [[1.0, 5.0, 0.0]]
    e = torch.zeros(100, dtype=torch.float32, device="cuda")
    tc.topk_gather(pl, x, e=e)
    torch.cuda.synchronize()
    assert tc.device_errors(clear=True) & tc.TC_KERR_BAD_INDEX
    ee = e.cpu()
    assert ee[1] == 0.0 and ee[5] == 0.0 and ee[2] == 2.0
