"""GPU: the in-process boundary module (Sec. 2.1) against the CPU oracle: the
forward output is the TopK receiver's tensor, the input gradient the
receiver's tensor of the gradient's message (at the activation's indices,
Sec. 3.2, or through its own TopK), with and without error feedback, bit for
bit over two steps; and a small model trains through it."""
import numpy as np
import pytest
import torch

from gpu_helpers import assert_bits_equal, raw
from paper_2401_07788_amd import boundary
from paper_2401_07788_amd import workloads as W

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("ef", [False, True])
@pytest.mark.parametrize("reuse", [True, False])
def test_boundary_matches_oracle(tc, orc, ef, reuse):
    n_seg, L = 6, 3000
    k = tc.topk_count(L, 1, 10)
    mod = boundary.TopkBoundary(1, 10, ef=ef, reuse_indices=reuse)
    e_f = np.zeros((n_seg, L), np.float32)
    e_b = np.zeros((n_seg, L), np.float32)
    for t in range(2):
        x = W.randn((n_seg, L), 21, t)
        gy = W.randn((n_seg, L), 22, t)
        xd = x.cuda().requires_grad_(True)
        y = mod(xd)
        y.backward(gy.cuda())
        torch.cuda.synchronize()
        assert tc.device_errors() == 0
        if ef:
            oi, ov, e_f = orc.ef_topk(raw(x), "f32", e_f, n_seg, L, k)
        else:
            oi, ov = orc.topk_compress(raw(x), "f32", n_seg, L, k)
        assert_bits_equal(raw(y.detach()), orc.topk_decompress(oi, ov, "f32", n_seg, L, k), f"forward step {t}")
        if reuse:
            if ef:
                gv, e_b = orc.topk_gather(raw(gy), "f32", oi, n_seg, L, k, e=e_b)
            else:
                gv = orc.topk_gather(raw(gy), "f32", oi, n_seg, L, k)
            gi = oi
        elif ef:
            gi, gv, e_b = orc.ef_topk(raw(gy), "f32", e_b, n_seg, L, k)
        else:
            gi, gv = orc.topk_compress(raw(gy), "f32", n_seg, L, k)
        assert_bits_equal(raw(xd.grad), orc.topk_decompress(gi, gv, "f32", n_seg, L, k), f"gradient step {t}")


def test_boundary_trains_a_small_model(tc):
    torch.manual_seed(0)
    net = torch.nn.Sequential(torch.nn.Linear(64, 256), torch.nn.ReLU(), boundary.TopkBoundary(3, 10, ef=True),
                              torch.nn.Linear(256, 10)).cuda()
    opt = torch.optim.SGD(net.parameters(), lr=0.1)
    xb = torch.randn(128, 64, device="cuda")
    yb = (xb[:, :10] > 0).float().argmax(dim=1)
    losses = []
    for _ in range(60):
        opt.zero_grad()
        loss = torch.nn.functional.cross_entropy(net(xb), yb)
        loss.backward()
        opt.step()
        losses.append(loss.item())
    torch.cuda.synchronize()
    assert tc.device_errors() == 0
    assert np.isfinite(losses).all() and losses[-1] < losses[0]
