"""GPU parity: EF-mixed (Sec. 2.4), half of the TopK budget on the input and
half on the error buffer, over several steps with the buffer carried on each
side: both lists bit for bit, the block tables, the receiver's dense tensor
(with and without block tables) and the binary32 buffer bit for bit.  The
full-size case is the CNN boundary the paper runs EF-mixed on: 128 samples of
32,768 post-ReLU fp32 activations, TopK 10 %, and the matching gradients."""
import numpy as np
import pytest
import torch

from gpu_helpers import DTN, TORCH, assert_bits_equal, check_block_table, raw
from paper_2401_07788_amd import workloads as W

pytestmark = pytest.mark.gpu


def efmix_steps(tc, orc, xs, n_seg, L, k, out_dt=None):
    dt = DTN[xs[0].dtype]
    out_dt = out_dt or dt
    e_gpu = torch.zeros(n_seg * L, dtype=torch.float32, device="cuda")
    e_orc = np.zeros((n_seg, L), np.float32)
    for t, x in enumerate(xs):
        px, pe = tc.efmix_step(x.cuda(), e_gpu, k, n_seg)
        y = tc.efmix_reconstruct(px, pe, L, out_dtype=TORCH[out_dt], use_blk=(t % 2 == 0))
        torch.cuda.synchronize()
        assert tc.device_errors() == 0
        ix, vx, ie, ve, e_orc = orc.efmix_send(raw(x), dt, e_orc, n_seg, L, k)
        assert_bits_equal(raw(px.idx), ix, f"idx_x step {t}")
        assert_bits_equal(raw(px.val), vx, f"val_x step {t}")
        assert_bits_equal(raw(pe.idx), ie, f"idx_e step {t}")
        assert_bits_equal(raw(pe.val), ve, f"val_e step {t}")
        check_block_table(px.blk, ix, L, f"blk_x step {t}")
        check_block_table(pe.blk, ie, L, f"blk_e step {t}")
        want = orc.efmix_recv(ix, vx, ie, ve, dt, n_seg, L, k, out_dt=out_dt)
        assert_bits_equal(raw(y), want, f"received step {t}")
        assert_bits_equal(raw(e_gpu).reshape(n_seg, L), e_orc, f"e step {t}")


def test_efmix_cnn_full(tc, orc):
    n_seg, L = 128, 32768
    k = tc.topk_count(L, 1, 10)
    acts = [W.relu_activation((n_seg, L), 31, t) for t in range(3)]
    efmix_steps(tc, orc, acts, n_seg, L, k)
    grads = [W.normal_gradient((n_seg, L), 1e-3, 31, 10 + t) for t in range(3)]
    efmix_steps(tc, orc, grads, n_seg, L, k)


@pytest.mark.parametrize("dt", ["f32", "bf16", "f16"])
@pytest.mark.parametrize("L", [1, 37, 1000, 4099, 16384, 32768])
def test_efmix_sizes(tc, orc, dt, L):
    # 4099 and 37: not a multiple of the 4-element pieces (element-wise path)
    xs = [W.randn((5, L), 9, t).to(TORCH[dt]) for t in range(3)]
    for num in (1, 3):
        efmix_steps(tc, orc, xs, 5, L, tc.topk_count(L, num, 10))


def test_efmix_wide_receiver(tc, orc):
    # bfloat16 wire, binary32 receiver: the sum at shared indices is not rounded
    xs = [W.transformer_hidden((4, 3072), 12, t) for t in range(3)]
    efmix_steps(tc, orc, xs, 4, 3072, tc.topk_count(3072, 1, 10), out_dt="f32")


@pytest.mark.parametrize("k", [0, 1, 2, 8191, 8192])
def test_efmix_k_edges(tc, orc, k):
    xs = [W.relu_activation((3, 8192), 13, t) for t in range(2)]
    efmix_steps(tc, orc, xs, 3, 8192, k)


def test_efmix_rejects_long_segments(tc):
    x = torch.zeros((1, 32769), dtype=torch.float32, device="cuda")
    e = torch.zeros_like(x)
    with pytest.raises(tc.TCError):
        tc.efmix_step(x, e, 100, 1)


def test_efmix_unaligned_buffers(tc, orc):
    # x and e start one element past a 16-byte boundary: element-wise loads
    # and stores throughout
    n_seg, L = 6, 8192
    k = tc.topk_count(L, 1, 10)
    xs = [W.relu_activation((n_seg, L), 14, t) for t in range(3)]
    xb = torch.empty(n_seg * L + 1, dtype=torch.float32, device="cuda")
    eb = torch.zeros(n_seg * L + 1, dtype=torch.float32, device="cuda")
    e_gpu = eb[1:]
    e_orc = np.zeros((n_seg, L), np.float32)
    for t, x in enumerate(xs):
        xb[1:] = x.reshape(-1).cuda()
        px, pe = tc.efmix_step(xb[1:].view(n_seg, L), e_gpu, k, n_seg)
        torch.cuda.synchronize()
        assert tc.device_errors() == 0
        ix, vx, ie, ve, e_orc = orc.efmix_send(raw(x), "f32", e_orc, n_seg, L, k)
        assert_bits_equal(raw(px.idx), ix, f"idx_x step {t}")
        assert_bits_equal(raw(pe.idx), ie, f"idx_e step {t}")
        assert_bits_equal(raw(pe.val), ve, f"val_e step {t}")
        assert_bits_equal(raw(e_gpu).reshape(n_seg, L), e_orc, f"e step {t}")


def test_efmix_more_segments_than_workgroups(tc, orc):
    # more segments than resident workgroups (one per compute unit): each
    # workgroup takes several segments in turn, LDS reused between them
    n_seg, L = 600, 3000
    k = tc.topk_count(L, 1, 10)
    xs = [W.randn((n_seg, L), 15, t) for t in range(2)]
    efmix_steps(tc, orc, xs, n_seg, L, k)
