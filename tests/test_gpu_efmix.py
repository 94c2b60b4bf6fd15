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


def _round_np(v, dt):
    """binary32 -> the wire dtype (RNE) -> binary32, with numpy alone"""
    v = np.asarray(v, np.float32)
    if dt == "f16":
        return v.astype(np.float16).astype(np.float32)
    b = v.view(np.uint32).astype(np.uint64)
    b = (b + 0x7FFF + ((b >> 16) & 1)) >> 16 << 16
    return b.astype(np.uint32).view(np.float32)


@pytest.mark.parametrize("dt", ["bf16", "f16"])
@pytest.mark.parametrize("L", [4000, 4099, 32768])
def test_efmix_shared_indices_conserve(tc, orc, dt, L):
    # multiples of 2^-6 below 2^9: every binary32 step is exact while the
    # wire keeps 8 (bf16) or 11 (f16) significant bits.  x is large where the
    # buffer is, so the two lists share indices whose sums fall off the wire
    # grid; with the receiver in the wire dtype, x + e == received + e' bit
    # for bit, on the GPU's own outputs and the oracle's alike
    rng = np.random.default_rng(L + (0 if dt == "bf16" else 1))
    n_seg = 3
    k = tc.topk_count(L, 2, 10)
    e_np = (rng.integers(-2 ** 12, 2 ** 12, (n_seg, L)) / 64.0).astype(np.float32)
    e_gpu = torch.from_numpy(e_np.copy()).reshape(-1).cuda()
    e_orc = e_np.copy()
    shared_off_grid = 0
    for t in range(3):
        x = _round_np((rng.integers(-2 ** 10, 2 ** 10, (n_seg, L)) / 64.0).astype(np.float32), dt)
        hot = np.argsort(-np.abs(e_orc), axis=1, kind="stable")[:, : k // 3]
        np.put_along_axis(x, hot, _round_np(np.take_along_axis(e_orc, hot, 1) * 0.75 + 3.0, dt), 1)
        xt = torch.from_numpy(x).to(TORCH[dt]).cuda()
        e_before = raw(e_gpu).reshape(n_seg, L).copy()
        px, pe = tc.efmix_step(xt, e_gpu, k, n_seg)
        y = tc.efmix_reconstruct(px, pe, L, out_dtype=TORCH[dt], use_blk=(t % 2 == 0))
        torch.cuda.synchronize()
        assert tc.device_errors() == 0
        ix, vx, ie, ve, e_orc = orc.efmix_send(raw(xt), dt, e_orc, n_seg, L, k)
        assert_bits_equal(raw(px.idx), ix, f"idx_x step {t}")
        assert_bits_equal(raw(pe.idx), ie, f"idx_e step {t}")
        assert_bits_equal(raw(px.val), vx, f"val_x step {t}")
        assert_bits_equal(raw(pe.val), ve, f"val_e step {t}")
        e_after = raw(e_gpu).reshape(n_seg, L)
        assert_bits_equal(e_after, e_orc, f"e step {t}")
        yf = y.float().cpu().numpy()
        lhs = (x + e_before).view(np.uint32)
        assert np.array_equal(lhs, (yf + e_after).view(np.uint32)), f"conservation step {t}"
        for s in range(n_seg):
            both = np.intersect1d(ix[s], ie[s])
            u = x[s, both] + _round_np(e_before[s, both], dt)
            shared_off_grid += int((_round_np(u, dt) != u).sum())
    assert shared_off_grid > 20
