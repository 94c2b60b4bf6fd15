"""GPU parity: TopK sender and receiver (Sec. 2.3) against the CPU oracle,
bit for bit (indices, kept values, dense reconstruction), over both kernel
layouts (one wavefront per short segment; several workgroups per long
segment), ragged tails, tie-heavy data and the k = 0 / k = seg_len edges."""
import numpy as np
import pytest
import torch

from gpu_helpers import DTN, TORCH, assert_bits_equal, check_block_table, raw
from paper_2401_07788_amd import workloads as W

pytestmark = pytest.mark.gpu


def make_input(kind, n_seg, L, dt, seed):
    z = W.randn((n_seg, L), seed, 11)
    if kind == "relu":
        z = torch.relu(z)
    elif kind == "ties":
        z = z.to(torch.bfloat16).to(torch.float32)
        g = torch.Generator().manual_seed(seed)
        u = torch.rand((n_seg, L), generator=g)
        z[u < 0.3] = 0.0
        z[(u >= 0.3) & (u < 0.4)] = -0.0
    elif kind == "const":
        z = torch.full((n_seg, L), 1.5)
    elif kind == "zeros":
        z = torch.zeros((n_seg, L))
        z[:, ::3] = -0.0
    return z.to(TORCH[dt]).contiguous()


def run_case(tc, orc, x, n_seg, L, k):
    dt = DTN[x.dtype]
    xd = x.cuda()
    p = tc.topk_compress(xd, k, n_seg)
    y = tc.topk_decompress(p, L)
    y_search = tc.topk_decompress(p, L, use_blk=False)
    torch.cuda.synchronize()
    assert tc.device_errors() == 0
    oi, ov = orc.topk_compress(raw(x), dt, n_seg, L, k)
    assert_bits_equal(raw(p.idx), oi, "idx")
    assert_bits_equal(raw(p.val), ov, "val")
    check_block_table(p.blk, oi, L)
    oy = orc.topk_decompress(oi, ov, dt, n_seg, L, k)
    assert_bits_equal(raw(y), oy, "dense")
    assert_bits_equal(raw(y_search), oy, "dense (index search)")


ROW_L = [1, 7, 64, 768, 1000, 2048]
BIG_L = [2049, 16384, 50001]


@pytest.mark.parametrize("dt", ["f32", "bf16", "f16"])
@pytest.mark.parametrize("L", ROW_L + BIG_L)
@pytest.mark.parametrize("kind", ["normal", "ties"])
def test_topk_parity(tc, orc, dt, L, kind):
    n_seg = 3 if L > 2048 else 5
    x = make_input(kind, n_seg, L, dt, seed=L)
    for num, den in [(1, 10), (3, 10)]:
        run_case(tc, orc, x, n_seg, L, tc.topk_count(L, num, den))


@pytest.mark.parametrize("dt", ["f32", "f16"])
def test_topk_group_aligned_ragged_tail(tc, orc, dt):
    """8 segments of 394,016 elements (whole 16-byte runs, not whole chunks):
    the most runs per thread, 33 workgroups per segment, more segments than
    resident groups, and a last chunk whose later runs lie wholly past the
    segment's end"""
    n_seg, L = 8, 394016
    x = make_input("normal", n_seg, L, dt, seed=7)
    run_case(tc, orc, x, n_seg, L, tc.topk_count(L, 1, 10))


@pytest.mark.parametrize("L", [768, 16384, 50001])
@pytest.mark.parametrize("kind", ["relu", "ties", "const", "zeros"])
def test_topk_edges(tc, orc, L, kind):
    n_seg = 2
    x = make_input(kind, n_seg, L, "f32", seed=7)
    for k in sorted({0, 1, 2, L // 2, L - 1, L}):
        run_case(tc, orc, x, n_seg, L, k)


def test_topk_many_segments_row_layout(tc, orc):
    # 4096 token rows of 768 (the transformer boundary): more segments than
    # resident wavefronts, so each wavefront loops
    x = W.transformer_hidden((8, 512, 768), seed=0, tensor_id=0).reshape(4096, 768)
    run_case(tc, orc, x, 4096, 768, tc.topk_count(768, 1, 10))


def test_topk_many_segments_group_layout(tc, orc):
    # more long segments than resident groups of workgroups (segments longer
    # than one workgroup's LDS holds take the group engine)
    x = make_input("relu", 200, 40000, "f32", seed=3)
    run_case(tc, orc, x, 200, 40000, tc.topk_count(40000, 1, 10))


# segments of 2049..32768 elements: one workgroup per segment, held in LDS
LDS_L = [4097, 32767, 32768]


@pytest.mark.parametrize("dt", ["f32", "bf16", "f16"])
@pytest.mark.parametrize("L", LDS_L)
@pytest.mark.parametrize("kind", ["normal", "relu", "ties", "zeros"])
def test_topk_lds_engine(tc, orc, dt, L, kind):
    x = make_input(kind, 3, L, dt, seed=L + 1)
    for k in sorted({0, 1, tc.topk_count(L, 1, 10), tc.topk_count(L, 3, 10), L - 1, L}):
        run_case(tc, orc, x, 3, L, k)


def test_topk_lds_engine_many_segments_unaligned(tc, orc):
    # more segments than resident workgroups, and an input that starts 4
    # bytes past a 16-byte boundary (element-wise loads)
    n_seg, L = 600, 12288
    x = make_input("relu", n_seg, L, "f32", seed=5)
    buf = torch.empty(n_seg * L + 1, dtype=torch.float32)
    buf[1:] = x.reshape(-1)
    xd = buf.cuda()[1:].view(n_seg, L)
    k = tc.topk_count(L, 1, 10)
    p = tc.topk_compress(xd, k, n_seg)
    torch.cuda.synchronize()
    assert tc.device_errors() == 0
    oi, ov = orc.topk_compress(raw(x), "f32", n_seg, L, k)
    assert_bits_equal(raw(p.idx), oi, "idx")
    assert_bits_equal(raw(p.val), ov, "val")
    check_block_table(p.blk, oi, L)


def test_decompress_rejects_bad_index_without_fault(tc):
    idx = torch.tensor([[0, 5, 1 << 20]], dtype=torch.int32, device="cuda")
    val = torch.ones((1, 3), dtype=torch.float32, device="cuda")
    tc.device_errors(clear=True)
    y = tc.topk_decompress(tc.TopkPayload(idx, val, None), 100)
    torch.cuda.synchronize()
    assert tc.device_errors(clear=True) & tc.TC_KERR_BAD_INDEX
    yy = y.cpu()
    assert yy[0, 0] == 1 and yy[0, 5] == 1 and yy.sum() == 2


def test_decompress_flags_unsorted_payload(tc):
    idx = torch.tensor([[0, 7, 5, 9]], dtype=torch.int32, device="cuda")
    val = torch.ones((1, 4), dtype=torch.float32, device="cuda")
    tc.device_errors(clear=True)
    tc.topk_decompress(tc.TopkPayload(idx, val, None), 100)
    torch.cuda.synchronize()
    assert tc.device_errors(clear=True) & tc.TC_KERR_BAD_INDEX


def test_decompress_flags_bad_block_table(tc):
    idx = torch.tensor([[0, 5, 9]], dtype=torch.int32, device="cuda")
    val = torch.ones((1, 3), dtype=torch.float32, device="cuda")
    blk = torch.tensor([[0, 7]], dtype=torch.int32, device="cuda")     # claims 7 entries, k is 3
    tc.device_errors(clear=True)
    tc.topk_decompress(tc.TopkPayload(idx, val, blk), 100)
    torch.cuda.synchronize()
    assert tc.device_errors(clear=True) & tc.TC_KERR_BAD_INDEX


@pytest.mark.parametrize("L", [1, 7, 37, 768, 2048, 2049])
@pytest.mark.parametrize("out_dt", ["f32", "f16"])
def test_decompress_rows_unaligned_output(tc, orc, L, out_dt):
    # the one-wavefront-per-row receiver (L <= 2048) and the chunk receiver
    # (2049) into an output that starts one element past a 16-byte boundary,
    # bf16 wire widened (f32) or converted (f16), many rows
    n_seg = 300
    x = make_input("ties", n_seg, L, "bf16", seed=L + 3)
    k = tc.topk_count(L, 1, 10)
    p = tc.topk_compress(x.cuda(), k, n_seg)
    buf = torch.empty(n_seg * L + 1, dtype=TORCH[out_dt], device="cuda")
    y = buf[1:].view(n_seg, L)
    tc.topk_decompress(p, L, out=y)
    torch.cuda.synchronize()
    assert tc.device_errors() == 0
    oi, ov = orc.topk_compress(raw(x), "bf16", n_seg, L, k)
    assert_bits_equal(raw(y), orc.topk_decompress(oi, ov, "bf16", n_seg, L, k, out_dt=out_dt), "dense")


def test_decompress_rows_several_per_wavefront(tc, orc):
    # more rows than the row receiver's wavefronts (8 workgroups of 4 per
    # compute unit): each wavefront builds several rows in its LDS slice
    n_seg, L = 9000, 37
    x = make_input("normal", n_seg, L, "f16", seed=21)
    k = tc.topk_count(L, 3, 10)
    p = tc.topk_compress(x.cuda(), k, n_seg)
    y = tc.topk_decompress(p, L)
    torch.cuda.synchronize()
    assert tc.device_errors() == 0
    oi, ov = orc.topk_compress(raw(x), "f16", n_seg, L, k)
    assert_bits_equal(raw(y), orc.topk_decompress(oi, ov, "f16", n_seg, L, k), "dense")


@pytest.mark.parametrize("dt", ["f32", "bf16"])
def test_topk_row_threshold_bin_shortcuts(tc, orc, dt):
    # rows where the bin chosen by the first digits holds a few keys with
    # ties among them (values 1 + j * 2^-20 share their top 16 key bits in
    # fp32; in bf16 they collapse to one value), swept over k so that the
    # selection ends needing one key of the bin, all of it, or something
    # in between
    n_seg, L = 6, 768
    g = torch.Generator().manual_seed(5)
    x = torch.rand((n_seg, L), generator=g) * 0.4 - 0.2
    pick = torch.rand((n_seg, L), generator=g) < 0.01
    j = torch.randint(0, 4, (n_seg, L), generator=g).to(torch.float64)
    x = torch.where(pick, (1.0 + j * 2.0 ** -20).to(torch.float32), x)
    x[:, 5] = 3.0
    x[:, 700] = -3.0
    x = x.to(TORCH[dt]).contiguous()
    n_big = int(pick.sum(dim=1).max()) + 2
    for k in range(1, n_big + 4):
        run_case(tc, orc, x, n_seg, L, k)


@pytest.mark.parametrize("L", [64, 768, 960])
@pytest.mark.parametrize("spread", [1.0, 30.0, 1e6])
def test_topk_row_first_digit_window(tc, orc, L, spread):
    # the first digit (the exponent) is counted for the eight binades below
    # the row's largest key; with a few entries `spread` times larger, T's
    # binade lies inside that window (1, 30) or far below it (1e6: the
    # histogram pass); rows of subnormal values and of exact zeros too
    n_seg = 8
    g = torch.Generator().manual_seed(int(L + spread))
    x = torch.randn((n_seg, L), generator=g)
    big = torch.rand((n_seg, L), generator=g) < 0.01
    x = torch.where(big, x * spread, x)
    x[6] = torch.randn(L, generator=g) * 1e-40
    x[7] = 0.0
    x = x.contiguous()
    for num, den in [(1, 100), (1, 10), (3, 10), (9, 10)]:
        run_case(tc, orc, x, n_seg, L, tc.topk_count(L, num, den))
