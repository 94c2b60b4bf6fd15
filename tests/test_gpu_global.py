"""GPU parity: TopK over segments too long to stay on chip, with error
feedback (Sec. 2.4), and TopK whose kept list is min-max quantized as one
group per segment (Sec. 2.2 applied to the TopK payload), the large language
model boundary: one bfloat16 micro-batch of 16 x 2048 x 4096 activations as a
single segment, TopK 10 %, 4-bit codes, the residual carried from one
micro-batch to the next.

Indices, codes and meta are compared bit for bit with the oracle, the binary32
residual within 1e-6 relative (and checked bit for bit), and the receiver's
dense tensor bit for bit.  At the full length the oracle runs on the first
micro-batch; the second is checked through properties computed from the
inputs alone (the exact threshold from a partition, the tie rule, the codes
of the selected values)."""
import numpy as np
import pytest
import torch

from gpu_helpers import DTN, TORCH, assert_bits_equal, assert_rel_close, check_block_table, raw
from paper_2401_07788_amd import workloads as W

pytestmark = pytest.mark.gpu


def f32_of(xr, dt):
    """binary32 values of raw element patterns"""
    if dt == "f32":
        return np.asarray(xr, np.float32)
    if dt == "bf16":
        return (np.asarray(xr, np.uint32) << 16).view(np.float32)
    return np.asarray(xr, np.uint16).view(np.float16).astype(np.float32)


def tq_steps(tc, orc, xs, n_seg, k, b):
    """EF + TopK + quantized kept list over successive tensors, against the oracle"""
    dt = DTN[xs[0].dtype]
    L = xs[0].numel() // n_seg
    e_gpu = torch.zeros(n_seg * L, dtype=torch.float32, device="cuda")
    e_orc = np.zeros((n_seg, L), np.float32)
    for t, x in enumerate(xs):
        p = tc.ef_step_topk_quant(x.cuda(), e_gpu, k, b, n_seg)
        y_blk = tc.topk_quant_decompress(p, L, TORCH[dt])
        y_srch = tc.topk_quant_decompress(p, L, TORCH[dt], use_blk=False)
        torch.cuda.synchronize()
        assert tc.device_errors() == 0, f"device errors step {t}"
        oi, oc, om, e_orc = orc.ef_topk_quant(raw(x), dt, e_orc, n_seg, L, k, b)
        assert_bits_equal(raw(p.idx), oi, f"idx step {t}")
        assert_bits_equal(raw(p.meta), om, f"meta step {t}")
        assert_bits_equal(raw(p.codes), oc, f"codes step {t}")
        check_block_table(p.blk, oi, L, f"blk step {t}")
        oy = orc.topk_quant_decompress(oi, oc, om, n_seg, L, k, b, dt)
        assert_bits_equal(raw(y_blk), oy, f"received step {t}")
        assert_bits_equal(raw(y_srch), oy, f"received (search) step {t}")
        eg = raw(e_gpu).reshape(n_seg, L)
        assert_rel_close(eg, e_orc, 1e-6, f"e step {t}")
        assert_bits_equal(eg, e_orc, f"e step {t} (bitwise)")


@pytest.mark.parametrize("b", [1, 4, 8, 32])
def test_topk_quant_small_f32(tc, orc, b):
    # one segment of 12411 elements (three full 4096 tiles and a ragged tail)
    L = 3 * 4096 + 123
    xs = [W.randn((L,), 7, t) for t in range(3)]
    tq_steps(tc, orc, xs, 1, tc.topk_count(L, 1, 10), b)


@pytest.mark.parametrize("b", [2, 4])
def test_topk_quant_segments_bf16(tc, orc, b):
    # three bfloat16 segments of 40000 with sparse outliers, TopK 10 %
    xs = [W.sparse_outlier_stream((3, 40000), 8, t) for t in range(3)]
    tq_steps(tc, orc, xs, 3, tc.topk_count(40000, 1, 10), b)


def test_topk_quant_ties_bf16(tc, orc):
    # values from {-3 .. 3}: the threshold bin holds thousands of ties, the
    # kept ones must be the lowest indices; zeros are never ahead of others
    L = 5 * 4096 + 1000
    g = torch.Generator().manual_seed(11)
    xs = [torch.randint(-3, 4, (L,), generator=g).to(torch.bfloat16) for _ in range(2)]
    for k in (1, 777, 3 * 4096, L - 5):
        tq_steps(tc, orc, xs, 1, k, 4)


@pytest.mark.parametrize("k", [0, 1, 4095, 4096, 4097, 9000])
def test_topk_quant_k_edges(tc, orc, k):
    L = 2 * 4096 + 808
    xs = [W.randn((L,), 12, t).to(torch.float16) for t in range(2)]
    tq_steps(tc, orc, xs, 1, min(k, L), 4)
    tq_steps(tc, orc, xs, 1, L, 3)


def test_topk_quant_constant_group(tc, orc):
    # every kept value equal (hi == lo): scale 0, all codes 0
    L = 4096 + 17
    xs = [torch.full((L,), -2.5, dtype=torch.float32), torch.full((L,), 0.0, dtype=torch.float32)]
    tq_steps(tc, orc, xs, 1, 100, 4)


def tie_sign_inputs():
    """ties of both signs at the threshold (1000 values of +-1), 300 of them
    kept; 200 larger values: +-5 (kept values beyond +|T| and -|T|), or all
    +5 (then which ties are kept decides the minimum of the kept list)"""
    L = 20000
    rng = np.random.default_rng(5)
    base = ((rng.random(L) - 0.5) * 0.9).astype(np.float32)
    pos = rng.permutation(L)
    both = base.copy()
    both[pos[:100]] = 5.0
    both[pos[100:200]] = -5.0
    both[pos[200:1200]] = np.where(np.arange(1000) % 2 == 0, 1.0, -1.0).astype(np.float32)
    one = both.copy()
    one[pos[100:200]] = 5.0
    return both, one


@pytest.mark.parametrize("case", [0, 1])
def test_topk_quant_tie_signs(tc, orc, case):
    x = tie_sign_inputs()[case]
    tq_steps(tc, orc, [torch.from_numpy(x), torch.from_numpy(x[::-1].copy())], 1, 500, 4)


def test_workspace_left_zero_across_lengths(tc, orc):
    """every call leaves the shared workspace zero-filled: a short segment
    with a long candidate list, then a longer one whose tile words lie
    where that list was, then a register-resident TopK on the same
    workspace"""
    short = [torch.full((4096 + 17,), -2.5, dtype=torch.float32)]
    tq_steps(tc, orc, short, 1, 100, 4)
    longer = [W.randn((6 * 4096 + 5,), 17, t) for t in range(2)]
    tq_steps(tc, orc, longer, 1, 2000, 4)
    x = W.randn((32, 16384), 17, 9)
    k = tc.topk_count(16384, 1, 10)
    p = tc.topk_compress(x.cuda(), k, 32)
    torch.cuda.synchronize()
    assert tc.device_errors() == 0
    oi, ov = orc.topk_compress(raw(x), "f32", 32, 16384, k, "f32")
    assert_bits_equal(raw(p.idx), oi, "resident idx")
    assert_bits_equal(raw(p.val), ov, "resident val")


# ------------------------------------------- plain and EF TopK, long segments
LONG = (1 << 24) + 777    # more workgroups than can be resident at once


def test_topk_long_segment_plain(tc, orc):
    x = W.randn((LONG,), 13, 0)
    k = tc.topk_count(LONG, 1, 100)
    p = tc.topk_compress(x.cuda(), k, 1)
    y = tc.topk_decompress(p, LONG)
    torch.cuda.synchronize()
    assert tc.device_errors() == 0
    oi, ov = orc.topk_compress(raw(x), "f32", 1, LONG, k, "f32")
    assert_bits_equal(raw(p.idx), oi, "idx")
    assert_bits_equal(raw(p.val), ov, "val")
    check_block_table(p.blk, oi, LONG, "blk")
    assert_bits_equal(raw(y), orc.topk_decompress(oi, ov, "f32", 1, LONG, k), "received")


def test_ef_topk_long_segment_bf16(tc, orc):
    xs = [W.sparse_outlier_stream((LONG,), 14, t) for t in range(2)]
    k = tc.topk_count(LONG, 1, 10)
    e_gpu = torch.zeros(LONG, dtype=torch.float32, device="cuda")
    e_orc = np.zeros((1, LONG), np.float32)
    for t, x in enumerate(xs):
        p = tc.ef_step_topk(x.cuda(), e_gpu, k, 1)
        torch.cuda.synchronize()
        assert tc.device_errors() == 0
        oi, ov, e_orc = orc.ef_topk(raw(x), "bf16", e_orc, 1, LONG, k)
        assert_bits_equal(raw(p.idx), oi, f"idx step {t}")
        assert_bits_equal(raw(p.val), ov, f"val step {t}")
        check_block_table(p.blk, oi, LONG, f"blk step {t}")
        assert_bits_equal(raw(e_gpu).reshape(1, LONG), e_orc, f"e step {t} (bitwise)")


def test_aqsgd_long_segment_rejected(tc):
    # the per-sample buffer update has no chain for segments this long: a clear error
    m = torch.zeros((2, LONG), dtype=torch.float16, device="cuda")
    a = torch.zeros((1, LONG), dtype=torch.float16, device="cuda")
    ids = torch.zeros(1, dtype=torch.int64, device="cuda")
    with pytest.raises(tc.TCError):
        tc.aqsgd_step(a, m, ids, 10)


# ------------------------------------------------------- the full length
def property_check(orc, x_f32, e_prev, k, b, p, e_gpu, y, dt):
    """TopK + quantized kept list checked from the inputs alone: X = x + e in
    binary32; kept = the k largest |X| with the lowest indices among ties;
    codes and meta = one min-max group over X at the kept indices (computed
    here with the oracle's quantizer on the independently selected list); the
    residual X - received; the receiver's tensor."""
    X = x_f32 + e_prev
    keys = X.view(np.uint32) & np.uint32(0x7FFFFFFF)
    L = keys.size
    T = np.partition(keys, L - k)[L - k]
    gt = np.flatnonzero(keys > T)
    eq = np.flatnonzero(keys == T)
    sel = np.sort(np.concatenate([gt, eq[: k - gt.size]])).astype(np.uint32)
    assert_bits_equal(raw(p.idx).reshape(-1), sel, "idx (threshold property)")
    oc, om = orc.quant_pack(X[sel], "f32", 1, k, b)
    assert_bits_equal(raw(p.meta), om, "meta")
    assert_bits_equal(raw(p.codes), oc, "codes")
    oy = orc.topk_quant_decompress(sel.reshape(1, -1), oc, om, 1, L, k, b, dt).reshape(-1)
    assert_bits_equal(raw(y).reshape(-1), oy, "received")
    e_exp = X - f32_of(oy, dt)
    assert_bits_equal(raw(e_gpu), e_exp, "e (bitwise)")
    return e_exp


@pytest.mark.timeout(300)
def test_topk_quant_full_length(tc, orc):
    shape = W.LM_STREAM["shape"]
    L = W.LM_STREAM["seg_len"]
    k = tc.topk_count(L, 1, 10)
    e_gpu = torch.zeros(L, dtype=torch.float32, device="cuda")
    # micro-batch 0: the oracle
    x0 = W.sparse_outlier_stream(shape, 15, 0)
    p = tc.ef_step_topk_quant(x0.cuda(), e_gpu, k, 4)
    y = tc.topk_quant_decompress(p, L, torch.bfloat16)
    torch.cuda.synchronize()
    assert tc.device_errors() == 0
    oi, oc, om, e_orc = orc.ef_topk_quant(raw(x0).reshape(1, -1), "bf16", np.zeros((1, L), np.float32), 1, L, k, 4)
    assert_bits_equal(raw(p.idx), oi, "idx mb0")
    assert_bits_equal(raw(p.meta), om, "meta mb0")
    assert_bits_equal(raw(p.codes), oc, "codes mb0")
    check_block_table(p.blk, oi, L, "blk mb0")
    oy = orc.topk_quant_decompress(oi, oc, om, 1, L, k, 4, "bf16")
    assert_bits_equal(raw(y), oy, "received mb0")
    assert_bits_equal(raw(e_gpu).reshape(1, L), e_orc, "e mb0 (bitwise)")
    del oi, oc, oy
    # micro-batch 1, residual carried: properties
    x1 = W.sparse_outlier_stream(shape, 15, 1)
    p = tc.ef_step_topk_quant(x1.cuda(), e_gpu, k, 4)
    y = tc.topk_quant_decompress(p, L, torch.bfloat16)
    torch.cuda.synchronize()
    assert tc.device_errors() == 0
    property_check(orc, f32_of(raw(x1).reshape(-1), "bf16"), e_orc.reshape(-1), k, 4, p, e_gpu, y, "bf16")


def test_topk_quant_two_streams(tc, orc):
    """micro-batch stream: compress(j+1) on one stream while decompress(j)
    runs on another; the residual is carried on the compress stream.  Every
    micro-batch's payload, received tensor and residual match the oracle's
    serial chain."""
    L = 1 << 22
    n_mb = 4
    k = tc.topk_count(L, 1, 10)
    xs = [W.sparse_outlier_stream((L,), 16, j).cuda() for j in range(n_mb)]
    sa, sb = torch.cuda.Stream(), torch.cuda.Stream()
    e_gpu = torch.zeros(L, dtype=torch.float32, device="cuda")
    torch.cuda.synchronize()
    pls, ys, es, done = [], [], [], []
    for j in range(n_mb):
        with torch.cuda.stream(sa):
            pls.append(tc.ef_step_topk_quant(xs[j], e_gpu, k, 4))
            es.append(e_gpu.clone())
            ev = torch.cuda.Event()
            ev.record(sa)
        with torch.cuda.stream(sb):
            sb.wait_event(ev)
            ys.append(tc.topk_quant_decompress(pls[j], L, torch.bfloat16))
    torch.cuda.synchronize()
    assert tc.device_errors() == 0
    e_orc = np.zeros((1, L), np.float32)
    for j in range(n_mb):
        oi, oc, om, e_orc = orc.ef_topk_quant(raw(xs[j]).reshape(1, -1), "bf16", e_orc, 1, L, k, 4)
        assert_bits_equal(raw(pls[j].idx), oi, f"idx mb{j}")
        assert_bits_equal(raw(pls[j].codes), oc, f"codes mb{j}")
        assert_bits_equal(raw(pls[j].meta), om, f"meta mb{j}")
        assert_bits_equal(raw(ys[j]), orc.topk_quant_decompress(oi, oc, om, 1, L, k, 4, "bf16"), f"received mb{j}")
        assert_bits_equal(raw(es[j]).reshape(1, L), e_orc, f"e mb{j}")
