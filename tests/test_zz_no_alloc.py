"""The allocation-free AQ-SGD sender (tc_aqsgd_step_noalloc): its kernels take
the library's own device scratch instead of a caller workspace, and its
results equal tc_aqsgd_step's bit for bit -- payload (indices, values, block
table) and the updated buffer rows -- on calls in a row of decreasing size,
so that each call finds the scratch as the previous one left it.  A shape that
needs more scratch than the library holds is refused with nothing written."""
import pytest
import torch

from gpu_helpers import assert_bits_equal, raw
from paper_2401_07788_amd import workloads as W

pytestmark = pytest.mark.gpu

# (n_samples, n_ids, seg_len, dtype): the 512x768 binary16 micro-batch of 8,
# then smaller ones (a ragged length, another dtype, a one-workgroup length)
CALLS = [
    (16, 8, 393216, torch.float16),
    (6, 3, 100003, torch.float16),
    (5, 2, 70001, torch.bfloat16),
    (4, 2, 50000, torch.float32),
    (3, 1, 3000, torch.float16),
]


def _one(tc, n_samples, n_ids, L, dtype, seed):
    k = tc.topk_count(L, 3, 10)
    m0 = W.randn((n_samples, L), seed, 0, device="cuda").to(dtype)
    ids = W.epoch_ids(n_samples, n_ids, seed=seed)[0].cuda()
    a = W.drifted_activation(m0, ids, seed, 1)
    m_ref, m_na = m0.clone(), m0.clone()
    p_ref = tc.aqsgd_step(a, m_ref, ids, k)
    out = tc.empty_topk_payload(n_ids, L, k, dtype, "cuda")
    out.idx.fill_(-1)
    p_na = tc.aqsgd_step_noalloc(a, m_na, ids, k, out=out)
    torch.cuda.synchronize()
    what = f"{n_ids}x{L} {dtype}"
    assert_bits_equal(raw(p_na.idx), raw(p_ref.idx), f"idx {what}")
    assert_bits_equal(raw(p_na.val), raw(p_ref.val), f"val {what}")
    assert_bits_equal(raw(p_na.blk), raw(p_ref.blk), f"blk {what}")
    assert_bits_equal(raw(m_na), raw(m_ref), f"m {what}")
    assert not torch.equal(raw_t(m_na), raw_t(m0)), f"{what}: the buffer was not updated"


def raw_t(t):
    return t.view(torch.int32) if t.dtype == torch.float32 else t.view(torch.int16)


def test_noalloc_equals_aqsgd_step_on_calls_in_a_row(tc):
    for i, (n_samples, n_ids, L, dtype) in enumerate(CALLS):
        print(f"noalloc call {i}: {n_ids}x{L} {dtype}", flush=True)
        _one(tc, n_samples, n_ids, L, dtype, seed=40 + i)
    # and back to the first shape: the scratch was left as it must be
    _one(tc, *CALLS[0], seed=50)
    assert tc.device_errors() == 0


def test_noalloc_refuses_a_shape_beyond_its_scratch(tc):
    n_samples, n_ids, L = 600, 600, 40000
    k = tc.topk_count(L, 3, 10)
    m = torch.zeros((n_samples, L), dtype=torch.float16, device="cuda")
    ids = torch.arange(n_ids, dtype=torch.int64, device="cuda")
    a = torch.ones((n_ids, L), dtype=torch.float16, device="cuda")
    out = tc.empty_topk_payload(n_ids, L, k, torch.float16, "cuda")
    out.idx.fill_(-7)
    with pytest.raises(tc.TCError) as ei:
        tc.aqsgd_step_noalloc(a, m, ids, k, out=out)
    assert ei.value.status == tc.TC_ERR_WORKSPACE and "scratch" in str(ei.value)
    torch.cuda.synchronize()
    assert int(m.abs().sum()) == 0 and bool((out.idx == -7).all())
    # the reference entry point, with its own workspace, takes the same shape
    p = tc.aqsgd_step(a, m, ids, k)
    torch.cuda.synchronize()
    assert int(p.idx[0, -1]) == k - 1
    assert tc.device_errors() == 0
