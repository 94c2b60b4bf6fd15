"""The Python binding refuses tensors whose shapes do not match the call
before anything reaches the C ABI: the library sees only pointers, so a
payload made for another k or segment count would otherwise let a kernel
write past its arrays.  These checks run on the CPU (they come before the
binding asks for GPU tensors)."""
import pytest
import torch

from paper_2401_07788_amd import tc


def payload(n_seg, k, L, dtype=torch.float16, blk=True):
    return tc.empty_topk_payload(n_seg, L, k, dtype, "cpu", blk)


def test_topk_compress_rejects_foreign_payload():
    x = torch.zeros((4, 5000), dtype=torch.float16)
    with pytest.raises(ValueError, match="idx"):
        tc.topk_compress(x, 100, 4, out=payload(4, 99, 5000))
    with pytest.raises(ValueError, match="idx"):
        tc.topk_compress(x, 100, 4, out=payload(3, 100, 5000))
    bad_val = payload(4, 100, 5000)._replace(val=torch.zeros((4, 50), dtype=torch.float16))
    with pytest.raises(ValueError, match="val"):
        tc.topk_compress(x, 100, 4, out=bad_val)
    with pytest.raises(TypeError, match="val"):
        tc.topk_compress(x, 100, 4, out=payload(4, 100, 5000, dtype=torch.float32))
    with pytest.raises(ValueError, match="blk"):
        tc.topk_compress(x, 100, 4, out=payload(4, 100, 50000))
    with pytest.raises(ValueError, match="segments"):
        tc.topk_compress(x, 100, 3)


def test_ef_step_topk_rejects_foreign_payload():
    x = torch.zeros((2, 8192))
    e = torch.zeros(2 * 8192)
    with pytest.raises(ValueError, match="idx"):
        tc.ef_step_topk(x, e, 10, 2, out=payload(2, 11, 8192, torch.float32))
    with pytest.raises(ValueError, match="blk"):
        tc.ef_step_topk(x, e, 10, 2, out=payload(2, 10, 4096, torch.float32))
    with pytest.raises(ValueError, match="segments"):
        tc.ef_step_topk(x, e, 10, 3)


def test_ef_step_topk_quant_rejects_foreign_payload():
    x = torch.zeros((1, 10000))
    e = torch.zeros(10000)
    good = tc.empty_topk_quant_payload(1, 10000, 1000, 4, "cpu")
    with pytest.raises(ValueError, match="bits"):
        tc.ef_step_topk_quant(x, e, 1000, 8, out=good)
    with pytest.raises(ValueError, match="idx"):
        tc.ef_step_topk_quant(x, e, 999, 4, out=good)
    short = good._replace(codes=torch.zeros((1, 10), dtype=torch.uint8))
    with pytest.raises(ValueError, match="codes"):
        tc.ef_step_topk_quant(x, e, 1000, 4, out=short)


def test_aqsgd_step_rejects_shapes():
    ids = torch.tensor([0, 1], dtype=torch.int64)
    a = torch.zeros((2, 6000), dtype=torch.float16)
    # a buffer of [n_samples, 512, 768] would silently compress the wrong segments
    with pytest.raises(ValueError, match="m must be"):
        tc.aqsgd_step(a, torch.zeros((4, 2, 3000), dtype=torch.float16), ids, 100)
    m = torch.zeros((4, 6000), dtype=torch.float16)
    with pytest.raises(ValueError, match="a must hold"):
        tc.aqsgd_step(torch.zeros((3, 6000), dtype=torch.float16), m, ids, 100)
    with pytest.raises(ValueError, match="ids"):
        tc.aqsgd_step(a, m, ids.view(2, 1), 100)
    with pytest.raises(TypeError):
        tc.aqsgd_step(a, m, ids.to(torch.int32), 100)
    with pytest.raises(ValueError, match="idx"):
        tc.aqsgd_step(a, m, ids, 100, out=payload(2, 101, 6000))
    with pytest.raises(ValueError, match="blk"):
        tc.aqsgd_step(a, m, ids, 100, out=payload(2, 100, 60000))


def test_aqsgd_reconstruct_rejects_shapes():
    ids = torch.tensor([0, 1], dtype=torch.int64)
    m_r = torch.zeros((4, 6000), dtype=torch.float16)
    with pytest.raises(ValueError, match="segments"):
        tc.aqsgd_reconstruct(payload(3, 100, 6000), m_r, ids)
    with pytest.raises(ValueError, match="blk"):
        tc.aqsgd_reconstruct(payload(2, 100, 10000), m_r, ids)
    with pytest.raises(TypeError, match="val"):
        tc.aqsgd_reconstruct(payload(2, 100, 6000, torch.bfloat16), m_r, ids)
    with pytest.raises(ValueError, match="m_r"):
        tc.aqsgd_reconstruct(payload(2, 100, 6000), m_r.view(4, 2, 3000), ids)
    with pytest.raises(ValueError, match="out"):
        tc.aqsgd_reconstruct(payload(2, 100, 6000), m_r, ids, out=torch.zeros((1, 6000), dtype=torch.float16))


def test_receivers_reject_mismatched_payloads():
    pl = payload(2, 100, 6000)
    with pytest.raises(ValueError, match="val"):
        tc.topk_decompress(pl._replace(val=torch.zeros((2, 99), dtype=torch.float16)), 6000)
    with pytest.raises(ValueError, match="blk"):
        tc.topk_decompress(pl, 9000)
    with pytest.raises(ValueError, match="segments"):
        tc.topk_gather(pl, torch.zeros(12001, dtype=torch.float16))
    with pytest.raises(ValueError, match="out"):
        tc.topk_gather(pl, torch.zeros((2, 6000), dtype=torch.float16), out=torch.zeros((2, 5), dtype=torch.float16))


def test_efmix_rejects_foreign_payloads():
    x = torch.zeros((2, 4096))
    e = torch.zeros(2 * 4096)
    kx, ke = tc.efmix_counts(41)
    good = (payload(2, kx, 4096, torch.float32), payload(2, ke, 4096, torch.float32))
    with pytest.raises(ValueError, match=r"out\[1\]"):
        tc.efmix_step(x, e, 41, 2, out=(good[0], payload(2, ke + 1, 4096, torch.float32)))
    with pytest.raises(ValueError, match="budget"):
        tc.efmix_reconstruct(good[0], payload(2, ke - 1, 4096, torch.float32), 4096)
