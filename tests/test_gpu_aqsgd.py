"""GPU parity: AQ-SGD with TopK (Sec. 2.5), sender and receiver, against the
CPU oracle: payload bit for bit, both copies of the per-example buffer bit for
bit (and equal to each other), rows outside the micro-batch untouched, and the
receiver's reconstruction bit for bit.  Includes the full-size workload (4096
examples x 512x768 binary16 buffer, micro-batches of 8, TopK 30% of the
per-sample change) in the launch layout the benchmark times."""
import numpy as np
import pytest
import torch

from gpu_helpers import DTN, TORCH, assert_bits_equal, check_block_table, raw
from paper_2401_07788_amd import workloads as W

pytestmark = pytest.mark.gpu


def aq_steps(tc, orc, m0, ids_list, acts, k, check_rows=None):
    """run AQ-SGD steps on GPU and oracle from the same buffer m0 (CPU tensor)"""
    dt = DTN[m0.dtype]
    m_s = m0.cuda()
    m_r = m_s.clone()
    mo = raw(m0).copy()
    mo_r = mo.copy()
    for t, (ids, a) in enumerate(zip(ids_list, acts)):
        idsd = ids.cuda()
        p = tc.aqsgd_step(a.cuda(), m_s, idsd, k)
        # alternate the receiver between the block table and the index search
        a_hat = tc.aqsgd_reconstruct(p, m_r, idsd, use_blk=(t % 2 == 0))
        torch.cuda.synchronize()
        assert tc.device_errors() == 0
        oi, ov = orc.aqsgd_send(raw(a), mo, dt, ids.numpy(), k)
        oa = orc.aqsgd_recv(oi, ov, mo_r, dt, ids.numpy(), k)
        assert_bits_equal(raw(p.idx), oi, f"idx step {t}")
        assert_bits_equal(raw(p.val), ov, f"val step {t}")
        check_block_table(p.blk, oi, m0.shape[1], f"blk step {t}")
        assert_bits_equal(raw(a_hat), oa, f"a_hat step {t}")
        rows = ids.numpy() if check_rows is None else np.union1d(ids.numpy(), check_rows)
        assert_bits_equal(raw(m_s[torch.from_numpy(rows).cuda()]), mo[rows], f"m_s rows step {t}")
        assert_bits_equal(raw(m_r[torch.from_numpy(rows).cuda()]), mo_r[rows], f"m_r rows step {t}")
    assert torch.equal(m_s.view(torch.int16) if m_s.dtype != torch.float32 else m_s.view(torch.int32),
                       m_r.view(torch.int16) if m_r.dtype != torch.float32 else m_r.view(torch.int32))


@pytest.mark.parametrize("dt", ["f16", "bf16", "f32"])
@pytest.mark.parametrize("L", [1000, 12289, 16384, 100003])
def test_aqsgd_small(tc, orc, dt, L):
    n_samples, B = 24, 4
    m0 = W.randn((n_samples, L), 1, 0).to(TORCH[dt])
    ids = W.epoch_ids(n_samples, B, seed=1)
    steps = 3
    acts = [W.drifted_activation(m0, ids[t], 1, 10 + t) for t in range(steps)]
    aq_steps(tc, orc, m0, [ids[t] for t in range(steps)], acts, tc.topk_count(L, 3, 10),
             check_rows=np.arange(n_samples))


def test_aqsgd_aligned_ragged_tail(tc, orc):
    """8 examples of 394,016 binary16 elements (a multiple of the 8-element
    run, not of the 12,288-element chunk): three runs per thread, 33
    workgroups per example, so the last chunk's later runs lie wholly past
    the example's end; more examples than resident groups, so a group takes
    a second example"""
    n_samples, L, B = 24, 394016, 8
    m0 = W.randn((n_samples, L), 3, 0).to(torch.float16)
    ids = W.epoch_ids(n_samples, B, seed=2)
    acts = [W.drifted_activation(m0, ids[t], 1, 20 + t) for t in range(2)]
    aq_steps(tc, orc, m0, [ids[t] for t in range(2)], acts, tc.topk_count(L, 3, 10),
             check_rows=np.arange(n_samples))


def test_aqsgd_revisit_and_k_edges(tc, orc):
    # the same ids again (the buffer has moved), and k = 0 / k = L
    n_samples, L = 8, 50000
    m0 = W.randn((n_samples, L), 2, 0).to(torch.float16)
    ids = torch.tensor([5, 1, 7], dtype=torch.int64)
    acts = [W.drifted_activation(m0, ids, 2, 10 + t) for t in range(2)]
    aq_steps(tc, orc, m0, [ids, ids], acts, tc.topk_count(L, 3, 10), check_rows=np.arange(n_samples))
    for k in (0, L):
        aq_steps(tc, orc, m0, [ids], acts[:1], k, check_rows=np.arange(n_samples))


def test_aqsgd_bad_id_is_flagged_not_faulted(tc):
    m = torch.zeros((4, 5000), dtype=torch.float16, device="cuda")
    a = torch.ones((2, 5000), dtype=torch.float16, device="cuda")
    ids = torch.tensor([1, 9], dtype=torch.int64, device="cuda")
    tc.device_errors(clear=True)
    tc.aqsgd_step(a, m, ids, 100)
    torch.cuda.synchronize()
    assert tc.device_errors(clear=True) & tc.TC_KERR_BAD_ID
    mm = m.float().cpu()
    assert mm[1].sum() == 100 and mm[[0, 2, 3]].abs().sum() == 0


def test_aqsgd_full_size(tc, orc):
    """4096 x 393216 binary16 buffers on both sides; two micro-batches of 8"""
    n_samples, L, B = W.AQSGD["n_samples"], W.AQSGD["seg_len"], W.AQSGD["batch"]
    k = tc.topk_count(L, 3, 10)
    m_s = W.aqsgd_buffer(n_samples, L, seed=0, device="cuda")
    m_r = m_s.clone()
    ids_all = W.epoch_ids(n_samples, B, seed=0)
    for t in range(2):
        ids = ids_all[t]
        rows0 = raw(m_s[ids.cuda()])                     # the oracle's copy of the touched rows
        a = W.drifted_activation(m_s, ids, 0, 100 + t)
        p = tc.aqsgd_step(a, m_s, ids.cuda(), k)
        a_hat = tc.aqsgd_reconstruct(p, m_r, ids.cuda(), use_blk=(t == 0))
        idx, val = p.idx, p.val
        torch.cuda.synchronize()
        assert tc.device_errors() == 0
        mo = rows0.copy()
        local = np.arange(B, dtype=np.int64)
        oi, ov = orc.aqsgd_send(raw(a), mo, "f16", local, k, threads=8)
        mo_r = rows0.copy()
        oa = orc.aqsgd_recv(oi, ov, mo_r, "f16", local, k)
        assert_bits_equal(raw(idx), oi, f"idx mb {t}")
        assert_bits_equal(raw(val), ov, f"val mb {t}")
        check_block_table(p.blk, oi, L, f"blk mb {t}")
        assert_bits_equal(raw(a_hat), oa, f"a_hat mb {t}")
        assert_bits_equal(raw(m_s[ids.cuda()]), mo, f"m_s rows mb {t}")
        assert_bits_equal(raw(m_r[ids.cuda()]), mo_r, f"m_r rows mb {t}")
    # an untouched row is unchanged on both sides
    untouched = int(ids_all[2][0])
    ref = W.aqsgd_buffer(n_samples, L, seed=0, device="cuda")[untouched]
    assert torch.equal(m_s[untouched].view(torch.int16), ref.view(torch.int16))
    del m_s, m_r
    torch.cuda.empty_cache()


@pytest.mark.parametrize("shape", [(128, 32768), (6, 100003)])
def test_ef21_parity(tc, orc, shape):
    # EF21 (Sec. 2.4): g <- g + TopK(x - g) on both sides, one row per segment
    B, L = shape
    k = tc.topk_count(L, 1, 10)
    g = torch.zeros((B, L), dtype=torch.float32, device="cuda")
    g_r = g.clone()
    go = np.zeros((B, L), np.float32)
    go_r = go.copy()
    ids = np.arange(B)
    for t in range(3):
        x = W.relu_activation((B, L), 3, t)
        p = tc.ef21_step(x.cuda(), g, k)
        out = tc.ef21_reconstruct(p, g_r)
        torch.cuda.synchronize()
        assert tc.device_errors() == 0
        oi, ov = orc.aqsgd_send(raw(x), go, "f32", ids, k)
        orc.aqsgd_recv(oi, ov, go_r, "f32", ids, k)
        assert_bits_equal(raw(p.idx), oi, f"idx step {t}")
        assert_bits_equal(raw(p.val), ov, f"val step {t}")
        assert_bits_equal(raw(g), go, f"g step {t}")
        assert_bits_equal(raw(g_r), go_r, f"g_r step {t}")
        assert_bits_equal(raw(out), go_r, f"received step {t}")


def test_aqsgd_per_token_row(tc, orc):
    # a second AQ-SGD workload: one buffer row per 768-element token row,
    # TopK 30 % of each row (k = 231); row ids = example id * rows + row
    n_ex, rows, H, B = 12, 64, 768, 4
    m0 = W.randn((n_ex * rows, H), 7, 0).to(torch.float16)
    ex_ids = W.epoch_ids(n_ex, B, seed=7)
    ids_list, acts = [], []
    for t in range(3):
        rid = (ex_ids[t].view(B, 1) * rows + torch.arange(rows).view(1, rows)).reshape(-1)
        ids_list.append(rid)
        acts.append(W.drifted_activation(m0, rid, 7, 20 + t))
    aq_steps(tc, orc, m0, ids_list, acts, tc.topk_count(H, 3, 10), check_rows=np.arange(n_ex * rows))


def test_aqsgd_rows_several_per_wavefront(tc, orc):
    # the one-wavefront-per-row receiver with more rows than wavefronts
    n_samples, L, n_ids = 10000, 64, 9000
    m0 = W.randn((n_samples, L), 16, 0).to(torch.float16)
    ids = torch.randperm(n_samples, generator=torch.Generator().manual_seed(16))[:n_ids]
    acts = [W.drifted_activation(m0, ids, 16, 1)]
    aq_steps(tc, orc, m0, [ids], acts, tc.topk_count(L, 3, 10))
