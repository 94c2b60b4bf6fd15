"""GPU parity on the edges of the floating-point readings and of the selection
paths, against the CPU oracle, bit for bit:

* quantization (Sec. 2.2) of groups whose range hi - lo is a binary32
  subnormal, of groups made of subnormals, and of binary16 / bfloat16
  subnormal inputs, with and without error feedback (Sec. 2.4);
* AQ-SGD (Sec. 2.5) with binary16 buffers holding subnormals and values near
  the binary16 maximum 65504, and wire values near it;
* error-feedback TopK and AQ-SGD on tie-heavy, constant and all-zero inputs at
  lengths that spread a segment over several workgroups, for every dtype, so
  that the exact fallback selection and the placement after it run with the
  residual and buffer epilogues;
* binary32 error feedback over many long segments (the plain placement path
  of the several-workgroup engine, segments looped over resident groups);
* AQ-SGD's first visit of an example from an all-zero buffer at the full
  workload size, which must equal plain TopK of the activation (Sec. 2.5)."""
import numpy as np
import pytest
import torch

from gpu_helpers import DTN, TORCH, assert_bits_equal, check_block_table, raw
from paper_2401_07788_amd import workloads as W

pytestmark = pytest.mark.gpu


def _gen(seed):
    return torch.Generator().manual_seed(seed)


# ------------------------------------------------------------ quantization
def subnormal_groups(n_grp, G, seed):
    """binary32 groups: [0] 2^-126 + j*2^-149 (normal values, subnormal range),
    [1] j*2^-149 (subnormal values), [2] a normal group, [3] constant subnormal"""
    g = _gen(seed)
    j = torch.randint(0, 1001, (n_grp, G), generator=g).to(torch.float64)
    x = torch.empty((n_grp, G), dtype=torch.float64)
    x[0] = 2.0 ** -126 + j[0] * 2.0 ** -149
    x[1] = (j[1] - 500) * 2.0 ** -149
    x[2] = torch.randn((G,), generator=g, dtype=torch.float64)
    x[3] = 37 * 2.0 ** -149
    return x[:n_grp].to(torch.float32).contiguous()


def half_subnormals(n_grp, G, dt, seed):
    """bfloat16 / binary16 groups of subnormal patterns of that format (and a
    group mixing them with normal values)"""
    g = _gen(seed)
    q = torch.randint(-127, 128, (n_grp, G), generator=g).to(torch.float64)
    step = 2.0 ** -133 if dt == "bf16" else 2.0 ** -24
    x = q * step
    x[-1, ::7] = torch.randn((len(range(0, G, 7)),), generator=g, dtype=torch.float64)
    return x.to(TORCH[dt]).contiguous()


def quant_case(tc, orc, x, n_grp, G, b):
    dt = DTN[x.dtype]
    codes, meta = tc.quant_pack(x.cuda(), b, n_grp)
    y = tc.quant_unpack(codes, meta, G, b, out_dtype=x.dtype)
    torch.cuda.synchronize()
    assert tc.device_errors() == 0
    oc, om = orc.quant_pack(raw(x), dt, n_grp, G, b)
    assert_bits_equal(raw(codes), oc, "codes")
    assert_bits_equal(raw(meta), om, "meta")
    assert_bits_equal(raw(y), orc.quant_unpack(oc, om, n_grp, G, b, dt), "dense")


def ef_quant_case(tc, orc, xs, n_grp, G, b):
    dt = DTN[xs[0].dtype]
    e = torch.zeros(n_grp * G, dtype=torch.float32, device="cuda")
    eo = np.zeros((n_grp, G), np.float32)
    for t, x in enumerate(xs):
        codes, meta = tc.ef_step_quant(x.cuda(), e, b, n_grp)
        torch.cuda.synchronize()
        assert tc.device_errors() == 0
        oc, om, eo = orc.ef_quant(raw(x), dt, eo, n_grp, G, b)
        assert_bits_equal(raw(codes), oc, f"codes step {t}")
        assert_bits_equal(raw(meta), om, f"meta step {t}")
        assert_bits_equal(raw(e).reshape(n_grp, G), eo, f"e step {t}")


@pytest.mark.parametrize("b", [2, 4, 8])
@pytest.mark.parametrize("G", [768, 40000])
def test_quant_subnormal_range_f32(tc, orc, b, G):
    x = subnormal_groups(4, G, seed=G + b)
    meta_range = x.double().amax(1) - x.double().amin(1)
    assert 0 < meta_range[0] < 2.0 ** -126 and 0 < meta_range[1] < 2.0 ** -126
    quant_case(tc, orc, x, 4, G, b)
    ef_quant_case(tc, orc, [x, subnormal_groups(4, G, seed=G + b + 1)], 4, G, b)


@pytest.mark.parametrize("dt", ["bf16", "f16"])
@pytest.mark.parametrize("G", [768, 40000])
def test_quant_half_subnormals(tc, orc, dt, G):
    xs = [half_subnormals(3, G, dt, seed=G + t) for t in range(2)]
    quant_case(tc, orc, xs[0], 3, G, 4)
    ef_quant_case(tc, orc, xs, 3, G, 4)


# ------------------------------------------------------------------ AQ-SGD
def aq_case(tc, orc, m0, ids, acts, k):
    """AQ-SGD steps on the GPU and the oracle from the same buffer (CPU tensor
    m0); payload, both buffers' rows and the reconstruction bit for bit"""
    dt = DTN[m0.dtype]
    m_s = m0.cuda()
    m_r = m_s.clone()
    mo = raw(m0).copy()
    mo_r = mo.copy()
    for t, a in enumerate(acts):
        idsd = ids.cuda()
        p = tc.aqsgd_step(a.cuda(), m_s, idsd, k)
        a_hat = tc.aqsgd_reconstruct(p, m_r, idsd, use_blk=(t % 2 == 0))
        torch.cuda.synchronize()
        assert tc.device_errors() == 0
        oi, ov = orc.aqsgd_send(raw(a), mo, dt, ids.numpy(), k, threads=8)
        oa = orc.aqsgd_recv(oi, ov, mo_r, dt, ids.numpy(), k)
        assert_bits_equal(raw(p.idx), oi, f"idx step {t}")
        assert_bits_equal(raw(p.val), ov, f"val step {t}")
        check_block_table(p.blk, oi, m0.shape[1], f"blk step {t}")
        assert_bits_equal(raw(a_hat), oa, f"a_hat step {t}")
        assert_bits_equal(raw(m_s), mo, f"m_s step {t}")
        assert_bits_equal(raw(m_r), mo_r, f"m_r step {t}")


def f16_extremes(n, L, seed):
    """binary16 buffer rows and an activation: 10 % of the entries near the
    binary16 maximum (changes near +-100, and some near +-64000 where the
    buffer sits at -+32000), 70 % subnormal buffers with subnormal changes,
    20 % unchanged"""
    g = _gen(seed)
    u = torch.rand((n, L), generator=g)
    sub = torch.randint(-1023, 1024, (n, L), generator=g).to(torch.float64) * 2.0 ** -24
    dsub = torch.randint(-300, 301, (n, L), generator=g).to(torch.float64) * 2.0 ** -24
    sign = torch.where(torch.rand((n, L), generator=g) < 0.5, -1.0, 1.0).to(torch.float64)
    big = sign * (60000.0 + torch.randint(0, 4000, (n, L), generator=g).to(torch.float64))
    dbig = -sign * torch.randint(0, 100, (n, L), generator=g).to(torch.float64)
    half = sign * 32000.0
    m = torch.where(u < 0.07, big, torch.where(u < 0.10, -half, sub))
    a = torch.where(u < 0.07, big + dbig, torch.where(u < 0.10, half, torch.where(u < 0.80, sub + dsub, sub)))
    m16, a16 = m.to(torch.float16), a.to(torch.float16)
    assert torch.isfinite(m16.float()).all() and torch.isfinite(a16.float()).all()
    # every change (and so every wire value) stays inside the binary16 range
    assert (a16.double() - m16.double()).abs().max() <= 65504
    return m16, a16


@pytest.mark.parametrize("shape", [(8, 393216), (3, 100003)])
def test_aqsgd_f16_subnormal_and_near_max(tc, orc, shape):
    B, L = shape
    m_rows, a = f16_extremes(B, L, seed=L)
    n_samples = B + 3
    m0 = torch.zeros((n_samples, L), dtype=torch.float16)
    ids = torch.randperm(n_samples, generator=_gen(L))[:B]
    m0[ids] = m_rows
    # second step: the same ids again, the activation drifted by subnormals
    a2 = (a.double() + torch.randint(-5, 6, (B, L), generator=_gen(L + 1)).double() * 2.0 ** -24).to(torch.float16)
    aq_case(tc, orc, m0, ids, [a, a2], tc.topk_count(L, 3, 10))


# ------------------------------------------- ties / constants / zeros, long
def special_input(kind, n_seg, L, dt, seed):
    g = _gen(seed)
    if kind == "ties":
        # values from {0, +-0.5, ..., +-3} with +0 and -0 both common
        z = torch.randint(-6, 7, (n_seg, L), generator=g).to(torch.float32) * 0.5
        u = torch.rand((n_seg, L), generator=g)
        z[u < 0.2] = -0.0
    elif kind == "const":
        z = torch.full((n_seg, L), -1.5)
    else:   # zeros of both signs
        z = torch.zeros((n_seg, L))
        z[:, ::3] = -0.0
    return z.to(TORCH[dt]).contiguous()


# (n_seg, L): one run per thread and many workgroups per segment; three runs
# per thread (binary32: six, where the exact fallback always runs)
LONG_SHAPES = [(3, 50001), (24, 131072)]


@pytest.mark.parametrize("dt", ["f32", "bf16", "f16"])
@pytest.mark.parametrize("kind", ["ties", "const", "zeros"])
@pytest.mark.parametrize("shape", LONG_SHAPES)
def test_ef_topk_special_long(tc, orc, dt, kind, shape):
    n_seg, L = shape
    k = tc.topk_count(L, 3, 10)
    e = torch.zeros(n_seg * L, dtype=torch.float32, device="cuda")
    eo = np.zeros((n_seg, L), np.float32)
    for t in range(2):
        x = special_input(kind, n_seg, L, dt, seed=L + t)
        p = tc.ef_step_topk(x.cuda(), e, k, n_seg)
        torch.cuda.synchronize()
        assert tc.device_errors() == 0
        oi, ov, eo = orc.ef_topk(raw(x), dt, eo, n_seg, L, k, threads=8)
        assert_bits_equal(raw(p.idx), oi, f"idx step {t}")
        assert_bits_equal(raw(p.val), ov, f"val step {t}")
        check_block_table(p.blk, oi, L, f"blk step {t}")
        assert_bits_equal(raw(e).reshape(n_seg, L), eo, f"e step {t}")


@pytest.mark.parametrize("dt", ["f32", "bf16", "f16"])
@pytest.mark.parametrize("kind", ["ties", "const", "zeros", "first"])
@pytest.mark.parametrize("shape", LONG_SHAPES)
def test_aqsgd_special_long(tc, orc, dt, kind, shape):
    B, L = shape
    n_samples = B + 2
    g = _gen(L)
    if kind == "first":
        # first visit: an all-zero buffer, so the change is the activation
        m0 = torch.zeros((n_samples, L)).to(TORCH[dt])
        acts = [W.randn((B, L), L, 1).to(TORCH[dt]), special_input("ties", B, L, dt, seed=L)]
    else:
        # a buffer on a coarse grid, so that a = m + change is exact and the
        # changes keep the input's ties (-0 as a buffer value too)
        m0 = (torch.randint(-8, 9, (n_samples, L), generator=g).to(torch.float32) * 0.25)
        m0[:, ::5] = -0.0
        m0 = m0.to(TORCH[dt])
        acts = []
        for t in range(2):
            d = special_input(kind, B, L, "f32", seed=L + t)
            ids_rows = m0[:B].to(torch.float32)
            acts.append((ids_rows + d).to(TORCH[dt]))
    ids = torch.arange(B, dtype=torch.int64)
    aq_case(tc, orc, m0, ids, acts, tc.topk_count(L, 3, 10))


def test_ef_topk_f32_many_long_segments(tc, orc):
    # 200 segments of 40,000 binary32: several workgroups per segment with six
    # runs per thread, more segments than resident groups
    n_seg, L = 200, 40000
    k = tc.topk_count(L, 1, 10)
    e = torch.zeros(n_seg * L, dtype=torch.float32, device="cuda")
    eo = np.zeros((n_seg, L), np.float32)
    for t in range(2):
        x = W.relu_activation((n_seg, L), 21, t) if t == 0 else special_input("ties", n_seg, L, "f32", 21)
        p = tc.ef_step_topk(x.cuda(), e, k, n_seg)
        y = tc.topk_decompress(p, L)
        torch.cuda.synchronize()
        assert tc.device_errors() == 0
        oi, ov, eo = orc.ef_topk(raw(x), "f32", eo, n_seg, L, k, threads=8)
        assert_bits_equal(raw(p.idx), oi, f"idx step {t}")
        assert_bits_equal(raw(p.val), ov, f"val step {t}")
        check_block_table(p.blk, oi, L, f"blk step {t}")
        assert_bits_equal(raw(e).reshape(n_seg, L), eo, f"e step {t}")
        assert_bits_equal(raw(y), orc.topk_decompress(oi, ov, "f32", n_seg, L, k), f"received step {t}")


def test_aqsgd_first_visit_full_size(tc, orc):
    """4096 x 393216 binary16 buffers, all zero on both sides; the first
    micro-batch of 8 is plain TopK 30 % of the activation"""
    n_samples, L, B = W.AQSGD["n_samples"], W.AQSGD["seg_len"], W.AQSGD["batch"]
    k = tc.topk_count(L, 3, 10)
    m_s = torch.zeros((n_samples, L), dtype=torch.float16, device="cuda")
    m_r = torch.zeros_like(m_s)
    ids = W.epoch_ids(n_samples, B, seed=5)[0]
    a = W.randn((B, L), 5, 2, device="cuda").to(torch.float16)
    p = tc.aqsgd_step(a, m_s, ids.cuda(), k)
    a_hat = tc.aqsgd_reconstruct(p, m_r, ids.cuda())
    torch.cuda.synchronize()
    assert tc.device_errors() == 0
    ti, tv = orc.topk_compress(raw(a), "f16", B, L, k, threads=8)
    assert_bits_equal(raw(p.idx), ti, "idx = TopK(a)")
    assert_bits_equal(raw(p.val), tv, "val = TopK(a)")
    dense = orc.topk_decompress(ti, tv, "f16", B, L, k)
    assert_bits_equal(raw(a_hat), dense, "a_hat = decompressed TopK(a)")
    assert_bits_equal(raw(m_s[ids.cuda()]), dense, "m_s rows")
    assert_bits_equal(raw(m_r[ids.cuda()]), dense, "m_r rows")
    # the same through the AQ-SGD oracle on zero rows
    mo = np.zeros((B, L), np.uint16)
    oi, ov = orc.aqsgd_send(raw(a), mo, "f16", np.arange(B), k, threads=8)
    assert_bits_equal(oi, ti, "oracle AQ-SGD = oracle TopK (idx)")
    assert_bits_equal(ov, tv, "oracle AQ-SGD = oracle TopK (val)")
    other = int(W.epoch_ids(n_samples, B, seed=5)[1][0])
    assert int(m_s[other].view(torch.int16).abs().sum()) == 0
    del m_s, m_r
    torch.cuda.empty_cache()
