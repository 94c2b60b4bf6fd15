"""GPU parity over a seeded sweep of random cases, against the CPU oracle,
bit for bit: TopK (Sec. 2.3) sender and receiver, TopK and min-max
quantization (Sec. 2.2) inside error feedback (Sec. 2.4) over two carried
steps, plain quantization, TopK with its kept list quantized, a tensor sent
at another's TopK indices (alone and inside EF), EF-mixed (Sec. 2.4), and
AQ-SGD (Sec. 2.5) over two micro-batches.
Each case draws its segment count and length (so that every engine runs:
rows of up to 2048 elements, segments held in LDS, segments spread over
several workgroups), its dtype, its K or bit width and the kind of data
(continuous, post-ReLU, heavily tied, tiny or huge magnitudes, a few
outliers) from its own seed, and prints them on failure."""
import numpy as np
import pytest
import torch

from gpu_helpers import DTN, TORCH, assert_bits_equal, check_block_table, raw

pytestmark = pytest.mark.gpu

N_CASES = 64
KINDS = ["normal", "relu", "ties", "tiny", "huge", "outliers"]


def draw(seed):
    r = np.random.default_rng(1000 + seed)
    band = r.integers(0, 3)
    if band == 0:
        L = int(r.integers(1, 2049))
        n_seg = int(r.integers(1, 40))
    elif band == 1:
        L = int(r.integers(2049, 32769))
        n_seg = int(r.integers(1, 9))
    else:
        L = int(r.integers(32769, 200001))
        n_seg = int(r.integers(1, 4))
    dt = ["f32", "bf16", "f16"][int(r.integers(0, 3))]
    kind = KINDS[int(r.integers(0, len(KINDS)))]
    u = r.random()
    k = 1 if u < 0.1 else L if u < 0.15 else max(1, int(L * r.uniform(0.01, 0.5)))
    bits = [1, 2, 3, 4, 5, 6, 7, 8, 32][int(r.integers(0, 9))]
    return dict(n_seg=n_seg, L=L, dt=dt, kind=kind, k=min(k, L), bits=bits, seed=seed)


def make(kind, shape, dt, seed):
    g = torch.Generator().manual_seed(seed)
    z = torch.randn(shape, generator=g)
    if kind == "relu":
        z = torch.relu(z)
    elif kind == "ties":
        z = torch.randint(-4, 5, shape, generator=g).to(torch.float32) * 0.25
        z[torch.rand(shape, generator=g) < 0.2] = -0.0
    elif kind == "tiny":
        z = z * (1e-6 if dt == "f16" else 1e-30)
    elif kind == "huge":
        z = z * (1e4 if dt == "f16" else 1e30)
    elif kind == "outliers":
        z[torch.rand(shape, generator=g) < 1e-3] *= 50.0
    return z.to(TORCH[dt]).contiguous()


@pytest.mark.parametrize("seed", range(N_CASES))
def test_sweep_topk_and_ef(tc, orc, seed):
    c = draw(seed)
    n_seg, L, dt, k = c["n_seg"], c["L"], c["dt"], c["k"]
    # plain TopK, then two carried EF steps
    x = make(c["kind"], (n_seg, L), dt, seed)
    p = tc.topk_compress(x.cuda(), k, n_seg)
    y = tc.topk_decompress(p, L)
    torch.cuda.synchronize()
    assert tc.device_errors() == 0, c
    oi, ov = orc.topk_compress(raw(x), dt, n_seg, L, k, threads=8)
    assert_bits_equal(raw(p.idx), oi, f"idx {c}")
    assert_bits_equal(raw(p.val), ov, f"val {c}")
    check_block_table(p.blk, oi, L, f"blk {c}")
    assert_bits_equal(raw(y), orc.topk_decompress(oi, ov, dt, n_seg, L, k), f"dense {c}")

    e = torch.zeros(n_seg * L, dtype=torch.float32, device="cuda")
    eo = np.zeros((n_seg, L), np.float32)
    for t in range(2):
        xt = make(c["kind"], (n_seg, L), dt, seed * 7 + t + 1)
        pe = tc.ef_step_topk(xt.cuda(), e, k, n_seg)
        torch.cuda.synchronize()
        assert tc.device_errors() == 0, c
        oi, ov, eo = orc.ef_topk(raw(xt), dt, eo, n_seg, L, k, threads=8)
        assert_bits_equal(raw(pe.idx), oi, f"EF idx step {t} {c}")
        assert_bits_equal(raw(pe.val), ov, f"EF val step {t} {c}")
        assert_bits_equal(raw(e).reshape(n_seg, L), eo, f"EF e step {t} {c}")


@pytest.mark.parametrize("seed", range(N_CASES))
def test_sweep_quant_and_ef(tc, orc, seed):
    c = draw(seed)
    n_grp, G, dt, b = c["n_seg"], c["L"], c["dt"], c["bits"]
    x = make(c["kind"], (n_grp, G), dt, seed)
    codes, meta = tc.quant_pack(x.cuda(), b, n_grp)
    y = tc.quant_unpack(codes, meta, G, b, out_dtype=x.dtype)
    torch.cuda.synchronize()
    assert tc.device_errors() == 0, c
    oc, om = orc.quant_pack(raw(x), dt, n_grp, G, b)
    assert_bits_equal(raw(codes), oc, f"codes {c}")
    assert_bits_equal(raw(meta), om, f"meta {c}")
    assert_bits_equal(raw(y), orc.quant_unpack(oc, om, n_grp, G, b, dt), f"dense {c}")

    e = torch.zeros(n_grp * G, dtype=torch.float32, device="cuda")
    eo = np.zeros((n_grp, G), np.float32)
    for t in range(2):
        xt = make(c["kind"], (n_grp, G), dt, seed * 7 + t + 1)
        cg, mg = tc.ef_step_quant(xt.cuda(), e, b, n_grp)
        torch.cuda.synchronize()
        assert tc.device_errors() == 0, c
        oc, om, eo = orc.ef_quant(raw(xt), dt, eo, n_grp, G, b)
        assert_bits_equal(raw(cg), oc, f"EF codes step {t} {c}")
        assert_bits_equal(raw(mg), om, f"EF meta step {t} {c}")
        assert_bits_equal(raw(e).reshape(n_grp, G), eo, f"EF e step {t} {c}")


@pytest.mark.parametrize("seed", range(N_CASES))
def test_sweep_aqsgd(tc, orc, seed):
    c = draw(seed)
    B, L, dt, k = c["n_seg"], c["L"], c["dt"], c["k"]
    if dt == "f32" and c["kind"] == "huge":
        c["kind"] = "normal"   # a - m of two 1e30-scale binary32 values may overflow to inf
    n_samples = 2 * B + 3
    g = torch.Generator().manual_seed(seed)
    m0 = make(c["kind"], (n_samples, L), dt, seed + 500)
    m_s = m0.cuda()
    m_r = m_s.clone()
    mo = raw(m0).copy()
    mo_r = mo.copy()
    perm = torch.randperm(n_samples, generator=g)
    for t in range(2):
        # the second micro-batch revisits some ids of the first
        ids = perm[t * (B // 2): t * (B // 2) + B].clone()
        drift = make("normal", (B, L), "f32", seed * 11 + t)
        a = (m0[ids].to(torch.float32) + 0.1 * drift).to(TORCH[dt]).contiguous()
        idsd = ids.cuda()
        p = tc.aqsgd_step(a.cuda(), m_s, idsd, k)
        a_hat = tc.aqsgd_reconstruct(p, m_r, idsd, use_blk=(t == 0))
        torch.cuda.synchronize()
        assert tc.device_errors() == 0, c
        oi, ov = orc.aqsgd_send(raw(a), mo, dt, ids.numpy(), k, threads=8)
        oa = orc.aqsgd_recv(oi, ov, mo_r, dt, ids.numpy(), k)
        assert_bits_equal(raw(p.idx), oi, f"idx step {t} {c}")
        assert_bits_equal(raw(p.val), ov, f"val step {t} {c}")
        assert_bits_equal(raw(a_hat), oa, f"a_hat step {t} {c}")
        assert_bits_equal(raw(m_s), mo, f"m_s step {t} {c}")
        assert_bits_equal(raw(m_r), mo_r, f"m_r step {t} {c}")


@pytest.mark.parametrize("seed", range(N_CASES))
def test_sweep_topk_quant_and_gather(tc, orc, seed):
    c = draw(seed)
    n_seg, L, dt, k, b = c["n_seg"], c["L"], c["dt"], c["k"], c["bits"]
    # TopK with the kept list quantized (one group per segment), inside EF
    n_q = min(n_seg, 4)
    e = torch.zeros(n_q * L, dtype=torch.float32, device="cuda")
    eo = np.zeros((n_q, L), np.float32)
    for t in range(2):
        xt = make(c["kind"], (n_q, L), dt, seed * 13 + t)
        pq = tc.ef_step_topk_quant(xt.cuda(), e, k, b, n_q)
        y = tc.topk_quant_decompress(pq, L, out_dtype=xt.dtype)
        torch.cuda.synchronize()
        assert tc.device_errors() == 0, c
        oi, oc, om, eo = orc.ef_topk_quant(raw(xt), dt, eo, n_q, L, k, b)
        assert_bits_equal(raw(pq.idx), oi, f"TopK-Q idx step {t} {c}")
        assert_bits_equal(raw(pq.codes), oc, f"TopK-Q codes step {t} {c}")
        assert_bits_equal(raw(pq.meta), om, f"TopK-Q meta step {t} {c}")
        assert_bits_equal(raw(e).reshape(n_q, L), eo, f"TopK-Q e step {t} {c}")
        assert_bits_equal(raw(y), orc.topk_quant_decompress(oi, oc, om, n_q, L, k, b, dt), f"TopK-Q dense {t} {c}")
    # a second tensor at the first one's TopK indices, alone and inside EF
    x = make(c["kind"], (n_seg, L), dt, seed)
    p = tc.topk_compress(x.cuda(), k, n_seg)
    oi, _ = orc.topk_compress(raw(x), dt, n_seg, L, k, threads=8)
    g0 = make("normal", (n_seg, L), dt, seed + 99)
    val = tc.topk_gather(p, g0.cuda())
    torch.cuda.synchronize()
    assert tc.device_errors() == 0, c
    assert_bits_equal(raw(val), orc.topk_gather(raw(g0), dt, oi, n_seg, L, k), f"gather {c}")
    e = torch.zeros(n_seg * L, dtype=torch.float32, device="cuda")
    eo = np.zeros((n_seg, L), np.float32)
    for t in range(2):
        gt = make("normal", (n_seg, L), dt, seed + 100 + t)
        val = tc.topk_gather(p, gt.cuda(), e=e, use_blk=(t == 0))
        torch.cuda.synchronize()
        assert tc.device_errors() == 0, c
        ov, eo = orc.topk_gather(raw(gt), dt, oi, n_seg, L, k, e=eo)
        assert_bits_equal(raw(val), ov, f"gather EF val step {t} {c}")
        assert_bits_equal(raw(e).reshape(n_seg, L), eo, f"gather EF e step {t} {c}")


@pytest.mark.parametrize("seed", range(N_CASES))
def test_sweep_efmix(tc, orc, seed):
    c = draw(seed)
    n_seg, dt = c["n_seg"], c["dt"]
    L = c["L"] if c["L"] <= 32768 else 1 + c["L"] % 32768   # one workgroup per segment
    k = min(c["k"], L)
    e = torch.zeros(n_seg * L, dtype=torch.float32, device="cuda")
    eo = np.zeros((n_seg, L), np.float32)
    for t in range(2):
        xt = make(c["kind"], (n_seg, L), dt, seed * 17 + t)
        px, pe = tc.efmix_step(xt.cuda(), e, k, n_seg)
        y = tc.efmix_reconstruct(px, pe, L)
        torch.cuda.synchronize()
        assert tc.device_errors() == 0, c
        oix, ovx, oie, ove, eo = orc.efmix_send(raw(xt), dt, eo, n_seg, L, k)
        assert_bits_equal(raw(px.idx), oix, f"EF-mixed idx_x step {t} {c}")
        assert_bits_equal(raw(px.val), ovx, f"EF-mixed val_x step {t} {c}")
        assert_bits_equal(raw(pe.idx), oie, f"EF-mixed idx_e step {t} {c}")
        assert_bits_equal(raw(pe.val), ove, f"EF-mixed val_e step {t} {c}")
        assert_bits_equal(raw(e).reshape(n_seg, L), eo, f"EF-mixed e step {t} {c}")
        assert_bits_equal(raw(y), orc.efmix_recv(oix, ovx, oie, ove, dt, n_seg, L, k, out_dt=dt),
                          f"EF-mixed dense step {t} {c}")
