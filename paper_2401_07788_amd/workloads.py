"""Seeded synthetic boundary tensors.

These stand in for the activations and gradients that cross a pipeline-stage
boundary in the paper's two workloads (ResNet-18 on 32x32 images, Sec. 3.1, and
GPT-2-small fine-tuning with hidden size 768 and batch 8, Sec. 3.2); the
datasets and trained weights are not used.  Shapes and value structure:

* CNN activations: ReLU outputs, so about half are exact zeros and the rest
  are half-normal; CNN gradients: N(0, sigma) with a small sigma.
* Transformer hidden states: N(0, 1) in bfloat16 with a few fixed outlier
  channels scaled up (the outlier structure of large language models noted in
  Sec. 4.2); gradients: small-sigma normal in bfloat16.
* AQ-SGD: a per-example binary16 buffer, a seeded permutation of the example
  ids cut into micro-batches, and activations that drift from the buffer by
  N(0, 0.1).
* Large LM stream: bfloat16 N(0, 1) with a sparse set of outliers.

Every tensor comes from its own torch.Generator seeded as seed*1000 + tensor_id.
Nothing here compresses anything: this module holds no arithmetic of the method
and serves both the GPU path and the oracle equally.
"""
from __future__ import annotations

from dataclasses import dataclass

import torch


def _gen(device, seed: int, tensor_id: int) -> torch.Generator:
    g = torch.Generator(device=device)
    g.manual_seed(seed * 1000 + tensor_id)
    return g


def randn(shape, seed: int, tensor_id: int, device="cpu") -> torch.Tensor:
    return torch.randn(shape, generator=_gen(device, seed, tensor_id), device=device, dtype=torch.float32)


def relu_activation(shape, seed: int, tensor_id: int, device="cpu") -> torch.Tensor:
    """post-ReLU activation: exact +0 where z < 0, else z (half-normal)"""
    return torch.relu(randn(shape, seed, tensor_id, device))


def normal_gradient(shape, sigma: float, seed: int, tensor_id: int, device="cpu",
                    dtype=torch.float32) -> torch.Tensor:
    return (randn(shape, seed, tensor_id, device) * sigma).to(dtype)


OUTLIER_CHANNELS = (0, 255, 511, 767)


def transformer_hidden(shape, seed: int, tensor_id: int, device="cpu",
                       channels=OUTLIER_CHANNELS, scale: float = 20.0) -> torch.Tensor:
    """bfloat16 N(0,1) hidden states whose last-dim channels in `channels` are scaled"""
    z = randn(shape, seed, tensor_id, device)
    z[..., list(channels)] *= scale
    return z.to(torch.bfloat16)


def sparse_outlier_stream(shape, seed: int, tensor_id: int, device="cpu",
                          p: float = 1e-3, scale: float = 50.0) -> torch.Tensor:
    """bfloat16 N(0,1) with Bernoulli(p) positions scaled by `scale`"""
    g = _gen(device, seed, tensor_id)
    z = torch.randn(shape, generator=g, device=device, dtype=torch.float32)
    hit = torch.rand(shape, generator=g, device=device) < p
    z[hit] *= scale
    return z.to(torch.bfloat16)


def aqsgd_buffer(n_samples: int, L: int, seed: int, tensor_id: int = 0, device="cpu",
                 chunk_rows: int = 256) -> torch.Tensor:
    """binary16 per-example buffer [n_samples, L] ~ N(0,1), filled chunk by chunk"""
    out = torch.empty((n_samples, L), dtype=torch.float16, device=device)
    g = _gen(device, seed, tensor_id)
    for r0 in range(0, n_samples, chunk_rows):
        r1 = min(n_samples, r0 + chunk_rows)
        out[r0:r1] = torch.randn((r1 - r0, L), generator=g, device=device, dtype=torch.float32).to(torch.float16)
    return out


def epoch_ids(n_samples: int, batch: int, seed: int, tensor_id: int = 1) -> torch.Tensor:
    """a seeded permutation of the example ids, [n_samples // batch, batch] int64 (CPU)"""
    perm = torch.randperm(n_samples, generator=_gen("cpu", seed, tensor_id))
    n_mb = n_samples // batch
    return perm[: n_mb * batch].reshape(n_mb, batch)


def drifted_activation(m: torch.Tensor, ids: torch.Tensor, seed: int, tensor_id: int,
                       drift: float = 0.1) -> torch.Tensor:
    """a[b] = fp16(m[ids[b]] + drift * z): the activation a sample produces this epoch"""
    rows = m.index_select(0, ids.to(m.device)).to(torch.float32)
    z = randn(rows.shape, seed, tensor_id, m.device)
    return (rows + drift * z).to(m.dtype)


# ---------------------------------------------------------------- workloads
@dataclass(frozen=True)
class Workload:
    """one boundary configuration: a segment layout and its K% / bit width"""
    name: str
    shape: tuple
    n_seg: int          # independent TopK segments (or quantization groups)
    seg_len: int
    dtype: torch.dtype
    k_num: int = 1      # TopK keeps ceil(seg_len * k_num / k_den) entries
    k_den: int = 10
    bits: int = 0       # quantization width, 0 when not quantizing


CNN_TINY = dict(shape=(32, 256, 8, 8), n_seg=32, seg_len=256 * 8 * 8)
CNN_RESNET18 = dict(shape=(128, 128, 16, 16), n_seg=128, seg_len=128 * 16 * 16)
TRANSFORMER = dict(shape=(8, 512, 768), n_seg=8 * 512, seg_len=768)
AQSGD = dict(n_samples=4096, seg_len=512 * 768, batch=8)
LM_STREAM = dict(shape=(16, 2048, 4096), n_seg=1, seg_len=16 * 2048 * 4096, n_micro=8)
