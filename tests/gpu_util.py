"""Helpers shared by the GPU tests: move generated layers to the device and
wrap them for the binding. Nothing here computes any part of the method."""
from __future__ import annotations

import functools
import sys

import numpy as np

from paper_2402_04925_amd import inputs

TOL_FP16 = 2e-3   # max|err| / max|ref| for fp16 outputs accumulated in fp32
# bf16 outputs: 2^-8 is one bf16 rounding of the output alone; the act-order
# and M-tiled kernels also round each dequantized weight to bf16 (2^-9
# relative), whose sum over K stays well inside 1e-2 of max|ref|
TOL_BF16 = 1e-2


def log(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def torch_dev():
    import torch
    if not torch.cuda.is_available():
        import pytest
        pytest.skip("no GPU visible")
    return torch.device("cuda:0")


def to_dev(a, dev, bf16=False):
    """numpy -> device tensor; bf16=True: float32 values that bfloat16 holds
    exactly (the generators' bf16 arrays) as a bfloat16 tensor."""
    import torch
    t = torch.from_numpy(np.ascontiguousarray(a))
    if bf16:
        t = t.to(torch.float32).to(torch.bfloat16)
    return t.to(dev)


def layer_to_dev(layer, dev, with_gidx=True):
    """inputs.QuantLinear -> binding QuantWeight on the device (bf16 scales
    when the layer was generated with them: float32 arrays)."""
    import paper_2402_04925_amd as tpdq
    bf16 = layer.scales.dtype == np.float32
    return tpdq.QuantWeight.from_tensors(
        to_dev(layer.qweight, dev), to_dev(layer.scales, dev, bf16), to_dev(layer.qzeros, dev),
        to_dev(layer.g_idx.astype(np.int32), dev) if with_gidx else None, layer.G)


def np_of(t):
    import torch
    t = t.detach().cpu()
    if t.dtype == torch.bfloat16:
        t = t.to(torch.float32)
    return t.numpy()


def sample_cols(N, rng, n_rand=48, edge=32):
    """First and last `edge` columns (tile edges, ragged tail) plus random ones."""
    cols = set(range(min(edge, N))) | set(range(max(0, N - edge), N))
    cols |= set(rng.choice(N, size=min(n_rand, N), replace=False).tolist())
    return np.array(sorted(cols), dtype=np.int64)


@functools.lru_cache(maxsize=2)
def workload_layers(name):
    """Global layers of a named workload (generated once per process)."""
    return inputs.make_workload(inputs.WORKLOADS[name])
