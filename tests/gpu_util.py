"""Helpers shared by the GPU tests: move generated layers to the device and
wrap them for the binding. Nothing here computes any part of the method."""
from __future__ import annotations

import functools
import sys

import numpy as np

from paper_2402_04925_amd import inputs

TOL_FP16 = 2e-3   # max|err| / max|ref| for fp16 outputs accumulated in fp32


def log(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def torch_dev():
    import torch
    if not torch.cuda.is_available():
        import pytest
        pytest.skip("no GPU visible")
    return torch.device("cuda:0")


def to_dev(a, dev):
    import torch
    return torch.from_numpy(np.ascontiguousarray(a)).to(dev)


def layer_to_dev(layer, dev, with_gidx=True):
    """inputs.QuantLinear -> binding QuantWeight on the device."""
    import paper_2402_04925_amd as tpdq
    return tpdq.QuantWeight.from_tensors(
        to_dev(layer.qweight, dev), to_dev(layer.scales, dev), to_dev(layer.qzeros, dev),
        to_dev(layer.g_idx.astype(np.int32), dev) if with_gidx else None, layer.G)


def np_of(t):
    return t.detach().cpu().numpy()


def sample_cols(N, rng, n_rand=48, edge=32):
    """First and last `edge` columns (tile edges, ragged tail) plus random ones."""
    cols = set(range(min(edge, N))) | set(range(max(0, N - edge), N))
    cols |= set(rng.choice(N, size=min(n_rand, N), replace=False).tolist())
    return np.array(sorted(cols), dtype=np.int64)


@functools.lru_cache(maxsize=2)
def workload_layers(name):
    """Global layers of a named workload (generated once per process)."""
    return inputs.make_workload(inputs.WORKLOADS[name])
