"""The device state hash against the oracle (hashlib SHA-256 over the same tree), digest for digest, on
tensors of every size class (empty, partial blocks, one and several leaves, misaligned bases) and on a
model state."""
import numpy as np
import pytest
import torch

import paper_2609_17380_amd.canon as C
import paper_2609_17380_amd.inputs as I
from gpu_util import DEV
from oracle import state_hash as H

pytestmark = pytest.mark.gpu


def device_digest(tensors):
    ws = torch.empty(max(1, C.state_hash_workspace_bytes(tensors)), dtype=torch.uint8, device=DEV)
    d = torch.zeros(32, dtype=torch.uint8, device=DEV)
    C.state_hash(tensors, d, ws)
    torch.cuda.synchronize()
    return bytes(d.cpu().numpy().tolist())


def host_bytes(t):
    return t.detach().contiguous().view(torch.uint8).cpu().numpy().tobytes() if t.numel() else b""


def test_size_classes_and_alignment():
    rng = np.random.default_rng(3)
    sizes = [0, 1, 63, 64, 65, 64 * 1024, 64 * 1024 + 1, 64 * 1024 * 3 + 17, 5_000_003]
    ts = [torch.from_numpy(rng.integers(0, 256, n, dtype=np.uint8)).to(DEV) for n in sizes]
    big = torch.from_numpy(rng.integers(0, 256, 300_000, dtype=np.uint8)).to(DEV)
    ts.append(big[3:])  # base off 16-byte alignment: byte loads
    print("state hash sizes", sizes, flush=True)
    assert device_digest(ts) == H.state_digest([host_bytes(t) for t in ts])


def test_model_state_and_sensitivity():
    params = [torch.from_numpy(p.view(np.int16)).to(DEV) for p in I.model_params(2, 256, 512, 1000, seed=1)]
    m = [torch.randn(p.shape, device=DEV) * 1e-3 for p in params]
    tensors = params + m
    d = device_digest(tensors)
    assert d == H.state_digest([host_bytes(t) for t in tensors])
    tensors[3].view(-1)[5] += 1  # one value of one tensor changes
    assert device_digest(tensors) != d
