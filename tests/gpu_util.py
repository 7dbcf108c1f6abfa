"""Helpers for the GPU parity tests: moving seeded host buffers to the device and comparing bits."""
import numpy as np
import torch

DEV = torch.device("cuda:0")


def dev_bf16(u16: np.ndarray) -> torch.Tensor:
    return torch.from_numpy(np.ascontiguousarray(u16).view(np.int16)).to(DEV).view(torch.bfloat16)


def dev_f32(x: np.ndarray) -> torch.Tensor:
    return torch.from_numpy(np.ascontiguousarray(x, dtype=np.float32)).to(DEV)


def dev_i32(x: np.ndarray) -> torch.Tensor:
    return torch.from_numpy(np.ascontiguousarray(x, dtype=np.int32)).to(DEV)


def host_u16(t: torch.Tensor) -> np.ndarray:
    return t.detach().view(torch.int16).cpu().numpy().view(np.uint16)


def host_f32(t: torch.Tensor) -> np.ndarray:
    return t.detach().cpu().numpy().astype(np.float32, copy=False)


def assert_bits(got: np.ndarray, want: np.ndarray, what: str):
    g = np.ascontiguousarray(got).view(np.uint32 if got.dtype == np.float32 else np.uint16)
    w = np.ascontiguousarray(want).view(np.uint32 if want.dtype == np.float32 else np.uint16)
    assert g.shape == w.shape, (what, g.shape, w.shape)
    bad = np.nonzero(g.ravel() != w.ravel())[0]
    if bad.size:
        i = bad[0]
        raise AssertionError(f"{what}: {bad.size}/{g.size} elements differ; first at {i}: "
                             f"gpu {got.ravel()[i]!r} (0x{int(g.ravel()[i]):x}) oracle {want.ravel()[i]!r} "
                             f"(0x{int(w.ravel()[i]):x})")


def poisoned_workspace(nbytes: int) -> torch.Tensor:
    """A workspace of all-ones bytes (NaN as bf16 and as fp32): a read of any part the library did not write
    first (outside the ranges its kernels mask) turns into NaN in the results, which the bit comparison sees."""
    return torch.full((max(int(nbytes), 1),), 255, dtype=torch.uint8, device=DEV)
