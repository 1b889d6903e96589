"""Helpers for the GPU tests: move seeded inputs to the device."""
import numpy as np
import pytest

torch = pytest.importorskip("torch")


def need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2203_00448_amd import binding
    binding.load_library()  # raises if the HIP library is missing: no silent fallback
    return binding


def dev(a, dtype):
    return torch.from_numpy(np.ascontiguousarray(a)).to(device="cuda", dtype=dtype)


def batch_to_device(batch):
    return (dev(batch.begin, torch.int64), dev(batch.num_ops, torch.int32),
            dev(batch.size, torch.int64), dev(batch.first, torch.int32), dev(batch.last, torch.int32))


def host(t):
    return t.cpu().numpy()
