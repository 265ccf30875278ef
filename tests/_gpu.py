"""GPU-test helpers: move seeded 16-bit inputs to the device and call the C ABI."""
import numpy as np
import pytest


def torch_dev():
    torch = pytest.importorskip("torch")
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    return torch


def to_dev(bits, in_dtype):
    torch = torch_dev()
    dt = torch.bfloat16 if in_dtype == 1 else torch.float16
    return torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).view(dt).to("cuda")


def flag_fmt(fmt):
    return 0 if fmt == 0 else 1


def say(*a):
    print(*a, flush=True)
