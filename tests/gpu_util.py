"""Device helpers for the GPU tests (marshalling only)."""
import numpy as np
import pytest


def torch_dev():
    torch = pytest.importorskip("torch")
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2607_24062_amd import acrl
    acrl.lib()  # fail loudly if the HIP library is missing
    return torch, torch.device("cuda:0")


def up_bf16(torch, dev, bits: np.ndarray):
    return torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).to(dev).view(torch.bfloat16)


def up(torch, dev, a: np.ndarray):
    return torch.from_numpy(np.ascontiguousarray(a)).to(dev)


def down(t) -> np.ndarray:
    return t.detach().cpu().numpy()


def bf16_bits(t) -> np.ndarray:
    return t.detach().cpu().view(dtype=__import__("torch").int16).numpy().view(np.uint16)
