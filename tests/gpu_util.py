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


def par_map(fn, items):
    """fn over items on a pool of threads, results in order.  For the
    oracle's one-row calls: ctypes releases the GIL while the C runs, so the
    rows proceed on separate cores (the oracle's functions share no state)."""
    import os
    from concurrent.futures import ThreadPoolExecutor
    items = list(items)
    workers = max(1, min(16, os.cpu_count() or 1, len(items)))
    with ThreadPoolExecutor(max_workers=workers) as ex:
        return list(ex.map(fn, items))
