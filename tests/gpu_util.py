"""Helpers for the GPU tests: host <-> device transfer of opaque words and the
batched pack/unpack sweep as the benchmark issues it."""
import numpy as np
import torch

SIGNED = {1: np.int8, 2: np.int16, 4: np.int32, 8: np.int64}
UNSIGNED = {1: np.uint8, 2: np.uint16, 4: np.uint32, 8: np.uint64}


def to_dev(arr: np.ndarray) -> torch.Tensor:
    """Upload words bit-exactly (as the same-width signed torch dtype; int32
    tables stay int32)."""
    a = np.ascontiguousarray(arr)
    return torch.from_numpy(a.view(SIGNED[a.itemsize])).cuda()


def to_host(t: torch.Tensor) -> np.ndarray:
    """Download a device tensor as unsigned words of the same width."""
    ints = {1: torch.int8, 2: torch.int16, 4: torch.int32, 8: torch.int64}
    t = t.detach().contiguous()
    a = t.view(ints[t.element_size()]).cpu().numpy()
    return a.view(UNSIGNED[a.itemsize])


def say(msg: str) -> None:
    print(msg, flush=True)
