"""Helpers shared by the GPU tests (no method arithmetic here)."""
import sys

import numpy as np
import pytest


def need_gpu():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    return torch.device("cuda:0")


def say(msg):
    """Name the case before a GPU step, so a failure can be attributed."""
    print(f"[gpu] {msg}", flush=True)
    sys.stdout.flush()


def bits(t):
    """Raw bytes of a CPU tensor as an unsigned numpy array (bit-exact compare)."""
    import torch
    a = t.detach().cpu().contiguous()
    if a.element_size() == 2:
        return a.view(torch.int16).numpy().view(np.uint16)
    if a.element_size() == 4:
        return a.view(torch.int32).numpy().view(np.uint32)
    if a.element_size() == 8:
        return a.view(torch.int64).numpy().view(np.uint64)
    return a.view(torch.uint8).numpy()
