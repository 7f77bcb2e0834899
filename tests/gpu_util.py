"""Helpers shared by the GPU tests."""
import sys

import numpy as np
import pytest
import torch


def need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2007_06563_amd import hobflops as hf
    hf.lib()  # fails loudly if the library is missing
    return hf


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def dev(x):
    return torch.from_numpy(np.ascontiguousarray(x)).cuda()


def codes_of(t):
    """int32 tensor of codes -> uint64 numpy."""
    return t.cpu().numpy().view(np.uint32).astype(np.uint64)
