"""Helpers shared by the GPU tests: device copies of numpy inputs and a
progress line flushed before each GPU step (so a failing case is named even
if the process dies)."""
import sys

import numpy as np
import torch


def say(*parts):
    print("[gpu-step]", *parts, flush=True)
    sys.stdout.flush()


def dev(a):
    if a is None:
        return None
    a = np.ascontiguousarray(a)
    if a.dtype == np.uint16:
        a = a.view(np.int16)
    return torch.from_numpy(a).to("cuda", non_blocking=False)


def host(t):
    torch.cuda.synchronize()
    return t.cpu().numpy()
