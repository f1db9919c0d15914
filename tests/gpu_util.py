"""Helpers shared by the GPU parity tests (marshalling only: no estimator arithmetic)."""
import sys

import numpy as np
import torch

import workloads as wl

DEV = "cuda:0"


def log(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def upload_meta(meta):
    return {
        "offsets": torch.from_numpy(meta.offsets).to(DEV),
        "rewards": torch.from_numpy(meta.rewards).to(DEV),
        "p": torch.from_numpy(meta.p).to(DEV),
    }


def scores_to_host(t):
    """Device scores -> numpy float32, or uint16 bf16 bit patterns."""
    t = t.detach().cpu().contiguous()
    if t.dtype == torch.bfloat16:
        return t.view(torch.int16).numpy().view(np.uint16)
    return t.numpy()


def scores_to_device(arr, w):
    if w.dtype == wl.F32:
        return torch.from_numpy(np.ascontiguousarray(arr)).to(DEV)
    return torch.from_numpy(np.ascontiguousarray(arr).view(np.int16)).to(DEV).view(torch.bfloat16)


def rel_l2(got, want):
    got = np.asarray(got, dtype=np.float64)
    want = np.asarray(want, dtype=np.float64)
    den = np.linalg.norm(want)
    num = np.linalg.norm(got - want)
    if den == 0.0:
        return 0.0 if num == 0.0 else np.inf
    return num / den
