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


def rel_l2(got, want, zero_ok=False):
    """Relative L2 error of `got` against `want`.  An identically zero
    reference would make the comparison vacuous, so it fails unless the
    caller expects that case (`zero_ok`: then 0 if `got` is exactly zero too,
    else inf)."""
    got = np.asarray(got, dtype=np.float64)
    want = np.asarray(want, dtype=np.float64)
    den = np.linalg.norm(want)
    num = np.linalg.norm(got - want)
    if den == 0.0:
        assert zero_ok, "the reference is identically zero: the comparison would be vacuous"
        return 0.0 if num == 0.0 else np.inf
    return num / den


def tile_columns(D, tile, rng, edge_every=16):
    """Columns that touch every `tile`-wide column tile of a D-wide row: one
    random column inside each tile, the first and last column of every
    `edge_every`-th tile, and the last 16 columns."""
    ntiles = (D + tile - 1) // tile
    starts = np.arange(ntiles, dtype=np.int64) * tile
    widths = np.minimum(tile, D - starts)
    cols = [starts + (rng.random(ntiles) * widths).astype(np.int64)]
    cols.append(starts[::edge_every])
    cols.append(starts[::edge_every] + widths[::edge_every] - 1)
    cols.append(np.arange(max(D - 16, 0), D, dtype=np.int64))
    cols = np.unique(np.concatenate(cols))
    assert np.array_equal(np.unique(cols // tile), np.arange(ntiles))
    return cols
