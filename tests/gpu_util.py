"""Helpers for the GPU parity tests: tensor conversion and error reporting."""
import numpy as np
import torch


def np64(t):
    """Exact float64 copy of a (GPU or CPU) tensor."""
    return t.detach().float().cpu().numpy().astype(np.float64)


def max_err(got, ref):
    return float(np.max(np.abs(np64(got) - np.asarray(ref, dtype=np.float64)))) if np.size(ref) else 0.0


def dev(*ts):
    out = tuple(None if t is None else t.cuda() for t in ts)
    return out if len(out) > 1 else out[0]


def log(msg):
    print(msg, flush=True)
