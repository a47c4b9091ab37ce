"""Helpers shared by the GPU tests: move seeded bf16 inputs to the device and
compare device outputs with the fp64 oracle."""

import sys

import numpy as np
import torch

from oracle import bf16_bits_to_f64

# Parity bar for bf16 inputs and outputs against the fp64 oracle.
MAX_ABS = 2e-2
MEAN_ABS = 2e-3


def say(msg: str) -> None:
    """Name the GPU step before it runs (flushed, so a fault still shows it)."""
    print(f"[gpu] {msg}", flush=True)
    sys.stdout.flush()


def to_dev(bits: np.ndarray) -> torch.Tensor:
    return torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).view(torch.bfloat16).cuda()


def dev_inputs(inp):
    q, k, v = to_dev(inp.q), to_dev(inp.k), to_dev(inp.v)
    cu = None if inp.cu_seqlens_k is None else torch.from_numpy(inp.cu_seqlens_k).cuda()
    return q, k, v, cu


def to_f64(t: torch.Tensor) -> np.ndarray:
    return bf16_bits_to_f64(t.detach().cpu().view(torch.int16).numpy().view(np.uint16))


def errors(gpu: np.ndarray, ref: np.ndarray):
    d = np.abs(gpu - ref)
    return float(d.max()) if d.size else 0.0, float(d.mean()) if d.size else 0.0


def assert_parity(gpu_out: torch.Tensor, ref: np.ndarray, what: str = "") -> None:
    g = to_f64(gpu_out)
    assert np.all(np.isfinite(g)), f"{what}: non-finite output"
    mx, mean = errors(g, ref)
    assert mx <= MAX_ABS and mean <= MEAN_ABS, f"{what}: max-abs {mx:.3e} mean-abs {mean:.3e}"


def fit_waves(p):
    """Keep an edited plan's wave count valid: two waves only with K/V through
    registers (kv_fetch 0 or 1), one V slice and the merge in a second
    launch; four otherwise (sharing CUs, as four-wave plans do)."""
    if p.group_waves == 2 and (p.kv_fetch == 2 or p.v_slices != 1 or p.combine != 0):
        p.group_waves, p.wg_per_cu = 4, 0
    return p
