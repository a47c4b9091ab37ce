"""Seeded synthetic inputs for single-query (L_Q = 1) decode attention.

This module is shared by the fp64 oracle tests, the GPU parity tests and the
benchmark.  It holds none of the attention arithmetic: it only draws seeded
normal variates and rounds them to bf16 bit patterns, so that the oracle and
the HIP path see exactly the same input bits.

Workloads follow the shapes the paper measures (shape tuple
(Batch, L_Q, L_K, H_Q, H_KV, D), bf16; Section 5.1 and Table 1) plus the
MI355X workload set built around them:

  1  MQA decode            B=1,  H_Q=8,  H_KV=1, L_K=128
  2  Llama-3.1-70B GQA     B=1,  H_Q=64, H_KV=8, L_K in {128,256,384,512}
  3  pure-MQA low-tile     B in {1,2,4} x L_K in {64,128,256,512}, H_Q=32, H_KV=1
  4  varlen batched GQA    B=16, H_Q=32, H_KV=4, L_b ~ U[32,512] (cu_seqlens)
  5  high-load             B=32, H_Q=64, H_KV=8, L_K=8192

Recipe: NumPy PCG64 with seed = 1000 * config_id + shape_idx, draw order
(varlen lengths) -> Q -> K -> V, each standard normal in float32, rounded to
bf16 by round-to-nearest-even.  head_dim is 128 throughout.
"""

from __future__ import annotations

from dataclasses import dataclass, field
from typing import List, Optional, Sequence

import numpy as np

HEAD_DIM = 128


def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round float32 values to bf16 (round-to-nearest-even); return uint16 bits.

    Finite inputs only (the generators never produce NaN or Inf)."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32).astype(np.uint64)
    lsb = (u >> np.uint64(16)) & np.uint64(1)
    r = (u + np.uint64(0x7FFF) + lsb) >> np.uint64(16)
    return r.astype(np.uint16)


@dataclass(frozen=True)
class Shape:
    """One decode-attention problem size (L_Q = 1)."""

    config_id: int
    shape_idx: int
    B: int
    H_Q: int
    H_KV: int
    L_K: int                      # fixed length, or max length when varlen
    D: int = HEAD_DIM
    varlen: bool = False
    name: str = ""

    @property
    def seed(self) -> int:
        return 1000 * self.config_id + self.shape_idx

    @property
    def group(self) -> int:
        return self.H_Q // self.H_KV


@dataclass
class Inputs:
    """bf16 bit patterns (uint16) of one problem, laid out as the C-ABI expects.

    q:  [B, H_Q, D]
    k,v: [B, L_K, H_KV, D] (fixed) or [sum L_b, H_KV, D] (varlen)
    cu_seqlens_k: None (fixed) or int32 [B+1] prefix sums of the lengths
    lengths: int64 [B], the per-sequence key counts in either layout
    """

    shape: Shape
    q: np.ndarray
    k: np.ndarray
    v: np.ndarray
    lengths: np.ndarray
    cu_seqlens_k: Optional[np.ndarray] = None
    extra: dict = field(default_factory=dict)

    @property
    def total_keys(self) -> int:
        return int(self.lengths.sum())


def _normal_bf16(rng: np.random.Generator, shape: Sequence[int], chunk_elems: int = 1 << 24) -> np.ndarray:
    """Draw float32 N(0,1) of `shape` from `rng` and round to bf16 bits.

    Drawn in consecutive chunks so the float32 staging stays small for the
    1 GiB high-load KV cache; the stream of variates is the same as a single
    draw of the whole array."""
    n = int(np.prod(shape))
    out = np.empty(n, dtype=np.uint16)
    pos = 0
    while pos < n:
        m = min(chunk_elems, n - pos)
        out[pos:pos + m] = f32_to_bf16_bits(rng.standard_normal(m, dtype=np.float32))
        pos += m
    return out.reshape(shape)


def make_inputs(shape: Shape, seed: Optional[int] = None,
                lengths: Optional[Sequence[int]] = None) -> Inputs:
    """Draw the inputs of `shape` from seed (default: the shape's own seed).

    For varlen shapes the per-sequence lengths are drawn first from the same
    stream as U[32, L_K] inclusive, unless `lengths` is given."""
    rng = np.random.default_rng(shape.seed if seed is None else seed)
    B, H_Q, H_KV, D = shape.B, shape.H_Q, shape.H_KV, shape.D
    if shape.varlen:
        if lengths is None:
            lens = rng.integers(32, shape.L_K + 1, size=B).astype(np.int64)
        else:
            lens = np.asarray(lengths, dtype=np.int64)
            assert lens.shape == (B,)
        cu = np.zeros(B + 1, dtype=np.int32)
        cu[1:] = np.cumsum(lens)
        q = _normal_bf16(rng, (B, H_Q, D))
        k = _normal_bf16(rng, (int(cu[-1]), H_KV, D))
        v = _normal_bf16(rng, (int(cu[-1]), H_KV, D))
        return Inputs(shape, q, k, v, lens, cu)
    lens = np.full(B, shape.L_K, dtype=np.int64)
    q = _normal_bf16(rng, (B, H_Q, D))
    k = _normal_bf16(rng, (B, shape.L_K, H_KV, D))
    v = _normal_bf16(rng, (B, shape.L_K, H_KV, D))
    return Inputs(shape, q, k, v, lens, None)


@dataclass
class PagedInputs:
    """The keys of an Inputs scattered into a pool of fixed-size pages.

    k_cache, v_cache: uint16 bf16 bits [num_pages, page_size, H_KV, D]
    block_table: int32 [B, max_pages]; key j of sequence b sits in page
        block_table[b, j // page_size], row j % page_size
    seq_lens: int32 [B]
    Rows and pages that hold no key of any sequence, and table entries past a
    sequence's last page, hold seeded noise (valid page ids of other
    sequences' pages), so a kernel that reads them gives a wrong answer."""

    k_cache: np.ndarray
    v_cache: np.ndarray
    block_table: np.ndarray
    seq_lens: np.ndarray
    page_size: int

    @property
    def num_pages(self) -> int:
        return int(self.k_cache.shape[0])

    @property
    def max_pages(self) -> int:
        return int(self.block_table.shape[1])


def sequence_rows(inp: Inputs, b: int, which: str = "k") -> np.ndarray:
    """Sequence b's key (or value) rows [L_b, H_KV, D] in either layout."""
    x = inp.k if which == "k" else inp.v
    if inp.cu_seqlens_k is None:
        return x[b]
    return x[int(inp.cu_seqlens_k[b]):int(inp.cu_seqlens_k[b + 1])]


def paged_layout(inp: Inputs, page_size: int, seed: int, spare_pages: int = 3,
                 max_pages: Optional[int] = None) -> PagedInputs:
    """Scatter the keys and values of `inp` into pages in a seeded random order.

    Draw order from PCG64(seed): K noise, V noise, page permutation, noise
    table entries.  Pure data movement: no attention arithmetic."""
    rng = np.random.default_rng(seed)
    B, H_KV, D = inp.shape.B, inp.shape.H_KV, inp.shape.D
    need = [-(-int(L) // page_size) for L in inp.lengths]
    mp = max(max(need, default=0), 1) if max_pages is None else max_pages
    assert mp >= max(need, default=0)
    n_pages = sum(need) + spare_pages
    k_cache = _normal_bf16(rng, (n_pages, page_size, H_KV, D))
    v_cache = _normal_bf16(rng, (n_pages, page_size, H_KV, D))
    order = rng.permutation(n_pages)
    table = rng.integers(0, n_pages, size=(B, mp)).astype(np.int32)
    pos = 0
    for b in range(B):
        kr, vr = sequence_rows(inp, b, "k"), sequence_rows(inp, b, "v")
        for j in range(need[b]):
            pid = int(order[pos])
            pos += 1
            table[b, j] = pid
            rows = slice(j * page_size, min((j + 1) * page_size, kr.shape[0]))
            n = rows.stop - rows.start
            k_cache[pid, :n] = kr[rows]
            v_cache[pid, :n] = vr[rows]
    return PagedInputs(k_cache, v_cache, table, inp.lengths.astype(np.int32), page_size)


def custom_shape(B: int, H_Q: int, H_KV: int, L_K: int, D: int = HEAD_DIM,
                 varlen: bool = False, name: str = "custom") -> Shape:
    """A shape outside the fixed workload set (edge cases, tests)."""
    return Shape(0, 0, B, H_Q, H_KV, L_K, D, varlen, name)


def config_shapes(config_id: int) -> List[Shape]:
    """The shapes of one workload, in shape_idx order."""
    if config_id == 1:
        return [Shape(1, 0, 1, 8, 1, 128, name="mqa_b1_h8_l128")]
    if config_id == 2:
        return [Shape(2, i, 1, 64, 8, L, name=f"llama70b_gqa_b1_l{L}")
                for i, L in enumerate((128, 256, 384, 512))]
    if config_id == 3:
        out = []
        idx = 0
        for B in (1, 2, 4):
            for L in (64, 128, 256, 512):
                out.append(Shape(3, idx, B, 32, 1, L, name=f"mqa32_b{B}_l{L}"))
                idx += 1
        return out
    if config_id == 4:
        return [Shape(4, 0, 16, 32, 4, 512, varlen=True, name="varlen_gqa_b16_h32_kv4")]
    if config_id == 5:
        return [Shape(5, 0, 32, 64, 8, 8192, name="highload_b32_h64_kv8_l8192")]
    raise ValueError(f"unknown config {config_id}")


ALL_CONFIG_IDS = (1, 2, 3, 4, 5)


def all_shapes() -> List[Shape]:
    return [s for c in ALL_CONFIG_IDS for s in config_shapes(c)]


def ragged_batches() -> List[tuple]:
    """Batches of mixed sequence lengths for the per-sequence schedule:
    (name, lengths, H_Q, H_KV).  Lengths are drawn from PCG64 with the
    stated seed; K/V values for timing are drawn separately (any values)."""
    def uniform(seed, B, lo, hi):
        return [int(x) for x in np.random.default_rng(seed).integers(lo, hi + 1, B)]

    def lognormal(seed, B, median, sigma, lo=16, hi=65536):
        x = np.random.default_rng(seed).lognormal(np.log(median), sigma, B)
        return [int(v) for v in np.clip(x, lo, hi)]

    return [
        ("ragged_highload_b32_h64_kv8", uniform(2024, 32, 1024, 16384), 64, 8),
        ("bimodal_b32_h64_kv8", [16384] * 4 + [512] * 28, 64, 8),
        ("one_long_mqa_b8_h8_kv1", [32768] + [256] * 7, 8, 1),
        ("lognormal_mqa_b128_h8_kv1", lognormal(106, 128, 1000, 1.0), 8, 1),
    ]


def schedule_batches(kind: str) -> List[tuple]:
    """Mixed-length batches for measuring the per-sequence schedule's cost
    model: "fit" (the batches its constants were fitted to) or "check"
    (batches drawn afterwards, never fitted).  (name, lengths, H_Q, H_KV)."""
    def U(seed, B, lo, hi):
        return [int(x) for x in np.random.default_rng(seed).integers(lo, hi + 1, B)]

    def LN(seed, B, median, sigma, lo=16, hi=65536):
        return [int(v) for v in np.clip(np.random.default_rng(seed).lognormal(np.log(median), sigma, B), lo, hi)]

    if kind == "fit":
        return [
            ("ragged_b32_gqa", U(1, 32, 1024, 16384), 64, 8),
            ("bimodal_b32_gqa", [16384] * 4 + [512] * 28, 64, 8),
            ("ragged_b64_gqa", U(3, 64, 256, 8192), 64, 8),
            ("ragged_b16_gqa", U(4, 16, 1024, 16384), 64, 8),
            ("ragged_b8_gqa", U(5, 8, 512, 32768), 64, 8),
            ("ragged_b4_gqa", U(6, 4, 256, 4096), 64, 8),
            ("ragged_b32_mqa", U(7, 32, 128, 16384), 8, 1),
            ("ragged_b16_mqa", U(8, 16, 128, 8192), 8, 1),
            ("ragged_b64_mqa", U(9, 64, 1024, 32768), 8, 1),
            ("one_long_mqa", [32768] + [256] * 7, 8, 1),
            ("one_long_gqa", [65536] + [1024] * 15, 64, 8),
            ("two_long_b32", [16384] * 2 + U(10, 30, 64, 1024), 32, 4),
            ("varlen_gqa_b16", U(4000, 16, 32, 512), 32, 4),
            ("ragged_b128_h32", U(11, 128, 32, 2048), 32, 4),
            ("ragged_b32_g16", U(12, 32, 512, 8192), 32, 2),
            ("ragged_b8_h128", U(13, 8, 512, 8192), 128, 2),
            ("geometric_b32", [int(x) for x in np.minimum(32768, 64 * 2 ** np.random.default_rng(14).uniform(0, 9, 32))],
             64, 8),
            ("ragged_b2_mqa", U(15, 2, 1024, 65536), 8, 1),
        ]
    if kind == "check":
        return [
            ("ragged_b32_gqa", U(101, 32, 512, 16384), 64, 8),
            ("lognorm_b64_gqa", LN(102, 64, 2000, 1.0), 64, 8),
            ("lognorm_b16_mqa", LN(103, 16, 4000, 1.2), 8, 1),
            ("ragged_b48_h32", U(104, 48, 64, 4096), 32, 4),
            ("bimodal_b16", [32768] * 2 + [256] * 14, 64, 8),
            ("one_long_b4", [50000, 300, 300, 300], 8, 1),
            ("ragged_b24_g16", U(105, 24, 256, 12000), 32, 2),
            ("lognorm_b128_mqa", LN(106, 128, 1000, 1.0), 8, 1),
            ("ragged_b6_h128", U(107, 6, 1024, 16384), 128, 2),
            ("lognorm_b32_gqa", LN(108, 32, 8000, 0.6), 64, 8),
            ("short_b64", U(109, 64, 16, 600), 32, 4),
            ("ragged_b12_gqa", U(110, 12, 128, 2048), 64, 8),
            ("equal_b32_gqa", [8192] * 32, 64, 8),
            ("equal_b1_gqa", [512], 64, 8),
        ]
    raise ValueError(kind)


def algorithmic_bytes(B: int, H_Q: int, H_KV: int, total_keys: int, D: int = HEAD_DIM,
                      varlen: bool = False) -> int:
    """Bytes the method must move once: K and V once, Q read, O written (bf16),
    plus the cu_seqlens metadata for the varlen layout."""
    kv = 2 * total_keys * H_KV * D * 2
    qo = 2 * B * H_Q * D * 2
    meta = 4 * (B + 1) if varlen else 0
    return kv + qo + meta
