"""The paper's sequence-aware split rule, written from its prose (Section 4),
and the evolved single-batch setting its search found (Section 3, Fig. 1).

TEST INFRASTRUCTURE ONLY.  It pins the planner's PAPER and EVOLVED policy
modes.

The rule works on two quantities: the number of key blocks of the sequence
(blocks of 128 keys on the paper's stack, so L_K <= 384 is at most 3 blocks
and L_K = 512 is 4 blocks; Section 4.2) and the aggregate work-tile count,
which for a single query reduces to Batch * H_KV (Section 4).

  * three blocks or fewer: keep one split (Guard 1);
  * four blocks with at least four tiles: keep one split (Guard 2);
  * four blocks with fewer than four tiles: three splits (the low-tile
    override the paper demonstrates);
  * more than four blocks: the rule does not apply, and the stack's own
    long-context choice is used (the paper does not define it).
"""

from __future__ import annotations

from typing import Optional


def paper_split_policy(L_K: int, B: int, H_KV: int, block_keys: int = 128) -> Optional[int]:
    """num_splits chosen by the paper's rule, or None when L_K exceeds four
    blocks and the rule defers to the long-context path."""
    if L_K <= 0 or B <= 0 or H_KV <= 0:
        raise ValueError("L_K, B and H_KV must be positive")
    blocks = -(-L_K // block_keys)
    tiles = B * H_KV
    if blocks <= 3:
        return 1
    if blocks == 4:
        return 1 if tiles >= 4 else 3
    return None


def evolved_split_policy(L_K: int, B: int) -> Optional[int]:
    """num_splits of the evolved heuristic fragment (Section 3, Fig. 1): for a
    single sequence, twelve splits, or sixteen below 256 keys, with GQA
    packing on and no reserved compute units.  The fragment covers batch 1
    only; None for larger batches (the stack's own choice applies)."""
    if L_K <= 0 or B <= 0:
        raise ValueError("L_K and B must be positive")
    if B != 1:
        return None
    return 16 if L_K < 256 else 12
