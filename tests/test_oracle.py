"""Pins for the fp64 oracle (CPU only).

Each check rests on something other than the oracle's own formula: mpmath
brute force without max subtraction, closed forms, invariants of softmax
attention, a library attention routine, and the paper's policy table."""

import json
import os

import mpmath
import numpy as np
import pytest
import torch

from oracle import (bf16_bits_to_f64, combine_partials, decode_attention, even_bounds,
                    evolved_split_policy, paper_split_policy, split_partials)
from oracle.brute import brute_attention
from workloads import config_shapes, custom_shape, f32_to_bf16_bits, make_inputs

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def bf16(x):
    """bf16 bits of x (scalar in, scalar out)."""
    arr = f32_to_bf16_bits(np.atleast_1d(np.asarray(x, dtype=np.float32)))
    return arr[0] if np.ndim(x) == 0 else arr


def rand_bf16(rng, shape, scale=1.0):
    return bf16(rng.standard_normal(shape).astype(np.float32) * scale)


# ---------------------------------------------------------------- brute force

BRUTE_CASES = [
    # B, H_Q, H_KV, L, D, input scale
    (1, 1, 1, 1, 4, 1.0),
    (1, 2, 1, 3, 8, 2.0),
    (2, 4, 2, 5, 8, 1.5),
    (1, 4, 4, 7, 4, 3.0),
    (2, 2, 1, 9, 1, 4.0),
]


@pytest.mark.parametrize("B,H_Q,H_KV,L,D,sc", BRUTE_CASES)
def test_brute_force_fixed(B, H_Q, H_KV, L, D, sc):
    rng = np.random.default_rng(7 + B * 100 + L)
    q = rand_bf16(rng, (B, H_Q, D), sc)
    k = rand_bf16(rng, (B, L, H_KV, D), sc)
    v = rand_bf16(rng, (B, L, H_KV, D))
    O, lse = decode_attention(q, k, v)
    Ob, lseb = brute_attention(q, k, v)
    for b in range(B):
        for h in range(H_Q):
            assert abs(float(lseb[b][h]) - lse[b, h]) <= 1e-13 * max(1.0, abs(lse[b, h]))
            for c in range(D):
                assert abs(float(Ob[b][h][c]) - O[b, h, c]) <= 1e-13


def test_brute_force_d128_scale():
    rng = np.random.default_rng(11)
    B, H_Q, H_KV, L, D = 1, 2, 1, 4, 128
    q = rand_bf16(rng, (B, H_Q, D))
    k = rand_bf16(rng, (B, L, H_KV, D))
    v = rand_bf16(rng, (B, L, H_KV, D))
    for scale in (None, 0.3):
        O, lse = decode_attention(q, k, v, scale=scale)
        Ob, lseb = brute_attention(q, k, v, scale=scale)
        err = max(abs(float(Ob[b][h][c]) - O[b, h, c])
                  for b in range(B) for h in range(H_Q) for c in range(D))
        assert err <= 1e-13


def test_brute_force_varlen_with_empty_sequence():
    rng = np.random.default_rng(12)
    lens = [3, 0, 5]
    cu = np.array([0, 3, 3, 8], dtype=np.int32)
    H_Q, H_KV, D = 4, 2, 8
    q = rand_bf16(rng, (3, H_Q, D), 2.0)
    k = rand_bf16(rng, (8, H_KV, D), 2.0)
    v = rand_bf16(rng, (8, H_KV, D))
    O, lse = decode_attention(q, k, v, lengths=np.array(lens), cu_seqlens=cu)
    Ob, lseb = brute_attention(q, k, v, cu_seqlens=cu)
    for b in range(3):
        for h in range(H_Q):
            if lens[b] == 0:
                assert lse[b, h] == -np.inf and lseb[b][h] == mpmath.mpf("-inf")
                assert np.all(O[b, h] == 0)
                continue
            assert abs(float(lseb[b][h]) - lse[b, h]) <= 1e-13
            for c in range(D):
                assert abs(float(Ob[b][h][c]) - O[b, h, c]) <= 1e-13


# ------------------------------------------------------------- closed forms

def test_single_key_gives_v_exactly():
    rng = np.random.default_rng(1)
    q = rand_bf16(rng, (2, 8, 128))
    k = rand_bf16(rng, (2, 1, 2, 128))
    v = rand_bf16(rng, (2, 1, 2, 128))
    O, lse = decode_attention(q, k, v)
    vf = bf16_bits_to_f64(v)
    for h in range(8):
        np.testing.assert_array_equal(O[:, h, :], vf[:, 0, h // 4, :])


def test_identical_keys_give_mean_v():
    rng = np.random.default_rng(2)
    L = 37
    q = rand_bf16(rng, (1, 4, 128))
    k1 = rand_bf16(rng, (1, 1, 1, 128))
    k = np.repeat(k1, L, axis=1)
    v = rand_bf16(rng, (1, L, 1, 128))
    O, lse = decode_attention(q, k, v)
    mean = bf16_bits_to_f64(v)[0, :, 0, :].mean(axis=0)
    for h in range(4):
        np.testing.assert_allclose(O[0, h], mean, rtol=0, atol=1e-14)


def test_zero_query_gives_mean_v_and_log_length():
    rng = np.random.default_rng(3)
    L = 50
    q = np.zeros((1, 2, 128), dtype=np.uint16)
    k = rand_bf16(rng, (1, L, 1, 128), 5.0)
    v = rand_bf16(rng, (1, L, 1, 128))
    O, lse = decode_attention(q, k, v)
    mean = bf16_bits_to_f64(v)[0, :, 0, :].mean(axis=0)
    np.testing.assert_allclose(O[0, 0], mean, atol=1e-14)
    np.testing.assert_allclose(lse[0], np.log(L), rtol=1e-15)


def test_constant_value_rows_reproduce_the_constant():
    # The softmax weights sum to one: any column of V that is constant over
    # the keys comes back exactly as that constant.
    rng = np.random.default_rng(4)
    L = 300
    q = rand_bf16(rng, (2, 8, 128), 2.0)
    k = rand_bf16(rng, (2, L, 2, 128), 2.0)
    const = rand_bf16(rng, (2, 1, 2, 128))
    v = np.repeat(const, L, axis=1)
    O, _ = decode_attention(q, k, v)
    cf = bf16_bits_to_f64(const)
    for h in range(8):
        np.testing.assert_allclose(O[:, h, :], cf[:, 0, h // 4, :], rtol=1e-14, atol=1e-15)


@pytest.mark.parametrize("alpha,scale", [(1.0, None), (4.0, None), (3.0, 0.5), (64.0, None)])
def test_two_level_weights_closed_form(alpha, scale):
    """One key aligned with q, the others orthogonal to it: scores are
    sigma*a*c for the aligned key and 0 for the rest, so
    O = (e^{s*} v* + sum_{j != *} v_j) / (e^{s*} + L - 1)."""
    rng = np.random.default_rng(5)
    L, D, star = 40, 128, 17
    a = 2.0
    q = np.zeros((1, 1, D), dtype=np.uint16)
    q[0, 0, 0] = bf16(a)
    k = np.zeros((1, L, 1, D), dtype=np.uint16)
    k[0, :, 0, 1:] = rand_bf16(rng, (L, D - 1))       # orthogonal to q
    k[0, star, 0, :] = 0
    k[0, star, 0, 0] = bf16(alpha)
    v = rand_bf16(rng, (1, L, 1, D))
    O, lse = decode_attention(q, k, v, scale=scale)
    sigma = 1 / np.sqrt(D) if scale is None else scale
    s_star = sigma * a * alpha
    vf = bf16_bits_to_f64(v)[0, :, 0, :]
    others = np.delete(vf, star, axis=0).sum(axis=0)
    expect = (np.exp(s_star) * vf[star] + others) / (np.exp(s_star) + L - 1)
    np.testing.assert_allclose(O[0, 0], expect, rtol=1e-13, atol=1e-14)
    np.testing.assert_allclose(lse[0, 0], np.log(np.exp(s_star) + L - 1), rtol=1e-14)


def test_large_alignment_selects_the_aligned_value():
    L, D, star = 16, 128, 5
    q = np.zeros((1, 1, D), dtype=np.uint16)
    q[0, 0, 0] = bf16(64.0)
    k = np.zeros((1, L, 1, D), dtype=np.uint16)
    k[0, star, 0, 0] = bf16(64.0)      # score 64*64/sqrt(128) ~ 362
    rng = np.random.default_rng(6)
    v = rand_bf16(rng, (1, L, 1, D))
    O, _ = decode_attention(q, k, v)
    np.testing.assert_allclose(O[0, 0], bf16_bits_to_f64(v)[0, star, 0], atol=1e-12)


def test_softmax_shift_invariance_large_scores():
    # Scores of order 1e3 would overflow a naive exp; the oracle must stay
    # finite and agree with the same problem at a small scale shift.
    L, D = 8, 128
    q = np.zeros((1, 1, D), dtype=np.uint16)
    q[0, 0, 0] = bf16(256.0)
    k = np.zeros((1, L, 1, D), dtype=np.uint16)
    k[0, :, 0, 0] = bf16(np.linspace(40, 48, L))
    rng = np.random.default_rng(8)
    v = rand_bf16(rng, (1, L, 1, D))
    O, lse = decode_attention(q, k, v)
    assert np.all(np.isfinite(O)) and np.isfinite(lse).all()
    s = 256.0 * bf16_bits_to_f64(k[0, :, 0, 0]) / np.sqrt(D)
    w = np.exp(s - s.max())
    w /= w.sum()
    np.testing.assert_allclose(O[0, 0], w @ bf16_bits_to_f64(v)[0, :, 0], rtol=1e-12, atol=1e-14)


# ------------------------------------------------------------- the partition

def balanced_partition_ok(cuts, L, s):
    """Whether `cuts` is a balanced partition of L keys into s chunks, as the
    split step defines it (chunks of floor(L/s) or ceil(L/s) keys, in order,
    covering every key once): checked from the definition, not the formula."""
    if len(cuts) != s + 1 or cuts[0] != 0 or cuts[-1] != L:
        return False
    sizes = [cuts[i + 1] - cuts[i] for i in range(s)]
    if min(sizes) < 0 or max(sizes) - min(sizes) > 1:
        return False
    # empty chunks only when there are more chunks than keys
    return L >= s or sizes.count(0) == s - L


def test_even_bounds_worked_examples():
    # chunk i is [floor(iL/s), floor((i+1)L/s)): worked out by hand
    assert even_bounds(10, 3) == [0, 3, 6, 10]
    assert even_bounds(5, 8) == [0, 0, 1, 1, 2, 3, 3, 4, 5]
    assert even_bounds(0, 4) == [0, 0, 0, 0, 0]
    assert even_bounds(7, 1) == [0, 7]
    assert even_bounds(64, 64) == list(range(65))


@pytest.mark.parametrize("L", [0, 1, 2, 5, 31, 32, 45, 127, 512, 1000, 8192])
def test_even_bounds_is_balanced(L):
    for s in range(1, 65):
        cuts = even_bounds(L, s)
        assert balanced_partition_ok(cuts, L, s), (L, s, cuts)
        # exactly L mod s chunks hold one key more than the others
        sizes = np.diff(cuts)
        assert int((sizes == L // s + 1).sum()) == L % s


def test_even_bounds_brute_force_tiny():
    """For tiny L and s, enumerate every non-decreasing cut vector and keep
    the balanced ones; the floor cuts must be among them, and for s <= L
    (no empty chunk) the chunk sizes are the unique multiset {q, q+1}."""
    import itertools
    for L in range(0, 7):
        for s in range(1, 6):
            balanced = [c for c in itertools.combinations_with_replacement(range(L + 1), s - 1)
                        if balanced_partition_ok([0, *c, L], L, s)]
            assert tuple(even_bounds(L, s)[1:-1]) in balanced
            q, r = divmod(L, s)
            assert sorted(np.diff(even_bounds(L, s)).tolist()) == [q] * (s - r) + [q + 1] * r


def test_partition_check_rejects_an_unbalanced_split():
    # a plausible mistake: every key in the last chunk, or cuts off by one
    assert not balanced_partition_ok([0, 0, 0, 10], 10, 3)
    assert not balanced_partition_ok([0, 4, 8, 10], 10, 3)
    assert not balanced_partition_ok([0, 3, 6, 9], 10, 3)
    assert not balanced_partition_ok([0, 0, 2, 2, 5], 5, 4)


# ------------------------------------------------------------- invariants

def test_convex_hull():
    sh = config_shapes(2)[0]
    inp = make_inputs(sh)
    O, _ = decode_attention(inp.q, inp.k, inp.v)
    vf = bf16_bits_to_f64(inp.v)[0]                       # [L, H_KV, D]
    lo, hi = vf.min(axis=0), vf.max(axis=0)               # [H_KV, D]
    for h in range(sh.H_Q):
        assert np.all(O[0, h] >= lo[h // sh.group] - 1e-15)
        assert np.all(O[0, h] <= hi[h // sh.group] + 1e-15)


@pytest.mark.parametrize("s", [1, 2, 3, 4, 7, 8, 16, 33, 64])
def test_split_then_combine_equals_unsplit(s):
    sh = custom_shape(2, 8, 2, 45)
    inp = make_inputs(sh, seed=100 + s)
    O, lse = decode_attention(inp.q, inp.k, inp.v)
    bounds = [even_bounds(45, s)] * 2
    op, mp, lp = split_partials(inp.q, inp.k, inp.v, bounds)
    Oc, lsec = combine_partials(op, mp, lp)
    np.testing.assert_allclose(Oc, O, rtol=0, atol=1e-12)
    np.testing.assert_allclose(lsec, lse, rtol=0, atol=1e-12)
    if s > 45:
        assert (lp == 0).any() and np.isneginf(mp).any()


def test_split_random_cut_points_varlen():
    sh = custom_shape(3, 8, 1, 64, varlen=True)
    inp = make_inputs(sh, seed=9, lengths=[64, 1, 33])
    O, lse = decode_attention(inp.q, inp.k, inp.v, inp.lengths, inp.cu_seqlens_k)
    rng = np.random.default_rng(10)
    for s in (2, 5, 9):
        bounds = []
        for L in inp.lengths:
            cuts = np.sort(rng.integers(0, L + 1, s - 1))
            bounds.append([0] + cuts.tolist() + [int(L)])
        op, mp, lp = split_partials(inp.q, inp.k, inp.v, bounds, inp.lengths, inp.cu_seqlens_k)
        Oc, lsec = combine_partials(op, mp, lp)
        np.testing.assert_allclose(Oc, O, atol=1e-12)
        np.testing.assert_allclose(lsec, lse, atol=1e-12)


def test_combine_edge_cases():
    rng = np.random.default_rng(13)
    o = rng.standard_normal((1, 2, 3, 4))
    m = rng.standard_normal((1, 2, 3))
    l = rng.random((1, 2, 3)) + 0.5
    O, lse = combine_partials(o, m, l)
    np.testing.assert_allclose(O, o[0] / l[0][..., None], rtol=1e-15)
    np.testing.assert_allclose(lse, m[0] + np.log(l[0]), rtol=1e-15)
    # every chunk empty -> O = 0, lse = -inf, no NaN
    Oe, lsee = combine_partials(np.zeros((3, 2, 4)), np.full((3, 2), -np.inf), np.zeros((3, 2)))
    assert np.all(Oe == 0) and np.all(np.isneginf(lsee))
    # chunk order does not matter
    o3 = rng.standard_normal((5, 2, 4))
    m3 = rng.standard_normal((5, 2)) * 10
    l3 = rng.random((5, 2)) + 0.1
    perm = rng.permutation(5)
    Oa, la = combine_partials(o3, m3, l3)
    Ob, lb = combine_partials(o3[perm], m3[perm], l3[perm])
    np.testing.assert_allclose(Oa, Ob, rtol=1e-14)
    np.testing.assert_allclose(la, lb, rtol=1e-14)


def test_varlen_equal_lengths_matches_fixed_layout():
    sh = custom_shape(3, 8, 2, 70)
    inp = make_inputs(sh, seed=14)
    cu = np.array([0, 70, 140, 210], dtype=np.int32)
    kv = inp.k.reshape(210, 2, 128)
    vv = inp.v.reshape(210, 2, 128)
    O1, l1 = decode_attention(inp.q, inp.k, inp.v)
    O2, l2 = decode_attention(inp.q, kv, vv, lengths=np.array([70, 70, 70]), cu_seqlens=cu)
    np.testing.assert_array_equal(O1, O2)
    np.testing.assert_array_equal(l1, l2)


# --------------------------------------------------------- library routine

@pytest.mark.parametrize("cfg", [1, 2, 3])
def test_matches_torch_sdpa_float64(cfg):
    sh = config_shapes(cfg)[0]
    inp = make_inputs(sh)
    O, _ = decode_attention(inp.q, inp.k, inp.v)
    q = torch.from_numpy(bf16_bits_to_f64(inp.q)).unsqueeze(2)              # [B,H,1,D]
    k = torch.from_numpy(bf16_bits_to_f64(inp.k)).permute(0, 2, 1, 3)       # [B,H_KV,L,D]
    v = torch.from_numpy(bf16_bits_to_f64(inp.v)).permute(0, 2, 1, 3)
    k = k.repeat_interleave(sh.group, dim=1).contiguous()
    v = v.repeat_interleave(sh.group, dim=1).contiguous()
    ref = torch.nn.functional.scaled_dot_product_attention(q, k, v)[:, :, 0, :].numpy()
    np.testing.assert_allclose(O, ref, rtol=0, atol=1e-12)


# ------------------------------------------------------------ paper policy

def test_paper_policy_matches_table():
    with open(os.path.join(GOLDEN, "paper_policy.json")) as f:
        table = json.load(f)
    for c in table["cases"]:
        assert paper_split_policy(c["L_K"], c["B"], c["H_KV"], table["block_keys"]) == c["s"], c


def test_evolved_policy_matches_figure():
    with open(os.path.join(GOLDEN, "evolved_policy.json")) as f:
        table = json.load(f)
    for c in table["cases"]:
        assert evolved_split_policy(c["L_K"], c["B"]) == c["s"], c


# ---------------------------------------------------------- input recipe

def test_bf16_rounding_matches_torch():
    rng = np.random.default_rng(15)
    x = np.concatenate([rng.standard_normal(100000).astype(np.float32) * 10,
                        np.array([1.00390625, 1.01171875, -1.00390625, 0.0, -0.0, 3.4e38], np.float32)])
    ours = f32_to_bf16_bits(x)
    ref = torch.from_numpy(x).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    np.testing.assert_array_equal(ours, ref)


def test_inputs_are_seeded_and_chunking_does_not_change_the_stream():
    from workloads import _normal_bf16
    sh = config_shapes(4)[0]
    a, b = make_inputs(sh), make_inputs(sh)
    for x, y in ((a.q, b.q), (a.k, b.k), (a.v, b.v), (a.cu_seqlens_k, b.cu_seqlens_k)):
        np.testing.assert_array_equal(x, y)
    assert a.lengths.min() >= 32 and a.lengths.max() <= 512
    r1 = np.random.default_rng(3)
    r2 = np.random.default_rng(3)
    np.testing.assert_array_equal(_normal_bf16(r1, (1000, 7)), _normal_bf16(r2, (1000, 7), chunk_elems=333))
