"""Host checks of the seeded input generators (no attention arithmetic)."""

import numpy as np

from workloads import custom_shape, make_inputs, paged_layout, sequence_rows


def gather(pg, b, L, cache):
    rows = [cache[pg.block_table[b, j // pg.page_size], j % pg.page_size] for j in range(L)]
    return np.array(rows).reshape((L,) + cache.shape[2:])


def test_paged_layout_round_trip():
    sh = custom_shape(4, 8, 2, 300, varlen=True)
    inp = make_inputs(sh, seed=5, lengths=[0, 1, 300, 64])
    for page, mp in ((32, None), (64, 12), (96, None)):
        pg = paged_layout(inp, page, seed=9, max_pages=mp)
        assert pg.max_pages == (mp or -(-300 // page))
        for b, L in enumerate(inp.lengths):
            assert np.array_equal(gather(pg, b, int(L), pg.k_cache), sequence_rows(inp, b, "k"))
            assert np.array_equal(gather(pg, b, int(L), pg.v_cache), sequence_rows(inp, b, "v"))
        # every sequence owns distinct pages, and the table holds only valid ids
        owned = [pg.block_table[b, j] for b, L in enumerate(inp.lengths) for j in range(-(-int(L) // page))]
        assert len(set(owned)) == len(owned)
        assert pg.block_table.min() >= 0 and pg.block_table.max() < pg.num_pages


def test_paged_layout_fixed_layout_and_seed():
    sh = custom_shape(2, 8, 1, 128)
    inp = make_inputs(sh, seed=3)
    a = paged_layout(inp, 32, seed=1)
    b = paged_layout(inp, 32, seed=1)
    assert np.array_equal(a.block_table, b.block_table) and np.array_equal(a.k_cache, b.k_cache)
    assert np.array_equal(gather(a, 1, 128, a.k_cache), inp.k[1])
    assert list(a.seq_lens) == [128, 128]


def test_ragged_batches_are_mixed_and_seeded():
    from workloads import ragged_batches
    a, b = ragged_batches(), ragged_batches()
    assert a == b
    names = [x[0] for x in a]
    assert len(set(names)) == len(names)
    for name, lens, H_Q, H_KV in a:
        assert H_Q % H_KV == 0 and len(set(lens)) > 1 and min(lens) >= 1 and max(lens) <= 65536


def test_split_masks_keep_cus_on_every_xcd():
    """Both masks leave CUs on each of the 8 XCDs whether mask bits map to
    XCDs in blocks of 32 or in turn."""
    import pytest
    from paper_2604_00028_amd.streams import split_masks
    for per in (8, 16, 24):
        res, dec = split_masks(256, per)
        bits = lambda w: [i for i in range(256) if (w[i // 32] >> (i % 32)) & 1]  # noqa: E731
        r, d = bits(res), bits(dec)
        assert len(r) == 8 * per and len(d) == 256 - 8 * per and not set(r) & set(d)
        for mapping in (lambda i: i // 32, lambda i: i % 8):
            assert {mapping(i) for i in r} == set(range(8)) and {mapping(i) for i in d} == set(range(8))
    for bad in (0, 4, 32):
        with pytest.raises(ValueError):
            split_masks(256, bad)
