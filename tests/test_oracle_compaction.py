"""Oracle pins for sequence compaction after pruning (App. H "Index map and
physical token accounting"): the index map iota deletes the visual positions
that were not kept and preserves the order of every retained position; the
boundary sequence takes the transported states at the retained visual
positions; prefix caches are gathered at the same original indices."""
import numpy as np
import pytest

from oracle import gmc_oracle as O


def test_hand_worked_index_map():
    # L = 8, visual tokens at positions 2..5, visual tokens 1 and 3 kept:
    # positions 2 and 4 are deleted, the rest close up in order
    iota, keep = O.index_map(8, 2, 4, [1, 3])
    assert keep.tolist() == [0, 1, 3, 5, 6, 7]
    assert iota.tolist() == [0, 1, -1, 2, -1, 3, 4, 5]


@pytest.mark.parametrize("seed", range(6))
def test_index_map_against_deletion(seed):
    rng = np.random.default_rng(seed)
    n = int(rng.integers(1, 40))
    k = int(rng.integers(1, n + 1))
    before, after = int(rng.integers(0, 9)), int(rng.integers(0, 9))
    seq = before + n + after
    kept = np.sort(rng.choice(n, size=k, replace=False))
    iota, keep = O.index_map(seq, before, n, kept)
    deleted = np.setdiff1d(np.arange(n), kept) + before
    assert np.array_equal(keep, np.delete(np.arange(seq), deleted))
    assert keep.size == seq - n + k and np.all(np.diff(keep) > 0)
    assert np.array_equal(iota[keep], np.arange(keep.size))
    assert np.all(iota[deleted] == -1)
    assert np.array_equal(iota[:before], np.arange(before))                       # prefix unmoved
    assert np.array_equal(iota[before + n:], np.arange(before + n, seq) - (n - k))  # suffix shifted


def test_index_map_identity_and_single():
    iota, keep = O.index_map(10, 3, 5, range(5))
    assert np.array_equal(keep, np.arange(10)) and np.array_equal(iota, np.arange(10))
    iota, keep = O.index_map(10, 0, 10, [7])
    assert keep.tolist() == [7] and iota[7] == 0 and np.sum(iota >= 0) == 1


def test_compact_sequence_rows_and_positions():
    rng = np.random.default_rng(3)
    before, n, after, d = 3, 9, 4, 5
    seq = before + n + after
    rows = rng.standard_normal((seq, d))
    pos = rng.integers(0, 50, size=(seq, 3))
    kept = np.array([0, 4, 8])
    vis = rng.standard_normal((3, d))
    iota, keep, out, opos = O.compact_sequence(rows, vis, pos, before, n, kept)
    assert out.shape == (seq - n + 3, d)
    assert np.array_equal(out[:before], rows[:before])                 # text keeps its states
    assert np.array_equal(out[before:before + 3], vis)                 # kept visual -> transported
    assert np.array_equal(out[before + 3:], rows[before + n:])
    assert np.array_equal(opos, pos[keep])                              # original ids retained
    assert np.array_equal(opos[before:before + 3], pos[before + kept])


def test_gather_cache_by_original_indices():
    rng = np.random.default_rng(4)
    cache = rng.standard_normal((2, 3, 11, 4))    # [layer][head][seq][dh]
    keep = np.array([0, 2, 3, 7, 10])
    got = O.gather_cache(cache, keep)
    for layer in range(2):
        for h in range(3):
            for j, i in enumerate(keep):
                assert np.array_equal(got[layer, h, j], cache[layer, h, i])
