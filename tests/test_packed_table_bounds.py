"""Sizing of the packed-row chunk table (CPU only).

With a device seq_idx (or host offsets) the fused kernels cut every sequence
of a packed row into chunks of its own, from its first token on (the last
one partial).  The workspace holds that table, the Gram / B^T buffers and
the flags for at most ceil(T/Q) + nseq - 1 chunks (and at most T), and a
state ring for the sequences longer than one chunk, at most min(nseq,
ceil(T/Q)) of them.  These tests check those bounds on random and extreme
partitions of a row, and that the workspace query covers the packed layout.
"""
import math

import numpy as np
import pytest

from paper_2405_21060_amd import ssd

Q = 256


def table(lens):
    """The chunk table the device builds, as (first token, length, sequence)."""
    out, t = [], 0
    for s, n in enumerate(lens):
        for k in range(math.ceil(n / Q)):
            out.append((t + k * Q, min(Q, n - k * Q), s))
        t += n
    return out


def check_bounds(lens):
    T, nseq = sum(lens), len(lens)
    nC = math.ceil(T / Q)
    tab = table(lens)
    assert len(tab) <= min(nC + nseq - 1, T)
    multi = sum(1 for n in lens if n > Q)
    assert multi <= min(nseq, nC)
    # every entry inside the row, no chunk holds two sequences, all tokens covered once
    covered = np.zeros(T, dtype=np.int64)
    for t0, L, s in tab:
        assert 1 <= L <= Q and 0 <= t0 and t0 + L <= T
        covered[t0:t0 + L] += 1
    assert np.all(covered == 1)


@pytest.mark.parametrize("seed", range(20))
def test_random_partitions(seed):
    rng = np.random.default_rng(seed)
    hi = [3, 40, 300, 700, 5000][seed % 5]
    lens = rng.integers(1, hi, rng.integers(1, 400)).tolist()
    check_bounds(lens)


@pytest.mark.parametrize("lens", [
    [1] * 1000,                     # one-token sequences: T chunks
    [Q + 1] * 50,                   # every sequence just over a chunk: the bound is reached
    [1, Q] * 30 + [5 * Q],          # chunk-length sequences behind one-token ones
    [65536],                        # one sequence
    [Q] * 64,                       # sequences on the chunk grid
])
def test_extreme_partitions(lens):
    check_bounds(lens)


def test_bound_is_reached():
    # sequences of Q + 1 tokens: 2 chunks each, ceil(T/Q) + nseq - 1 in all
    lens = [Q + 1] * 50
    T = sum(lens)
    assert len(table(lens)) == math.ceil(T / Q) + len(lens) - 1


def test_workspace_covers_the_packed_layout():
    ssd.load_library()

    def ws(nseq, T=32768):
        return ssd.ssd_workspace_bytes(ssd.make_problem(1, T, 64, 64, 128, 8, 256, ssd.SSD_DTYPE_BF16, nseq))

    plain = ws(0)
    # more sequences: more table entries and ring rows, so never less workspace
    sizes = [ws(n) for n in (1, 17, 500, 5000)]
    assert all(a <= b for a, b in zip(sizes, sizes[1:]))
    assert sizes[-1] > plain
    # nseq beyond T is invalid for a packed row and adds nothing
    assert ws(40000, T=32768) == plain


def depth_order(lens):
    """The order in which the chunk kernel takes the table's entries when a
    row holds several sequences: by each entry's index within its sequence
    (every sequence's first chunk, then every second chunk, ...)."""
    tab = table(lens)
    starts = np.concatenate([[0], np.cumsum(lens)])
    depth = [(t0 - starts[s]) // Q for t0, _, s in tab]
    return sorted(range(len(tab)), key=lambda e: depth[e]), tab


@pytest.mark.parametrize("seed", range(10))
def test_depth_order_follows_every_chain(seed):
    """A permutation of the table in which every chunk comes after the chunk
    before it in its sequence (what keeps the persistent kernel free of
    deadlock), whatever the order among the entries of one index."""
    rng = np.random.default_rng(100 + seed)
    lens = rng.integers(1, [300, 2000, 5000][seed % 3], rng.integers(2, 60)).tolist()
    order, tab = depth_order(lens)
    assert sorted(order) == list(range(len(tab)))
    pos = {e: i for i, e in enumerate(order)}
    for e in range(1, len(tab)):
        if tab[e][2] == tab[e - 1][2]:   # the same sequence: e - 1 is the chunk before e
            assert pos[e - 1] < pos[e]
    # the first entries taken are the sequences' first chunks, one per sequence
    assert [tab[e][2] for e in order[:len(lens)]] == list(range(len(lens)))
