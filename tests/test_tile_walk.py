"""CPU model of the kernels' chunk-table walk (TileIter in the HIP source): which key tiles each decode wave and
each prefill workgroup processes.  Every visible tile of a request must be processed exactly once, whatever order
the records' positions take in the table (positions, not table indices, decide visibility, so a record placed after
the query may precede visible ones).

The model follows the device code statement by statement: a split owns tiles lo..hi-1 of the request's tiles
(record after record, ceil(len / TK) tiles each); step() moves to the next tile, seek() passes over invisible tiles
one at a time (prefill, sequential walk), and the decode waves start at tile `wave` of the split and move 4 tiles at
a time, passing over invisible tiles 4 at a time (seek_strided), so each wave keeps its own residue class.
"""
import numpy as np
import pytest


class TileIter:
    def __init__(self, recs, tk, split, splits):
        self.recs, self.tk = recs, tk
        nt = [(n + tk - 1) // tk for n, _ in recs]
        ntiles = sum(nt)
        lo = ntiles * split // splits
        hi = ntiles * (split + 1) // splits
        self.left = hi - lo
        self.i, self.j0 = len(recs), 0
        if self.left <= 0:
            return
        acc = 0
        for i, t in enumerate(nt):
            if acc + t > lo:
                self.i, self.j0 = i, (lo - acc) * tk
                break
            acc += t

    def pos(self):
        return self.recs[self.i][1] + self.j0

    def step(self):
        self.left -= 1
        self.j0 += self.tk
        while self.left > 0 and self.j0 >= self.recs[self.i][0]:
            self.i += 1
            self.j0 = 0

    def skip(self, n):
        for _ in range(n):
            if self.left <= 0:
                break
            self.step()

    def seek(self, causal, qmax):
        while self.left > 0:
            if not causal or self.pos() <= qmax:
                return True
            self.step()
        return False

    def seek_strided(self, causal, qmax, stride):
        while self.left > 0:
            if not causal or self.pos() <= qmax:
                return True
            self.skip(stride)
        return False


def decode_tiles(recs, q_pos, splits, causal=True, strided=True, tk=32, waves=4):
    """(record, j0) of every tile the decode waves process, in any order."""
    done = []
    for split in range(splits):
        for wave in range(waves):
            it = TileIter(recs, tk, split, splits)
            it.skip(wave)
            have = it.seek_strided(causal, q_pos, waves) if strided else it.seek(causal, q_pos)
            while have:
                done.append((it.i, it.j0))
                it.skip(waves)
                have = it.seek_strided(causal, q_pos, waves) if strided else it.seek(causal, q_pos)
    return done


def prefill_tiles(recs, q_max, splits, causal=True, tk=64):
    done = []
    for split in range(splits):
        it = TileIter(recs, tk, split, splits)
        have = it.seek(causal, q_max)
        while have:
            done.append((it.i, it.j0))
            it.step()
            have = it.seek(causal, q_max)
    return done


def visible_tiles(recs, q_pos, causal, tk):
    return sorted((i, j0) for i, (n, p) in enumerate(recs) for j0 in range(0, n, tk) if not causal or p + j0 <= q_pos)


def test_reviewed_counterexample_double_counts_with_plain_seek():
    """A record after the query placed before the visible one: with a per-wave seek of one tile at a time the four
    waves converge on the same tiles (tiles 3, 7, 11, 15 four times each, the other twelve never); the strided seek
    processes each visible tile once."""
    recs = [(70, 1000), (500, 0)]
    old = decode_tiles(recs, 600, 1, strided=False)
    assert sorted(old) != visible_tiles(recs, 600, True, 32)
    assert max(old.count(t) for t in set(old)) == 4
    assert sorted(decode_tiles(recs, 600, 1)) == visible_tiles(recs, 600, True, 32)
    recs = [(64, 0), (100, 900), (512, 64)]
    assert sorted(decode_tiles(recs, 700, 3)) == visible_tiles(recs, 700, True, 32)


@pytest.mark.parametrize("seed", range(40))
def test_every_visible_tile_once_random_tables(seed):
    rng = np.random.default_rng(seed)
    n = int(rng.integers(1, 30))
    recs = [(int(rng.integers(1, 300)), int(rng.integers(0, 5000))) for _ in range(n)]
    q_pos = int(rng.integers(0, 5500))
    for causal in (True, False):
        for splits in (1, 2, 3, 7):
            got = decode_tiles(recs, q_pos, splits, causal)
            assert sorted(got) == visible_tiles(recs, q_pos, causal, 32), (seed, causal, splits)
            got = prefill_tiles(recs, q_pos, splits, causal)
            assert sorted(got) == visible_tiles(recs, q_pos, causal, 64), (seed, causal, splits)
