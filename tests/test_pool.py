"""Page pool (the K/V lifecycle of a fork) on the host: reference counts, fork / reserve / drop /
promote, and what every live sequence reads through its page table (CPU only).

The pool's contents are simulated on the host: every position a sequence owns is tagged with
(context id, position), written through the layout the kernels use (prefix position p at index
p // 16, suffix position j at ceil(Lp / 16) + j // 16; dense after a promote).  After every
operation each live row must read its own context back, so a page given to two writers, or freed
while still read, shows up as a wrong tag."""
import numpy as np
import pytest

P = 16


@pytest.fixture(scope="module")
def fa():
    from paper_2608_13667_amd import forkattn
    return forkattn


class World:
    def __init__(self, fa, n_pages, rows, max_pages):
        self.fa, self.pool = fa, fa.Pool(n_pages)
        self.n_pages, self.max_pages = n_pages, max_pages
        self.table = np.full((rows, max_pages), -1, np.int32)
        self.content = np.full((n_pages, P), -1, np.int64)  # tag per (page, slot)
        self.rows = {}   # row -> [prefix_len, expected tags (prefix then suffix)]
        self.next_ctx = 1

    def tag(self, ctx, pos):
        return ctx * 100000 + pos

    def where(self, r, q):
        lp = self.rows[r][0]
        if q < lp:
            return self.table[r, q // P], q % P
        j = q - lp
        return self.table[r, -(-lp // P) + j // P], j % P

    def check(self):
        held = np.zeros(self.n_pages, np.int64)
        for r in range(self.table.shape[0]):
            for pg in self.table[r]:
                if pg >= 0:
                    held[pg] += 1
        for pg in range(self.n_pages):
            assert self.pool.refcount(pg) == held[pg], (pg, self.pool.refcount(pg), held[pg])
        assert self.pool.free_pages() == int((held == 0).sum())
        for r, (lp, tags) in self.rows.items():
            got = [self.content[self.where(r, q)] for q in range(len(tags))]
            assert got == tags, f"row {r} reads a wrong context"

    def free_rows(self):
        return [r for r in range(self.table.shape[0]) if r not in self.rows]

    def new_snapshot(self, lp, rows):
        ids = self.pool.alloc(-(-lp // P))
        ctx = self.next_ctx
        self.next_ctx += 1
        tags = [self.tag(ctx, q) for q in range(lp)]
        for q in range(lp):
            self.content[ids[q // P], q % P] = tags[q]
        self.fork(ids, lp, tags, rows)
        self.pool.release(ids)  # the rows hold the snapshot now

    def fork(self, ids, lp, tags, rows):
        for r in rows:
            self.pool.fork(ids, self.table, r, 1)
            self.rows[r] = [lp, list(tags)]

    def append(self, r):
        lp, tags = self.rows[r]
        j = len(tags) - lp
        self.pool.reserve(self.table, r, lp, j + 1)
        tags.append(self.tag(self.next_ctx, 0))
        self.next_ctx += 1
        self.content[self.where(r, lp + j)] = tags[-1]

    def drop(self, r):
        self.pool.drop(self.table, r)
        del self.rows[r]

    def promote(self, r, fork_rows):
        lp, tags = self.rows[r]
        dense, frm = self.pool.promote(self.table, r, lp, len(tags) - lp)
        del self.rows[r]
        assert frm == (lp // P) * P and len(dense) == -(-len(tags) // P)
        for q in range(frm, len(tags)):  # the scatter, from the gathered copy
            self.content[dense[q // P], q % P] = tags[q]
        self.fork(dense, len(tags), tags, fork_rows)
        self.pool.release(dense)


@pytest.mark.parametrize("seed", [1, 2, 3, 4])
def test_pool_lifecycle_random(fa, seed):
    rng = np.random.default_rng(seed)
    w = World(fa, n_pages=48, rows=10, max_pages=14)
    for _ in range(400):
        op = rng.integers(0, 10)
        live = sorted(w.rows)
        try:
            if op == 0 and len(w.free_rows()) >= 1:
                k = int(rng.integers(1, min(5, len(w.free_rows())) + 1))
                w.new_snapshot(int(rng.integers(0, 90)), list(rng.choice(w.free_rows(), k, replace=False)))
            elif op <= 5 and live:
                w.append(int(rng.choice(live)))
            elif op <= 7 and live:
                w.drop(int(rng.choice(live)))
            elif op <= 9 and live:
                r = int(rng.choice(live))
                rest = [x for x in w.free_rows() if x != r] + [r]
                k = int(rng.integers(0, min(4, len(rest)) + 1))
                w.promote(r, list(rng.choice(rest, k, replace=False)) if k else [])
        except fa.FkaError as e:
            assert e.status in (-4, -1), e  # no room (pages or max_pages): nothing changed
        w.check()
    for r in list(w.rows):
        w.drop(r)
    w.check()
    assert w.pool.free_pages() == 48


def test_fork_turn_cycle(fa):
    """Fork 5 sequences off a 40-token snapshot, decode 20 tokens each, harvest (drop the four
    branches), promote the main sequence to the next snapshot and fork again."""
    w = World(fa, n_pages=64, rows=10, max_pages=8)
    w.new_snapshot(40, [0, 1, 2, 3, 4])
    shared_last = w.table[0, 2]
    assert w.pool.refcount(shared_last) == 5  # the partly filled prefix page, read by all five
    for _ in range(20):
        for r in range(5):
            w.append(r)
    w.check()
    assert w.pool.free_pages() == 64 - 3 - 5 * 2
    for r in (1, 2, 3, 4):
        w.drop(r)
    assert w.pool.refcount(shared_last) == 1
    old = w.table[0].copy()
    w.promote(0, [5, 6, 7, 8, 9])
    w.check()
    # 60 tokens: the two full prefix pages keep their ids, the partial one and the suffix pages
    # are refilled, one suffix page is left over and freed
    assert list(w.table[5, :2]) == list(old[:2]) and w.table[5, 2] == old[2] and w.table[5, 3] == old[3]
    assert w.pool.free_pages() == 64 - 4


def test_errors_change_nothing(fa):
    w = World(fa, n_pages=6, rows=3, max_pages=4)
    w.new_snapshot(20, [0, 1])
    before = ([w.pool.refcount(i) for i in range(6)], w.table.copy())
    with pytest.raises(fa.FkaError) as e:
        w.pool.alloc(5)
    assert e.value.status == -4
    with pytest.raises(fa.FkaError):
        w.pool.reserve(w.table, 0, 20, 16 * 3)  # 2 + 3 pages > max_pages 4
    with pytest.raises(fa.FkaError):
        w.pool.release(np.array([5], np.int32))  # not live
    with pytest.raises(fa.FkaError):
        w.pool.release(np.array([0, 0, 0], np.int32))  # two references only
    with pytest.raises(fa.FkaError):
        w.pool.fork(np.array([0], np.int32), w.table, 1, 1)  # row 1 holds pages
    with pytest.raises(fa.FkaError):
        w.pool.retain(np.array([4], np.int32))
    assert ([w.pool.refcount(i) for i in range(6)], w.table.tolist()) == (before[0], before[1].tolist())
    w.check()
