"""Random operation traces over a slice state, for invariant and parity tests.

A ``Cache`` keeps the canonical block tables of a batch (``tables[l][b][j]``,
unified ids, -1 padding; the owner of row b is sequence b) consistent with a
backend while random operations run: sequences grow and finish, blocks migrate
between pools, prefetches run, the lender lends and reclaims.

Backends expose: alloc_blocks(where, owners) -> ids, free_blocks(ids),
lend(n) -> added, migrate(src, dst), prefetch(src, dst), writeback(src, dst),
reclaim(n, tables) -> dict, owners() -> (own_local, own_slice, lim).
Errors are raised as exceptions carrying ``.code``.
"""
import numpy as np

LOCAL, SLICE = 0, 1
STAGING = -2


class OracleBackend:
    validating = True     # rejects invalid id lists (device backends may not)

    def __init__(self, st):
        self.st = st

    def alloc_blocks(self, where, owners):
        return self.st.alloc_blocks(where, owners)

    def free_blocks(self, ids):
        self.st.free_blocks(ids)

    def lend(self, n):
        return self.st.lend(n)

    def migrate(self, src, dst):
        self.st.migrate(src, dst)

    def prefetch(self, src, dst):
        self.st.prefetch(src, dst)

    def writeback(self, src, dst):
        self.st.writeback(src, dst)

    def reclaim(self, n, tables):
        r = self.st.reclaim(n, tables)
        return {k: r[k] for k in ("reclaimed", "moved", "written_back", "victims", "lim")} | {
            "moves": r["moves"]}

    def owners(self):
        return self.st.own_local.copy(), self.st.own_slice.copy(), self.st.lim

    @property
    def n_local(self):
        return self.st.n_local


class Cache:
    def __init__(self, backends, layers, batch, maxblk, rng, write_data=None):
        self.backends = backends
        self.L, self.B, self.maxblk = layers, batch, maxblk
        self.tables = np.full((layers, batch, maxblk), -1, dtype=np.int64)
        self.nb = np.zeros((layers, batch), dtype=np.int64)
        self.rng = rng
        self.write_data = write_data     # callback(u) fills fresh blocks (oracle data)
        self.log = []

    def _all(self, name, *args):
        outs = []
        errs = []
        for be in self.backends:
            try:
                outs.append(getattr(be, name)(*args))
                errs.append(None)
            except Exception as e:        # noqa: BLE001  compare error codes across backends
                outs.append(None)
                errs.append(getattr(e, "code", repr(e)))
        if len(set(map(str, errs))) != 1:
            raise AssertionError(f"{name}{args}: backends disagree on errors: {errs}")
        if errs[0] is not None:
            return None, errs[0]
        for o in outs[1:]:
            _assert_same(outs[0], o, name)
        return outs[0], None

    # ---- operations ------------------------------------------------------------
    def grow(self, l, b, where, k):
        k = int(min(k, self.maxblk - self.nb[l, b]))
        if k <= 0:
            return
        ids, err = self._all("alloc_blocks", where, np.full(k, b))
        self.log.append(("grow", l, b, where, k, err))
        if err is not None:
            return
        j0 = self.nb[l, b]
        self.tables[l, b, j0:j0 + k] = ids
        self.nb[l, b] += k
        if self.write_data is not None:
            for u in ids:
                self.write_data(int(u))

    def finish(self, b):
        ids = self.tables[:, b][self.tables[:, b] >= 0]
        self.log.append(("finish", b, len(ids)))
        if len(ids):
            _, err = self._all("free_blocks", ids)
            assert err is None, err
        self.tables[:, b] = -1
        self.nb[:, b] = 0

    def lend(self, n):
        self.log.append(("lend", n))
        self._all("lend", n)

    def migrate(self, l, b, j, where):
        u = int(self.tables[l, b, j])
        if u < 0:
            return
        new, err = self._all("alloc_blocks", where, [b])
        self.log.append(("migrate", l, b, j, where, err))
        if err is not None:
            return
        _, err = self._all("migrate", [u], [int(new[0])])
        assert err is None, err
        _, err = self._all("free_blocks", [u])
        assert err is None, err
        self.tables[l, b, j] = int(new[0])

    def prefetch_layer(self, l, check=None):
        row = self.tables[l]
        n_local = self.n_local
        src = [int(u) for u in row.reshape(-1) if u >= n_local]
        if not src:
            return
        dst, err = self._all("alloc_blocks", LOCAL, np.full(len(src), STAGING))
        self.log.append(("prefetch", l, len(src), err))
        if err is not None:
            return
        _, err = self._all("prefetch", src, [int(u) for u in dst])
        assert err is None, err
        if check is not None:
            check(src, [int(u) for u in dst])
        # the staged copies go back (a decode step that wrote them); where every
        # backend validates ids, a wrong direction is refused by all alike
        _, err = self._all("writeback", [int(u) for u in dst], src)
        assert err is None, err
        if all(getattr(be, "validating", False) for be in self.backends):
            _, err = self._all("writeback", src, [int(u) for u in dst])
            assert err is not None, "writeback from a slice block into staging was accepted"
        _, err = self._all("free_blocks", dst)
        assert err is None, err

    def reclaim(self, n):
        per = []
        for be in self.backends:
            t = self.tables.copy()
            per.append((be.reclaim(n, t), t))
        r0, t0 = per[0]
        for r, t in per[1:]:
            _assert_same(r0, r, "reclaim")
            assert np.array_equal(t0, t), "reclaim: rewritten tables differ"
        self.log.append(("reclaim", n, r0["moved"], r0["victims"]))
        self.tables = t0
        for v in r0["victims"]:
            assert np.all(self.tables[:, v] == -1), "victim row not cleared by the rewrite"
            self.nb[:, v] = 0
        return r0

    @property
    def n_local(self):
        return self.backends[0].n_local


def _assert_same(a, b, what):
    if isinstance(a, dict):
        assert set(a) == set(b), what
        for k in a:
            _assert_same(a[k], b[k], f"{what}.{k}")
    elif isinstance(a, (list, tuple, np.ndarray)):
        # pair lists compare flattened, so [] equals an empty [0][2] array
        assert np.array_equal(np.asarray(a, dtype=np.int64).reshape(-1),
                              np.asarray(b, dtype=np.int64).reshape(-1)), f"{what}: {a} != {b}"
    else:
        assert a == b, f"{what}: {a} != {b}"


def random_trace(cache, steps, rng, on_step=None):
    """Drive `steps` random operations. Weighted toward growth early on."""
    L, B = cache.L, cache.B
    for step in range(steps):
        op = rng.choice(["grow", "grow", "grow", "finish", "lend", "reclaim", "migrate",
                         "prefetch"])
        if op == "grow":
            cache.grow(int(rng.integers(L)), int(rng.integers(B)), int(rng.integers(2)),
                       int(rng.integers(1, 4)))
        elif op == "finish":
            cache.finish(int(rng.integers(B)))
        elif op == "lend":
            cache.lend(int(rng.integers(0, 6)))
        elif op == "reclaim":
            cache.reclaim(int(rng.integers(0, 8)))
        elif op == "migrate":
            l, b = int(rng.integers(L)), int(rng.integers(B))
            if cache.nb[l, b]:
                cache.migrate(l, b, int(rng.integers(cache.nb[l, b])), int(rng.integers(2)))
        elif op == "prefetch":
            cache.prefetch_layer(int(rng.integers(L)))
        if on_step is not None:
            on_step(step, op)
