"""Host logic of the paged-pool tests: gathering a sequence's records out of a pool inverts
scattering them in, record by record with its own index arithmetic."""
import numpy as np

import oracle
from parity import gather_paged


class _S:
    """The part of parity.Setup that gather_paged reads (the oracle's layout)."""

    def __init__(self, L, H, d, kinds):
        self.L, self.H, self.d = L, H, d
        self.orc = oracle.Codec(L, H, d, kinds, np.ones((L, d), np.int8))


def test_gather_inverts_scatter():
    rng = np.random.default_rng(0)
    kinds = [oracle.Kind(64, oracle.NORM_LINEAR, 8), oracle.Kind(64, oracle.NORM_LOG, 4),
             oracle.Kind(48, oracle.NORM_F32, 32), oracle.Kind(256, oracle.NORM_LINEAR, 8)]
    s = _S(2, 3, 64, kinds)
    P, n_blocks, max_blocks = 32, 9, 3
    table = np.array([[4, 0, 7], [2, -1, 12]], np.int32)      # -1 and 12 name no pool block
    cap = max_blocks * P
    pool_total, pool_off = s.orc.layout(n_blocks, P)
    pool = np.full(pool_total, 0xAB, np.uint8)
    want = []
    for b in range(2):
        total, off = s.orc.layout(1, cap)
        c = rng.integers(0, 256, total, dtype=np.uint8)
        want.append(c)
        for l in range(s.L):
            for kind in range(2):
                rec = s.orc.record_bytes(l, kind)
                for p in range(3):
                    for h in range(s.H):
                        for t in range(cap):
                            blk = table[b, t // P]
                            if not 0 <= blk < n_blocks:
                                continue
                            src = off[l, kind, p] + (h * cap + t) * rec[p]
                            dst = pool_off[l, kind, p] + ((blk * s.H + h) * P + t % P) * rec[p]
                            pool[dst:dst + rec[p]] = c[src:src + rec[p]]
    for b in range(2):
        got = gather_paged(pool, s, n_blocks, P, table[b], 0xCD)
        total, off = s.orc.layout(1, cap)
        for l in range(s.L):
            for kind in range(2):
                rec = s.orc.record_bytes(l, kind)
                for p in range(3):
                    n = s.H * cap * rec[p]
                    g = got[off[l, kind, p]: off[l, kind, p] + n].reshape(s.H, cap, rec[p])
                    w = want[b][off[l, kind, p]: off[l, kind, p] + n].reshape(s.H, cap, rec[p])
                    for i in range(max_blocks):
                        sl = slice(i * P, (i + 1) * P)
                        if 0 <= table[b, i] < n_blocks:
                            assert np.array_equal(g[:, sl], w[:, sl])
                        else:
                            assert np.all(g[:, sl] == 0xCD)
