"""Oracle ground truth over whole power-law corpora (test infrastructure).

The 1,000,000 x 1536 power-law corpus is coded by the oracle in full --
every row, at b = 2, 3, 4 and 8 from one float64 rotation per row -- with the
library's float32 rotation and exported tables (the parameters of the encode
definition, section II-B steps 1-4).  Every score of every vector against the
checked queries is then computed by the oracle (section II-B step 5), so
each GPU top-k list is compared with the brute-force result over the whole
corpus (section IV-A), not over a sample.  The 999K corpus is the first
999,000 rows of the same stream with the same queries, so its ground truth is
the first 999,000 columns of the same score rows.

Nothing here does method arithmetic: codes, scales and scores come from
oracle/ alone.
"""
from __future__ import annotations

import time

import numpy as np

import oracle
import synth
from tests.parity import oracle_tables

D = 1536
ROWS_PER_CHUNK = 65536


def _log(msg):
    print("[fullsize] %s" % msg, flush=True)


class PowerlawCorpus:
    """Rows of a power-law workload, the library parameters, and the oracle's
    codes, scales and score rows (computed on first use)."""

    def __init__(self, name: str, nq: int, bits=(4,)):
        """nq: the queries (the first nq of the workload's) whose results
        the oracle checks; all of the workload's queries are in Qall."""
        import paper_2607_16973_amd as tq
        t = time.time()
        self.X, self.Qall = synth.workload(name, d=D)
        self.n = self.X.shape[0]
        self.Q = np.ascontiguousarray(self.Qall[:nq])
        _log("%s: %d rows generated in %.1f s" % (name, self.n, time.time() - t))
        self.rot = tq.Rotation(D, 42)
        self.R32 = self.rot.matrix()
        self.cb = {b: tq.Codebook(D, b) for b in bits}
        self.ocb = {b: oracle_tables(self.cb[b]) for b in bits}
        self.qrot = oracle.rotate_queries(self.R32, self.Q)
        self.qn = np.linalg.norm(self.Q.astype(np.float64), axis=1)
        self.codes, self.scales, self._scores = {}, {}, {}
        self._encode(bits)

    def _encode(self, bits):
        """oracle.encode of every row at the first bit width (float64
        rotation, norms), then oracle.quantise_rotated of the same rotated
        rows at the others; one chunk of rows at a time."""
        t = time.time()
        n = self.n
        for b in bits:
            self.codes[b] = np.empty((n, D), dtype=np.uint8)
            self.scales[b] = np.empty(n, dtype=np.float32)
        first, rest = bits[0], bits[1:]
        for s in range(0, n, ROWS_PER_CHUNK):
            e = min(n, s + ROWS_PER_CHUNK)
            c, nrm, sc, S = oracle.encode(self.X[s:e], self.R32, self.ocb[first],
                                          return_rotated=True)
            self.codes[first][s:e], self.scales[first][s:e] = c, sc
            for b in rest:
                self.codes[b][s:e], self.scales[b][s:e] = oracle.quantise_rotated(S, nrm,
                                                                                  self.ocb[b])
            del S
            if (s // ROWS_PER_CHUNK) % 4 == 3:
                _log("oracle encode: %d of %d rows, %.1f s" % (e, n, time.time() - t))
        _log("oracle encode of %d rows at b=%s: %.1f s" % (n, list(bits), time.time() - t))

    def scores(self, bits: int) -> np.ndarray:
        """Oracle scores of every vector against every checked query, float64
        [nq, n]."""
        if bits not in self._scores:
            t = time.time()
            self._scores[bits] = oracle.score_all(self.codes[bits], self.scales[bits],
                                                  self.ocb[bits].cents, self.qrot)
            _log("oracle scores b=%d: %.1f s" % (bits, time.time() - t))
        return self._scores[bits]

    def topk(self, bits, k, n=None, tenants=None, allow=None):
        """The oracle's top-k of the checked queries over the first n rows
        (all by default)."""
        sc = self.scores(bits)
        if n is not None:
            sc = sc[:, :n]
        return oracle.topk_from_scores(sc, k, tenants=tenants, allow=allow)


def assert_index_codes_equal(idx, codes_or, bits, rows=None):
    """The index's canonical codes (tq_index_export) equal the oracle's codes
    of the same rows bit for bit, compared a chunk of rows at a time."""
    codes, _, _ = idx.export()
    n = codes.shape[0] if rows is None else rows
    for s in range(0, n, ROWS_PER_CHUNK):
        e = min(n, s + ROWS_PER_CHUNK)
        got = oracle.unpack_codes(codes[s:e].cpu().numpy(), D, bits)
        bad = np.argwhere(got != codes_or[s:e])
        assert bad.size == 0, ("code mismatches", len(bad), (bad[:5] + [s, 0]).tolist())
    del codes
