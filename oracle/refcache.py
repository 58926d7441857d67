"""Oracle: adaptive reference cache with int8 residuals and reference release
(Sec. 3.4, "Memory-efficient Cache Management").

TEST INFRASTRUCTURE ONLY: the plain CPU definition the GPU path is checked
against.  Only tests, the smoke check and the benchmark's CPU-baseline leg may
import this module; the product path never does.

What the paper states: a latent's cached output x_l is compared with the
current reference cache r by cosine similarity <x_l, r> / (|x_l|_2 |r|_2);
above the threshold tau only the residual x_l - r is kept, quantized to int8,
otherwise x_l itself is stored in full precision and becomes the new
reference.  A residual entry is read back as r + dequantized residual,
converted to the compute precision.  Before new entries are written, the old
entries are deleted and a reference that no latent depends on any more is
released.

Readings (the paper leaves these open):

* the "current reference" runs along chains of adjacent latents: the tokens
  of one spatial row of the latent grid (chain_len consecutive token
  indices), visited in index order; chains are independent;
* a chain's current reference persists across writes; a chain that has none
  yet makes its first written token a reference;
* a reference is stored in the activation dtype; the similarity is taken in
  fp64 between the fresh fp32 output and the stored reference, as
  dot / (sqrt(<y, y>) * sqrt(<r, r>)), and is 0 when either norm is 0; the
  token becomes a residual iff sim > tau;
* the residual res = fp32(y - r) is quantized with the per-token symmetric
  absmax code of the residual cache (oracle.cache.quantize_rows) and read back
  as cast(fp32(r + fp32(scale * code)));
* a reference is held by every entry that uses it (its own token's entry and
  the residual entries against it) and by the chain while it is the chain's
  current reference; it is released when nothing holds it.  Rewriting a
  token first drops its old entry's hold, for all rewritten tokens, and then
  scans the chains.
"""
from __future__ import annotations

import numpy as np

from oracle.cache import cast_act, dequantize_rows, quantize_rows

NONE, REFERENCE, RESIDUAL = 0, 1, 2


def cosine(y: np.ndarray, r: np.ndarray) -> float:
    """Cosine similarity in fp64; 0 when either vector is zero."""
    y = np.asarray(y, np.float64)
    r = np.asarray(r, np.float64)
    yy = float(np.dot(y, y))
    rr = float(np.dot(r, r))
    if yy == 0.0 or rr == 0.0:
        return 0.0
    return float(np.dot(y, r)) / (np.sqrt(yy) * np.sqrt(rr))


class RefCache:
    """Cache of L token outputs of width D, chains of chain_len tokens."""

    def __init__(self, L: int, D: int, chain_len: int, tau: float, dtype: str):
        assert L % chain_len == 0
        # the threshold is an fp32 value (the boundary passes it as a float)
        self.L, self.D, self.chain_len, self.dtype = L, D, chain_len, dtype
        self.tau = float(np.float32(tau))
        self.refs: dict[int, np.ndarray] = {}   # reference id -> stored row (fp32 values)
        self.holds: dict[int, int] = {}         # reference id -> number of holders
        self.kind = np.zeros(L, np.int8)
        self.ref_of = np.full(L, -1, np.int64)
        self.codes = np.zeros((L, D), np.int8)
        self.scale = np.zeros(L, np.float32)
        self.chain_ref = np.full(L // chain_len, -1, np.int64)
        self._next = 0
        self.sims: dict[int, float] = {}        # token -> similarity of its last write (nan: none)

    # -- holds ---------------------------------------------------------------
    def _hold(self, rid: int) -> None:
        self.holds[rid] += 1

    def _drop(self, rid: int) -> None:
        self.holds[rid] -= 1
        if self.holds[rid] == 0:
            del self.holds[rid]
            del self.refs[rid]

    def _new_ref(self, row: np.ndarray) -> int:
        rid = self._next
        self._next += 1
        self.refs[rid] = cast_act(row, self.dtype)
        self.holds[rid] = 0
        return rid

    # -- write ---------------------------------------------------------------
    def write(self, idx, y_sel) -> None:
        """Store the fresh outputs y_sel [K, D] (fp32) of the tokens idx [K]
        (ascending, distinct)."""
        idx = np.asarray(idx, np.int64)
        y_sel = np.asarray(y_sel, np.float32)
        assert np.all(np.diff(idx) > 0)
        for l in idx:                      # old entries go first
            if self.kind[l] != NONE:
                self._drop(int(self.ref_of[l]))
                self.kind[l] = NONE
                self.ref_of[l] = -1
        for j, l in enumerate(idx):        # chains in order, tokens in index order
            c = int(l) // self.chain_len
            y = y_sel[j]
            r = int(self.chain_ref[c])
            sim = cosine(y, self.refs[r]) if r >= 0 else float("nan")
            self.sims[int(l)] = sim
            if r >= 0 and sim > self.tau:
                res = (y - self.refs[r]).astype(np.float32)
                codes, scale = quantize_rows(res[None, :])
                self.codes[l] = codes[0]
                self.scale[l] = scale[0]
                self.kind[l] = RESIDUAL
                self.ref_of[l] = r
                self._hold(r)
            else:
                rid = self._new_ref(y)
                self._hold(rid)            # the token's own entry
                self._hold(rid)            # the chain's current reference
                if r >= 0:
                    self._drop(r)          # the chain lets go of its old reference
                self.chain_ref[c] = rid
                self.codes[l] = 0
                self.scale[l] = 0.0
                self.kind[l] = REFERENCE
                self.ref_of[l] = rid

    # -- read ----------------------------------------------------------------
    def read(self, rows=None) -> np.ndarray:
        """Cached outputs of the given tokens (all by default) in the
        activation dtype (as fp32 values); a token without an entry reads 0."""
        rows = np.arange(self.L) if rows is None else np.asarray(rows, np.int64)
        out = np.zeros((len(rows), self.D), np.float32)
        for o, l in enumerate(rows):
            k = self.kind[l]
            if k == REFERENCE:
                out[o] = self.refs[int(self.ref_of[l])]
            elif k == RESIDUAL:
                r = self.refs[int(self.ref_of[l])]
                out[o] = cast_act(dequantize_rows(r[None, :], self.codes[l:l + 1], self.scale[l:l + 1]),
                                  self.dtype)[0]
        return out

    def live_refs(self) -> int:
        return len(self.refs)

    def check_holds(self) -> None:
        """Every live reference's hold count equals a recount of its holders,
        and every entry's reference is live."""
        count: dict[int, int] = {}
        for l in range(self.L):
            if self.kind[l] != NONE:
                rid = int(self.ref_of[l])
                assert rid in self.refs, ("entry of a released reference", l)
                count[rid] = count.get(rid, 0) + 1
        for rid in self.chain_ref:
            if rid >= 0:
                assert int(rid) in self.refs, ("chain holds a released reference", int(rid))
                count[int(rid)] = count.get(int(rid), 0) + 1
        assert count == self.holds, (count, self.holds)


def step_update(cache: RefCache, x, idx, y_sel, xref):
    """One step's write and mask fusion: returns (y [L, D] in the activation
    dtype, xref').  Selected tokens output their fresh y_sel (cast) and
    record their current input as the saliency reference; the others read
    their cache entry."""
    x = np.asarray(x, np.float32)
    idx = np.asarray(idx, np.int64)
    y = cache.read()                       # entries before this write
    cache.write(idx, y_sel)
    xref2 = np.array(xref, np.float32, copy=True)
    if len(idx):
        y[idx] = cast_act(y_sel, cache.dtype)
        xref2[idx] = x[idx]
    return y, xref2
