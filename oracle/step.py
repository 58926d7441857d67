"""Oracle: one cached block step (Sec. 3.3 and Sec. 3.4 composed).

TEST INFRASTRUCTURE ONLY: the plain CPU definition the GPU path is checked
against.  Only tests, the smoke check and the benchmark's CPU-baseline leg may
import this module; the product path never does.

step = saliency -> top-K selection -> block on the selected rows -> cache
update with reuse of every other row.  The first ("init") step selects every
token, which fills the whole cache and equals the dense block.
"""
from __future__ import annotations

import numpy as np

from . import block as _block
from . import cache as _cache
from . import select as _select


def cached_step(params, x, cache, frame_weight, N: int, H: int, K: int, dtype: str,
                xi: float = 1e-6):
    """Returns dict(idx, s, y_sel (fp32), y, cache=(xref, codes, scale), step_delta)."""
    xref, codes, scale = cache
    s, num, den = _select.saliency(x, xref, frame_weight, N, xi)
    idx = _select.select_topk(s, K)
    y_sel = _block.block_partial(params, x, idx, H).astype(np.float32)
    y, xref2, codes2, scale2 = _cache.cache_update(x, idx, y_sel, xref, codes, scale, dtype)
    return {"idx": idx, "s": s, "y_sel": y_sel, "y": y,
            "cache": (xref2, codes2, scale2), "step_delta": _select.step_delta(num, den, xi)}


def init_step(params, x, H: int, dtype: str):
    """Recompute every token and fill the cache from an empty one."""
    L, D = np.asarray(x).shape
    idx = np.arange(L, dtype=np.int32)
    y_sel = _block.block_partial(params, x, idx, H).astype(np.float32)
    y, xref, codes, scale = _cache.cache_update(x, idx, y_sel, *_cache.empty_cache(L, D), dtype)
    return {"idx": idx, "y_sel": y_sel, "y": y, "cache": (xref, codes, scale)}
