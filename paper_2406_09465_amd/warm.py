"""Pre-compiles (hipRTC, gfx950, no GPU needed) the kernels of the standard plans
of every workload so a GPU run finds them in the code-object cache."""

from __future__ import annotations

import time

from . import graphs
from ._abi import KorchError

# Sizes run by the test suite, smoke() and bench.py.
SIZES = {
    "attention": [{}, dict(n=50, d=24)],
    "mlp": [{}, dict(m=300, d=96, h=200), dict(m=256, d=128, h=256)],
    "sra": [{}, dict(hh=40, ww=24, c=16, r=8)],
    "conv": [{}, dict(hh=37, ww=29, cin=8, cout=24)],
    "linattn": [{}, dict(heads=3, n=300, d=16)],
}


def warm_cache(verbose=False):
    t0 = time.time()
    failures = []
    for w, sizes in SIZES.items():
        for sz in sizes:
            wl = graphs.build(w, **sz)
            for pn in ("unfused", "layered", "fused"):
                try:
                    wl.plan(pn).compile()
                except KorchError as e:
                    failures.append((w, sz, pn, str(e)[:200]))
    if verbose:
        print(f"warm_cache: {time.time() - t0:.1f}s, {len(failures)} plans not compiled")
        for f in failures:
            print("  ", f)
    return failures
