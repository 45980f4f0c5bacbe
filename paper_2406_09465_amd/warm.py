"""Pre-compiles (hipRTC, gfx950, no GPU needed) the kernels of the standard plans
of every workload, and of the seeded sampled plans the GPU tests run, so a GPU
run finds them in the code-object cache."""

from __future__ import annotations

import time

from . import graphs, search
from ._abi import KorchError

# Sizes run by the test suite, smoke() and bench.py.
SIZES = {
    "attention": [{}, dict(n=50, d=24)],
    "mlp": [{}, dict(m=300, d=96, h=200), dict(m=256, d=128, h=256)],
    "sra": [{}, dict(hh=40, ww=24, c=16, r=8)],
    "conv": [{}, dict(hh=37, ww=29, cin=8, cout=24)],
    "linattn": [{}, dict(heads=3, n=300, d=16)],
}
# (sizes, number of plans, seed) of the sampled-plan GPU tests.
SAMPLED = {
    "attention": (dict(n=96, d=32), 6, 7),
    "mlp": (dict(m=256, d=128, h=192), 6, 7),
    "sra": (dict(hh=32, ww=32, c=32, r=8), 6, 7),
    "conv": (dict(hh=24, ww=20, cin=16, cout=32), 6, 7),
    "linattn": (dict(heads=4, n=512, d=16), 6, 7),
}


def prune(before):
    """Delete cached code objects not used since ``before`` (a time.time())."""
    import os
    d = os.environ.get("KORCH_CACHE_DIR")
    if not d or not os.path.isdir(d):
        return 0
    n = 0
    for f in os.listdir(d):
        p = os.path.join(d, f)
        if f.endswith(".co") and os.path.getmtime(p) < before - 1:
            os.remove(p)
            n += 1
    return n


def warm_cache(verbose=False, prune_stale=True):
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
    for w, (sz, n, seed) in SAMPLED.items():
        wl = graphs.build(w, **sz)
        for i, ks in enumerate(search.sampled_plans(wl.graph, n, seed)):
            try:
                graphs.Plan(wl.graph, ks).compile()
            except KorchError as e:
                failures.append((w, sz, f"sampled {i}", str(e)[:200]))
    removed = prune(t0) if prune_stale and not failures else 0
    if verbose:
        print(f"warm_cache: {time.time() - t0:.1f}s, {len(failures)} plans not compiled, {removed} stale removed")
        for f in failures:
            print("  ", f)
    return failures
