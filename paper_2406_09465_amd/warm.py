"""Pre-compiles (hipRTC, gfx950, no GPU needed) the kernels of the standard plans
of every workload, of the seeded sampled plans the GPU tests run, and every
supported candidate kernel the measured-cost chooser profiles, so a GPU run
finds them in the code-object cache."""

from __future__ import annotations

import time

from . import graphs, search
from ._abi import KorchError

# Sizes run by the test suite, smoke() and bench.py.
SIZES = {
    "attention": [{}, dict(n=50, d=24)],
    "mlp": [{}, dict(m=300, d=96, h=200), dict(m=256, d=128, h=256), dict(m=256, d=128, h=192)],
    "sra": [{}, dict(hh=40, ww=24, c=16, r=8)],
    "conv": [{}, dict(hh=37, ww=29, cin=8, cout=24)],
    "linattn": [{}, dict(heads=3, n=300, d=16)],
    "instnorm": [{}, dict(hh=13, ww=11, c=24)],
}
# (sizes, number of plans, seed) of the sampled-plan GPU tests.
SAMPLED = {
    "attention": (dict(n=96, d=32), 6, 7),
    "mlp": (dict(m=256, d=128, h=192), 6, 7),
    "sra": (dict(hh=32, ww=32, c=32, r=8), 6, 7),
    "conv": (dict(hh=24, ww=20, cin=16, cout=32), 6, 7),
    "linattn": (dict(heads=4, n=512, d=16), 6, 7),
    "instnorm": (dict(hh=40, ww=36, c=16), 6, 7),
}

# Shapes of the convolution-kernel GPU tests, each run with the direct kernel
# allowed and with the implicit-GEMM kernel forced (KORCH_CONV_DIRECT=0).
CONV_CASES = [
    dict(hh=37, ww=29, cin=8, cout=24),
    dict(hh=15, ww=13, cin=48, cout=16),
    dict(hh=10, ww=50, cin=16, cout=48),
    dict(hh=21, ww=40, cin=16, cout=16, k=5),
    dict(hh=9, ww=70, cin=32, cout=128),
]

# MLP shapes of the GEMM-kernel GPU tests (GEMM2 wider than 128 columns, with one tile per compute
# unit and a long contraction: an odd and an even number of k-tiles), each run
# with the intra-workgroup split of K and without it (KORCH_GEMM_NO_KSPLIT=1).
GEMM_CASES = [
    dict(m=500, d=256, h=1056),
    dict(m=256, d=192, h=2048),
]

# An MLP block whose first product takes 128 x 192 tiles: ragged rows (4000)
# and a ragged contraction (176 = 5.5 k-tiles of 32).
WIDE_TILE_CASE = dict(m=4000, d=176, h=1536)

# An MLP block whose first product takes 256 x 192 tiles of eight waves
# (16 x 16 = 256 tiles): ragged rows (4000 = 15.6 row tiles) and a ragged
# contraction (720 = 11.25 k-tiles of 64).
BIG_TILE_CASE = dict(m=4000, d=720, h=3072)

# MLP shapes of the direct-to-LDS staging GPU tests (the layered plan's first
# product takes it): bf16 with 64 x 64 tiles and three right-operand stages;
# a contraction of two k-tiles (two stages).  Each runs with the path switched
# off too (KORCH_GEMM_DMA=0), and the full MLP block also with two stages
# forced (KORCH_GEMM_DMA_2STAGE=1).
DMA_CASES = [
    dict(m=1024, d=256, h=768, dtype="bf16"),
    dict(m=512, d=128, h=512),
]

# MLP shapes whose second product, asked for eight waves over the whole
# contraction with three direct-to-LDS stages of each operand
# (KORCH_GEMM_DMA8=1; 128-row tiles dividing the problem, at most one per
# compute unit), takes them: odd numbers of k-tiles (31, and 17 in bf16 over
# 240 tiles).  Each also runs register-staged without the split.
DMA8_CASES = [
    dict(m=4096, d=768, h=1984),
    dict(m=3840, d=768, h=1088, dtype="bf16"),
]

# MLP shapes of the folded-LayerNorm GPU tests: plans whose first kernel holds
# the LayerNorm, the first product and (or not) the GELU.
LN_FOLD_CASES = [{}, dict(m=1024, d=256, h=768)]
LN_FOLD_PLANS = {
    "gelu": [(["mu", "D", "D2", "var", "ve", "r", "Xh", "Yg", "Y", "H0", "Hg"], ["Hg"]), (["Zo", "out"], ["out"])],
    "product": [(["mu", "D", "D2", "var", "ve", "r", "Xh", "Yg", "Y", "H0"], ["H0"]), (["Hg"], ["Hg"]),
                (["Zo", "out"], ["out"])],
}

# InstanceNorm shapes of the column-moments GPU tests (the split-moments
# transformation, then the two-kernel plan graphs.moments_plan builds): the
# full size (196 splits of the reduced axis, two-level arrival), 1600 rows (3
# splits), and one workgroup with ragged channels (24) or fewer rows than a
# workgroup has row lanes (15).  Each also with the mean and the reciprocal
# deviation as extra outputs.
MOMENTS_CASES = [{}, dict(hh=40, ww=40, c=16), dict(hh=13, ww=11, c=24), dict(hh=3, ww=5, c=8)]

# Attention shapes of the attention-kernel GPU tests (few query rows: the keys
# are split over the waves; fp32 and fp16, padded keys), each run with the key
# split and without it (KORCH_ATTN_NO_KEY_SPLIT=1).
ATTN_CASES = [
    ("attention", dict(n=50, d=16)),
    ("attention", dict(n=128, d=64)),
    ("sra", dict(hh=16, ww=32, c=32, r=2)),
    ("sra", dict(hh=8, ww=56, c=16, r=2)),
]

# Bit-exact layout GPU tests.  In place: the unfused plan of a workload with
# each listed layout node and its operand (when computed) as extra graph
# outputs, at the full and a ragged size.
LAYOUT_IN_PLACE = {
    "attention": [("KT", "K")],
    "sra": [("Xt", "X"), ("KT", "ln_Y")],
    "linattn": [("KrT", "Kr"), ("sKT", "sK")],
    "instnorm": [("out", "R")],
}
LAYOUT_SIZES = {w: SIZES[w][:2] for w in LAYOUT_IN_PLACE}
# Stand-alone layout primitives (graphs.layout_probe): (op, dtype, input shapes, attributes).
LAYOUT_STANDALONE = [
    # the product-merging transformation at full workload sizes
    ("concat", "f16", [(256, 64)], dict(axis=1, fill=1.0)),
    ("concat", "bf16", [(16, 4096, 16)], dict(axis=2, fill=1.0)),
    ("concat", "f32", [(128, 64)], dict(axis=1, fill=1.0)),
    ("slice", "f16", [(16384, 65)], dict(begin=(0, 0), end=(16384, 64))),
    ("slice", "f16", [(16384, 65)], dict(begin=(0, 64), end=(16384, 65))),
    ("slice", "bf16", [(16, 4096, 17)], dict(begin=(0, 0, 0), end=(16, 4096, 16))),
    ("slice", "bf16", [(16, 4096, 17)], dict(begin=(0, 0, 16), end=(16, 4096, 17))),
    ("slice", "bf16", [(16, 16, 17)], dict(begin=(0, 0, 0), end=(16, 16, 16))),
    ("slice", "f32", [(128, 65)], dict(begin=(0, 64), end=(128, 65))),
    # layout variants of product operands (transposes of the last two axes)
    ("transpose", "f16", [(4096, 768)], dict(perm=(1, 0))),
    ("transpose", "f16", [(16384, 256)], dict(perm=(1, 0))),
    ("transpose", "bf16", [(16, 16, 4096)], dict(perm=(0, 2, 1))),
    # ragged shapes, several axes, two inputs, a non-zero pad value
    ("transpose", "f16", [(37, 29, 8)], dict(perm=(2, 0, 1))),
    ("transpose", "f32", [(50, 24)], dict(perm=(1, 0))),
    ("transpose", "bf16", [(3, 5, 7, 9)], dict(perm=(3, 1, 0, 2))),
    ("slice", "f16", [(33, 17, 5)], dict(begin=(3, 2, 1), end=(30, 17, 4))),
    ("pad", "f16", [(13, 11, 24)], dict(lo=(1, 2, 0), hi=(2, 1, 0), value=0.0)),
    ("pad", "bf16", [(7, 9)], dict(lo=(0, 3), hi=(5, 0), value=-2.5)),
    ("pad", "f32", [(5, 6, 3)], dict(lo=(1, 1, 1), hi=(1, 1, 1), value=7.0)),
    ("concat", "f16", [(9, 5), (9, 3)], dict(axis=1)),
    ("concat", "bf16", [(4, 6, 2), (3, 6, 2)], dict(axis=0)),
]


# Workloads whose computed product operands get layout variants.
LAYOUT_WORKLOADS = ("attention", "mlp", "sra", "linattn")

# Sizes at which the chooser profiles every supported candidate (bench.py's
# measured-cost plan at full size; the chooser GPU test at the sampled sizes).
CHOOSER = {w: [{}, SAMPLED[w][0]] for w in SAMPLED}
CHOOSER_LIMITS = dict(max_prims=64, max_outs=3)


def _jobs():
    """Independent compile jobs: (kind, workload, sizes, extra)."""
    jobs = []
    for w, sizes in SIZES.items():
        for sz in sizes:
            jobs.append(("plans", w, sz, None))
    for w, (sz, n, seed) in SAMPLED.items():
        jobs.append(("sampled", w, sz, (n, seed)))
        if w in LAYOUT_WORKLOADS:
            jobs.append(("sampled_layouts", w, sz, (n, seed)))
    for sz in CONV_CASES + [{}]:
        for direct in ("1", "0"):
            jobs.append(("env_plans", "conv", sz, ("KORCH_CONV_DIRECT", direct)))
    for sz in GEMM_CASES:
        for flag in ("", "1"):
            jobs.append(("env_plans", "mlp", sz, ("KORCH_GEMM_NO_KSPLIT", flag)))
    jobs.append(("plans", "mlp", WIDE_TILE_CASE, None))
    jobs.append(("plans", "mlp", BIG_TILE_CASE, None))
    for sz in DMA8_CASES + [{}]:
        jobs.append(("env_plans", "mlp", sz, ("KORCH_GEMM_DMA8", "1")))
        jobs.append(("env_plans", "mlp", sz, (("KORCH_GEMM_DMA8", "1"), ("KORCH_GEMM_DMA_STAGES", "5"))))
    for sz in DMA_CASES + DMA8_CASES + [{}]:
        if sz:
            jobs.append(("plans", "mlp", sz, None))
        jobs.append(("env_plans", "mlp", sz, ("KORCH_GEMM_DMA", "0")))
        jobs.append(("env_plans", "mlp", sz, (("KORCH_GEMM_NO_KSPLIT", "1"),)))
        jobs.append(("env_plans", "mlp", sz, (("KORCH_GEMM_NO_KSPLIT", "1"), ("KORCH_GEMM_DMA", "0"))))
    for sz in LN_FOLD_CASES:
        jobs.append(("ln_fold", "mlp", sz, None))
    for sz in MOMENTS_CASES:
        jobs.append(("moments", "instnorm", sz, None))
    jobs.append(("env_plans", "mlp", {}, ("KORCH_GEMM_DMA_2STAGE", "1")))
    jobs.append(("env_plans", "mlp", {}, (("KORCH_GEMM_NO_KSPLIT", "1"), ("KORCH_GEMM_DMA_2STAGE", "1"))))
    jobs.append(("env_plans", "mlp", {}, ("KORCH_GEMM_DMA_KSPLIT", "1")))
    for wl, sz in ATTN_CASES:
        for flag in ("", "1"):
            jobs.append(("env_plans", wl, sz, ("KORCH_ATTN_NO_KEY_SPLIT", flag)))
    for w, sizes in LAYOUT_SIZES.items():
        for sz in sizes:
            jobs.append(("layout_in_place", w, sz, None))
    for i in range(len(LAYOUT_STANDALONE)):
        jobs.append(("layout_probe", None, {}, i))
    for w, sizes in CHOOSER.items():
        for sz in sizes:
            jobs.append(("candidates", w, sz, None))
            jobs.append(("candidates", w, sz, "rewritten"))
            if w in LAYOUT_WORKLOADS:
                jobs.append(("candidates", w, sz, "layouts"))
    return jobs


def _run_job(job, part=0, parts=1):
    """Compiles this process's share of one job; returns the failures."""
    kind, w, sz, extra = job
    failures = []
    if kind in ("layout_in_place", "layout_probe"):
        if kind == "layout_probe":
            op, dt, shapes, attrs = LAYOUT_STANDALONE[extra]
            wl = graphs.layout_probe(op, dt, shapes, **attrs)
        else:
            names = [n for pair in LAYOUT_IN_PLACE[w] for n in pair]
            wl = graphs.build(w, **sz)
            names = [n for n in names if n not in wl.input_names]
            wl = graphs.build(w, extra_outputs=names, **sz)
        try:
            wl.plan("unfused").compile()
        except KorchError as e:
            failures.append((w, sz, f"{kind} {extra}", str(e)[:200]))
        return failures
    if kind == "moments":
        for extra in ((), ("mu", "r")):
            w2, _ = graphs.rewritten(graphs.build(w, extra_outputs=extra, **sz))
            try:
                graphs.Plan(w2.graph, graphs.moments_plan(w2)).compile()
            except KorchError as e:
                failures.append((w, sz, f"moments {extra}", str(e)[:200]))
        return failures
    wl = graphs.build(w, **sz)
    if kind == "ln_fold":
        for name, ks in LN_FOLD_PLANS.items():
            try:
                graphs.Plan(wl.graph, [([wl.ids[n] for n in p], [wl.ids[n] for n in o]) for p, o in ks]).compile()
            except KorchError as e:
                failures.append((w, sz, f"ln_fold {name}", str(e)[:200]))
        return failures
    if kind == "plans":
        for pn in ("unfused", "layered", "fused"):
            try:
                wl.plan(pn).compile()
            except KorchError as e:
                failures.append((w, sz, pn, str(e)[:200]))
    elif kind == "env_plans":
        import os
        pairs = (extra,) if isinstance(extra[0], str) else extra  # one (var, value) or several
        prev = {var: os.environ.get(var) for var, _ in pairs}
        for var, val in pairs:
            if val:
                os.environ[var] = val
            else:
                os.environ.pop(var, None)
        tag = " ".join(f"{var}={val}" for var, val in pairs)
        try:
            for pn in ("layered", "fused"):
                try:
                    wl.plan(pn).compile()
                except KorchError as e:
                    failures.append((w, sz, f"{pn} {tag}", str(e)[:200]))
        finally:
            for var, old in prev.items():
                if old is None:
                    os.environ.pop(var, None)
                else:
                    os.environ[var] = old
    elif kind in ("sampled", "sampled_layouts"):
        if kind == "sampled_layouts":
            from ._abi import RW_LAYOUT_VARIANTS
            wl, _ = graphs.rewritten(wl, RW_LAYOUT_VARIANTS)
        for i, ks in enumerate(search.sampled_plans(wl.graph, *extra)):
            try:
                graphs.Plan(wl.graph, ks).compile()
            except KorchError as e:
                failures.append((w, sz, f"sampled {i}", str(e)[:200]))
    else:
        if extra in ("rewritten", "layouts"):
            from ._abi import RW_LAYOUT_VARIANTS
            wl, n = graphs.rewritten(wl, RW_LAYOUT_VARIANTS if extra == "layouts" else None)
            if n == 0:
                return failures
        cands = wl.graph.candidates(only_supported=True, **CHOOSER_LIMITS)
        for c in cands[part::parts]:
            try:
                wl.graph.compile_candidate(*c)
            except KorchError as e:
                failures.append((w, sz, f"candidate {c}", str(e)[:200]))
    return failures


def _worker(args):
    return _run_job(*args)


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


def warm_cache(verbose=False, prune_stale=True, processes=None):
    """Compiles every job; hipRTC serializes compiles within one process, so the
    jobs are spread over worker processes (spawned, each loading the library)."""
    import concurrent.futures as cf
    import multiprocessing as mp
    import os
    t0 = time.time()
    procs = processes or min(8, os.cpu_count() or 1)
    tasks = []
    for job in _jobs():
        parts = procs if job[0] == "candidates" else 1
        tasks.extend((job, i, parts) for i in range(parts))
    failures = []
    if procs <= 1:
        for t in tasks:
            failures.extend(_worker(t))
    else:
        with cf.ProcessPoolExecutor(max_workers=procs, mp_context=mp.get_context("spawn")) as ex:
            for f in ex.map(_worker, tasks):
                failures.extend(f)
    removed = prune(t0) if prune_stale and not failures else 0
    if verbose:
        print(f"warm_cache: {time.time() - t0:.1f}s, {len(failures)} plans not compiled, {removed} stale removed")
        for f in failures:
            print("  ", f)
    return failures
