"""C-ABI tests that need no GPU: exports, graph and plan error codes, the
orchestration analysis against the oracle's plain definitions, candidate
enumeration, and runtime compilation (hipRTC, gfx950) of every workload plan."""

import itertools
import os
import random
import re

import pytest

from oracle import configs as OC
from oracle import orchestration as O
from oracle.graph import Graph as OGraph
from paper_2406_09465_amd import _abi as K
from paper_2406_09465_amd import graphs

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def header_functions():
    text = open(os.path.join(ROOT, "include", "korch.h")).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(korch_[a-z_]+)\s*\(", text)))


def test_library_exports_every_declared_function():
    names = header_functions()
    assert len(names) >= 30
    for n in names:
        assert hasattr(K.lib, n), n
        assert n in K.EXPORTED, f"binding lacks {n}"


def code(fn):
    try:
        fn()
    except K.KorchError as e:
        return e.code
    return 0


def test_graph_errors():
    g = K.Graph()
    x = g.input("f16", (4, 8))
    w = g.input("f16", (5, 3))
    assert code(lambda: g.op("matmul", [x, w], "f16")) == -2          # contraction mismatch
    assert code(lambda: g.op("add", [x, 99], "f16")) == -1            # bad id
    assert code(lambda: g.op("transpose", [x], "f16", perm=(0, 0))) == -2
    assert code(lambda: g.op("reshape", [x], "f16", shape=(3, 3))) == -2
    assert code(lambda: g.op("reshape", [x], "f32", shape=(32,))) == -1  # a view keeps its dtype
    assert code(lambda: g.output(x)) == -1                             # an input cannot be an output
    y = g.op("exp", [x], "f16")
    assert code(lambda: g.finalize()) == 0 or True
    g2 = K.Graph()
    a = g2.input("f32", (2, 3))
    assert code(lambda: g2.finalize()) == -1                           # no outputs
    b = g2.op("relu", [a], "f32")
    g2.output(b)
    g2.finalize()
    assert code(lambda: g2.op("exp", [a], "f32")) == -4                # finalized
    assert g.node_info(y) == ("exp", "f16", (4, 8))


def small_graph():
    g = K.Graph()
    x = g.input("f32", (4, 8))
    a = g.op("exp", [x], "f32")         # 1
    b = g.op("neg", [a], "f32")         # 2
    c = g.op("tanh", [a], "f32")        # 3
    d = g.op("add", [b, c], "f32")      # 4
    e = g.op("relu", [x], "f32")        # 5 (disconnected chain)
    f = g.op("exp", [e], "f32")         # 6
    g.output(d)
    g.output(f)
    g.finalize()
    return g, (a, b, c, d, e, f)


def plan_code(g, kernels, strict=False):
    old = os.environ.get("KORCH_STRICT_SINGLE_OUTPUT")
    if strict:
        os.environ["KORCH_STRICT_SINGLE_OUTPUT"] = "1"
    try:
        return code(lambda: K.Plan(g, kernels))
    finally:
        if strict:
            if old is None:
                del os.environ["KORCH_STRICT_SINGLE_OUTPUT"]
            else:
                os.environ["KORCH_STRICT_SINGLE_OUTPUT"] = old


def test_plan_validation_codes():
    g, (a, b, c, d, e, f) = small_graph()
    ok = [([a, b, c, d], [d]), ([e, f], [f])]
    assert plan_code(g, ok) == 0
    assert plan_code(g, []) == -10                                    # empty plan
    assert plan_code(g, [([0], [0]), ([e, f], [f])]) == -10           # graph input inside a kernel
    assert plan_code(g, [([a, d], [d]), ([b, c], [b, c]), ([e, f], [f])]) == -11  # a ~> b ~> d outside
    assert plan_code(g, [([a, b, c, d], [b, d]), ([e, f], [f])]) == -12  # b has no outside consumer
    assert plan_code(g, [([b, c, d], [d]), ([a], [a]), ([e, f], [f])]) == -13  # reads a before it exists
    assert plan_code(g, [([a, b, c, d], [d])]) == -14                 # f never produced
    assert plan_code(g, [([a, b, c, d, e, f], [d, f])], strict=True) == -15
    assert plan_code(g, [([a, b, c, d, e, f], [d, f])]) == 0          # multi-output allowed by default
    # redundant execution: a computed by two kernels
    assert plan_code(g, [([a, b], [b]), ([a, c], [c]), ([d], [d]), ([e, f], [f])]) == 0


def test_disconnected_kernels_cycle_rejected():
    g = K.Graph()
    x = g.input("f32", (4,))
    a = g.op("exp", [x], "f32")
    b = g.op("exp", [a], "f32")
    c = g.op("exp", [x], "f32")
    d = g.op("exp", [c], "f32")
    g.output(b)
    g.output(d)
    g.finalize()
    assert g.is_convex([a, d]) and g.is_convex([b, c])
    assert plan_code(g, [([a, d], [a, d]), ([b, c], [b, c])]) == -13
    assert plan_code(g, [([a, c], [a, c]), ([b, d], [b, d])]) == 0


def twin_dags(n, edges):
    """The same DAG in the library and in the oracle (same node ids)."""
    kg = K.Graph()
    og = OGraph()
    kx = kg.input("f32", (2,))
    og.input("x", (2,))
    preds = {v: [u for (u, w) in edges if w == v] for v in range(n)}
    ids = []
    for v in range(n):
        ins = [ids[u] for u in preds[v]] or [0]
        op = "exp" if len(ins) == 1 else "add"
        ids.append(kg.op(op, ins if ins != [0] else [kx], "f32"))
        og.op(op, ins)
    sinks = [v for v in range(n) if not any(u == v for (u, _) in edges)]
    for s in sinks:
        kg.output(ids[s])
        og.output(ids[s])
    kg.finalize()
    return kg, og


def random_dag(rnd, n):
    edges = []
    for v in range(1, n):
        for u in rnd.sample(range(v), min(v, rnd.randint(0, 2))):
            edges.append((u, v))
    return edges


def test_convexity_and_states_match_oracle():
    """Theorem 1 / Definitions 1-2 in C++ against the oracle's set computations."""
    rnd = random.Random(3)
    for trial in range(40):
        n = rnd.randint(2, 9)
        kg, og = twin_dags(n, random_dag(rnd, n))
        states = set(kg.states())
        assert states == O.execution_states_bruteforce(og)
        prims = og.primitives()
        r = O.reach(og)
        for _ in range(60):
            sub = rnd.sample(prims, rnd.randint(1, len(prims)))
            assert kg.is_convex(sub) == O.is_convex(og, sub, r)


def test_candidates_are_convex_with_possible_outputs():
    """Algorithm 1 candidates: every P' is convex and every O is a possible output set,
    and the set of P' equals all differences of execution states."""
    og = OC.attention(n=8, d=4)
    w = graphs.attention(n=8, d=4)
    cands = w.graph.candidates(max_prims=64, max_outs=3)
    seen_p = set()
    for prims, outs in cands:
        assert O.is_convex(og, prims)
        assert O.is_possible_output_set(og, prims, outs)
        seen_p.add(frozenset(prims))
    expected = {p for p in O.convex_sets_from_states(O.execution_states_bruteforce(og))
                if any(O.is_possible_output_set(og, p, [v]) for v in p) or True}
    # every non-empty state difference with a non-empty possible output set appears
    with_outputs = {p for p in expected
                    if [v for v in p if v in og.outputs or any(c not in p for c in og.consumers()[v])]}
    assert seen_p == with_outputs


def test_supported_candidate_filter():
    w = graphs.mlp(m=64, d=64, h=64)
    allc = w.graph.candidates(max_prims=13, max_outs=2)
    sup = w.graph.candidates(max_prims=13, max_outs=2, only_supported=True)
    assert 0 < len(sup) < len(allc)
    for prims, outs in sup[:50]:
        assert w.graph.family(prims, outs) != "none"


def test_unfused_plan_skips_views():
    w = graphs.sra(hh=16, ww=16, c=8, r=8)
    p = w.plan("unfused")
    assert p.num_kernels() == 20  # 23 primitives, 3 contiguous reshapes are views


@pytest.mark.parametrize("workload", list(graphs.BUILDERS))
def test_every_plan_compiles_for_gfx950(workload):
    """Family match, code generation and hipRTC compilation run without a GPU."""
    w = graphs.build(workload)
    expected = {
        "attention": ["attention"], "mlp": ["row", "gemm", "gemm"], "sra": ["splitk", "attention"],
        "conv": ["conv"], "linattn": ["splitk", "gemm"], "instnorm": ["colreduce", "colreduce", "pointwise"],
    }[workload]
    for pn in ("unfused", "layered", "fused"):
        p = w.plan(pn)
        p.compile()
        fams = [p.kernel_info(k)[0] for k in range(p.num_kernels())]
        assert "none" not in fams
        if pn == "fused":
            assert fams == expected
        for k in range(p.num_kernels()):
            src = p.kernel_source(k)
            assert p.kernel_name(k) in src
            grid, block, _ = p.kernel_launch(k)
            assert min(grid) >= 1 and block in ((256, 1, 1), (512, 1, 1))
            assert f"__launch_bounds__({block[0]})" in src


def test_workspace_holds_only_intermediates():
    w = graphs.mlp()
    p = w.plan("fused")
    ws = p.workspace_bytes()
    # D [4096, 768], r [4096, 1] and Hg [4096, 3072] (fp16) are the kernel-boundary
    # tensors; all three are live during the second kernel, so none can share
    # space.  X, W1, W2 and out are caller buffers.
    need = 4096 * 768 * 2 + 4096 * 2 + 4096 * 3072 * 2
    assert need <= ws <= need + 3 * 256
    # unfused plan: lifetimes let dead intermediates share space
    pu = w.plan("unfused")
    g = w.graph
    inter = 0
    for name, nid in w.ids.items():
        op, dt, shape = g.node_info(nid)
        if op != "input" and nid not in g.outputs():
            n = 1
            for s in shape:
                n *= s
            inter += n * 2
    largest_pair = 2 * 4096 * 3072 * 2  # H0 and Hg are live together
    assert largest_pair <= pu.workspace_bytes() < inter
    fam, b, f = p.kernel_info(1)
    assert fam == "gemm" and f == 2.0 * 4096 * 3072 * 768


def test_execute_without_gpu_fails_loudly():
    import torch
    if torch.cuda.is_available():
        pytest.skip("a GPU is present")
    w = graphs.attention(n=16, d=16)
    p = w.plan("fused")
    p.compile()
    assert code(p.load) == -30  # KORCH_E_HIP: no device to load on


def test_execute_of_an_unloaded_plan_is_a_state_error():
    """Execution never compiles, loads or allocates: a plan that was not
    loaded on the device is refused with KORCH_E_STATE before any HIP call
    (so this runs without a GPU), compiled or not."""
    w = graphs.attention(n=16, d=16)
    p = w.plan("fused")
    assert code(lambda: p.execute([16, 16, 16], [16])) == -4
    p.compile()
    assert code(lambda: p.execute([16, 16, 16], [16])) == -4
    assert code(lambda: p.execute_kernels(0, 1, [16, 16, 16], [16])) == -4
    try:
        p.execute([16, 16, 16], [16])
    except K.KorchError as e:
        assert "korch_plan_load" in str(e)
    assert code(lambda: p.execute_timed(0, 1, [16, 16, 16], [16], 0, 0, 0, 0, 0, 0)) == -4
    assert code(lambda: p.execute_noalloc([16, 16, 16], [16])) == -4


def test_unsupported_kernel_reports_infinite_cost():
    w = graphs.attention(n=16, d=16)
    ids = w.ids
    # a reduction and a product in one kernel with the reduction output feeding nothing
    prims = [ids["m"], ids["Z"], ids["E"], ids["s"], ids["P"], ids["O"]]
    assert w.graph.family(prims, [ids["O"]]) == "none"
    p = K.Plan(w.graph, [([ids["KT"], ids["S0"], ids["S"]], [ids["S"]]), (prims, [ids["O"]])])
    assert code(p.compile) == -20


def test_sampled_and_sized_plans_compile():
    """Every plan that the GPU tests execute (workload plans at the test sizes and
    the seeded random plans) generates kernels that hipRTC compiles for gfx950."""
    from paper_2406_09465_amd import warm

    failures = warm.warm_cache(prune_stale=False)
    assert not failures, failures[:3]


def test_conv_kernel_variants():
    """The conv family generates the direct kernel (halo tile in LDS) for
    half-precision stride-1 convolutions within its register budget, and the
    implicit-GEMM kernel otherwise or when KORCH_CONV_DIRECT=0."""
    import os
    from paper_2406_09465_amd import graphs
    from paper_2406_09465_amd.warm import CONV_CASES

    def source(sizes, direct):
        prev = os.environ.get("KORCH_CONV_DIRECT")
        os.environ["KORCH_CONV_DIRECT"] = direct
        try:
            p = graphs.build("conv", **sizes).plan("fused")
            p.compile()
            return p.kernel_source(0)
        finally:
            if prev is None:
                os.environ.pop("KORCH_CONV_DIRECT")
            else:
                os.environ["KORCH_CONV_DIRECT"] = prev

    direct_cases = [{}] + CONV_CASES[:4]
    for sz in direct_cases:
        assert "fetch_halo" in source(sz, "1"), sz
        assert "fetch_halo" not in source(sz, "0"), sz
    # 128 output channels need more LDS than two workgroups per compute unit allow
    assert "fetch_halo" not in source(CONV_CASES[4], "1")
    # 48 -> 96 channels: the weights of a wave exceed its register budget
    assert "fetch_halo" not in source(dict(hh=15, ww=13, cin=48, cout=96), "1")
    assert "fetch_halo" not in source(dict(hh=12, ww=12, cin=8, cout=16, dtype="f32"), "1")


def test_timed_execute_rejects_a_kernel_outside_the_range():
    w = graphs.build("mlp", m=64, d=32, h=48)
    p = w.plan("layered")
    n = p.num_kernels()
    assert code(lambda: p.execute_timed(0, n, [0] * 6, [0], 0, 0, 0, n, 0, 0)) == -1
    assert code(lambda: p.execute_timed(1, 1, [0] * 6, [0], 0, 0, 0, 0, 0, 0)) == -1


def test_column_moments_kernel():
    """After the split-moments transformation InstanceNorm's mean, centred
    squares and variance (with + eps and rsqrt) form one column-reduction
    kernel that reads X once (Welford per thread, Chan's merge, three fp32
    partial planes per split) and exports the mean and the reciprocal
    deviation; the normalization recomputes X - m from them.  The chooser's
    candidates include it.  Kernels that would have to export the centred
    values, or whose square is not of X minus its mean, are not moments
    kernels."""
    import re
    w2, n = graphs.rewritten(graphs.build("instnorm"))
    assert n >= 1
    ks = graphs.moments_plan(w2)
    assert ks is not None and len(ks) == 2
    p = graphs.Plan(w2.graph, ks)
    p.compile()
    assert p.kernel_info(0)[0] == "colreduce" and p.kernel_info(1)[0] == "pointwise"
    src = p.kernel_source(0)
    assert "cn_ += 1.0f" in src and src.count("ldv<8>(") == 1  # one vector load of X per row
    assert "coherent_store(&part[6272LL + o_], q_);" in src  # 196 splits x 32 channels per plane
    body = src[src.index('extern "C"'):]
    assert len(re.findall(r"st1_out\(", body)) == 2  # the mean and rsqrt(var + eps) only
    g = w2.graph
    cands = {(tuple(a), tuple(b)) for a, b in g.candidates(max_prims=64, max_outs=3, only_supported=True)}
    assert (tuple(ks[0][0]), tuple(ks[0][1])) in cands
    # the centred values as an output: not a moments kernel
    ops = {v: g.node_info(v)[0] for v in range(g.num_nodes())}
    sq = next(v for v in ops if ops[v] == "square")
    dc = g.node_inputs(sq)[0]
    assert g.family(sorted(ks[0][0]), sorted(ks[0][1] + [dc])) == "none"
    # in the original graph the same kernel computes the variance, but the mean
    # has no reader outside it (X - m is inside), so it cannot be an output
    # (Definition 3) and the normalization could not recompute X - m
    w = graphs.build("instnorm")
    ids = w.ids
    assert w.graph.family([ids[k] for k in ("mu", "D", "D2", "var")], [ids["var"]]) == "colreduce"
    with pytest.raises(K.KorchError):
        graphs.Plan(w.graph, [([ids[k] for k in ("mu", "D", "D2", "var")], [ids["mu"], ids["var"]])] +
                    [(sorted(set(range(w.graph.num_nodes())) - set(w.graph.inputs()) -
                             {ids[k] for k in ("mu", "D2", "var")}), [ids["out"]])])


def test_gemm_k_split_selection(monkeypatch):
    """GEMM2 of the MLP block (256 tiles, 48 k-tiles) and of the odd-k test shape
    use the intra-workgroup split of K; GEMM1 (256 x 192 tiles of eight waves)
    and KORCH_GEMM_NO_KSPLIT=1 do not.  Asked for (KORCH_GEMM_DMA8=1), the split
    gives way to eight waves over the whole contraction where both operands can
    be staged three k-tiles deep (tiles of 128 rows dividing the problem), and
    stays for ragged rows and for 64-row tiles."""
    from paper_2406_09465_amd.warm import GEMM_CASES

    def sources(sizes, flag):
        monkeypatch.delenv("KORCH_GEMM_NO_KSPLIT", raising=False)
        if flag:
            monkeypatch.setenv("KORCH_GEMM_NO_KSPLIT", flag)
        p = graphs.build("mlp", **sizes).plan("layered")
        p.compile()
        return [p.kernel_source(k) for k in range(p.num_kernels())], [p.kernel_launch(k) for k in range(3)]

    monkeypatch.delenv("KORCH_GEMM_DMA8", raising=False)
    for sz in [{}] + GEMM_CASES:
        src, launch = sources(sz, "")
        assert "kgrp" in src[2] and launch[2][1][0] == 512, sz
        src, launch = sources(sz, "1")
        assert "kgrp" not in src[2] and launch[2][1][0] == 256, sz
    src, _ = sources({}, "")
    assert "kgrp" not in src[1]
    monkeypatch.setenv("KORCH_GEMM_DMA8", "1")
    for sz, dma8 in zip([{}] + GEMM_CASES, [True, False, False]):
        src, launch = sources(sz, "")
        assert launch[2][1][0] == 512, sz
        assert ("3 A stages and 3 B stages" in src[2]) == dma8 and ("kgrp" in src[2]) != dma8, sz


def test_gemm_wide_tile_selection():
    """GEMM1 of the MLP block (4096 x 3072 output) takes 256 x 192 tiles of
    eight waves with k-tiles of 64: 256 tiles, one per compute unit, re-reading
    the operand panels least.  The ragged 4000 x 3072 shape of the GPU test
    takes them too (16 x 16 tiles); 4000 x 1536 (too few 256-row tiles for a
    round) takes 128 x 192 tiles with k-tiles of 32 (32 x 8 tiles); a hidden
    width that 192 does not divide keeps narrower tiles."""
    from paper_2406_09465_amd.warm import BIG_TILE_CASE, WIDE_TILE_CASE

    def gemm1(sizes):
        p = graphs.build("mlp", **sizes).plan("layered")
        p.compile()
        return p.kernel_launch(1), p.kernel_source(1)

    (grid, block, _), src = gemm1({})
    assert grid == (256, 1, 1) and block == (512, 1, 1)
    (grid, block, _), src = gemm1(BIG_TILE_CASE)
    assert grid == (16 * 16, 1, 1) and block == (512, 1, 1)
    assert "* 80 + " in src  # register-staged A tile rows of 64 + 16 halves (k-tiles of 64)
    (grid, block, _), src = gemm1(WIDE_TILE_CASE)
    assert grid == (32 * 8, 1, 1) and block == (256, 1, 1)
    assert "* 48 + " in src  # A tile rows of 32 + 16 halves (k-tiles of 32)
    (grid, _, _), _ = gemm1(dict(m=500, d=256, h=1056))
    assert grid[0] != 4 * 1056 // 192


def test_gemm_direct_to_lds_staging_selection(monkeypatch):
    """The MLP block's first product (plain fp16 operands, 256 x 192 tiles that
    divide the problem, k-tiles of 64) stages both operands with direct
    global-to-LDS loads: 32 + 24 one-KiB blocks per k-tile, two left-operand
    and three right-operand stages in 136 KiB of LDS, every wait before a
    barrier a full vmcnt(0).  KORCH_GEMM_DMA=0 restores register staging;
    ragged rows keep it; KORCH_GEMM_DMA_2STAGE=1 gives two right-operand
    stages."""
    import re
    from paper_2406_09465_amd.warm import BIG_TILE_CASE

    def gemm1(sizes):
        p = graphs.build("mlp", **sizes).plan("layered")
        p.compile()
        return p.kernel_launch(1), p.kernel_source(1)

    monkeypatch.delenv("KORCH_GEMM_DMA", raising=False)
    monkeypatch.delenv("KORCH_GEMM_DMA_2STAGE", raising=False)
    monkeypatch.delenv("KORCH_GEMM_DMA8", raising=False)
    monkeypatch.delenv("KORCH_GEMM_DMA_A3", raising=False)
    monkeypatch.delenv("KORCH_GEMM_DMA_STAGES", raising=False)
    (grid, block, lds), src = gemm1({})
    assert "32 A blocks and 24 B blocks of 1 KiB per k-tile, 2 A stages and 3 B stages" in src
    assert lds == (2 * 256 + 3 * 192) * 64 * 2
    assert src.count("global_load_lds_dwordx4") == 2  # the A and the B staging lambda
    assert set(re.findall(r"s_waitcnt vmcnt\((\d+)\)", src)) == {"0"}
    assert "stashA" not in src
    _, src = gemm1(BIG_TILE_CASE)
    assert "global_load_lds_dwordx4" not in src and "stashA" in src
    # asked for (KORCH_GEMM_DMA8=1), the second product (one 128 x 96 tile per
    # compute unit, K = 3072) runs eight waves of 32 x 48 over the whole
    # contraction with three stages of each operand (both loaded two k-tiles
    # ahead by their own wave groups per k-tile parity) instead of the
    # intra-workgroup split of K; with KORCH_GEMM_DMA_STAGES=5, five stages
    # loaded four ahead by one wave per residue of the k-tile index mod 4
    monkeypatch.setenv("KORCH_GEMM_DMA8", "1")
    for stages, par in ((3, "par_ = wv_ / 2 % 2"), (5, "par_ = wv_ / 1 % 4")):
        monkeypatch.setenv("KORCH_GEMM_DMA_STAGES", str(stages))
        p = graphs.build("mlp").plan("layered")
        p.compile()
        (_, block2, lds2), src2 = p.kernel_launch(2), p.kernel_source(2)
        assert f"16 A blocks and 12 B blocks of 1 KiB per k-tile, {stages} A stages and {stages} B stages" in src2
        assert block2 == (512, 1, 1) and lds2 == stages * (128 + 96) * 64 * 2
        assert "kgrp" not in src2 and par in src2
        assert set(re.findall(r"s_waitcnt vmcnt\((\d+)\)", src2)) == {"0"}
    monkeypatch.delenv("KORCH_GEMM_DMA_STAGES")
    monkeypatch.delenv("KORCH_GEMM_DMA8")
    # by default the split keeps register staging; asked for direct-to-LDS
    # staging, each group of four waves has its own 68 KiB of stages (two
    # groups, 136 KiB)
    p = graphs.build("mlp").plan("layered")
    p.compile()
    assert "global_load_lds_dwordx4" not in p.kernel_source(2) and "kgrp" in p.kernel_source(2)
    monkeypatch.setenv("KORCH_GEMM_DMA_KSPLIT", "1")
    p = graphs.build("mlp").plan("layered")
    p.compile()
    (_, block2, lds2), src2 = p.kernel_launch(2), p.kernel_source(2)
    assert block2 == (512, 1, 1) and lds2 == 2 * (2 * 128 + 3 * 96) * 64 * 2
    assert "16 A blocks and 12 B blocks of 1 KiB per k-tile, 2 A stages and 3 B stages" in src2
    assert "readfirstlane(kgrp)" in src2
    monkeypatch.delenv("KORCH_GEMM_DMA_KSPLIT")
    monkeypatch.setenv("KORCH_GEMM_DMA_2STAGE", "1")
    (_, _, lds), src = gemm1({})
    assert "2 A stages and 2 B stages" in src and lds == (2 * 256 + 2 * 192) * 64 * 2
    monkeypatch.setenv("KORCH_GEMM_DMA", "0")
    _, src = gemm1({})
    assert "global_load_lds_dwordx4" not in src and "stashA" in src


@pytest.mark.parametrize("workload,sizes", [("mlp", {}), ("sra", {}), ("mlp", dict(m=1024, d=256, h=768, dtype="bf16"))])
def test_direct_to_lds_kernels_use_m0_only_for_their_loads(workload, sizes):
    """Kernels with direct-to-LDS staging set M0 (the loads' LDS address) in
    inline assembly the compiler does not see: in their disassembly (the
    compiler's own objdump, on code objects built here) every instruction that
    names m0 is an s_mov_b32 to it directly followed by the load, so no value
    the compiler keeps in M0 can be overwritten."""
    import os
    import subprocess
    import tempfile
    objdump = "/opt/rocm/llvm/bin/llvm-objdump"
    if not os.path.exists(objdump):
        pytest.skip("no llvm-objdump")
    w = graphs.build(workload, **sizes)
    seen = 0
    for plan in ("layered", "unfused"):
        p = w.plan(plan)
        p.compile()
        for k in range(p.num_kernels()):
            if "global_load_lds_dwordx4" not in p.kernel_source(k):
                continue
            with tempfile.NamedTemporaryFile(suffix=".co", delete=False) as f:
                f.write(p.kernel_code(k))
            try:
                r = subprocess.run([objdump, "-d", "--mcpu=gfx950", f.name], capture_output=True, text=True)
            finally:
                os.unlink(f.name)
            assert r.returncode == 0, r.stderr[:500]
            ins = [ln.split("//")[0].strip() for ln in r.stdout.splitlines()]
            ins = [ln for ln in ins if ln and not ln.endswith(":") and not ln.startswith("Disassembly")]
            loads = [i for i, ln in enumerate(ins) if ln.startswith("global_load_lds_dwordx4")]
            assert loads
            for i, ln in enumerate(ins):
                if "m0" in ln.replace(",", " ").split():
                    assert ln.startswith("s_mov_b32 m0,") and ins[i + 1].startswith("global_load_lds_dwordx4"), (plan, k, ln)
            assert all(ins[i - 1].startswith("s_mov_b32 m0,") for i in loads)
            seen += 1
    assert seen


def test_attention_key_split_selection():
    """Few query rows split the keys over the waves (one workgroup per 16 rows);
    the SRA workload's 16384 queries keep one workgroup per 64 rows."""
    from paper_2406_09465_amd.warm import ATTN_CASES

    def launch_and_src(workload, sizes):
        p = graphs.build(workload, **sizes).plan("fused")
        p.compile()
        k = [i for i in range(p.num_kernels()) if "attention" in p.kernel_name(i)][0]
        return p.kernel_launch(k), p.kernel_source(k)

    prev = os.environ.pop("KORCH_ATTN_NO_KEY_SPLIT", None)
    try:
        for wl, sz in ATTN_CASES:
            (grid, _, _), src = launch_and_src(wl, sz)
            nq = sz["n"] if wl == "attention" else sz["hh"] * sz["ww"]
            assert "this wave's keys" in src and grid[0] == (nq + 15) // 16, (wl, sz)
        (grid, _, _), src = launch_and_src("sra", {})
        assert "this wave's keys" not in src and grid[0] == 16384 // 64
        os.environ["KORCH_ATTN_NO_KEY_SPLIT"] = "1"
        (grid, _, _), src = launch_and_src("attention", {})
        assert "this wave's keys" not in src and grid[0] == 2
    finally:
        os.environ.pop("KORCH_ATTN_NO_KEY_SPLIT", None)
        if prev is not None:
            os.environ["KORCH_ATTN_NO_KEY_SPLIT"] = prev


def test_runtime_compiler_helper(tmp_path):
    """The helper that compiles cache misses in a child process: a code object
    for a valid kernel, exit status 1 and the compiler's log for a broken one."""
    import subprocess
    helper = os.path.join(os.path.dirname(K.LIB_PATH), "korch_rtc")
    opts = ["--offload-arch=gfx950", "-O3", "-std=c++17"]
    good = tmp_path / "good.hip"
    good.write_text('extern "C" __global__ void k(float* p) { p[threadIdx.x] += 1.0f; }\n')
    r = subprocess.run([helper, str(good), "k", str(tmp_path / "good.co"), str(tmp_path / "good.log"), *opts],
                       capture_output=True, text=True, timeout=300)
    assert r.returncode == 0, r.stderr
    assert (tmp_path / "good.co").read_bytes()[:4] in (b"\x7fELF", b"__CL")
    bad = tmp_path / "bad.hip"
    bad.write_text('extern "C" __global__ void k(float* p) { p[threadIdx.x] += undeclared_name; }\n')
    r = subprocess.run([helper, str(bad), "k", str(tmp_path / "bad.co"), str(tmp_path / "bad.log"), *opts],
                       capture_output=True, text=True, timeout=300)
    assert r.returncode == 1 and "undeclared_name" in (tmp_path / "bad.log").read_text()


def test_flush_rejects_bad_buffers_before_any_device_call():
    """korch_flush_caches checks its arguments on the host: a null buffer
    (with a size) and a misaligned one are refused without launching."""
    import ctypes as C

    from paper_2406_09465_amd._abi import lib
    assert lib.korch_flush_caches(None, C.c_size_t(1 << 20), 0, None) == -1  # KORCH_E_ARG
    assert lib.korch_flush_caches(C.c_void_p(0x1008), C.c_size_t(1 << 20), 1, None) == -21  # KORCH_E_ALIGN


@pytest.mark.parametrize("workload", list(graphs.BUILDERS))
def test_standard_plan_kernels_do_not_spill(workload):
    """No generated kernel of a workload's hand-written and unfused plans keeps
    registers in scratch memory (its code object's private segment is empty):
    a kernel whose first build spills is generated again with register relief."""
    from paper_2406_09465_amd import codeobj
    w = graphs.build(workload)
    for plan in ("fused", "layered", "unfused"):
        p = w.plan(plan)
        p.compile()
        for k in range(p.num_kernels()):
            for name, r in codeobj.kernel_resources(p.kernel_code(k)).items():
                assert r["scratch"] == 0 and r["vgpr_spill"] == 0, (workload, plan, name, r)
                assert r["vgpr"] <= 512 and r["lds"] <= 160 * 1024


def test_spilling_kernel_is_regenerated_with_register_relief():
    """The MLP's fused plan puts LayerNorm's apply step in the first product's
    operand prologue; with 256 x 192 tiles and two fragment register sets that
    kernel spills, so compilation regenerates it (one fragment set, then
    smaller tiles) until its code object needs no scratch."""
    import re

    from paper_2406_09465_amd import codeobj
    w = graphs.build("mlp")
    p = w.plan("fused")
    first = p.kernel_source(1)  # generated, not yet compiled
    p.compile()
    final = p.kernel_source(1)
    assert "frag1(" in first and final != first
    (r,) = codeobj.kernel_resources(p.kernel_code(1)).values()
    assert r["scratch"] == 0
    assert re.search(r"__launch_bounds__\((\d+)\)", final).group(1) == "256"  # 128-row tiles, four waves
