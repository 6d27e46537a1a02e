"""The C ABI on the host: the library loads, exports every symbol the header
declares, and rejects bad arguments before touching any device (no GPU needed:
every call here fails validation before anything is enqueued)."""
import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "skip.h")


@pytest.fixture(scope="module")
def b():
    from paper_2607_25422_amd import binding
    return binding


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(skip_[a-z_]+)\s*\(", text)))


def test_header_declares_the_three_entry_points():
    names = declared_functions()
    for n in ("skip_prune_topk", "skip_bipartite_xattn", "skip_route_fused"):
        assert n in names


def test_library_exports_every_declared_symbol(b):
    for name in declared_functions():
        assert hasattr(b.LIB, name), name
    assert set(b.ENTRY_POINTS) == set(declared_functions())


def test_version_and_status_strings(b):
    assert b.abi_version() == 7
    for s in range(5):
        assert b.status_string(s).startswith("SKIP_")
    assert "UNKNOWN" in b.status_string(99)


def test_problem_struct_layout(b):
    # 14 int32, a double at offset 56, a float and three int32 after it, a
    # double at 80 (the library asserts the same layout at compile time)
    assert ctypes.sizeof(b.SkipProblem) == 88
    assert b.SkipProblem.avg_degree.offset == 56
    assert b.SkipProblem.edge_rule.offset == 72
    assert b.SkipProblem.edge_metric.offset == 76
    assert b.SkipProblem.edge_beta.offset == 80


def _problem(b, **kw):
    base = dict(B=2, N=576, d=1024, H=16, d_h=64, q_offsets=[0, 3, 7],
                kept_offsets=[0, 96, 192], passage_offsets=[0, 10, 20, 30],
                query_passages=[0, 2, 3], sm_scale=0.125)
    base.update(kw)
    return b.make_problem("bf16", **base)


def test_workspace_bytes(b):
    p = _problem(b)
    n = b.workspace_bytes(p)
    # u + z + kbar + edge partials (4 slices of 256 columns) + row-norm and
    # key-norm partials + rowmask + the attention work list (16 bytes per
    # workgroup id: 8 ids per run of 8 (question, head) groups, 2 * 16 groups,
    # one chunk of <= 192 rows) + one prune counter per question, each rounded
    # to 256 bytes
    S = 4
    parts = [2 * 1024 * 8, 2 * 576 * 8, 3 * 1024 * 8, 2 * S * 96 * 2 * 8, 2 * S * 96 * 8,
             2 * S * 2 * 8, 192 * 8, 4 * 8 * 16, 2 * 4]
    assert n == sum((x + 255) // 256 * 256 for x in parts)
    with pytest.raises(b.SkipError):
        b.workspace_bytes(_problem(b, B=0, q_offsets=[0], kept_offsets=[0], query_passages=[0]))


FAKE = 1 << 40   # never dereferenced: every call below fails validation


def _prune(b, p, ws_bytes=1 << 30, **ptrs):
    args = dict(V=FAKE, Qtok=FAKE, q_off=FAKE, w=None, k_off=FAKE, idx=FAKE, scores=None,
                vk=None, ws=FAKE)
    args.update(ptrs)
    return b.LIB.skip_prune_topk(ctypes.byref(p), args["V"], args["Qtok"], args["q_off"],
                                 args["w"], args["k_off"], args["idx"], args["scores"],
                                 args["vk"], args["ws"], ws_bytes, None)


def test_prune_rejects_bad_arguments(b):
    p = _problem(b)
    assert _prune(b, p, V=None) == b.SKIP_ERR_INVALID_ARG
    assert _prune(b, p, idx=None) == b.SKIP_ERR_INVALID_ARG
    assert _prune(b, p, ws=None) == b.SKIP_ERR_INVALID_ARG
    assert _prune(b, p, ws_bytes=16) == b.SKIP_ERR_WORKSPACE
    assert _prune(b, _problem(b, kept_offsets=[0, 600, 700])) == b.SKIP_ERR_INVALID_ARG  # k > N
    assert _prune(b, _problem(b, N=20000)) == b.SKIP_ERR_UNSUPPORTED
    assert _prune(b, _problem(b, d=1020, H=15, d_h=68)) == b.SKIP_ERR_UNSUPPORTED
    q = _problem(b)
    q.o_f32 = 2
    assert _prune(b, q) == b.SKIP_ERR_INVALID_ARG
    q = _problem(b)
    q.dtype = 7
    assert _prune(b, q) == b.SKIP_ERR_INVALID_ARG
    q = _problem(b)
    q.total_qtok = 1          # fewer question tokens than questions
    assert _prune(b, q) == b.SKIP_ERR_INVALID_ARG


def _xattn(b, p, ws_bytes=1 << 30, **ptrs):
    a = dict(Qh=FAKE, k_off=FAKE, Kh=FAKE, Vh=FAKE, p_off=FAKE, qp=FAKE, pk=None, erp=None,
             ecol=None, O=FAKE, lse=None, rp_out=None, col_out=None, ws=FAKE)
    a.update(ptrs)
    return b.LIB.skip_bipartite_xattn(ctypes.byref(p), a["Qh"], a["k_off"], a["Kh"], a["Vh"],
                                      a["p_off"], a["qp"], a["pk"], a["erp"], a["ecol"], a["O"],
                                      a["lse"], a["rp_out"], a["col_out"], a["ws"], ws_bytes,
                                      None)


def test_mlp_scorer_struct_and_validation(b):
    assert ctypes.sizeof(b.SkipQvsMlp) == 40
    assert b.SkipQvsMlp.b2.offset == 32
    p = _problem(b)
    n = b.workspace_bytes_mlp(p, 512)
    assert n > b.workspace_bytes(p)
    assert b.workspace_bytes_mlp(p, 1024) > n

    def call(q, m=None, ws_bytes=1 << 30, **kw):
        m = m if m is not None else b.SkipQvsMlp(512, 0, FAKE, None, FAKE, 0.5)
        args = dict(V=FAKE, Qtok=FAKE, qo=FAKE, ko=FAKE, idx=FAKE)
        args.update(kw)
        return b.LIB.skip_prune_topk_mlp(ctypes.byref(q), ctypes.byref(m) if m is not False else None,
                                         args["V"], args["Qtok"], args["qo"], args["ko"],
                                         args["idx"], None, None, FAKE, ws_bytes, None)
    assert call(p, m=False) == b.SKIP_ERR_INVALID_ARG                      # no scorer
    assert call(p, V=None) == b.SKIP_ERR_INVALID_ARG
    assert call(p, m=b.SkipQvsMlp(512, 1, FAKE, None, FAKE, 0.0)) == b.SKIP_ERR_INVALID_ARG
    assert call(p, m=b.SkipQvsMlp(512, 0, None, None, FAKE, 0.0)) == b.SKIP_ERR_INVALID_ARG
    assert call(p, m=b.SkipQvsMlp(512, 0, FAKE, None, FAKE, float("inf"))) == b.SKIP_ERR_INVALID_ARG
    assert call(p, m=b.SkipQvsMlp(384, 0, FAKE, None, FAKE, 0.0)) == b.SKIP_ERR_UNSUPPORTED
    assert call(p, m=b.SkipQvsMlp(8192, 0, FAKE, None, FAKE, 0.0)) == b.SKIP_ERR_UNSUPPORTED
    q = b.make_problem("f32", B=2, N=576, d=1024, q_offsets=[0, 3, 7], kept_offsets=[0, 96, 192])
    assert call(q) == b.SKIP_ERR_UNSUPPORTED                              # bf16 only
    q = b.make_problem("bf16", B=2, N=576, d=1000, q_offsets=[0, 3, 7], kept_offsets=[0, 96, 192])
    assert call(q) == b.SKIP_ERR_UNSUPPORTED                              # d % 32
    assert call(p, ws_bytes=n - 1) == b.SKIP_ERR_WORKSPACE
    with pytest.raises(b.SkipError):
        b.workspace_bytes_mlp(p, 100)


def test_xattn_rejects_bad_arguments(b):
    p = _problem(b)
    assert _xattn(b, p, O=None) == b.SKIP_ERR_INVALID_ARG
    assert _xattn(b, p, Kh=None) == b.SKIP_ERR_INVALID_ARG
    assert _xattn(b, p, rp_out=FAKE) == b.SKIP_ERR_INVALID_ARG          # one of a pair
    assert _xattn(b, p, erp=FAKE, rp_out=FAKE, col_out=FAKE) == b.SKIP_ERR_INVALID_ARG
    assert _xattn(b, p, ws_bytes=0) == b.SKIP_ERR_WORKSPACE
    assert _xattn(b, _problem(b, d_h=32, H=32)) == b.SKIP_ERR_UNSUPPORTED
    assert _xattn(b, _problem(b, H=8)) == b.SKIP_ERR_INVALID_ARG          # H*d_h != d
    many = list(range(0, 70 * 10 + 1, 10))
    assert _xattn(b, _problem(b, passage_offsets=many, query_passages=[0, 65, 70])) \
        == b.SKIP_ERR_UNSUPPORTED                                           # P > 64
    q = _problem(b)
    q.avg_degree = float("nan")
    assert _xattn(b, q) == b.SKIP_ERR_INVALID_ARG
    q = _problem(b)
    q.total_tokens = 1        # fewer tokens than passages
    assert _xattn(b, q) == b.SKIP_ERR_INVALID_ARG
    for field, value in (("edge_rule", 3), ("edge_rule", -1), ("edge_metric", 2)):
        q = _problem(b)
        setattr(q, field, value)
        assert _xattn(b, q) == b.SKIP_ERR_INVALID_ARG, (field, value)
    for beta in (0.0, -0.5, 1.5, float("nan")):
        q = _problem(b, edge_rule="fraction", edge_beta=beta)
        assert _xattn(b, q) == b.SKIP_ERR_INVALID_ARG, beta
    q = _problem(b, edge_rule="question", edge_beta=0.0)    # beta unused: accepted
    assert _xattn(b, q, ws_bytes=0) == b.SKIP_ERR_WORKSPACE


def test_misaligned_element_arrays_are_rejected(b):
    """Element arrays are read with 16-byte vector and direct-to-LDS loads:
    each one shifted by 8 bytes is an argument error, found before anything
    is enqueued."""
    MIS = FAKE + 8
    p = _problem(b)
    for name in ("V", "Qtok", "w", "vk"):
        assert _prune(b, p, **{name: MIS}) == b.SKIP_ERR_INVALID_ARG, name
    for name in ("Qh", "Kh", "Vh", "O"):
        assert _xattn(b, p, **{name: MIS}) == b.SKIP_ERR_INVALID_ARG, name

    def fused(V=FAKE, Qtok=FAKE, w=None, Kh=FAKE, Vh=FAKE, pk=None, O=FAKE):
        return b.LIB.skip_route_fused(ctypes.byref(p), V, Qtok, FAKE, w, FAKE, Kh, Vh, FAKE,
                                      FAKE, pk, FAKE, O, None, FAKE, 1 << 30, None)
    for name in ("V", "Qtok", "w", "Kh", "Vh", "pk", "O"):
        assert fused(**{name: MIS}) == b.SKIP_ERR_INVALID_ARG, name
    # the float passage-key table is read with 16-byte loads too
    assert _xattn(b, p, pk=MIS) == b.SKIP_ERR_INVALID_ARG
    assert _xattn(b, p, pk=FAKE, ws_bytes=0) == b.SKIP_ERR_WORKSPACE     # aligned: passes
    m = b.SkipQvsMlp(512, 0, MIS, None, FAKE, 0.5)
    assert b.LIB.skip_prune_topk_mlp(ctypes.byref(p), ctypes.byref(m), FAKE, FAKE, FAKE, FAKE,
                                     FAKE, None, None, FAKE, 1 << 30, None) \
        == b.SKIP_ERR_INVALID_ARG                                          # W1


def test_fused_requires_matching_head_split(b):
    p = _problem(b, H=8)      # 8 * 64 != 1024
    st = b.LIB.skip_route_fused(ctypes.byref(p), FAKE, FAKE, FAKE, None, FAKE, FAKE, FAKE,
                                FAKE, FAKE, None, FAKE, FAKE, None, FAKE, 1 << 30, None)
    assert st == b.SKIP_ERR_INVALID_ARG
    p = _problem(b)
    st = b.LIB.skip_route_fused(ctypes.byref(p), FAKE, FAKE, FAKE, None, FAKE, FAKE, FAKE,
                                FAKE, FAKE, None, None, FAKE, None, FAKE, 1 << 30, None)
    assert st == b.SKIP_ERR_INVALID_ARG                                   # kept_idx NULL


def test_gate_struct_and_validation(b):
    assert ctypes.sizeof(b.SkipSkvGate) == 56
    assert b.SkipSkvGate.b2.offset == 32
    assert b.SkipSkvGate.rho.offset == 48
    p = _problem(b)
    n = b.workspace_bytes_gate(p, 256)
    assert n > b.workspace_bytes(p)
    assert b.workspace_bytes_gate(p, 512) > n

    def gate(h=256, reserved=0, W=FAKE, w2=FAKE, b2=0.0, tau=0.5, rho=0.5):
        return b.SkipSkvGate(h, reserved, W, None, w2, b2, tau, rho)

    def call(q, g=None, ws_bytes=1 << 30, **kw):
        g = g if g is not None else gate()
        a = dict(Qtok=FAKE, qo=FAKE, Vk=FAKE, ko=FAKE, Kh=FAKE, po=FAKE, qp=FAKE, pk=None,
                 logits=None, keep=FAKE)
        a.update(kw)
        return b.LIB.skip_skv_gate(ctypes.byref(q), ctypes.byref(g) if g is not False else None,
                                   a["Qtok"], a["qo"], a["Vk"], a["ko"], a["Kh"], a["po"],
                                   a["qp"], a["pk"], a["logits"], a["keep"], FAKE, ws_bytes,
                                   None)
    # every call fails validation (the last ones on the workspace size)
    assert call(p, g=False) == b.SKIP_ERR_INVALID_ARG
    assert call(p, Qtok=None) == b.SKIP_ERR_INVALID_ARG
    assert call(p, keep=None) == b.SKIP_ERR_INVALID_ARG
    assert call(p, Vk=None) == b.SKIP_ERR_INVALID_ARG
    assert call(p, Kh=None) == b.SKIP_ERR_INVALID_ARG        # keys neither given nor poolable
    assert call(p, g=gate(reserved=1)) == b.SKIP_ERR_INVALID_ARG
    assert call(p, g=gate(W=None)) == b.SKIP_ERR_INVALID_ARG
    assert call(p, g=gate(W=FAKE + 8)) == b.SKIP_ERR_INVALID_ARG        # 16-byte alignment
    assert call(p, g=gate(b2=float("nan"))) == b.SKIP_ERR_INVALID_ARG
    for tau in (0.0, 1.0, -0.1, float("nan")):
        assert call(p, g=gate(tau=tau)) == b.SKIP_ERR_INVALID_ARG, tau
    for rho in (0.0, 1.5, float("nan")):
        assert call(p, g=gate(rho=rho)) == b.SKIP_ERR_INVALID_ARG, rho
    assert call(p, g=gate(h=96)) == b.SKIP_ERR_UNSUPPORTED
    assert call(p, g=gate(h=8192)) == b.SKIP_ERR_UNSUPPORTED
    q = b.make_problem("f32", B=2, N=576, d=1024, H=16, d_h=64, q_offsets=[0, 3, 7],
                       kept_offsets=[0, 96, 192], passage_offsets=[0, 10, 20, 30],
                       query_passages=[0, 2, 3], sm_scale=0.125)
    assert call(q) == b.SKIP_ERR_UNSUPPORTED                              # bf16 only
    assert call(p, ws_bytes=b.workspace_bytes_gate(p, 256) - 1) == b.SKIP_ERR_WORKSPACE
    assert call(p, Kh=None, pk=FAKE, ws_bytes=0) == b.SKIP_ERR_WORKSPACE  # given keys: no Kh
    assert call(p, Kh=None, pk=FAKE + 4, ws_bytes=0) == b.SKIP_ERR_INVALID_ARG  # misaligned
    with pytest.raises(b.SkipError):
        b.workspace_bytes_gate(p, 100)


def test_masked_xattn_validation(b):
    p = _problem(b)

    def call(q, keep=FAKE, ws_bytes=1 << 30, O=FAKE):
        return b.LIB.skip_bipartite_xattn_masked(ctypes.byref(q), FAKE, FAKE, FAKE, FAKE, FAKE,
                                                 FAKE, None, keep, O, None, None, None, FAKE,
                                                 ws_bytes, None)
    assert call(p, keep=None) == b.SKIP_ERR_INVALID_ARG
    assert call(p, O=None) == b.SKIP_ERR_INVALID_ARG
    assert call(p, ws_bytes=0) == b.SKIP_ERR_WORKSPACE
    assert call(_problem(b, H=8)) == b.SKIP_ERR_INVALID_ARG


def test_region_kmeans_validation(b):
    p = _problem(b)
    n = b.workspace_bytes_regions(p, 8)
    assert n > 0 and b.workspace_bytes_regions(p, 16) > n
    with pytest.raises(b.SkipError):
        b.workspace_bytes_regions(p, 0)
    with pytest.raises(b.SkipError):
        b.workspace_bytes_regions(p, 17)

    def call(q, rows=FAKE, ko=FAKE, idx=None, r_max=8, n_iter=10, region=FAKE, cent=FAKE,
             ws=FAKE, ws_bytes=1 << 30):
        return b.LIB.skip_region_kmeans(ctypes.byref(q), rows, ko, idx, r_max, n_iter, region,
                                        cent, None, ws, ws_bytes, None)
    # every call fails validation
    assert call(p, rows=None) == b.SKIP_ERR_INVALID_ARG
    assert call(p, ko=None) == b.SKIP_ERR_INVALID_ARG
    assert call(p, region=None) == b.SKIP_ERR_INVALID_ARG
    assert call(p, cent=None) == b.SKIP_ERR_INVALID_ARG
    assert call(p, ws=None) == b.SKIP_ERR_INVALID_ARG
    for r_max in (0, 17, -1):
        assert call(p, r_max=r_max) == b.SKIP_ERR_INVALID_ARG, r_max
    for n_iter in (0, 1001):
        assert call(p, n_iter=n_iter) == b.SKIP_ERR_INVALID_ARG, n_iter
    assert call(p, rows=FAKE + 8) == b.SKIP_ERR_INVALID_ARG     # rows 16-byte aligned
    q = _problem(b)
    q.k_max = 600             # kept rows read through kept_idx need k_max <= N
    q.total_kept = 1200
    assert call(q, idx=FAKE) == b.SKIP_ERR_INVALID_ARG
    assert call(p, ws_bytes=n - 1) == b.SKIP_ERR_WORKSPACE


def test_projection_and_edge_rows_validation(b):
    p = _problem(b)
    n = b.workspace_bytes_project(p, 256)
    assert n == 256 * 1024 * 2
    with pytest.raises(b.SkipError):
        b.workspace_bytes_project(p, 100)

    def proj(q, rows=FAKE, W=FAKE, d_out=256, Y=FAKE, f32=0, idx=None, ws_bytes=1 << 30):
        return b.LIB.skip_gather_project(ctypes.byref(q), rows, FAKE, idx, W, d_out, Y, f32,
                                         FAKE, ws_bytes, None)
    # every call fails validation
    assert proj(p, rows=None) == b.SKIP_ERR_INVALID_ARG
    assert proj(p, W=None) == b.SKIP_ERR_INVALID_ARG
    assert proj(p, Y=None) == b.SKIP_ERR_INVALID_ARG
    assert proj(p, f32=2) == b.SKIP_ERR_INVALID_ARG
    assert proj(p, W=FAKE + 8) == b.SKIP_ERR_INVALID_ARG
    assert proj(p, d_out=300) == b.SKIP_ERR_UNSUPPORTED
    assert proj(p, d_out=0) == b.SKIP_ERR_INVALID_ARG
    q = b.make_problem("f32", B=2, N=576, d=1024, q_offsets=[0, 3, 7], kept_offsets=[0, 96, 192])
    assert proj(q) == b.SKIP_ERR_UNSUPPORTED
    assert proj(p, ws_bytes=n - 1) == b.SKIP_ERR_WORKSPACE

    # packing once and multiplying with the packed copy
    def pack(q, W=FAKE, d_out=256, packed=FAKE, nbytes=1 << 30):
        return b.LIB.skip_pack_projection(ctypes.byref(q), W, d_out, packed, nbytes, None)
    assert pack(p, W=None) == b.SKIP_ERR_INVALID_ARG
    assert pack(p, packed=None) == b.SKIP_ERR_INVALID_ARG
    assert pack(p, packed=FAKE + 8) == b.SKIP_ERR_INVALID_ARG
    assert pack(p, d_out=300) == b.SKIP_ERR_UNSUPPORTED
    assert pack(q) == b.SKIP_ERR_UNSUPPORTED
    assert pack(p, nbytes=n - 1) == b.SKIP_ERR_WORKSPACE

    def packed_call(q, rows=FAKE, packed=FAKE, d_out=256, Y=FAKE, f32=0):
        return b.LIB.skip_gather_project_packed(ctypes.byref(q), rows, FAKE, None, packed, d_out,
                                                Y, f32, None)
    assert packed_call(p, packed=None) == b.SKIP_ERR_INVALID_ARG
    assert packed_call(p, rows=None) == b.SKIP_ERR_INVALID_ARG
    assert packed_call(p, Y=FAKE + 2) == b.SKIP_ERR_INVALID_ARG
    assert packed_call(p, f32=3) == b.SKIP_ERR_INVALID_ARG
    assert packed_call(p, d_out=512 + 128) == b.SKIP_ERR_UNSUPPORTED

    def xp(q, edge=FAKE, keys=FAKE, ws_bytes=0):
        return b.LIB.skip_bipartite_xattn_proj(ctypes.byref(q), FAKE, edge, FAKE, FAKE, FAKE,
                                               FAKE, FAKE, keys, None, FAKE, None, None, None,
                                               FAKE, ws_bytes, None)
    assert xp(p, edge=None) == b.SKIP_ERR_INVALID_ARG
    assert xp(p, keys=None) == b.SKIP_ERR_INVALID_ARG
    assert xp(p) == b.SKIP_ERR_WORKSPACE


def test_noalloc_route_validation(b):
    """The route without allocation checks everything on the host first: bad
    arguments and problems whose workspace exceeds the library's scratch are
    rejected before any HIP call (no GPU here)."""
    def call(q, V=FAKE, O=FAKE, pk=None):
        return b.LIB.skip_route_fused_noalloc(ctypes.byref(q), V, FAKE, FAKE, None, FAKE, FAKE,
                                              FAKE, FAKE, FAKE, pk, FAKE, O, None, None)
    p = _problem(b)
    assert b.workspace_bytes(p) <= b.NOALLOC_SCRATCH_BYTES
    assert call(p, V=None) == b.SKIP_ERR_INVALID_ARG
    assert call(p, O=FAKE + 8) == b.SKIP_ERR_INVALID_ARG
    assert call(p, pk=FAKE + 4) == b.SKIP_ERR_INVALID_ARG
    assert call(_problem(b, H=8)) == b.SKIP_ERR_INVALID_ARG
    # 8 questions x 40 passages of width 8192: the float64 passage keys alone
    # take 21 MB, above the 16 MiB scratch
    big = b.make_problem("bf16", B=8, N=576, d=8192, H=64, d_h=128,
                         q_offsets=list(range(0, 9 * 4, 4)),
                         kept_offsets=list(range(0, 9 * 96, 96)),
                         passage_offsets=list(range(0, 321 * 16, 16)),
                         query_passages=list(range(0, 321, 40)), sm_scale=0.125)
    assert b.workspace_bytes(big) > b.NOALLOC_SCRATCH_BYTES
    assert call(big) == b.SKIP_ERR_WORKSPACE
