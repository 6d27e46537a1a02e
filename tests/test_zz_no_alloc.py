"""The route without allocation (skip_route_fused_noalloc), through the C
ABI, against the route with a caller workspace: kept indices, attention
outputs and LSE bitwise equal (the two share every kernel), on two calls in a
row, the second with a smaller batch (the library's scratch then holds the
first call's values)."""
import sys

import pytest
import torch

from paper_2607_25422_amd import workloads as wls

pytestmark = pytest.mark.gpu


def say(*a):
    print(*a, file=sys.stderr, flush=True)


@pytest.fixture(scope="module")
def B():
    assert torch.cuda.is_available(), "GPU tests need a HIP device"
    from paper_2607_25422_amd import binding
    return binding


def _outputs(B, db):
    p = db.p
    dev = db.V.device
    n = max(p.total_kept, 1)
    return (torch.full((n,), -7, dtype=torch.int32, device=dev),
            torch.full((n, p.H, p.d_h), float("nan"), dtype=db.V.dtype, device=dev),
            torch.full((n, p.H), float("nan"), dtype=torch.float32, device=dev))


def _noalloc(B, db, out):
    p = db.p
    kept_idx, O, lse = out
    B.skip_route_fused_noalloc(p, db.V, db.Qtok, db.q_offsets, db.w_bias, db.kept_offsets,
                               db.Kh, db.Vh, db.passage_offsets, db.query_passages, kept_idx,
                               O, lse)


def _same(a, b):
    return torch.equal(a.view(torch.uint8) if a.dtype != torch.int32 else a,
                       b.view(torch.uint8) if b.dtype != torch.int32 else b)


@pytest.mark.parametrize("first,second", [(("highres_bf16", 16), ("highres_bf16", 5)),
                                          (("longctx_bf16", 4), ("llava_bf16", 3))])
def test_noalloc_matches_workspace_route(B, first, second):
    for name, nb in (first, second):
        say(f"[noalloc] {name} B={nb}")
        batch = wls.make_batch(name, 2026, B=nb)
        db = B.to_device(batch)
        assert B.workspace_bytes(db.p) <= B.NOALLOC_SCRATCH_BYTES
        ref = _outputs(B, db)
        got = _outputs(B, db)
        B.route_fused(db, out=ref)
        _noalloc(B, db, got)
        torch.cuda.synchronize()
        k = db.p.total_kept
        for r, g, what in zip(ref, got, ("kept_idx", "O", "lse")):
            assert _same(r[:k], g[:k]), f"{name} B={nb}: {what} differs"
        # a repeat on the same inputs gives the same bits again
        _noalloc(B, db, got)
        torch.cuda.synchronize()
        for r, g, what in zip(ref, got, ("kept_idx", "O", "lse")):
            assert _same(r[:k], g[:k]), f"{name} B={nb}: repeat {what} differs"


def test_noalloc_rejects_a_problem_above_the_scratch(B):
    batch = wls.make_batch("mixed_bf16", 2026, B=16)
    db = B.to_device(batch)
    assert B.workspace_bytes(db.p) > B.NOALLOC_SCRATCH_BYTES
    with pytest.raises(B.SkipError) as e:
        _noalloc(B, db, _outputs(B, db))
    assert e.value.status == B.SKIP_ERR_WORKSPACE
