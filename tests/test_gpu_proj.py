"""GPU parity of the learned row projection (gathered GEMM on the matrix
cores) and of the graph cut on separate edge rows, through the C ABI,
against the CPU oracle.

Bars:
* projection: |y - y_ref| <= (K/16 + 2) 2^-24 sum_k |x_k w_k| (float32 sums
  of exact bf16 products, one rounding per 16-product MFMA step), plus half a
  bf16 ulp of |y_ref| when Y is stored as bf16;
* graph on given edge rows and keys (both inputs, computed by the oracle):
  edge sets identical, attention as in the other attention tests.
"""
import sys

import numpy as np
import pytest
import torch

import oracle as orc
from paper_2607_25422_amd import workloads as wls

from test_gpu_parity import check_attention, check_graph, f64, queries_from_batch
from test_gpu_regions import kept_oracle

pytestmark = pytest.mark.gpu


def say(*a):
    print(*a, file=sys.stderr, flush=True)


@pytest.fixture(scope="module")
def B():
    assert torch.cuda.is_available(), "GPU tests need a HIP device"
    from paper_2607_25422_amd import binding
    return binding


def check_projection(X, W, Y, bf16_out, rows=None, tag=""):
    """X [M, d] and W [d_out, d] as float64 numpy; Y the GPU output."""
    Xs = X if rows is None else X[rows]
    ref = orc.project_rows(Xs, W)
    mag = np.abs(Xs) @ np.abs(W).T
    K = X.shape[1]
    got = Y.cpu().double().numpy()
    if rows is not None:
        got = got[rows]
    bound = (K / 16 + 2) * 2.0 ** -24 * mag + (2.0 ** -8 * np.abs(ref) if bf16_out else 0.0)
    excess = np.abs(got - ref) - bound
    worst = float(np.max(np.abs(got - ref) / np.maximum(mag, 1e-300)))
    say(f"{tag}: max |y - y_ref| / sum|x w| = {worst:.2e}")
    assert np.all(excess <= 0), f"{tag}: projection error beyond the bound"


def kept_rows(batch, kept):
    return torch.cat([batch.V[b][torch.from_numpy(kept[b].astype(np.int64))]
                      for b in range(batch.B)]).contiguous()


@pytest.mark.parametrize("d_out", [256, 512])
@pytest.mark.parametrize("seed", wls.SEEDS)
def test_project_small_ragged(B, seed, d_out):
    batch = wls.make_batch("llava_bf16", seed, B=5, N=300, H=4, d_h=64, T=(1, 3),
                           k=(0, 1, 7, 33, 64, 130))
    say(f"projection small seed={seed} d_out={d_out} k={batch.k.tolist()}")
    kept = kept_oracle(batch)
    rows = kept_rows(batch, kept)
    W = wls.make_projection(d_out, batch.wl.d, seed)
    db = B.to_device(batch)
    Wd = W.cuda()
    idx = torch.from_numpy(np.concatenate(kept).astype(np.int32)).cuda()
    y_rows = B.gather_project(db, rows.cuda(), Wd)
    y_idx = B.gather_project(db, db.V, Wd, kept_idx=idx)
    y32 = B.gather_project(db, db.V, Wd, kept_idx=idx, out_f32=True)
    torch.cuda.synchronize()
    assert torch.equal(y_rows, y_idx), "rows in place and gathered rows disagree"
    X = rows.double().numpy()
    Wn = W.double().numpy()
    check_projection(X, Wn, y_idx, True, tag=f"bf16 out d_out={d_out}")
    check_projection(X, Wn, y32, False, tag=f"f32 out d_out={d_out}")
    # the bf16 output is the rounding of the float32 one
    assert torch.equal(y32.to(torch.bfloat16), y_idx)


@pytest.mark.parametrize("d_out", [256, 512])
def test_project_permutation_exact(B, d_out):
    """W selecting one input column per output (a permutation of the d
    columns, repeated and scaled by 2 past the first d outputs): every output
    is one exact product, so Y equals the selected, scaled columns of the
    kept rows bit for bit, through the one-call and the packed paths (eq.
    (bsca)'s W_v x with a W whose product is known exactly)."""
    batch = wls.make_batch("llava_bf16", 11, B=4, N=300, H=4, d_h=64, T=(1, 3),
                           k=(0, 7, 64, 130))
    d = batch.wl.d
    rng = np.random.default_rng(11)
    perm = rng.permutation(d)
    W = torch.zeros((d_out, d), dtype=torch.float32)
    for o in range(d_out):
        W[o, perm[o % d]] = 1.0 if o < d else 2.0
    W = W.to(torch.bfloat16)
    say(f"projection permutation d_out={d_out} k={batch.k.tolist()}")
    kept = kept_oracle(batch)
    rows = kept_rows(batch, kept)
    cols = torch.from_numpy(np.array([perm[o % d] for o in range(d_out)], dtype=np.int64))
    scale = torch.tensor([1.0 if o < d else 2.0 for o in range(d_out)], dtype=torch.float32)
    want = rows.float()[:, cols] * scale
    db = B.to_device(batch)
    Wd = W.cuda()
    idx = torch.from_numpy(np.concatenate(kept).astype(np.int32)).cuda()
    packed = B.pack_projection(db, Wd)
    outs = [B.gather_project(db, db.V, Wd, kept_idx=idx, out_f32=True),
            B.gather_project_packed(db, rows.cuda(), packed, d_out, out_f32=True),
            B.gather_project(db, rows.cuda(), Wd).float()]
    torch.cuda.synchronize()
    for i, y in enumerate(outs):
        assert torch.equal(y.cpu(), want), f"output {i} is not the selected columns"


@pytest.mark.parametrize("d_out", [256, 768])
def test_project_packed_matches_one_call(B, d_out):
    """Weights packed once and reused: every output bitwise equal to the
    one-call projection (bf16 and float outputs, rows in place and through
    the kept indices), on two batches in a row."""
    W = wls.make_projection(d_out, 256, 3)
    Wd = W.cuda()
    for seed, k in ((3, (0, 5, 64, 130)), (4, (1, 33))):
        batch = wls.make_batch("llava_bf16", seed, B=len(k), N=300, H=4, d_h=64, T=(1, 3), k=k)
        say(f"projection packed seed={seed} d_out={d_out} k={batch.k.tolist()}")
        kept = kept_oracle(batch)
        db = B.to_device(batch)
        packed = B.pack_projection(db, Wd)
        idx = torch.from_numpy(np.concatenate(kept).astype(np.int32)).cuda()
        rows = kept_rows(batch, kept).cuda()
        for out_f32 in (False, True):
            one = B.gather_project(db, db.V, Wd, kept_idx=idx, out_f32=out_f32)
            two = B.gather_project_packed(db, db.V, packed, d_out, kept_idx=idx, out_f32=out_f32)
            three = B.gather_project_packed(db, rows, packed, d_out, out_f32=out_f32)
            torch.cuda.synchronize()
            assert torch.equal(one, two) and torch.equal(one, three), (seed, out_f32)


def test_project_full_size(B):
    """highres_bf16: 3072 kept rows read in place through the kept indices,
    W 4096 x 4096; 64 sampled rows checked against the oracle, all columns."""
    batch = wls.make_batch("highres_bf16", 2026, threads=16)
    say("projection full size highres_bf16 4096 x 4096")
    kept = kept_oracle(batch)
    W = wls.make_projection(4096, batch.wl.d, 2026)
    db = B.to_device(batch)
    idx = torch.from_numpy(np.concatenate(kept).astype(np.int32)).cuda()
    y = B.gather_project(db, db.V, W.cuda(), kept_idx=idx)
    torch.cuda.synchronize()
    rows = np.sort(np.random.default_rng(0).choice(int(batch.k.sum()), 64, replace=False))
    X = kept_rows(batch, kept).double().numpy()
    check_projection(X, W.double().numpy(), y, True, rows=rows, tag="highres")


@pytest.mark.parametrize("rule", ["question", "row"])
@pytest.mark.parametrize("seed", wls.SEEDS)
def test_xattn_on_projected_edge_rows(B, seed, rule):
    """Edge rows W_v v_i and keys W_k k_j made by the oracle (and rounded the
    way the library takes them: rows to bf16, keys to float32); attention on
    the unprojected kept rows."""
    batch = wls.make_batch("llava_bf16", seed, B=5, N=300, H=2, d_h=128, T=(1, 3),
                           k=(0, 7, 33, 64), P=(0, 1, 3, 6), L_p=(1, 5, 64))
    say(f"xattn on projected edge rows seed={seed} rule={rule} P={batch.P.tolist()}")
    d = batch.wl.d
    Wv = wls.make_projection(d, d, seed + 1).double().numpy()
    Wk = wls.make_projection(d, d, seed + 2).double().numpy()
    Qh = queries_from_batch(batch)
    E = orc.round_bf16(orc.project_rows(Qh.reshape(-1, d).double().numpy(), Wv))
    keys = []
    for j in range(int(batch.P.sum())):
        a, e = int(batch.passage_offsets[j]), int(batch.passage_offsets[j + 1])
        keys.append(batch.Kh[a:e].double().numpy().reshape(e - a, -1).mean(axis=0))
    K = (orc.project_rows(np.stack(keys), Wk).astype(np.float32) if keys
         else np.zeros((0, d), np.float32))
    db = B.to_device(batch, edge_rule=rule)
    O, L, rp, col = B.bipartite_xattn_proj(
        db, Qh.cuda(), torch.from_numpy(E).to(torch.bfloat16).cuda(),
        torch.from_numpy(K).cuda() if len(K) else None)
    torch.cuda.synchronize()
    _, adj, O_ref, L_ref = orc.bipartite_xattn(
        Qh, batch.kept_offsets, batch.Kh, batch.Vh, batch.passage_offsets, batch.query_passages,
        batch.wl.scale, batch.wl.avg_degree, passage_key_table=K.astype(np.float64),
        edge_rule=rule, edge_rows=E)
    check_graph(batch, rp, col, adj)
    check_attention(f64(O), f64(L), np.concatenate(O_ref), np.concatenate(L_ref), "bf16",
                    f"proj {rule}")


@pytest.mark.parametrize("d_out", [256, 768])
@pytest.mark.parametrize("seed", wls.SEEDS)
def test_project_passage_keys_bound(B, seed, d_out):
    """h_k = W_k k~_j on the device (eq. bsca; Def. B.3): k~ the bf16
    rounding of the pooled key (mean of the passage's token keys) or of a
    caller's float key; float output, held to the float32 bound of the row
    projection."""
    batch = wls.make_batch("llava_bf16", seed, B=5, N=300, H=4, d_h=64, T=(1, 3),
                           k=(0, 7, 33, 64), P=(0, 1, 3, 6), L_p=(1, 5, 64, 100))
    n_p = int(batch.P.sum())
    say(f"passage-key projection seed={seed} d_out={d_out} passages={n_p}")
    d = batch.wl.d
    Wk = wls.make_projection(d_out, d, seed + 2)
    db = B.to_device(batch)
    got = B.project_passage_keys(db, Wk.cuda())
    given = np.random.default_rng(seed).standard_normal((n_p, d)).astype(np.float32)
    got_given = B.project_passage_keys(db, Wk.cuda(), passage_keys=torch.from_numpy(given).cuda())
    torch.cuda.synchronize()
    po = batch.passage_offsets
    kbar = orc.passage_keys(batch.Kh.double().numpy(),
                            [(int(po[j]), int(po[j + 1])) for j in range(n_p)])
    Wn = Wk.double().numpy()
    check_projection(orc.round_bf16(kbar), Wn, got, False, tag=f"pooled keys d_out={d_out}")
    check_projection(orc.round_bf16(given.astype(np.float64)), Wn, got_given, False,
                     tag=f"given keys d_out={d_out}")


def test_project_passage_keys_no_passages(B):
    batch = wls.make_batch("llava_bf16", 42, B=3, N=64, H=4, d_h=64, T=1, k=(0, 5), P=(0,))
    db = B.to_device(batch)
    got = B.project_passage_keys(db, wls.make_projection(256, batch.wl.d, 1).cuda())
    torch.cuda.synchronize()
    assert got.shape == (0, 256)


@pytest.mark.parametrize("rule", ["question", "row"])
@pytest.mark.parametrize("seed", wls.SEEDS)
def test_projected_route_chain(B, seed, rule):
    """The projected route end to end on the device: kept rows from the
    top-k, edge rows W_v v_i (skip_gather_project), keys h_k = W_k k~_j
    (skip_project_passage_keys), queries W_Q v_i (skip_gather_project), then
    the graph on the edge rows and attention on the queries
    (skip_bipartite_xattn_proj); against the oracle's chain
    (project_rows, bf16 rounding, bipartite_xattn on edge_rows).

    Inputs on a grid, so that every float32 sum on the device is exact and
    both sides round the same values to bf16: token values and keys are
    multiples of 1/8 in [-2, 2], passages hold 1, 4, 16 or 64 tokens (the
    pooled keys are multiples of 2^-9), weights are multiples of 1/64 in
    [-1/8, 1/8].  The projected rows and keys then match the oracle bit for
    bit, the graphs exactly, and attention to the usual bar."""
    batch = wls.make_batch("llava_bf16", seed, B=5, N=300, H=2, d_h=128, T=(1, 3),
                           k=(0, 7, 33, 64), P=(0, 1, 3, 6), L_p=(1, 4, 16, 64))
    rng = np.random.default_rng([seed, 77])

    def grid(shape, lo, hi, den):
        return torch.from_numpy(rng.integers(lo, hi + 1, size=shape) / den).to(torch.bfloat16)

    batch.V = grid(tuple(batch.V.shape), -16, 16, 8.0)
    batch.Kh = grid(tuple(batch.Kh.shape), -16, 16, 8.0)
    d, H, d_h = batch.wl.d, batch.Kh.shape[1], batch.Kh.shape[2]
    Wv, Wk, Wq = (grid((d, d), -8, 8, 64.0) for _ in range(3))
    say(f"projected route chain seed={seed} rule={rule} k={batch.k.tolist()} "
        f"P={batch.P.tolist()}")
    db = B.to_device(batch, edge_rule=rule)
    idx, _, _ = B.prune_topk(db, want_scores=False, want_rows=False)
    E = B.gather_project(db, db.V, Wv.cuda(), kept_idx=idx)
    Kp = B.project_passage_keys(db, Wk.cuda())
    Q = B.gather_project(db, db.V, Wq.cuda(), kept_idx=idx).view(-1, H, d_h)
    O, L, rp, col = B.bipartite_xattn_proj(db, Q, E, Kp if Kp.shape[0] else None)
    torch.cuda.synchronize()

    kept = kept_oracle(batch)
    assert idx.cpu().numpy().tolist() == np.concatenate(kept).tolist(), "kept sets"
    X = kept_rows(batch, kept).double().numpy()
    E_ref = orc.round_bf16(orc.project_rows(X, Wv.double().numpy()))
    Q_ref = orc.round_bf16(orc.project_rows(X, Wq.double().numpy()))
    po = batch.passage_offsets
    n_p = int(batch.P.sum())
    kbar = orc.passage_keys(batch.Kh.double().numpy(),
                            [(int(po[j]), int(po[j + 1])) for j in range(n_p)])
    K_ref = orc.project_rows(orc.round_bf16(kbar), Wk.double().numpy())
    np.testing.assert_array_equal(E.cpu().double().numpy(), E_ref)
    np.testing.assert_array_equal(Q.cpu().double().numpy().reshape(-1, d), Q_ref)
    np.testing.assert_array_equal(Kp.cpu().double().numpy(), K_ref)
    _, adj, O_ref, L_ref = orc.bipartite_xattn(
        Q_ref.reshape(-1, H, d_h), batch.kept_offsets, batch.Kh, batch.Vh, batch.passage_offsets,
        batch.query_passages, batch.wl.scale, batch.wl.avg_degree, passage_key_table=K_ref,
        edge_rule=rule, edge_rows=E_ref)
    check_graph(batch, rp, col, adj)
    check_attention(f64(O), f64(L), np.concatenate(O_ref), np.concatenate(L_ref), "bf16",
                    f"projected chain {rule}")
