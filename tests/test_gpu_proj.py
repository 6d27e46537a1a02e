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
