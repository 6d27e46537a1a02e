"""GPU parity of the passage verification gate and of the graph + attention
on the verified passages, through the C ABI, against the CPU oracle.

Inputs shared by both sides: the seeded batch, the gate weights, and the kept
visual rows, chosen by the oracle's own stage 1 (plain salience, top-k).

Bars:
* logits within a float32-accumulation bound of the float64 oracle
  (|dz| <= 1e-4 (1 + max |z|); the inputs are the same bf16 values on both
  sides, so only the order of the float32 sums differs);
* the kept mask equal to the oracle's cut applied to the GPU's own logits
  (the cut is exact), and equal to the oracle's cut of its own logits except
  inside the tie band around the threshold or the cap (reported, never silent);
* on a given mask: edge sets identical, attention as in the unmasked tests.
"""
import math
import sys

import numpy as np
import pytest
import torch

import oracle as orc
from paper_2607_25422_amd import workloads as wls

from test_gpu_parity import check_attention, check_graph, f64, queries_from_batch, sample_rows

pytestmark = pytest.mark.gpu


def say(*a):
    print(*a, file=sys.stderr, flush=True)


@pytest.fixture(scope="module")
def B():
    assert torch.cuda.is_available(), "GPU tests need a HIP device"
    from paper_2607_25422_amd import binding
    return binding


def kept_rows_oracle(batch):
    """Kept rows V[b][top-k of the oracle's salience] per question, as one
    [total_kept, d] tensor in the batch's element type."""
    rows = []
    for b in range(batch.B):
        k = int(batch.k[b])
        Q = batch.Qtok[int(batch.q_offsets[b]):int(batch.q_offsets[b + 1])].double().numpy()
        z = orc.qvs_logits(batch.V[b].double().numpy(), orc.mean_pool_question(Q), None)
        idx = orc.qvs_topk(z, k) if k else np.zeros(0, dtype=np.int64)
        rows.append(batch.V[b][torch.from_numpy(np.asarray(idx, dtype=np.int64))])
    return torch.cat(rows, 0).contiguous()


def gate_oracle(batch, w, Vk, keys=None):
    """Per question: the oracle's logits (float64) of its passages."""
    W, b1, w2 = w.W.double().numpy(), w.b1.double().numpy(), w.w2.double().numpy()
    Vk = Vk.double().numpy()
    out = []
    for b in range(batch.B):
        p0, p1 = int(batch.query_passages[b]), int(batch.query_passages[b + 1])
        if p1 == p0:
            out.append(np.zeros(0))
            continue
        Q = batch.Qtok[int(batch.q_offsets[b]):int(batch.q_offsets[b + 1])].double().numpy()
        k0, k1 = int(batch.kept_offsets[b]), int(batch.kept_offsets[b + 1])
        vbar = Vk[k0:k1].mean(axis=0) if k1 > k0 else np.zeros(batch.wl.d)
        if keys is None:
            t0 = int(batch.passage_offsets[p0])
            ranges = [(int(batch.passage_offsets[j]) - t0, int(batch.passage_offsets[j + 1]) - t0)
                      for j in range(p0, p1)]
            Kq = batch.Kh[t0:int(batch.passage_offsets[p1])].double().numpy()
            E = orc.passage_keys(Kq, ranges)
        else:
            E = keys[p0:p1].double().numpy()
        out.append(orc.skv_logits(orc.mean_pool_question(Q), vbar, E, W, b1, w2, w.b2))
    return out


def check_gate(batch, w, logits, keep, ref, tau, rho, tag=""):
    lg = logits.cpu().double().numpy()
    kp = keep.cpu().numpy().astype(bool)
    events = 0
    for b in range(batch.B):
        p0, p1 = int(batch.query_passages[b]), int(batch.query_passages[b + 1])
        if p1 == p0:
            continue
        z_ref = ref[b]
        z = lg[p0:p1]
        err = float(np.max(np.abs(z - z_ref)))
        tol = 1e-4 * (1.0 + float(np.max(np.abs(z_ref))))
        assert err <= tol, f"{tag} q{b}: logit error {err:.3e} > {tol:.3e}"
        got = kp[p0:p1]
        assert np.array_equal(got, orc.skv_keep(z, tau, rho)), \
            f"{tag} q{b}: kept mask is not the cut of its own logits"
        want = orc.skv_keep(z_ref, tau, rho)
        if not np.array_equal(got, want):
            # a difference is allowed only for passages whose oracle logit sits
            # within the logit error of the threshold or of the cap's value
            t = math.log(tau) - math.log1p(-tau)
            ver = np.sort(z_ref[z_ref >= t])[::-1]
            cap = int(math.ceil(rho * (p1 - p0) - 1e-9))
            cuts = [t] + ([0.5 * (ver[cap - 1] + ver[cap])] if len(ver) > cap else [])
            diff = np.nonzero(got != want)[0]
            band = min(np.max(np.abs(z_ref[diff] - c)) for c in cuts)
            say(f"{tag} q{b}: tie-band event, passages {diff.tolist()} at {band:.2e} from a cut")
            assert band <= 2 * err, f"{tag} q{b}: kept mask differs outside the tie band"
            events += 1
    return events


def gate_device(B, w, tau, rho, b1=True):
    return B.SkvGate(w.W.cuda(), w.b1.cuda() if b1 else None, w.w2.cuda(), w.b2, tau, rho)


@pytest.mark.parametrize("hidden", [64, 256])
@pytest.mark.parametrize("seed", wls.SEEDS)
def test_gate_small_ragged(B, hidden, seed):
    batch = wls.make_batch("llava_bf16", seed, B=6, N=300, H=4, d_h=64, T=(1, 3, 8),
                           k=(0, 7, 33, 64), P=(0, 1, 3, 6, 17), L_p=(1, 5, 64, 100))
    w = wls.make_gate_weights(batch.wl, hidden, seed)
    say(f"gate small h={hidden} seed={seed} k={batch.k.tolist()} P={batch.P.tolist()}")
    db = B.to_device(batch)
    Vk = kept_rows_oracle(batch)
    ref = gate_oracle(batch, w, Vk)
    for tau, rho in ((0.5, 0.5), (0.3, 1.0), (0.7, 0.25)):
        keep, logits = B.skv_gate(db, gate_device(B, w, tau, rho), Vk.cuda())
        torch.cuda.synchronize()
        check_gate(batch, w, logits, keep, ref, tau, rho, tag=f"h{hidden} tau={tau} rho={rho}")


@pytest.mark.parametrize("hidden", [128, 4096])
@pytest.mark.parametrize("given_keys", [False, True])
def test_gate_many_questions_odd_group_count(B, given_keys, hidden):
    """40 questions (two 32-row tiles of question blocks), 275 passages (a
    ragged last passage tile) and d = 192: the passage blocks' 3d columns
    are an odd number of 64-column groups (a wave's last round has spare
    slots), the question blocks' 2d columns fewer, so the two kinds of tile
    take different group counts.  At h = 4096 (the largest gate) every
    thread of the final kernel sums eight hidden units."""
    batch = wls.make_batch("llava_bf16", 42, B=40, N=120, H=3, d_h=64, T=(1, 3, 8),
                           k=(0, 7, 33, 64), P=(0, 1, 3, 6, 17), L_p=(1, 5, 40))
    w = wls.make_gate_weights(batch.wl, hidden, 42)
    say(f"gate 40 questions d=192 h={hidden} given_keys={given_keys} P={batch.P.tolist()}")
    assert batch.wl.d == 192 and batch.B == 40
    db = B.to_device(batch)
    Vk = kept_rows_oracle(batch)
    keys = None
    if given_keys:
        rng = np.random.default_rng(42)
        keys = torch.from_numpy((rng.standard_normal((int(batch.P.sum()), batch.wl.d)) * 0.5)
                                .astype(np.float32))
    ref = gate_oracle(batch, w, Vk, keys)
    for tau, rho in ((0.5, 0.5), (0.3, 1.0)):
        keep, logits = B.skv_gate(db, gate_device(B, w, tau, rho), Vk.cuda(),
                                  passage_keys=None if keys is None else keys.cuda())
        torch.cuda.synchronize()
        check_gate(batch, w, logits, keep, ref, tau, rho, tag=f"d192 tau={tau} rho={rho}")


def test_gate_given_keys_no_b1_repeatable(B):
    batch = wls.make_batch("llava_bf16", 7, B=4, N=200, H=2, d_h=128, T=(2, 9), k=(5, 40),
                           P=(2, 9, 64), L_p=(3, 20))
    w = wls.make_gate_weights(batch.wl, 128, 7)
    w0 = wls.GateWeights(w.W, torch.zeros_like(w.b1), w.w2, w.b2)
    rng = np.random.default_rng(7)
    keys = torch.from_numpy((rng.standard_normal((int(batch.P.sum()), batch.wl.d)) * 0.5)
                            .astype(np.float32))
    say(f"gate given keys P={batch.P.tolist()}")
    db = B.to_device(batch)
    Vk = kept_rows_oracle(batch)
    g = gate_device(B, w, 0.5, 0.5, b1=False)
    a = B.skv_gate(db, g, Vk.cuda(), passage_keys=keys.cuda())
    b = B.skv_gate(db, g, Vk.cuda(), passage_keys=keys.cuda())
    torch.cuda.synchronize()
    for x, y in zip(a, b):
        assert torch.equal(x, y)
    check_gate(batch, w0, a[1], a[0], gate_oracle(batch, w0, Vk, keys), 0.5, 0.5, tag="keys")


def test_gate_full_size(B):
    """highres_bf16 (16 questions of 10 passages, d = 4096) with a 512-unit
    gate on the kept rows of the oracle's stage 1: every passage checked."""
    batch = wls.make_batch("highres_bf16", 2026, threads=16)
    w = wls.make_gate_weights(batch.wl, 512, 2026)
    say("gate full size highres_bf16 h=512")
    db = B.to_device(batch)
    Vk = kept_rows_oracle(batch)
    keep, logits = B.skv_gate(db, gate_device(B, w, 0.5, 0.5), Vk.cuda())
    torch.cuda.synchronize()
    ref = gate_oracle(batch, w, Vk)
    check_gate(batch, w, logits, keep, ref, 0.5, 0.5, tag="highres")
    kept = int(keep.sum())
    say(f"highres gate keeps {kept} of {int(batch.P.sum())} passages")
    assert 0 < kept < int(batch.P.sum())


def seeded_masks(batch, seed):
    """Per-passage 0/1 masks: random, with one question all dropped and one all
    kept where the batch has them."""
    rng = np.random.default_rng(seed)
    m = (rng.random(int(batch.P.sum())) < 0.5).astype(np.uint8)
    qs = [b for b in range(batch.B) if batch.P[b] > 0]
    if qs:
        p0, p1 = int(batch.query_passages[qs[0]]), int(batch.query_passages[qs[0] + 1])
        m[p0:p1] = 0
    if len(qs) > 1:
        p0, p1 = int(batch.query_passages[qs[-1]]), int(batch.query_passages[qs[-1] + 1])
        m[p0:p1] = 1
    return m


@pytest.mark.parametrize("rule,metric,beta", [("question", "cosine", 0.1), ("row", "cosine", 0.1),
                                               ("fraction", "dot", 0.3)])
@pytest.mark.parametrize("seed", wls.SEEDS)
def test_masked_xattn_small_ragged(B, rule, metric, beta, seed):
    batch = wls.make_batch("llava_bf16", seed, B=5, N=300, H=2, d_h=128, T=(1, 3),
                           k=(0, 7, 33, 64), P=(0, 1, 3, 6, 17), L_p=(1, 5, 64))
    mask = seeded_masks(batch, seed)
    say(f"masked xattn {rule}/{metric} seed={seed} P={batch.P.tolist()} kept={int(mask.sum())}")
    db = B.to_device(batch, avg_degree=4.0, edge_rule=rule, edge_metric=metric, edge_beta=beta)
    Qh = queries_from_batch(batch)
    O, L, rp, col = B.bipartite_xattn_masked(db, Qh.cuda(), torch.from_numpy(mask).cuda())
    torch.cuda.synchronize()
    _, adj, O_ref, L_ref = orc.bipartite_xattn(
        Qh, batch.kept_offsets, batch.Kh, batch.Vh, batch.passage_offsets, batch.query_passages,
        batch.wl.scale, 4.0, edge_rule=rule, edge_metric=metric, edge_beta=beta,
        passage_keep=mask.astype(bool))
    check_graph(batch, rp, col, adj)
    for b in range(batch.B):
        p0, p1 = int(batch.query_passages[b]), int(batch.query_passages[b + 1])
        assert not adj[b][:, mask[p0:p1] == 0].any()
    check_attention(f64(O), f64(L), np.concatenate(O_ref), np.concatenate(L_ref), "bf16",
                    f"masked {rule}")


def test_masked_all_kept_equals_unmasked(B):
    batch = wls.make_batch("llava_bf16", 3, B=4, N=300, H=2, d_h=128, T=(2,), k=(7, 64),
                           P=(1, 6, 17), L_p=(5, 64))
    db = B.to_device(batch)
    Qh = queries_from_batch(batch).cuda()
    ones = torch.ones(int(batch.P.sum()), dtype=torch.uint8, device="cuda")
    a = B.bipartite_xattn_masked(db, Qh, ones)
    b = B.bipartite_xattn(db, Qh)
    torch.cuda.synchronize()
    for x, y in zip(a[:3], b[:3]):
        assert torch.equal(x, y)
    n = int(a[2][-1])        # the column buffer past the last edge is not written
    assert torch.equal(a[3][:n], b[3][:n])


def test_gate_then_masked_xattn_full_size(B):
    """The verify step feeding the graph at highres_bf16 scale: the GPU gate's
    mask (already checked against the oracle above) drives the masked graph;
    edges checked for every question, attention on sampled rows."""
    batch = wls.make_batch("highres_bf16", 2026, threads=16)
    w = wls.make_gate_weights(batch.wl, 512, 2026)
    db = B.to_device(batch)
    Vk = kept_rows_oracle(batch)
    keep, logits = B.skv_gate(db, gate_device(B, w, 0.5, 0.5), Vk.cuda())
    torch.cuda.synchronize()
    ref = gate_oracle(batch, w, Vk)
    check_gate(batch, w, logits, keep, ref, 0.5, 0.5, tag="highres chain")
    mask = keep.cpu().numpy().astype(bool)
    H, d_h = batch.Kh.shape[1], batch.Kh.shape[2]
    Qh = Vk.reshape(-1, H, d_h).contiguous()
    O, L, rp, col = B.bipartite_xattn_masked(db, Qh.cuda(), keep)
    torch.cuda.synchronize()
    rows = {b: [0, 5, int(batch.k[b]) - 1] for b in range(0, batch.B, 5)}
    _, adj, O_ref, L_ref = orc.bipartite_xattn(
        Qh, batch.kept_offsets, batch.Kh, batch.Vh, batch.passage_offsets, batch.query_passages,
        batch.wl.scale, batch.wl.avg_degree, passage_keep=mask, attn_rows=rows)
    check_graph(batch, rp, col, adj)
    Of, Lf = f64(O), f64(L)
    got_O, got_L, want_O, want_L = [], [], [], []
    for b, rs in rows.items():
        k0 = int(batch.kept_offsets[b])
        for r in rs:
            got_O.append(Of[k0 + r]); got_L.append(Lf[k0 + r])
            want_O.append(O_ref[b][r]); want_L.append(L_ref[b][r])
    check_attention(np.stack(got_O), np.stack(got_L), np.stack(want_O), np.stack(want_L),
                    "bf16", "highres masked")


# --------------------------------------------------------------------------- fused route with the gate

def gate_dict(w, tau, rho):
    return dict(W=w.W.double().numpy(), b1=w.b1.double().numpy(), w2=w.w2.double().numpy(),
                b2=w.b2, tau=tau, rho=rho)


def matching_questions(batch, keep, ref_keep):
    kp = keep.cpu().numpy().astype(bool)
    same = []
    for b in range(batch.B):
        p0, p1 = int(batch.query_passages[b]), int(batch.query_passages[b + 1])
        if np.array_equal(kp[p0:p1], ref_keep[b]):
            same.append(b)
        else:
            say(f"q{b}: gate tie-band event, downstream comparison skipped")
    return same


@pytest.mark.parametrize("seed", wls.SEEDS)
def test_route_fused_gated_small_ragged(B, seed):
    batch = wls.make_batch("llava_bf16", seed, B=6, N=300, H=4, d_h=64, T=(1, 3, 8),
                           k=(0, 7, 33, 64), P=(0, 1, 3, 6, 17), L_p=(1, 5, 64),
                           with_bias=True)
    w = wls.make_gate_weights(batch.wl, 256, seed)
    say(f"fused gated small seed={seed} k={batch.k.tolist()} P={batch.P.tolist()}")
    db = B.to_device(batch)
    idx, keep, logits, O, L = B.route_fused_gated(db, gate_device(B, w, 0.5, 0.5))
    torch.cuda.synchronize()
    ref = orc.route(batch.V, batch.Qtok, batch.q_offsets, batch.kept_offsets, batch.Kh,
                    batch.Vh, batch.passage_offsets, batch.query_passages, batch.wl.scale,
                    batch.wl.avg_degree, w_bias=batch.w_bias, gate=gate_dict(w, 0.5, 0.5))
    idx = idx.cpu().numpy()
    for b in range(batch.B):
        k0, k1 = batch.kept_offsets[b], batch.kept_offsets[b + 1]
        assert idx[k0:k1].tolist() == ref.kept_idx[b].tolist(), f"q{b} kept set"
    check_gate(batch, w, logits, keep, ref.gate_logits, 0.5, 0.5, tag=f"fused seed={seed}")
    Of, Lf = f64(O), f64(L)
    for b in matching_questions(batch, keep, ref.keep):
        k0, k1 = int(batch.kept_offsets[b]), int(batch.kept_offsets[b + 1])
        check_attention(Of[k0:k1], Lf[k0:k1], ref.O[b], ref.LSE[b], "bf16", f"fused gated q{b}")


def test_route_fused_gated_full_size_equals_staged(B):
    """highres_bf16 with a 512-unit gate: the fused gated route bitwise equal to
    the staged calls (prune, gate on the gathered rows, masked graph and
    attention); the oracle checks the gate on every passage, the graph on
    every question and attention on sampled rows."""
    batch = wls.make_batch("highres_bf16", 2026, threads=16)
    w = wls.make_gate_weights(batch.wl, 512, 2026)
    say("fused gated highres_bf16 h=512")
    db = B.to_device(batch)
    g = gate_device(B, w, 0.5, 0.5)
    fidx, fkeep, flog, fO, fL = B.route_fused_gated(db, g)
    idx, _, Vk = B.prune_topk(db, want_scores=False)
    keep, logits = B.skv_gate(db, g, Vk)
    Qh = Vk.view(-1, batch.Kh.shape[1], batch.Kh.shape[2])
    O, L, rp, col = B.bipartite_xattn_masked(db, Qh, keep)
    torch.cuda.synchronize()
    assert torch.equal(fidx, idx)
    assert torch.equal(fkeep, keep) and torch.equal(flog, logits), "fused gate != staged gate"
    assert torch.equal(fO, O) and torch.equal(fL, L), "fused attention != staged"
    rows = sample_rows(batch, 8)
    ref = orc.route(batch.V, batch.Qtok, batch.q_offsets, batch.kept_offsets, batch.Kh,
                    batch.Vh, batch.passage_offsets, batch.query_passages, batch.wl.scale,
                    batch.wl.avg_degree, attn_rows=rows, gate=gate_dict(w, 0.5, 0.5))
    idx = idx.cpu().numpy()
    for b in range(batch.B):
        k0, k1 = batch.kept_offsets[b], batch.kept_offsets[b + 1]
        assert idx[k0:k1].tolist() == ref.kept_idx[b].tolist(), f"q{b} kept set"
    check_gate(batch, w, logits, keep, ref.gate_logits, 0.5, 0.5, tag="fused highres")
    same = matching_questions(batch, keep, ref.keep)
    assert len(same) >= batch.B - 2
    rpn, coln = rp.cpu().numpy(), col.cpu().numpy()
    Of, Lf = f64(O), f64(L)
    got_O, got_L, want_O, want_L = [], [], [], []
    for b in same:
        k0, k1 = int(batch.kept_offsets[b]), int(batch.kept_offsets[b + 1])
        want_rp, want_col = orc.adjacency_to_csr(ref.adj[b])
        assert (rpn[k0:k1 + 1] - rpn[k0]).tolist() == want_rp.tolist(), f"q{b} row pointers"
        assert coln[rpn[k0]:rpn[k1]].tolist() == want_col.tolist(), f"q{b} columns"
        for r in rows.get(b, []):
            got_O.append(Of[k0 + r]); got_L.append(Lf[k0 + r])
            want_O.append(ref.O[b][r]); want_L.append(ref.LSE[b][r])
    check_attention(np.stack(got_O), np.stack(got_L), np.stack(want_O), np.stack(want_L),
                    "bf16", "fused gated highres")


@pytest.mark.parametrize("workload,seed", [("llava_bf16", s) for s in wls.SEEDS] +
                         [("highres_bf16", 2026)])
def test_route_fused_gated_keeping_all_equals_plain(B, workload, seed):
    """A gate that keeps every passage (threshold far below every logit,
    rho = 1: Def. B.4's cut then drops nothing) leaves the route of Alg. 1
    unchanged: kept sets, outputs and log-sum-exps bitwise equal to the
    plain fused route on the same batch."""
    if workload == "llava_bf16":
        batch = wls.make_batch(workload, seed, B=6, N=300, H=4, d_h=64, T=(1, 3, 8),
                               k=(0, 7, 33, 64), P=(0, 1, 3, 6, 17), L_p=(1, 5, 64),
                               with_bias=True)
    else:
        batch = wls.make_batch(workload, seed, threads=16)
    w = wls.make_gate_weights(batch.wl, 256, seed)
    say(f"gated keeping all {workload} seed={seed} P={batch.P.tolist()}")
    db = B.to_device(batch)
    idx, keep, logits, O, L = B.route_fused_gated(db, gate_device(B, w, 1e-300, 1.0))
    pidx, pO, pL = B.route_fused(db)
    torch.cuda.synchronize()
    assert bool((keep == 1).all()), "a passage was dropped"
    assert bool(torch.isfinite(logits).all())
    assert torch.equal(idx, pidx), "kept sets differ"
    assert torch.equal(O, pO) and torch.equal(L, pL), "gated route != plain route"


@pytest.mark.parametrize("rule,metric,beta", [("row", "cosine", 0.1), ("fraction", "dot", 0.3),
                                               ("question", "dot", 0.1)])
def test_route_fused_gated_edge_rules(B, rule, metric, beta):
    """The fused gated route under the other edge cuts and compatibilities
    (Sec. 3.5, eq. (bsca) and its quantile cut; per-row top-Δ): kept sets,
    the gate and the attention of every kept row against the oracle's route
    with the same gate and cut."""
    seed = 42
    batch = wls.make_batch("llava_bf16", seed, B=6, N=300, H=4, d_h=64, T=(1, 3, 8),
                           k=(0, 7, 33, 64), P=(0, 1, 3, 6, 17), L_p=(1, 5, 64),
                           with_bias=True)
    w = wls.make_gate_weights(batch.wl, 256, seed)
    say(f"fused gated {rule}/{metric} k={batch.k.tolist()} P={batch.P.tolist()}")
    db = B.to_device(batch, avg_degree=4.0, edge_rule=rule, edge_metric=metric, edge_beta=beta)
    idx, keep, logits, O, L = B.route_fused_gated(db, gate_device(B, w, 0.5, 0.5))
    torch.cuda.synchronize()
    ref = orc.route(batch.V, batch.Qtok, batch.q_offsets, batch.kept_offsets, batch.Kh,
                    batch.Vh, batch.passage_offsets, batch.query_passages, batch.wl.scale, 4.0,
                    w_bias=batch.w_bias, edge_rule=rule, edge_metric=metric, edge_beta=beta,
                    gate=gate_dict(w, 0.5, 0.5))
    idx = idx.cpu().numpy()
    for b in range(batch.B):
        k0, k1 = batch.kept_offsets[b], batch.kept_offsets[b + 1]
        assert idx[k0:k1].tolist() == ref.kept_idx[b].tolist(), f"q{b} kept set"
    check_gate(batch, w, logits, keep, ref.gate_logits, 0.5, 0.5, tag=f"fused {rule}/{metric}")
    Of, Lf = f64(O), f64(L)
    for b in matching_questions(batch, keep, ref.keep):
        k0, k1 = int(batch.kept_offsets[b]), int(batch.kept_offsets[b + 1])
        check_attention(Of[k0:k1], Lf[k0:k1], ref.O[b], ref.LSE[b], "bf16",
                        f"fused gated {rule}/{metric} q{b}")
