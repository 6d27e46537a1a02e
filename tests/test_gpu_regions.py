"""GPU parity of the regions of the kept tokens (approximate k-means), through
the C ABI, against the CPU oracle.

Inputs shared by both sides: the seeded batch and the kept rows, chosen by
the oracle's own stage 1 (plain salience, top-k).

Bars: region of every kept row and region sizes identical (both sides decide
in float64); centroids equal to the float32 rounding of the oracle's float64
centroids within 2 ulp of float32 at the centroid's scale (the float64 means
differ only in summation order).
"""
import sys

import numpy as np
import pytest
import torch

import oracle as orc
from paper_2607_25422_amd import workloads as wls

pytestmark = pytest.mark.gpu


def say(*a):
    print(*a, file=sys.stderr, flush=True)


@pytest.fixture(scope="module")
def B():
    assert torch.cuda.is_available(), "GPU tests need a HIP device"
    from paper_2607_25422_amd import binding
    return binding


def kept_oracle(batch):
    """Per question the oracle's kept indices (stage 1, plain salience)."""
    out = []
    for b in range(batch.B):
        k = int(batch.k[b])
        Q = batch.Qtok[int(batch.q_offsets[b]):int(batch.q_offsets[b + 1])].double().numpy()
        z = orc.qvs_logits(batch.V[b].double().numpy(), orc.mean_pool_question(Q), batch.w_bias
                           if batch.w_bias is None else batch.w_bias.double().numpy())
        out.append(orc.qvs_topk(z, k) if k else np.zeros(0, dtype=np.int64))
    return out


def check_regions(batch, kept, region, cent, sizes, r_max, n_iter, tag=""):
    region = region.cpu().numpy()
    cent = cent.cpu().numpy()
    sizes = sizes.cpu().numpy()
    for b in range(batch.B):
        k0, k = int(batch.kept_offsets[b]), int(batch.k[b])
        R = orc.region_count(k, r_max)
        if R == 0:
            assert np.all(cent[b] == 0) and np.all(sizes[b] == 0), f"{tag} q{b}: empty question"
            continue
        Vhat = batch.V[b].double().numpy()[kept[b]]
        a, C, n = orc.region_kmeans(Vhat, R, n_iter)
        assert region[k0:k0 + k].tolist() == a.tolist(), f"{tag} q{b}: regions differ"
        assert sizes[b, :R].tolist() == n.tolist() and np.all(sizes[b, R:] == 0), f"{tag} q{b}"
        want = C.astype(np.float32)
        scale = np.maximum(np.abs(want).max(axis=1, keepdims=True), 1e-30)
        err = np.max(np.abs(cent[b, :R] - want) / scale)
        assert err <= 2.0 ** -22, f"{tag} q{b}: centroid error {err:.2e}"
        assert np.all(cent[b, R:] == 0)


@pytest.mark.parametrize("r_max,n_iter", [(8, 10), (16, 3), (3, 1)])
@pytest.mark.parametrize("seed", wls.SEEDS)
def test_regions_small_ragged(B, seed, r_max, n_iter):
    batch = wls.make_batch("llava_bf16", seed, B=6, N=300, H=4, d_h=64, T=(1, 3, 8),
                           k=(0, 1, 3, 7, 33, 64, 300))
    say(f"regions small seed={seed} r_max={r_max} n_iter={n_iter} k={batch.k.tolist()}")
    kept = kept_oracle(batch)
    db = B.to_device(batch)
    rows = torch.cat([batch.V[b][torch.from_numpy(kept[b].astype(np.int64))]
                      for b in range(batch.B)]).contiguous().cuda()
    region, cent, sizes = B.region_kmeans(db, rows, r_max=r_max, n_iter=n_iter)
    idx = torch.from_numpy(np.concatenate(kept).astype(np.int32)).cuda()
    region2, cent2, sizes2 = B.region_kmeans(db, db.V, kept_idx=idx, r_max=r_max, n_iter=n_iter)
    torch.cuda.synchronize()
    for x, y in ((region, region2), (cent, cent2), (sizes, sizes2)):
        assert torch.equal(x, y), "rows in place and gathered rows disagree"
    check_regions(batch, kept, region, cent, sizes, r_max, n_iter, f"seed={seed}")


@pytest.mark.parametrize("wl,H,d_h,r_max", [("llava_bf16", 5, 64, 4), ("tiny_fp32", 5, 40, 16),
                                              ("llava_bf16", 10, 40, 8)])
def test_regions_ragged_slice(B, wl, H, d_h, r_max):
    """d = 320, 200 or 400: the last 256-column slice is partly empty (64,
    200 or 144 columns), so some waves of it own no columns at all."""
    batch = wls.make_batch(wl, 11, B=4, N=400, H=H, d_h=d_h, T=(2, 5), k=(5, 70, 200, 400))
    say(f"regions ragged slice {wl} d={H * d_h} r_max={r_max} k={batch.k.tolist()}")
    kept = kept_oracle(batch)
    db = B.to_device(batch)
    idx = torch.from_numpy(np.concatenate(kept).astype(np.int32)).cuda()
    region, cent, sizes = B.region_kmeans(db, db.V, kept_idx=idx, r_max=r_max, n_iter=6)
    torch.cuda.synchronize()
    check_regions(batch, kept, region, cent, sizes, r_max, 6, f"{wl} d={H * d_h}")


def test_regions_fp32_and_repeatable(B):
    batch = wls.make_batch("tiny_fp32", 5, B=3, N=200, k=(4, 40, 120))
    kept = kept_oracle(batch)
    db = B.to_device(batch)
    rows = torch.cat([batch.V[b][torch.from_numpy(kept[b].astype(np.int64))]
                      for b in range(batch.B)]).contiguous().cuda()
    a = B.region_kmeans(db, rows, r_max=8, n_iter=20)
    b = B.region_kmeans(db, rows, r_max=8, n_iter=20)
    torch.cuda.synchronize()
    for x, y in zip(a, b):
        assert torch.equal(x, y)
    check_regions(batch, kept, *a, 8, 20, "fp32")


def test_regions_full_size(B):
    """highres_bf16 (16 questions of 192 kept rows, d = 4096): R = 8, ten
    iterations, rows read in place through the kept indices."""
    batch = wls.make_batch("highres_bf16", 2026, threads=16)
    say("regions full size highres_bf16")
    kept = kept_oracle(batch)
    db = B.to_device(batch)
    idx = torch.from_numpy(np.concatenate(kept).astype(np.int32)).cuda()
    region, cent, sizes = B.region_kmeans(db, db.V, kept_idx=idx, r_max=8, n_iter=10)
    torch.cuda.synchronize()
    check_regions(batch, kept, region, cent, sizes, 8, 10, "highres")
    assert int(sizes.sum()) == int(batch.k.sum())
