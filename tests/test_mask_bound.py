"""CPU checks of the ReLU-decision bound the GPU step tests use
(gpu_helpers.product_bound / checked_masks): it holds for float32
accumulation and bfloat16 operands on data shaped like the layers'
(non-negative activations, zero-mean Glorot weights), and a forward pass
that zeroes small activations, which the normwise check of H lets through,
is caught by it."""
import numpy as np
import pytest

from tests.gpu_helpers import checked_masks, narrow_bound, product_bound


def _bf16(x):
    u = np.asarray(x, np.float32).view(np.uint32).astype(np.uint64)
    r = ((u + 0x7FFF + ((u >> 16) & 1)) >> 16) << 16
    return r.astype(np.uint32).view(np.float32)


def _layer(rng, n, K, h):
    H = np.maximum(rng.standard_normal((n, K)), 0).astype(np.float32)
    W = (rng.standard_normal((K, h)) * np.sqrt(2.0 / (K + h))).astype(np.float32)
    return H, W


@pytest.mark.parametrize("K", [50, 1024])
def test_bound_covers_sequential_fp32_accumulation(K):
    rng = np.random.default_rng(K)
    H, W = _layer(rng, 200, K, 48)
    acc = np.zeros((200, 48), np.float32)
    for k in range(K):   # one rounding per added term, in index order
        acc = (acc + H[:, k:k + 1] * W[k:k + 1, :]).astype(np.float32)
    Z = H.astype(np.float64) @ W.astype(np.float64)
    r = np.abs(acc - Z) / product_bound(H, H, W)
    assert r.max() < 0.5, r.max()


def test_bound_covers_bf16_operands():
    rng = np.random.default_rng(5)
    H, W = _layer(rng, 2000, 300, 64)
    Zb = _bf16(H).astype(np.float64) @ _bf16(W).astype(np.float64)
    Z = H.astype(np.float64) @ W.astype(np.float64)
    assert (np.abs(Zb - Z) / product_bound(H, H, W, bf16=True)).max() < 0.5


def test_bound_covers_aggregated_products():
    from oracle import gcn as og
    rng = np.random.default_rng(6)
    n = 300
    src = rng.integers(0, n, 3000)
    dst = rng.integers(0, n, 3000)
    from oracle import graph as gr
    rp, cl = gr.subgraph_build(n, src, dst)
    P = rng.standard_normal((n, 32)).astype(np.float32)
    # float32 sums of each row's neighbours, then the scale
    Z32 = np.zeros((n, 32), np.float32)
    for w in range(n):
        s = np.zeros(32, np.float32)
        for c in cl[rp[w]:rp[w + 1]]:
            s = (s + P[c]).astype(np.float32)
        d = rp[w + 1] - rp[w]
        Z32[w] = s * np.float32(1.0 / d) if d else 0.0
    Z = og.aggregate(rp, cl, P)
    bd = narrow_bound(rp, cl, P, P.astype(np.float64))
    ok = bd > 0
    assert (np.abs(Z32 - Z)[ok] / bd[ok]).max() < 0.5
    assert np.array_equal(Z32[~ok], np.zeros_like(Z32[~ok]))


def test_planted_zeroing_of_small_activations_is_caught():
    # a forward pass that zeroes every pre-activation below 1e-4 max|Z|
    # passes the normwise tolerance on H but not the decision check
    rng = np.random.default_rng(7)
    H, W = _layer(rng, 4000, 256, 64)
    Z = H.astype(np.float64) @ W.astype(np.float64)
    Zg = (H @ W).astype(np.float64)
    wrong = np.where(Zg > 1e-4 * np.abs(Zg).max(), Zg, 0.0)
    Hg, Href = np.maximum(wrong, 0), np.maximum(Z, 0)
    assert np.abs(Hg - Href).max() / np.abs(Href).max() < 1e-4
    bd = product_bound(H, H, W)
    checked_masks([Z], [Zg > 0], [bd], "float32 product")   # the honest kernel passes
    with pytest.raises(AssertionError, match="beyond rounding"):
        checked_masks([Z], [wrong > 0], [bd], "planted")
