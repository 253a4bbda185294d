"""Shared set-up for the GPU parity tests: seeded inputs on the device, the
oracle's float64 result beside them, and the normwise error metric.

Tolerance (normwise max relative error, per tensor):
    rel(T) = max|T_gpu - T_ref| / max(max|T_ref|, 1e-30)
fp32 GEMMs accumulate K <= ~10^4 products with a per-step rounding of
2^-24; a worst-case bound K * 2^-24 ~ 6e-4 is far above what random signs
give (~sqrt(K) * 2^-24 ~ 6e-6), so 1e-4 leaves an order of magnitude of
margin while catching any dropped term, sign or index (errors of order 1).
Aggregations sum at most a few thousand rows: 1e-5.
The bf16 variant of the dense products rounds every operand to 8 significant
bits (relative error up to 2^-9 each): 2e-2 against the float64 oracle, and
the fp32 bound against the oracle with the same operands rounded.
"""
import sys

import numpy as np
import pytest

from oracle import graph as gr
from oracle import reduction as rd

torch = pytest.importorskip("torch")

FP32_TOL = 1e-4
AGG_TOL = 1e-5
BF16_TOL = 2e-2


def need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def rel(gpu, ref):
    g = gpu.detach().cpu().double().numpy() if hasattr(gpu, "detach") else np.asarray(gpu, float)
    r = np.asarray(ref, dtype=np.float64)
    assert g.shape == r.shape, (g.shape, r.shape)
    if r.size == 0:
        return 0.0
    return float(np.abs(g - r).max() / max(np.abs(r).max(), 1e-30))


def dev(x, ld=None, fill=float("nan")):
    """float32 device matrix with leading dimension ld (padding = fill)."""
    x = np.asarray(x, dtype=np.float32)
    if x.ndim == 1:
        return torch.from_numpy(x.copy()).cuda()
    n, f = x.shape
    ld = ld or ((f + 3) // 4 * 4)
    buf = torch.full((n, ld), fill, dtype=torch.float32)
    buf[:, :f] = torch.from_numpy(x)
    return buf.cuda()[:, :f]


def empty(n, f, ld=None, fill=float("nan")):
    ld = ld or ((f + 3) // 4 * 4)
    return torch.full((n, ld), fill, dtype=torch.float32, device="cuda")[:, :f]


def padding_of(t):
    """The padding columns of a strided view (to check they are untouched)."""
    full = torch.as_strided(t, (t.shape[0], t.stride(0)), (t.stride(0), 1))
    return full[:, t.shape[1]:]


class GraphCase:
    """Subgraph + reduction on the host library, its device image, and the
    oracle's CSR of the same subgraph."""

    def __init__(self, n, src, dst, theta=2, rounds=5, max_aux=-1, seg_len=0):
        from paper_2001_02498_amd import gcn
        self.gcn = gcn
        self.n = n
        self.rp, self.cl = gr.subgraph_build(n, src, dst)
        g = gcn.subgraph_build(n, src, dst)
        self.red = gcn.redundancy_reduce(g, theta=theta, max_rounds=rounds, max_aux=max_aux)
        self.info = self.red.info()
        self.dg = gcn.DeviceGraph(self.red, seg_len=seg_len)
        torch.cuda.synchronize()

    def oracle_reduced(self):
        i = self.info
        return dict(rowptr=i["rowptr"], col=i["col"], pairs=i["pairs"],
                    round_offsets=i["round_offsets"], naux=i["naux"], n=i["n"])


# ------------------------------------------------------------ ReLU decisions
# The oracle takes its own ReLU decisions, [Z > 0] on its float64 Z. The
# kernels decide from their float32 (or bfloat16) Z, which differs from Z by
# rounding, so an entry within that rounding of zero may fall on the other
# side. Every such disagreement is checked against a bound on
# |Z_gpu - Z_ref| (Section 2.1, Eq. 1 and Eq. 2a-2c), and only those entries
# take the kernel's decision.
#
# Z_gpu = fl(Hg W + b), Hg the kernel's own layer input (read back), so
#   Z_gpu - Z_ref = (Hg - H_ref) W + e,
# where e is the rounding of the product. The first term is bounded
# rigorously by |Hg - H_ref| |W|. For e the bound is probabilistic (rounding
# errors independent with mean zero, as in Higham and Mary's probabilistic
# rounding-error analysis, SIAM J. Sci. Comput. 2019): to first order
# e = sum_k delta_k S_k with |delta_k| <= u and S_k the partial sums, so by
# Hoeffding's inequality |e| <= lam u sqrt(sum_k S_k^2) except with
# probability 2 exp(-lam^2 / 2); terms h_k w_k of random sign (zero-mean
# weights) make the partial sums a random walk, sum_k S_k^2 ~ K ||t||_2^2 with
# ||t||_2^2 = sum_k (h_k w_k)^2 + b^2. With bfloat16 operands each term also
# carries |delta_h + delta_w| <= 2 u16 + u16^2, independent over k:
# lam (2 u16 + u16^2) ||t||_2 more. lam = 8 (exceedance 2.5e-14 per entry)
# and a factor 2 for second-order terms:
#   bound = |Hg - H_ref| |W| + 2 lam (sqrt(K + 2) u + [bf16] (2 u16 + u16^2)) ||t||_2.
# A narrow-order neighbour half Z = fl(D^-1 A P_gpu), P_gpu = fl(Hg W): the
# mean of d_w rows adds lam u sqrt(D^-1 A P^2) by the same argument:
#   bound = D^-1 A |P_gpu - H_ref W| + 2 lam u sqrt(D^-1 A P_gpu^2).
# For K = 1024, unit weights scale this is ~2e-5 of a typical |Z|, so a
# kernel that zeroed small activations (which the normwise check of H would
# let pass) shows up here as disagreements far outside it.
U32 = 2.0 ** -24
U16 = 2.0 ** -8
LAM = 8.0


def product_bound(Hg, H_ref, W, b=None, bf16=False):
    Hg = np.asarray(Hg, np.float64)
    W = np.asarray(W, np.float64)
    K = Hg.shape[1]
    t2 = (Hg * Hg) @ (W * W)
    if b is not None:
        t2 = t2 + np.square(np.asarray(b, np.float64))[None, :]
    gam = np.sqrt(K + 2.0) * U32 + ((2 * U16 + U16 * U16) if bf16 else 0.0)
    return np.abs(Hg - np.asarray(H_ref, np.float64)) @ np.abs(W) + 2 * LAM * gam * np.sqrt(t2)


def narrow_bound(rp, cl, Pg, P_ref):
    from oracle import gcn as og
    Pg = np.asarray(Pg, np.float64)
    err = og.aggregate(rp, cl, np.abs(Pg - P_ref))
    return err + 2 * LAM * U32 * np.sqrt(og.aggregate(rp, cl, Pg * Pg))


def checked_masks(Z_ref, gpu_masks, bounds, tag=""):
    """Per layer: the oracle's [Z_ref > 0]; wherever the kernel decided
    otherwise, assert |Z_ref| <= bound there and take the kernel's
    decision at exactly those entries. Returns (masks, flip counts)."""
    masks, flips = [], []
    for l, (Z, mg, bd) in enumerate(zip(Z_ref, gpu_masks, bounds)):
        mine = Z > 0.0
        mg = np.asarray(mg, bool)
        diff = mine != mg
        nd = int(diff.sum())
        if nd:
            z, lim = np.abs(Z[diff]), bd[diff]
            assert (z <= lim).all(), (
                f"{tag} layer {l}: {int((z > lim).sum())} of {nd} ReLU decisions differ "
                f"from the oracle's beyond rounding (worst |Z| {z.max():.3e}, "
                f"bound there {lim[np.argmax(z)]:.3e})")
        masks.append(np.where(diff, mg, mine))
        flips.append(nd)
    say(f"{tag} ReLU decisions differing from the oracle's, per layer "
        f"(each within its rounding bound): {flips}")
    return masks, flips
