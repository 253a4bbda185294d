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
