"""GPU parity of the full training step (gcn_train_step) against the oracle,
on the seeded workloads at full size and on small ragged cases.

The oracle takes its own ReLU decisions from its float64 pre-activations.
Where the kernel's float32 decision differs, the entry's |Z| must lie within
a stated rounding bound of zero (gpu_helpers.checked_masks), and only there
does the oracle follow the kernel; the tiny and small ragged steps use the
oracle's decisions everywhere. The updated
weights are compared as W_new - W_old against -lr dW, with the float32
rounding of storing W added to the tolerance (lr dW can sit below the
spacing of W's float32 values)."""
import numpy as np
import pytest

from oracle import gcn as og
from oracle import graph as gr
from paper_2001_02498_amd import synth
from tests.gpu_helpers import (FP32_TOL, GraphCase, checked_masks, dev, narrow_bound,
                               need_gpu, product_bound, rel, say, torch)

pytestmark = pytest.mark.gpu


class StepRun:
    """Runs one gcn_train_step on a workload and keeps every tensor."""

    def __init__(self, wl, inp=None, bias=False, seg_len=0, precision=0, order=0):
        from paper_2001_02498_amd import gcn
        self.gcn, self.wl = gcn, wl
        self.precision = precision
        self.order = order
        self.inp = inp or synth.make_inputs(wl)
        rounds = wl.rounds if wl.reduce else 0
        self.case = GraphCase(wl.n, self.inp.src, self.inp.dst, theta=wl.theta,
                              rounds=rounds, max_aux=wl.max_aux, seg_len=seg_len)
        rng = np.random.default_rng(7)
        self.b = [(rng.standard_normal(2 * wl.h) * 0.1).astype(np.float32)
                  for _ in range(wl.L)] if bias else None
        self.bc = (rng.standard_normal(wl.C) * 0.1).astype(np.float32) if bias else None
        self.bias = bias

    def params_dev(self):
        wl, inp = self.wl, self.inp
        Ws = [dev(w, wl.h) for w in inp.W_self]
        Wn = [dev(w, wl.h) for w in inp.W_neigh]
        Wc = torch.from_numpy(inp.W_cls.copy()).cuda()
        b = [dev(x) for x in self.b] if self.bias else None
        bc = dev(self.bc) if self.bias else None
        return Ws, Wn, Wc, b, bc

    def run(self):
        gcn, wl, inp = self.gcn, self.wl, self.inp
        X = dev(inp.X)
        self.X = X
        Ws, Wn, Wc, b, bc = self.params_dev()
        self.dev_params = (Ws, Wn, Wc, b, bc)
        P = gcn.make_params(Ws, Wn, Wc, b, bc)
        gWs = [torch.zeros_like(w) for w in Ws]
        gWn = [torch.zeros_like(w) for w in Wn]
        gWc = torch.zeros_like(Wc)
        gb = [torch.zeros_like(x) for x in b] if self.bias else None
        gbc = torch.zeros_like(bc) if self.bias else None
        self.grads_dev = (gWs, gWn, gWc, gb, gbc)
        Gp = gcn.make_params(gWs, gWn, gWc, gb, gbc)
        desc = gcn.model_desc(wl.L, wl.f_in, wl.h, wl.C, wl.loss, X.stride(0),
                              has_bias=self.bias, precision=self.precision,
                              order=self.order)
        self.layout = gcn.workspace_layout(self.case.dg, desc)
        ws = gcn.alloc_ws(gcn.workspace_bytes(self.case.dg, desc))
        self.ws = ws
        labels = torch.from_numpy(inp.labels).cuda()
        loss = torch.zeros(1, device="cuda")
        say("train_step", wl.name, "n", wl.n, "L", wl.L, "f_in", wl.f_in, "h", wl.h,
            "C", wl.C, "naux", self.case.info["naux"], "bias", self.bias,
            "precision", self.precision, "order", self.order)
        gcn.train_step(self.case.dg, desc, P, X, labels, wl.lr, loss, ws, grads=Gp)
        torch.cuda.synchronize()
        self.loss = loss.item()
        return self

    def narrow(self, l):
        """Layer l transforms before it aggregates (narrow-side order)."""
        F = self.wl.f_in if l == 0 else 2 * self.wl.h
        return self.order == 1 and F > self.wl.h

    def act(self, off, rows, cols, ld):
        t = self.ws[off:off + 4 * rows * ld].view(torch.float32).view(rows, ld)
        return t[:, :cols]

    def act16(self, off, rows, cols, ld):
        """A bf16 region of the workspace, as bf16."""
        t = self.ws[off:off + 2 * rows * ld].view(torch.bfloat16).view(rows, ld)
        return t[:, :cols]

    def ah(self, l, rows, cols):
        """Layer l's AH region as float32 (the bf16 step keeps it in bf16)."""
        lay = self.layout
        off, ld = lay.AH[l], lay.ld_AH[l]
        if lay.ah_bytes == 4:
            return self.act(off, rows, cols, ld)
        return self.act16(off, rows, cols, ld).float()

    def H(self, l):
        """Layer l's output as float32: the fp32 activations, or in the bf16
        step on operand copies their bf16 copy where no fp32 one is kept
        (the layout reports -1: outputs no aggregation reads)."""
        wl, lay = self.wl, self.layout
        if lay.H[l] < 0:
            return self.act16(lay.H16[l], wl.n, 2 * wl.h, lay.ld_H).float()
        return self.act(lay.H[l], wl.n, 2 * wl.h, lay.ld_H)

    def masks(self):
        """The ReLU decisions the kernels took: from the fp32 activations, or
        in the bf16 step on operand copies from their bf16 copies."""
        wl, lay = self.wl, self.layout
        if lay.ah_bytes == 2:
            return [self.act16(lay.H16[l], wl.n, 2 * wl.h, lay.ld_H).float().cpu().numpy() > 0
                    for l in range(wl.L)]
        return [self.act(lay.H[l], wl.n, 2 * wl.h, lay.ld_H).cpu().numpy() > 0
                for l in range(wl.L)]

    def params_np(self):
        wl, inp = self.wl, self.inp
        return dict(W_self=inp.W_self, W_neigh=inp.W_neigh,
                    b=self.b if self.bias else [None] * wl.L, W_cls=inp.W_cls,
                    b_cls=self.bc)

    def mask_bounds(self, fw, params):
        """Per layer, the bound on |Z_gpu - Z_ref| at every entry (see
        gpu_helpers): from the kernel's own layer input and aggregated input
        (or, in the narrow order, the product it aggregates) as read back
        from the workspace."""
        wl, lay, h = self.wl, self.layout, self.wl.h
        bf16 = self.precision == 1
        out = []
        for l in range(wl.L):
            F = wl.f_in if l == 0 else 2 * h
            Hg = self.inp.X if l == 0 else self.H(l - 1).cpu().numpy()
            b = params["b"][l]
            bs, bn = (None, None) if b is None else (b[:h], b[h:])
            Ws, Wn = params["W_self"][l], params["W_neigh"][l]
            self_b = product_bound(Hg, fw["H"][l], Ws, bs, bf16)
            if self.narrow(l):
                Pg = self.act(lay.AH[l], wl.n, h, lay.ld_AH[l]).cpu().numpy()
                neigh_b = narrow_bound(self.case.rp, self.case.cl, Pg,
                                       fw["H"][l] @ np.asarray(Wn, np.float64))
            else:
                AHg = self.ah(l, wl.n, F).cpu().numpy()
                neigh_b = product_bound(AHg, fw["AH"][l], Wn, bn, bf16)
            out.append(np.concatenate([self_b, neigh_b], axis=1))
        return out

    def oracle(self, unconditioned=False, **kw):
        """The oracle's step on the same inputs. Its ReLU decisions are its
        own; unless `unconditioned`, entries where the kernel decided
        otherwise are checked to lie within rounding of zero and only those
        follow the kernel (checked_masks)."""
        wl, inp = self.wl, self.inp
        params = self.params_np()
        fw = og.forward(self.case.rp, self.case.cl, inp.X, params)
        masks = None
        self.flips = None
        if not unconditioned:
            masks, self.flips = checked_masks(fw["Z"], self.masks(),
                                              self.mask_bounds(fw, params), wl.name)
        return og.train_step(self.case.rp, self.case.cl, inp.X, params, inp.labels,
                             wl.loss, wl.lr, masks=masks, fw=fw, **kw)


def _update_err(new_dev, old, d_ref, lr):
    """max|(W_new - W_old) - (-lr dW)| relative to max|lr dW|, after removing
    the half-ulp of float32 storage of W_new."""
    new = new_dev.detach().cpu().double().numpy()
    want = old.astype(np.float64) - lr * d_ref
    ulp = np.spacing(np.abs(want).astype(np.float32)).astype(np.float64)
    excess = np.maximum(np.abs(new - want) - ulp, 0.0)
    return float(excess.max() / max(np.abs(lr * d_ref).max(), 1e-30))


def check_step(run, tol=FP32_TOL, unconditioned=False):
    ref = run.oracle(unconditioned=unconditioned)
    wl, lay = run.wl, run.layout
    errs = {}
    for l in range(wl.L):
        F = wl.f_in if l == 0 else 2 * wl.h
        if run.narrow(l):
            # the region holds H W_neigh, the product the layer aggregates
            Z = ref["fw"]["H"][l] @ run.inp.W_neigh[l].astype(np.float64)
            errs[f"Z{l}"] = rel(run.act(lay.AH[l], wl.n, wl.h, lay.ld_AH[l]), Z)
        else:
            errs[f"AH{l}"] = rel(run.ah(l, wl.n, F), ref["fw"]["AH"][l])
        errs[f"H{l}"] = rel(run.H(l), ref["fw"]["H"][l + 1])
    errs["logits"] = rel(run.act(lay.logits, wl.n, wl.C, lay.ld_C), ref["fw"]["logits"])
    errs["dlogits"] = rel(run.act(lay.dlogits, wl.n, wl.C, lay.ld_C), ref["dlogits"])
    errs["loss"] = abs(run.loss - ref["loss"]) / max(abs(ref["loss"]), 1e-30)
    # masked gradients still resident: the last two written (layers 0 and 1)
    h = wl.h
    for l in range(min(2, wl.L)):
        G_ref = ref["grads"]["G"][l]
        if lay.ah_bytes == 4:
            errs[f"G{l}"] = rel(run.act(lay.G[l], wl.n, 2 * h, lay.ld_H), G_ref)
            continue
        # bf16 step on operand copies: the full gradient in bf16, the fp32
        # one only where the fp32 aggregation reads it
        errs[f"G16_{l}"] = rel(run.act16(lay.G16[l], wl.n, 2 * h, lay.ld_H).float(), G_ref)
        if l >= 1:
            errs[f"G{l}n"] = rel(run.act(lay.G[l], wl.n, 2 * h, lay.ld_H)[:, h:], G_ref[:, h:])
    if lay.ah_bytes == 2:
        for l in [l for l in range(wl.L) if lay.H[l] >= 0]:
            H = run.act(lay.H[l], wl.n, 2 * h, lay.ld_H)
            assert torch.equal(run.act16(lay.H16[l], wl.n, 2 * h, lay.ld_H),
                               H.to(torch.bfloat16)), l
    gWs, gWn, gWc, gb, gbc = run.grads_dev
    Ws, Wn, Wc, b, bc = run.dev_params
    g = ref["grads"]
    for l in range(wl.L):
        errs[f"dWs{l}"] = rel(gWs[l], g["dW_self"][l])
        errs[f"dWn{l}"] = rel(gWn[l], g["dW_neigh"][l])
        errs[f"Ws{l}"] = rel(Ws[l], ref["params"]["W_self"][l])
        errs[f"dWs_upd{l}"] = _update_err(Ws[l], run.inp.W_self[l], g["dW_self"][l], wl.lr)
        errs[f"dWn_upd{l}"] = _update_err(Wn[l], run.inp.W_neigh[l], g["dW_neigh"][l], wl.lr)
        if run.bias:
            errs[f"db{l}"] = rel(gb[l], g["db"][l])
            errs[f"db_upd{l}"] = _update_err(b[l], run.b[l], g["db"][l], wl.lr)
    errs["dWc"] = rel(gWc, g["dW_cls"])
    errs["dWc_upd"] = _update_err(Wc, run.inp.W_cls, g["dW_cls"], wl.lr)
    if run.bias:
        errs["dbc"] = rel(gbc, g["db_cls"])
    worst = max(errs, key=errs.get)
    say("max error", worst, errs[worst])
    bad = {k: v for k, v in errs.items() if not v < tol}
    assert not bad, bad
    return errs


def test_step_tiny_reduced():
    # the oracle's own ReLU decisions throughout
    need_gpu()
    check_step(StepRun(synth.WORKLOADS["tiny"]).run(), unconditioned=True)


@pytest.mark.parametrize("L,loss,bias", [(2, synth.SIGMOID_BCE, True),
                                         (3, synth.SOFTMAX_CE, False),
                                         (1, synth.SOFTMAX_CE, True)])
def test_step_ragged_small(L, loss, bias):
    need_gpu()
    wl = synth.small_workload(437, 9, L, 29, 36, 7, loss, (L, loss, int(bias)))
    check_step(StepRun(wl, bias=bias, seg_len=4).run(), unconditioned=True)


@pytest.mark.parametrize("name", ["ppi8k", "reddit8k", "yelp10k", "stream8k"])
def test_step_workloads(name):
    need_gpu()
    check_step(StepRun(synth.WORKLOADS[name]).run())


def test_step_ppi_direct_matches_reduced():
    """The same step on G_s and on G_s^#: the direct one checked against
    the oracle like every step, and the two within tolerance of each
    other."""
    need_gpu()
    import dataclasses
    wl = synth.WORKLOADS["ppi8k"]
    inp = synth.make_inputs(wl)
    a = StepRun(dataclasses.replace(wl, reduce=False), inp=inp).run()
    assert a.case.info["naux"] == 0
    check_step(a)
    b = StepRun(wl, inp=inp).run()
    assert b.case.info["naux"] > 0
    assert abs(a.loss - b.loss) <= 1e-5 * abs(a.loss)
    for l in range(wl.L):
        assert rel(a.grads_dev[0][l], b.grads_dev[0][l].cpu().double().numpy()) < FP32_TOL


def test_step_deterministic():
    need_gpu()
    wl = synth.WORKLOADS["tiny"]
    a = StepRun(wl).run()
    b = StepRun(wl).run()
    assert a.loss == b.loss
    for x, y in zip(a.grads_dev[0] + a.grads_dev[1] + [a.grads_dev[2]],
                    b.grads_dev[0] + b.grads_dev[1] + [b.grads_dev[2]]):
        assert torch.equal(x, y)


@pytest.mark.parametrize("name", ["tiny", "ppi8k", "reddit8k", "yelp10k"])
def test_step_narrow_order(name):
    """Aggregating H W_neigh instead of H (the product reassociated) gives
    the paper-order step's results within tolerance."""
    need_gpu()
    check_step(StepRun(synth.WORKLOADS[name], order=1).run())


@pytest.mark.parametrize("L,f_in,h", [(1, 37, 28), (2, 20, 28), (3, 61, 16)])
def test_step_narrow_ragged(L, f_in, h):
    need_gpu()
    wl = synth.small_workload(437, 9, L, f_in, h, 7, synth.SOFTMAX_CE, (L, f_in, h, 5))
    check_step(StepRun(wl, seg_len=4, order=1).run())


def test_step_narrow_bf16():
    need_gpu()
    from tests.gpu_helpers import BF16_TOL
    run = StepRun(synth.WORKLOADS["ppi8k"], order=1, precision=1).run()
    check_step(run, tol=BF16_TOL)


def test_step_narrow_rejects_bias():
    need_gpu()
    from paper_2001_02498_amd import gcn
    wl = synth.WORKLOADS["tiny"]
    run = StepRun(wl, bias=True, order=1)
    desc = gcn.model_desc(wl.L, wl.f_in, wl.h, wl.C, wl.loss, wl.f_in, has_bias=True,
                          order=1)
    with pytest.raises(gcn.GcnError) as e:
        gcn.workspace_bytes(run.case.dg, desc)
    assert e.value.code == gcn.E_UNSUPPORTED


def _inputs_with_edges(wl, src, dst, seed):
    """Seeded features, weights and labels of `wl` on a given edge list."""
    rng = np.random.default_rng(seed)
    F = [wl.f_in] + [2 * wl.h] * (wl.L - 1)
    Ws = [synth.glorot(rng, f, wl.h) for f in F]
    Wn = [synth.glorot(rng, f, wl.h) for f in F]
    Wc = synth.glorot(rng, 2 * wl.h, wl.C)
    X = rng.standard_normal((wl.n, wl.f_in), dtype=np.float32)
    if wl.loss == synth.SOFTMAX_CE:
        y = rng.integers(0, wl.C, wl.n).astype(np.int32)
    else:
        y = (rng.random((wl.n, wl.C)) < 0.3).astype(np.uint8)
    return synth.Inputs(wl, np.asarray(src, np.int64), np.asarray(dst, np.int64), X, Ws, Wn,
                        Wc, y)


@pytest.mark.parametrize("shape", ["edgeless", "single", "bipartite"])
def test_step_degenerate_graphs(shape):
    # no edge at all (every aggregated row is zero); one vertex; K_{3,50},
    # whose 50 identical lists give three pairs of weight 50 for the
    # reduction (one is taken per round, the later rounds see new ids)
    need_gpu()
    if shape == "edgeless":
        wl = synth.small_workload(37, 0, 2, 13, 12, 5, synth.SOFTMAX_CE, (91,))
        src, dst = [], []
    elif shape == "single":
        wl = synth.small_workload(1, 0, 2, 6, 8, 3, synth.SIGMOID_BCE, (92,))
        src, dst = [], []
    else:
        wl = synth.small_workload(53, 0, 3, 10, 16, 4, synth.SOFTMAX_CE, (93,))
        src = [a for a in range(3) for _ in range(3, 53)]
        dst = [b for _ in range(3) for b in range(3, 53)]
    inp = _inputs_with_edges(wl, src, dst, 5)
    run = StepRun(wl, inp=inp, bias=True, seg_len=8).run()
    if shape == "bipartite":
        assert run.case.red.info()["naux"] >= 1
    check_step(run)
