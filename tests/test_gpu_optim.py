"""GPU parity of gcn_train_step_optim (momentum and Adam fused into the
weight-gradient reduction) against the oracle's update rules.

The optimiser states start from seeded values shaped like the weights
(scaled to the oracle's gradient of each tensor, as a mid-training state
would be), or from zero for Adam's first step. States are compared
normwise; updated weights as W_new - W_old against the oracle's update,
as in the plain-descent step tests."""
import numpy as np
import pytest

from oracle import gcn as og
from oracle import optim as oo
from paper_2001_02498_amd import synth
from tests.gpu_helpers import BF16_TOL, FP32_TOL, dev, need_gpu, rel, say, torch
from tests.test_gpu_step import StepRun, _update_err

pytestmark = pytest.mark.gpu

KEYS = ("W_self", "W_neigh", "b")


def _named(run):
    """(key, layer or None) of every tensor the model updates."""
    out = []
    for l in range(run.wl.L):
        out += [("W_self", l), ("W_neigh", l)] + ([("b", l)] if run.bias else [])
    return out + [("W_cls", None)] + ([("b_cls", None)] if run.bias else [])


def _get(d, key, l):
    return d[key][l] if l is not None else d[key]


class OptRun(StepRun):
    def __init__(self, wl, kind, step=1, zero_state=False, seed=3, **kw):
        super().__init__(wl, **kw)
        self.kind, self.step, self.zero_state, self.seed = kind, step, zero_state, seed
        self.hp = dict(lr=wl.lr, momentum=0.9, beta1=0.9, beta2=0.999, eps=1e-8)

    def params_np(self):
        inp = self.inp
        return dict(W_self=inp.W_self, W_neigh=inp.W_neigh,
                    b=self.b if self.bias else [None] * self.wl.L, W_cls=inp.W_cls,
                    b_cls=self.bc)

    def make_state(self):
        """Seeded optimiser states; their scale follows the oracle's gradient
        of each tensor (masks from the oracle's own activations)."""
        nkeys = 2 if self.kind == oo.ADAM else 1
        st = [dict(W_self=[None] * self.wl.L, W_neigh=[None] * self.wl.L,
                   b=[None] * self.wl.L, W_cls=None, b_cls=None) for _ in range(nkeys)]
        if not self.zero_state:
            fw = og.forward(self.case.rp, self.case.cl, self.inp.X, self.params_np())
            _, dz = og.loss_and_grad(self.wl.loss, fw["logits"], self.inp.labels)
            g = og.backward(self.case.rp, self.case.cl, self.params_np(), fw, dz)
        rng = np.random.default_rng(self.seed)
        for key, l in _named(self):
            shape = np.shape(_get(self.params_np(), key, l))
            for i in range(nkeys):
                if self.zero_state:
                    x = np.zeros(shape)
                else:
                    sigma = float(np.sqrt(np.mean(_get(g, "d" + key, l) ** 2))) + 1e-12
                    x = (rng.standard_normal(shape) * sigma if i == 0 else
                         (rng.uniform(0.5, 1.5, shape) * sigma) ** 2)
                x = x.astype(np.float32)
                if l is None:
                    st[i][key] = x
                else:
                    st[i][key][l] = x
        return st

    def run(self):
        gcn, wl, inp = self.gcn, self.wl, self.inp
        self.state_np = self.make_state()
        X = dev(inp.X)
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

        def to_dev(s):
            t = dict(W_self=[torch.from_numpy(x.copy()).cuda() for x in s["W_self"]],
                     W_neigh=[torch.from_numpy(x.copy()).cuda() for x in s["W_neigh"]],
                     b=[torch.from_numpy(x.copy()).cuda() for x in s["b"]] if self.bias
                     else None,
                     W_cls=torch.from_numpy(s["W_cls"].copy()).cuda(),
                     b_cls=torch.from_numpy(s["b_cls"].copy()).cuda() if self.bias else None)
            return t, gcn.make_params(t["W_self"], t["W_neigh"], t["W_cls"], t["b"], t["b_cls"])

        self.state_dev = [to_dev(s) for s in self.state_np]
        S = [p for _, p in self.state_dev] + [None, None]
        desc = gcn.model_desc(wl.L, wl.f_in, wl.h, wl.C, wl.loss, X.stride(0),
                              has_bias=self.bias, precision=self.precision)
        self.layout = gcn.workspace_layout(self.case.dg, desc)
        ws = gcn.alloc_ws(gcn.workspace_bytes(self.case.dg, desc))
        self.ws = ws
        labels = torch.from_numpy(inp.labels).cuda()
        loss = torch.zeros(1, device="cuda")
        opt = gcn.optim(self.kind, self.hp["lr"], step=self.step, momentum=self.hp["momentum"],
                        beta1=self.hp["beta1"], beta2=self.hp["beta2"], eps=self.hp["eps"])
        say("train_step_optim", wl.name, "kind", self.kind, "step", self.step, "zero_state",
            self.zero_state, "bias", self.bias, "n", wl.n)
        gcn.train_step_optim(self.case.dg, desc, P, X, labels, opt, loss, ws, state1=S[0],
                             state2=S[1], grads=Gp)
        torch.cuda.synchronize()
        self.loss = loss.item()
        return self

    def oracle(self, unconditioned=False):
        opt = oo.Optim(self.kind, lr=self.hp["lr"], step=self.step,
                       momentum=self.hp["momentum"], beta1=self.hp["beta1"],
                       beta2=self.hp["beta2"], eps=self.hp["eps"])
        s1 = self.state_np[0]
        s2 = self.state_np[1] if len(self.state_np) > 1 else None
        return super().oracle(unconditioned=unconditioned, opt=opt, state1=s1, state2=s2)


def _dev_tensor(run, key, l):
    Ws, Wn, Wc, b, bc = run.dev_params
    return {"W_self": lambda: Ws[l], "W_neigh": lambda: Wn[l], "b": lambda: b[l],
            "W_cls": lambda: Wc, "b_cls": lambda: bc}[key]()


def check_opt(run, first_step_bound=False, tol=FP32_TOL):
    ref = run.oracle()
    errs = {}
    for key, l in _named(run):
        tag = f"{key}{'' if l is None else l}"
        W_old = _get(run.params_np(), key, l)
        W_ref = _get(ref["params"], key, l)
        W_new = _dev_tensor(run, key, l)
        d_ref = (np.asarray(W_old, np.float64) - W_ref) / run.wl.lr   # the update direction
        for i, sname in enumerate(("state1", "state2")[:len(run.state_dev)]):
            t, _ = run.state_dev[i]
            errs[f"{sname}_{tag}"] = rel(_get(t, key, l), _get(ref[sname], key, l))
        if not first_step_bound:
            errs[f"upd_{tag}"] = _update_err(W_new, W_old, d_ref, run.wl.lr)
            continue
        # Adam's first step from zero state moves each weight by
        # lr g/(|g|+eps): insensitive to the gradient's rounding unless |g|
        # is within that rounding of zero, where the sign may differ.
        g = _get(ref["grads"], "d" + key, l)
        delta = 2.0 * FP32_TOL * np.abs(g).max()
        s_dev = (np.asarray(W_old, np.float64) - W_new.detach().cpu().double().numpy()) / run.wl.lr
        ulp = np.spacing(np.abs(W_ref).astype(np.float32)).astype(np.float64) / run.wl.lr
        firm = np.abs(g) > 2 * delta
        excess = np.maximum(np.abs(s_dev - d_ref) - ulp, 0.0)
        errs[f"upd_{tag}"] = float(excess[firm].max()) if firm.any() else 0.0
        assert np.all(np.abs(s_dev[~firm]) <= 1.0 + 1e-6 + ulp[~firm]), tag
        say(tag, "firm", int(firm.sum()), "of", firm.size)
    worst = max(errs, key=errs.get)
    say("max error", worst, errs[worst])
    bad = {k: v for k, v in errs.items() if not v < tol}
    assert not bad, bad
    return errs


@pytest.mark.parametrize("name", ["tiny", "ppi8k"])
def test_momentum_step(name):
    need_gpu()
    check_opt(OptRun(synth.WORKLOADS[name], oo.MOMENTUM).run())


@pytest.mark.parametrize("name", ["tiny", "ppi8k", "yelp10k"])
def test_adam_step_mid_training(name):
    need_gpu()
    check_opt(OptRun(synth.WORKLOADS[name], oo.ADAM, step=5).run())


def test_adam_first_step_from_zero():
    need_gpu()
    check_opt(OptRun(synth.WORKLOADS["tiny"], oo.ADAM, step=1, zero_state=True).run(),
              first_step_bound=True)


@pytest.mark.parametrize("kind", [oo.MOMENTUM, oo.ADAM])
def test_optim_ragged_with_bias(kind):
    need_gpu()
    wl = synth.small_workload(437, 9, 2, 29, 36, 7, synth.SIGMOID_BCE, (2, kind, 9))
    check_opt(OptRun(wl, kind, step=3, bias=True, seg_len=4).run())


def test_optim_sgd_equals_train_step():
    """GCN_OPT_SGD through the optimiser entry is the plain step, bit for bit."""
    need_gpu()
    wl = synth.WORKLOADS["tiny"]
    a = StepRun(wl).run()
    b = OptRun(wl, oo.SGD, zero_state=True).run()
    assert a.loss == b.loss
    for x, y in zip(a.dev_params[0] + a.dev_params[1] + [a.dev_params[2]],
                    b.dev_params[0] + b.dev_params[1] + [b.dev_params[2]]):
        assert torch.equal(x, y)


def test_optim_errors_before_launch():
    need_gpu()
    from paper_2001_02498_amd import gcn
    wl = synth.WORKLOADS["tiny"]
    run = OptRun(wl, oo.ADAM)
    inp = run.inp
    X = dev(inp.X)
    Ws, Wn, Wc, b, bc = run.params_dev()
    P = gcn.make_params(Ws, Wn, Wc)
    S = gcn.make_params([torch.zeros_like(w) for w in Ws], [torch.zeros_like(w) for w in Wn],
                        torch.zeros_like(Wc))
    desc = gcn.model_desc(wl.L, wl.f_in, wl.h, wl.C, wl.loss, X.stride(0))
    ws = gcn.alloc_ws(gcn.workspace_bytes(run.case.dg, desc))
    labels = torch.from_numpy(inp.labels).cuda()
    loss = torch.zeros(1, device="cuda")
    before = [w.clone() for w in Ws]
    cases = [(gcn.optim(7, 0.01), S, S),                             # unknown kind
             (gcn.optim(gcn.OPT_ADAM, 0.01, step=0), S, S),          # step < 1
             (gcn.optim(gcn.OPT_ADAM, 0.01), S, None),               # no second moment
             (gcn.optim(gcn.OPT_MOMENTUM, 0.01), None, None),        # no velocity
             (gcn.optim(gcn.OPT_MOMENTUM, 0.01, momentum=1.0), S, None),
             (gcn.optim(gcn.OPT_ADAM, 0.01, beta2=1.0), S, S),
             (gcn.optim(gcn.OPT_ADAM, 0.01, eps=0.0), S, S)]
    for opt, s1, s2 in cases:
        with pytest.raises(gcn.GcnError) as e:
            gcn.train_step_optim(run.case.dg, desc, P, X, labels, opt, loss, ws, state1=s1,
                                 state2=s2)
        assert e.value.code == gcn.E_INVALID_ARG, (opt.kind, e.value)
    torch.cuda.synchronize()
    for w0, w in zip(before, Ws):
        assert torch.equal(w0, w)


@pytest.mark.parametrize("name,kind", [("ppi8k", oo.ADAM), ("tiny", oo.MOMENTUM)])
def test_optim_bf16_step(name, kind):
    """Optimisers in the bf16 step on operand copies: the weights' copies are
    taken before their in-place update."""
    need_gpu()
    from paper_2001_02498_amd import gcn
    run = OptRun(synth.WORKLOADS[name], kind, step=5, precision=gcn.PREC_BF16).run()
    assert run.layout.ah_bytes == 2
    check_opt(run, tol=BF16_TOL)


def test_optim_bf16_ragged_with_bias():
    need_gpu()
    from paper_2001_02498_amd import gcn
    wl = synth.small_workload(437, 9, 2, 29, 40, 7, synth.SIGMOID_BCE, (2, 9, 16))
    run = OptRun(wl, oo.ADAM, step=3, bias=True, seg_len=4, precision=gcn.PREC_BF16).run()
    check_opt(run, tol=BF16_TOL)
