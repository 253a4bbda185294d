"""A training step captured into a HIP graph (stream capture) and replayed.

gcn_train_step only launches kernels on the caller's stream (no allocation,
copy, fill or host wait on the way), which is what capture needs. Each
replay must equal the eager step from the same state bit for bit: the same
kernels run in the same order on the same buffers. The replays are separated
by eager work of the program's own and synchronisations, and every one of
them is checked, loss and updated weights."""
import pytest

from paper_2001_02498_amd import synth
from tests.gpu_helpers import dev, need_gpu, say, torch
from tests.test_gpu_step import StepRun

pytestmark = pytest.mark.gpu

STEPS = 3


def _setup(run):
    """Fresh weights, workspace and loss for the run's workload and graph."""
    gcn, wl, inp = run.gcn, run.wl, run.inp
    Ws, Wn, Wc, b, bc = run.params_dev()
    weights = Ws + Wn + [Wc] + (b if b else []) + ([bc] if bc is not None else [])
    P = gcn.make_params(Ws, Wn, Wc, b, bc)
    X = dev(inp.X)
    desc = gcn.model_desc(wl.L, wl.f_in, wl.h, wl.C, wl.loss, X.stride(0),
                          has_bias=run.bias, precision=run.precision, order=run.order)
    ws = gcn.alloc_ws(gcn.workspace_bytes(run.case.dg, desc))
    labels = torch.from_numpy(inp.labels).cuda()
    loss = torch.zeros(1, device="cuda")

    def step():
        gcn.train_step(run.case.dg, desc, P, X, labels, wl.lr, loss, ws)

    return step, weights, loss


@pytest.mark.parametrize("name,precision,order,bias",
                         [("tiny", 0, 0, False), ("tiny", 1, 0, True), ("ppi8k", 0, 0, False),
                          ("reddit8k", 0, 1, False)])
def test_graph_replay_equals_eager(name, precision, order, bias):
    need_gpu()
    from paper_2001_02498_amd import gcn
    prec = gcn.PREC_BF16 if precision else gcn.PREC_FP32
    run = StepRun(synth.WORKLOADS[name], bias=bias, precision=prec, order=order)
    say("graph replay", name, "precision", prec, "order", order, "bias", bias)

    step, weights, loss = _setup(run)
    eager = []
    for _ in range(STEPS):
        step()
        torch.cuda.synchronize()
        eager.append(([w.clone() for w in weights], loss.clone()))

    step, weights, loss = _setup(run)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    side = torch.cuda.Stream()
    with torch.cuda.stream(side):
        graph.capture_begin()
        step()
        graph.capture_end()
    torch.cuda.synchronize()
    # capture records the launches without running them: the weights are
    # still the initial ones
    for w, w0 in zip(weights, _setup(run)[1]):
        assert torch.equal(w, w0)
    other = torch.randn(512, 512, device="cuda")
    for k in range(STEPS):
        graph.replay()
        other = torch.tanh(other @ other.T.contiguous() / 512)   # eager work between replays
        torch.cuda.synchronize()
        ref_w, ref_loss = eager[k]
        assert torch.equal(loss, ref_loss), (k, loss.item(), ref_loss.item())
        for i, (w, r) in enumerate(zip(weights, ref_w)):
            assert torch.equal(w, r), (k, i, (w - r).abs().max().item())
