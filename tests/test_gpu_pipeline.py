"""GPU: the overlapped schedule (host workers preparing -- reducing on the
host or driving the device reduction on streams of their own -- copy-stream
uploads into two device slots, compute stream waiting on copy events) trains
to the same weights, bit for bit, as preparing and uploading each subgraph
first."""
import collections

import numpy as np
import pytest

from paper_2001_02498_amd import synth
from tests.gpu_helpers import dev, need_gpu, say, torch

pytestmark = pytest.mark.gpu


class _D:
    def __init__(self, d):
        self.desc = d


def _model(gcn, wl, inp):
    Ws = [dev(w, wl.h) for w in inp.W_self]
    Wn = [dev(w, wl.h) for w in inp.W_neigh]
    Wc = torch.from_numpy(inp.W_cls.copy()).cuda()
    return Ws, Wn, Wc


@pytest.mark.parametrize("device_reduce", [False, True, "mixed"])
def test_pipelined_stream_matches_sequential(device_reduce):
    need_gpu()
    from paper_2001_02498_amd import gcn
    import dataclasses
    K = 6
    wls = [dataclasses.replace(synth.stream_workload(i), n=1500, f_in=40, h=32, C=10)
           for i in range(K)]
    wl = wls[0]
    inps = [synth.make_inputs(w) for w in wls]
    Xs = [dev(inp.X) for inp in inps]
    Ys = [torch.from_numpy(inp.labels).cuda() for inp in inps]
    desc = gcn.model_desc(wl.L, wl.f_in, wl.h, wl.C, wl.loss, Xs[0].stride(0))
    loss = torch.zeros(1, device="cuda")

    # sequential reference
    Ws, Wn, Wc = _model(gcn, wl, inps[0])
    P = gcn.make_params(Ws, Wn, Wc)
    dgs = []
    for inp in inps:
        red = gcn.redundancy_reduce(gcn.subgraph_build(wl.n, inp.src, inp.dst), theta=wl.theta,
                                    max_rounds=wl.rounds, max_aux=wl.max_aux)
        dgs.append(gcn.DeviceGraph(red))
    ws = gcn.alloc_ws(max(gcn.workspace_bytes(d, desc) for d in dgs))
    for i in range(K):
        gcn.train_step(dgs[i], desc, P, Xs[i], Ys[i], wl.lr, loss, ws)
    torch.cuda.synchronize()
    ref = [w.clone() for w in Ws + Wn + [Wc]]
    say("sequential loss", loss.item())

    # overlapped schedule
    Ws, Wn, Wc = _model(gcn, wl, inps[0])
    P = gcn.make_params(Ws, Wn, Wc)
    slots = [gcn.alloc_ws(max(d.nbytes for d in dgs)) for _ in range(2)]
    copy = torch.cuda.Stream()
    comp = torch.cuda.current_stream()
    slot_free = [None, None]
    held = collections.deque()
    # the GPU-reducing workers' device workspace, sized up front
    gs = [gcn.subgraph_build(wl.n, inp.src, inp.dst) for inp in inps]
    rr = dict(theta=wl.theta, max_rounds=wl.rounds, max_aux=wl.max_aux)
    if device_reduce == "mixed":
        # two host and two GPU-reducing workers share the queue
        dws = gcn.alloc_ws(gcn.device_reduce_bytes(gs, 2, **rr))
        pipe = gcn.Pipeline(**rr, workers=2, device_workers=2, depth=4, pinned=True,
                            device_ws=dws)
    else:
        dws = gcn.alloc_ws(gcn.device_reduce_bytes(gs, 3, **rr)) if device_reduce else None
        pipe = gcn.Pipeline(**rr, workers=3, depth=4, pinned=True, device_reduce=device_reduce,
                            device_ws=dws)
    try:
        for inp in inps:
            pipe.submit(wl.n, inp.src, inp.dst)
        for i in range(K):
            jid, ptr, nb, info = pipe.next()
            assert jid == i and nb == dgs[i].nbytes
            slot = i % 2
            with torch.cuda.stream(copy):
                if slot_free[slot] is not None:
                    copy.wait_event(slot_free[slot])
                d = gcn.upload_image(ptr, nb, slots[slot], stream=copy)
                copied = torch.cuda.Event()
                copied.record(copy)
            comp.wait_event(copied)
            gcn.train_step(_D(d), desc, P, Xs[i], Ys[i], wl.lr, loss, ws)
            done = torch.cuda.Event()
            done.record(comp)
            slot_free[slot] = done
            held.append((jid, copied))
            while len(held) > 1:
                j, e = held.popleft()
                e.synchronize()
                pipe.release(j)
        torch.cuda.synchronize()
        for j, _ in held:
            pipe.release(j)
    finally:
        pipe.close()
    for a, b in zip(ref, Ws + Wn + [Wc]):
        assert torch.equal(a, b)


def _np_weights(Ws, Wn, Wc):
    return ([w.cpu().numpy().copy() for w in Ws], [w.cpu().numpy().copy() for w in Wn],
            Wc.cpu().numpy().copy())


def test_full_stream_pipelined_matches_sequential_and_oracle():
    # eight subgraphs of the 64-subgraph stream at full size (8,000
    # vertices, 3 layers, 256 + 256 per layer, 64 classes): the overlapped
    # schedule reaches the sequential run's weights bit for bit, and
    # subgraphs 0 and 7, each from the weights the stream had reached,
    # match the oracle's step
    need_gpu()
    import dataclasses
    from paper_2001_02498_amd import gcn
    from tests.test_gpu_step import StepRun, check_step
    K = 8
    wls = [synth.stream_workload(i) for i in range(K)]
    wl = wls[0]
    inps = [synth.make_inputs(w) for w in wls]
    Xs = [dev(inp.X) for inp in inps]
    Ys = [torch.from_numpy(inp.labels).cuda() for inp in inps]
    desc = gcn.model_desc(wl.L, wl.f_in, wl.h, wl.C, wl.loss, Xs[0].stride(0))
    loss = torch.zeros(1, device="cuda")
    rr = dict(theta=wl.theta, max_rounds=wl.rounds, max_aux=wl.max_aux)

    # sequential: prepare and upload each subgraph, then step
    Ws, Wn, Wc = _model(gcn, wl, inps[0])
    P = gcn.make_params(Ws, Wn, Wc)
    gs = [gcn.subgraph_build(wl.n, inp.src, inp.dst) for inp in inps]
    dgs = [gcn.DeviceGraph(gcn.redundancy_reduce(g, **rr)) for g in gs]
    ws = gcn.alloc_ws(max(gcn.workspace_bytes(d, desc) for d in dgs))
    snap = {}
    for i in range(K):
        if i == K - 1:
            torch.cuda.synchronize()
            snap["before_last"] = _np_weights(Ws, Wn, Wc)
        say("sequential step", i, "n", wl.n, "naux", dgs[i].desc.naux)
        gcn.train_step(dgs[i], desc, P, Xs[i], Ys[i], wl.lr, loss, ws)
        if i == 0:
            torch.cuda.synchronize()
            snap["after_first"] = [w.clone() for w in Ws + Wn + [Wc]]
    torch.cuda.synchronize()
    ref = [w.clone() for w in Ws + Wn + [Wc]]

    # overlapped: three host workers and one GPU-reducing worker prepare
    # ahead, uploads on a copy stream into two slots
    Ws, Wn, Wc = _model(gcn, wl, inps[0])
    P = gcn.make_params(Ws, Wn, Wc)
    slots = [gcn.alloc_ws(max(d.nbytes for d in dgs)) for _ in range(2)]
    copy = torch.cuda.Stream()
    comp = torch.cuda.current_stream()
    slot_free = [None, None]
    held = collections.deque()
    dws = gcn.alloc_ws(gcn.device_reduce_bytes(gs, 1, **rr))
    pipe = gcn.Pipeline(**rr, workers=3, device_workers=1, depth=5, pinned=True, device_ws=dws)
    try:
        for inp in inps:
            pipe.submit(wl.n, inp.src, inp.dst)
        for i in range(K):
            jid, ptr, nb, info = pipe.next()
            assert jid == i and nb == dgs[i].nbytes
            slot = i % 2
            with torch.cuda.stream(copy):
                if slot_free[slot] is not None:
                    copy.wait_event(slot_free[slot])
                d = gcn.upload_image(ptr, nb, slots[slot], stream=copy)
                copied = torch.cuda.Event()
                copied.record(copy)
            comp.wait_event(copied)
            gcn.train_step(_D(d), desc, P, Xs[i], Ys[i], wl.lr, loss, ws)
            done = torch.cuda.Event()
            done.record(comp)
            slot_free[slot] = done
            held.append((jid, copied))
            while len(held) > 1:
                j, e = held.popleft()
                e.synchronize()
                pipe.release(j)
        torch.cuda.synchronize()
        for j, _ in held:
            pipe.release(j)
    finally:
        pipe.close()
    for a, b in zip(ref, Ws + Wn + [Wc]):
        assert torch.equal(a, b)

    # subgraph 0 from the initial weights, subgraph K-1 from the weights
    # before its step: the oracle's step, and the same update as the stream's
    L = wl.L
    for i, start, want in ((0, None, snap["after_first"]), (K - 1, snap["before_last"], ref)):
        inp = inps[i]
        if start is not None:
            inp = dataclasses.replace(inp, W_self=start[0], W_neigh=start[1], W_cls=start[2])
        run = StepRun(wls[i], inp=inp).run()
        check_step(run)
        Ws_i, Wn_i, Wc_i, _, _ = run.dev_params
        for a, b in zip(want, Ws_i + Wn_i + [Wc_i]):
            assert torch.equal(a, b), f"subgraph {i}: the step alone differs from the stream's"
        assert len(Ws_i) == L
