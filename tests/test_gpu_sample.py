"""GPU: minibatches sampled from a full graph (Section 3.1). The device row
gather against indexing (bit-exact, every copy width), and a training step
on a sampled minibatch -- pipeline job (walk, induced subgraph, reduction,
packed image with the sampled ids after it), one upload, gathers of the
features and labels from full-graph arrays resident on the device -- against
the oracle's step on the oracle's walk and induced subgraph."""
import dataclasses

import numpy as np
import pytest

from oracle import gcn as og
from oracle import graph as ograph
from oracle import sample as osample
from paper_2001_02498_amd import synth
from tests.gpu_helpers import (FP32_TOL, checked_masks, dev, empty, need_gpu, product_bound,
                               rel, say, torch)

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("dtype,width,ld", [
    (torch.float32, 256, 256),     # 16-byte copies
    (torch.float32, 50, 52),       # 4-byte copies (200-byte rows)
    (torch.uint8, 121, 121),       # byte copies (multi-hot label rows)
    (torch.int32, 1, 1),           # class ids
])
def test_gather_rows(dtype, width, ld):
    need_gpu()
    from paper_2001_02498_amd import gcn
    rng = np.random.default_rng(width)
    n_src, n = 3000, 777
    say("gather", dtype, width, ld)
    if dtype == torch.float32:
        full = torch.from_numpy(rng.standard_normal((n_src, ld)).astype(np.float32))
    else:
        full = torch.from_numpy(rng.integers(0, 120, (n_src, ld)).astype(np.int64)).to(dtype)
    src = full.cuda()[:, :width]
    idx = rng.integers(0, n_src, n).astype(np.int32)
    idx[5] = n_src          # out of range: row left untouched
    idx[6] = -1
    d_idx = torch.from_numpy(idx).cuda()
    dst = torch.full((n, ld), 7, dtype=dtype, device="cuda")[:, :width]
    gcn.gather_rows(src, d_idx, dst)
    torch.cuda.synchronize()
    got = torch.as_strided(dst, (n, ld), (ld, 1)).cpu()
    ok = (idx >= 0) & (idx < n_src)
    want = torch.full((n, ld), 7, dtype=dtype)
    want[torch.from_numpy(ok), :width] = full[torch.from_numpy(idx[ok]).long(), :width]
    assert torch.equal(got, want)
    # nothing to do
    gcn.gather_rows(src, d_idx[:0], dst)
    torch.cuda.synchronize()


def test_sampled_minibatch_step():
    need_gpu()
    from paper_2001_02498_amd import gcn
    n_full, m, budget = 20000, 40, 1500
    wl = dataclasses.replace(synth.SAMPLED["yelpfull"], f_in=40, h=32, C=10)
    fi = synth.make_full_inputs(wl, n_full=n_full)
    full = gcn.subgraph_build(n_full, fi.src, fi.dst)
    X_full = dev(fi.X)
    Y_full = torch.from_numpy(fi.labels).cuda()
    Ws = [dev(w, wl.h) for w in fi.W_self]
    Wn = [dev(w, wl.h) for w in fi.W_neigh]
    Wc = torch.from_numpy(fi.W_cls.copy()).cuda()
    gWc = torch.zeros_like(Wc)
    P = gcn.make_params(Ws, Wn, Wc)
    G = gcn.make_params([None] * wl.L, [None] * wl.L, gWc)
    seed = wl.sample_seed(3)

    pipe = gcn.Pipeline(theta=wl.theta, max_rounds=wl.rounds, max_aux=wl.max_aux, workers=2,
                        depth=2, pinned=True)
    try:
        pipe.submit_sample(full, m, budget, seed, wl.max_steps)
        jid, ptr, nb, info = pipe.next()
        say("sampled job: n", info.n, "nnz", info.nnz_direct, "naux", info.naux,
            "steps", info.steps)
        slot = gcn.alloc_ws(nb)
        d = gcn.upload_image(ptr, nb, slot)
        torch.cuda.synchronize()
        pipe.release(jid)
    finally:
        pipe.close()
    n = info.n
    vidx = slot[info.vertices_offset:info.vertices_offset + 4 * n].view(torch.int32)
    X = empty(n, wl.f_in)
    Y = torch.empty(n, dtype=torch.int32, device="cuda")
    gcn.gather_rows(X_full, vidx, X)
    gcn.gather_rows(Y_full, vidx, Y)

    class _D:
        desc = d
    desc = gcn.model_desc(wl.L, wl.f_in, wl.h, wl.C, wl.loss, X.stride(0))
    ws = gcn.alloc_ws(gcn.workspace_bytes(_D, desc))
    lay = gcn.workspace_layout(_D, desc)
    loss = torch.zeros(1, device="cuda")
    gcn.train_step(_D, desc, P, X, Y, wl.lr, loss, ws, grads=G)
    torch.cuda.synchronize()

    # the oracle: its own walk and induced subgraph of the same full graph
    rp, cl = ograph.subgraph_build(n_full, fi.src, fi.dst)
    V = osample.frontier_sample([int(x) for x in rp], [int(x) for x in cl], m, budget, seed,
                                wl.max_steps)
    assert np.array_equal(vidx.cpu().numpy(), np.asarray(V, np.int32))
    assert torch.equal(X.cpu(), torch.from_numpy(fi.X[V]))
    assert np.array_equal(Y.cpu().numpy(), fi.labels[V])
    srp, scl = osample.induce(rp, cl, V)
    def region(off, cols, ld):
        return ws[off:off + 4 * n * ld].view(torch.float32).view(n, ld)[:, :cols].cpu().numpy()

    H = [region(lay.H[l], 2 * wl.h, lay.ld_H) for l in range(wl.L)]
    params = dict(W_self=fi.W_self, W_neigh=fi.W_neigh, b=[None] * wl.L, W_cls=fi.W_cls,
                  b_cls=None)
    # the oracle's own ReLU decisions; the kernel's may differ only within
    # rounding of zero (checked), and only there does the oracle follow them
    fw = og.forward(srp, scl, fi.X[V], params)
    bounds = []
    for l in range(wl.L):
        F = wl.f_in if l == 0 else 2 * wl.h
        Hg = fi.X[V] if l == 0 else H[l - 1]
        AHg = region(lay.AH[l], F, lay.ld_AH[l])
        bounds.append(np.concatenate(
            [product_bound(Hg, fw["H"][l], fi.W_self[l]),
             product_bound(AHg, fw["AH"][l], fi.W_neigh[l])], axis=1))
    masks, _ = checked_masks(fw["Z"], [x > 0 for x in H], bounds, "sampled")
    ref = og.train_step(srp, scl, fi.X[V], params, fi.labels[V], wl.loss, wl.lr,
                        masks=masks, fw=fw)
    e_loss = abs(loss.item() - ref["loss"]) / abs(ref["loss"])
    e_dw = rel(gWc, ref["grads"]["dW_cls"])
    errs = [rel(w, ref["params"]["W_self"][l]) for l, w in enumerate(Ws)]
    errs += [rel(w, ref["params"]["W_neigh"][l]) for l, w in enumerate(Wn)]
    errs += [rel(Wc, ref["params"]["W_cls"])]
    say(f"loss {loss.item():.6f} oracle {ref['loss']:.6f}; rel loss {e_loss:.2e} "
        f"dW_cls {e_dw:.2e} W {max(errs):.2e}")
    assert e_loss < FP32_TOL and e_dw < FP32_TOL and max(errs) < FP32_TOL


@pytest.mark.parametrize("mode", ["device", "mixed"])
def test_sampled_jobs_reduced_on_gpu_match_host(mode):
    # sampled jobs whose reduction runs on the GPU (all workers, or one of
    # two) give byte-identical buffers (image and ids) to host-reduced jobs
    need_gpu()
    import ctypes
    from paper_2001_02498_amd import gcn
    wl = synth.SAMPLED["yelpfull"]
    fi = synth.make_full_inputs(wl, n_full=30000)
    full = gcn.subgraph_build(30000, fi.src, fi.dst)
    jobs = [(60, 2000, wl.sample_seed(i), wl.max_steps) for i in range(5)]

    # the GPU-reducing workers' device workspace, sized up front from the
    # same walks taken on the host
    rr = dict(theta=wl.theta, max_rounds=wl.rounds, max_aux=wl.max_aux)
    gs = [gcn.subgraph_induce(full, gcn.sample_frontier(full, *j)[0]) for j in jobs]
    dws = gcn.alloc_ws(gcn.device_reduce_bytes(gs, 2, **rr))

    def buffers(**kw):
        if kw.get("device_reduce") or kw.get("device_workers"):
            kw["device_ws"] = dws
        pipe = gcn.Pipeline(**rr, depth=3, pinned=True, **kw)
        out = []
        try:
            for j in jobs:
                pipe.submit_sample(full, *j)
            for _ in jobs:
                jid, ptr, nb, info = pipe.next()
                out.append(bytes((ctypes.c_uint8 * nb).from_address(ptr)))
                pipe.release(jid)
        finally:
            pipe.close()
        return out

    host = buffers(workers=2)
    if mode == "device":
        dev_ = buffers(workers=2, device_reduce=True)
    else:
        dev_ = buffers(workers=1, device_workers=1)
    say("sampled job buffers", [len(b) for b in host])
    assert host == dev_
