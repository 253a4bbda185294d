"""The host preparation pipeline (worker threads building, reducing and
packing subgraphs ahead of the device) on the CPU: results in submission
order, images identical to direct packing, failures reported per job, and
the hold limit that keeps a misused pipeline from waiting forever."""
import ctypes
import os

import numpy as np
import pytest

from paper_2001_02498_amd import synth

gcn = pytest.importorskip("paper_2001_02498_amd.gcn")
ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _direct_image(n, src, dst, theta, rounds, seg_len):
    red = gcn.redundancy_reduce(gcn.subgraph_build(n, src, dst), theta=theta,
                                max_rounds=rounds)
    nb = gcn.image_bytes(red, seg_len)
    buf = np.zeros(nb, dtype=np.uint8)
    gcn.pack(red, buf.ctypes.data, nb, seg_len)
    return buf, red.info()


def _image_bytes(ptr, nb):
    return np.frombuffer((ctypes.c_uint8 * nb).from_address(ptr), dtype=np.uint8).copy()


@pytest.mark.parametrize("workers", [1, 3, 8])
def test_pipeline_order_and_images(workers):
    rng = np.random.default_rng(workers)
    graphs = []
    for i in range(12):
        n = int(rng.integers(20, 300))
        s, d = synth.random_edges(n, int(rng.integers(0, 8 * n)), rng)
        graphs.append((n, s, d))
    pipe = gcn.Pipeline(theta=1, max_rounds=3, seg_len=7, workers=workers, depth=4, pinned=False)
    try:
        ids = [pipe.submit(n, s, d) for (n, s, d) in graphs]
        assert ids == list(range(12))
        for i, (n, s, d) in enumerate(graphs):
            jid, ptr, nb, info = pipe.next()
            assert jid == i
            want, winfo = _direct_image(n, s, d, 1, 3, 7)
            assert nb == want.size
            assert np.array_equal(_image_bytes(ptr, nb), want)
            assert info.n == n and info.naux == winfo["naux"] and info.nnz == winfo["nnz"]
            assert info.reduce_ms >= 0.0 and info.build_ms >= 0.0
            pipe.release(jid)
    finally:
        pipe.close()


def test_pipeline_reports_failed_job_and_continues():
    rng = np.random.default_rng(5)
    pipe = gcn.Pipeline(workers=2, depth=3, pinned=False)
    try:
        s, d = synth.random_edges(50, 200, rng)
        pipe.submit(50, s, d)
        pipe.submit(10, np.array([0, 99]), np.array([1, 2]))   # endpoint out of range
        pipe.submit(50, s, d)
        jid, ptr, nb, info = pipe.next()
        assert jid == 0 and nb > 0
        pipe.release(jid)
        with pytest.raises(gcn.GcnError) as ei:
            pipe.next()
        assert ei.value.code == gcn.E_INVALID_ARG and "job 1" in str(ei.value)
        pipe.release(1)
        jid, ptr, nb, info = pipe.next()
        assert jid == 2 and nb > 0
        pipe.release(jid)
    finally:
        pipe.close()


def test_pipeline_hold_limit():
    rng = np.random.default_rng(6)
    pipe = gcn.Pipeline(workers=2, depth=2, pinned=False)
    try:
        for _ in range(4):
            s, d = synth.random_edges(40, 120, rng)
            pipe.submit(40, s, d)
        a = pipe.next()
        b = pipe.next()
        with pytest.raises(gcn.GcnError) as ei:      # holding `depth` jobs
            pipe.next()
        assert ei.value.code == gcn.E_INVALID_ARG
        pipe.release(a[0])
        c = pipe.next()
        assert c[0] == 2
        pipe.release(b[0])
        pipe.release(c[0])
        d_ = pipe.next()
        assert d_[0] == 3
        pipe.release(d_[0])
        with pytest.raises(gcn.GcnError):             # nothing left
            pipe.next()
        with pytest.raises(gcn.GcnError):             # double release
            pipe.release(d_[0])
    finally:
        pipe.close()


def test_pipeline_destroy_with_pending_jobs():
    rng = np.random.default_rng(7)
    pipe = gcn.Pipeline(workers=2, depth=1, pinned=False)
    for _ in range(6):
        s, d = synth.random_edges(100, 500, rng)
        pipe.submit(100, s, d)
    pipe.next()
    pipe.close()          # held job, prepared-ahead job and queued jobs all freed


def test_pipeline_argument_errors():
    with pytest.raises(gcn.GcnError):
        gcn.Pipeline(workers=0)
    with pytest.raises(gcn.GcnError):
        gcn.Pipeline(depth=0)
    with pytest.raises(gcn.GcnError):
        gcn.Pipeline(max_rounds=gcn.MAX_ROUNDS + 1)


def test_mixed_pipeline_host_only_and_rejects():
    # the mixed form with no GPU-reducing worker is the host pipeline
    rng = np.random.default_rng(11)
    graphs = []
    for _ in range(5):
        n = int(rng.integers(50, 200))
        s, d = synth.random_edges(n, 6 * n, rng)
        graphs.append((n, s, d))
    pipe = gcn.Pipeline(theta=1, max_rounds=2, seg_len=5, workers=3, device_workers=0, depth=3,
                        pinned=False)
    try:
        for n, s, d in graphs:
            pipe.submit(n, s, d)
        for i, (n, s, d) in enumerate(graphs):
            jid, ptr, nb, info = pipe.next()
            want, _ = _direct_image(n, s, d, 1, 2, 5)
            assert jid == i and np.array_equal(_image_bytes(ptr, nb), want)
            pipe.release(jid)
    finally:
        pipe.close()
    for hw, dw in ((0, 0), (-1, 1), (200, 100)):
        with pytest.raises(gcn.GcnError):
            gcn.Pipeline(workers=hw, device_workers=dw, pinned=False)


def test_device_workers_need_a_workspace():
    # GPU-reducing workers take their device workspace from the caller up
    # front; without one the pipeline is refused before any worker starts
    for kw in (dict(device_workers=1), dict(device_reduce=True)):
        with pytest.raises(gcn.GcnError) as e:
            gcn.Pipeline(workers=1, pinned=False, **kw)
        assert e.value.code == gcn.E_INVALID_ARG
        assert "device workspace" in str(e.value)


def test_handles_survive_interpreter_teardown():
    # graphs, reductions and pipelines still alive at exit are freed by
    # their __del__ after the module's globals are gone, without errors
    import subprocess
    import sys
    code = ("import numpy as np\n"
            "from paper_2001_02498_amd import gcn\n"
            "g = gcn.subgraph_build(4, np.array([0, 1, 2]), np.array([1, 2, 3]))\n"
            "r = gcn.redundancy_reduce(g, theta=0)\n"
            "p = gcn.Pipeline(workers=1, pinned=False)\n"
            "keep = [g, r, p]\n")
    out = subprocess.run([sys.executable, "-c", code], capture_output=True, text=True,
                         cwd=ROOT, timeout=120)
    assert out.returncode == 0, out.stderr
    assert "Exception ignored" not in out.stderr and "Error" not in out.stderr, out.stderr
