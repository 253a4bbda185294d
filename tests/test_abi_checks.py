"""Argument checks of the device entry points, on the CPU.

Every check of gcn_act.h's device calls runs before the first launch, so a
call with a bad argument returns its error code, and names the problem in
gcn_last_error, without touching a GPU. The graphs and tensors here are
descriptors holding made-up device addresses that no check dereferences;
each call is one that must fail its checks (none reaches a launch)."""
import pytest

gcn = pytest.importorskip("paper_2001_02498_amd.gcn")

FAKE = 0x7f0000000000   # a 256-byte aligned address no check reads


class _Graph:
    """What the binding's entry points take: an object with `.desc`."""

    def __init__(self, n=100, naux=0):
        g = gcn.DGraph()
        g.n, g.naux, g.rounds, g.seg_len = n, naux, 0, 32
        g.nseg, g.nbins, g.nmulti, g.max_row = n, (n + 15) // 16, 0, 8
        g.nnz, g.exp_nnz = 4 * n, 0
        for f in ("rowptr", "col", "inv_deg", "seg", "bins"):
            setattr(g, f, FAKE)
        self.desc = g


class _T:
    """A stand-in tensor: a device address, a shape and a row stride."""

    def __init__(self, rows, cols, ld=None, ptr=FAKE, nbytes=None):
        self.shape = (rows, cols)
        self._ld = ld if ld is not None else cols
        self._ptr = ptr
        self._n = nbytes if nbytes is not None else 4 * rows * self._ld

    def data_ptr(self):
        return self._ptr

    def stride(self, i):
        return self._ld if i == 0 else 1

    def numel(self):
        return self._n

    def dim(self):
        return 2


def _code(fn, *a, **k):
    with pytest.raises(gcn.GcnError) as e:
        fn(*a, **k)
    return e.value.code, str(e.value)


def _desc(**kw):
    d = dict(L=2, f_in=50, h=64, C=16, loss_kind=gcn.LOSS_SOFTMAX_CE, ld_x=52)
    d.update(kw)
    return gcn.model_desc(d["L"], d["f_in"], d["h"], d["C"], d["loss_kind"], d["ld_x"],
                          precision=d.get("precision", gcn.PREC_FP32),
                          has_bias=d.get("has_bias", False), order=d.get("order", 0))


def test_workspace_size_is_host_arithmetic():
    g = _Graph()
    assert gcn.workspace_bytes(g, _desc()) > 0
    lay = gcn.workspace_layout(g, _desc(L=3, has_bias=True))
    assert lay.scratch <= lay.status < lay.total_bytes and lay.status % 4 == 0


@pytest.mark.parametrize("bad,what", [(dict(L=0), "L=0"),
                                      (dict(L=gcn.MAX_LAYERS + 1), "L="),
                                      (dict(f_in=0), "f_in"),
                                      (dict(h=6), "h=6"),
                                      (dict(C=0), "C < 1"),
                                      (dict(loss_kind=9), "loss"),
                                      (dict(ld_x=50), "ld_x"),
                                      (dict(precision=7), "precision"),
                                      (dict(order=4), "order")])
def test_model_descriptor_checks(bad, what):
    code, msg = _code(gcn.workspace_bytes, _Graph(), _desc(**bad))
    assert code == gcn.E_INVALID_ARG
    assert what in msg


def test_narrow_order_with_bias_unsupported():
    code, _ = _code(gcn.workspace_bytes, _Graph(), _desc(order=1, f_in=200, has_bias=True,
                                                         ld_x=200))
    assert code == gcn.E_UNSUPPORTED


def test_graph_descriptor_checks():
    g = _Graph()
    g.desc.rounds = 2   # the last round offset must equal naux (0 here)
    g.desc.round_offsets[2] = 5
    code, msg = _code(gcn.workspace_bytes, g, _desc())
    assert code == gcn.E_INVALID_ARG
    g = _Graph()
    g.desc.rowptr = None
    code, msg = _code(gcn.workspace_bytes, g, _desc())
    assert code == gcn.E_INVALID_ARG
    g = _Graph()
    g.desc.bins = None
    code, msg = _code(gcn.workspace_bytes, g, _desc())
    assert code == gcn.E_INVALID_ARG
    g = _Graph()
    g.desc.nmulti = g.desc.nbins + 1   # more bins with split rows than bins
    code, msg = _code(gcn.workspace_bytes, g, _desc())
    assert code == gcn.E_INVALID_ARG and "malformed" in msg
    g = _Graph()
    g.desc.nhub = 1                    # a hub bin outside the split-row bins
    code, msg = _code(gcn.workspace_bytes, g, _desc())
    assert code == gcn.E_INVALID_ARG and "malformed" in msg


def _params(L):
    P = gcn.Params()
    for l in range(L):
        P.W_self[l] = FAKE + 4096 * l
        P.W_neigh[l] = FAKE + 65536 + 4096 * l
    P.W_cls = FAKE + 2 * 65536
    return P


def test_train_step_checks_before_launch():
    g, d = _Graph(), _desc()
    X = _T(100, 50, 52)
    # a weight pointer missing
    code, msg = _code(gcn.train_step, g, d, gcn.Params(), X, X, 0.01, X,
                      _T(1, 1, nbytes=1 << 30), stream=0)
    assert code == gcn.E_INVALID_ARG and "NULL" in msg
    P = _params(2)
    need = gcn.workspace_bytes(g, d)
    small = _T(1, 1, nbytes=need - 256)
    # workspace too small
    code, msg = _code(gcn.train_step, g, d, P, X, X, 0.01, X, small, stream=0)
    assert code == gcn.E_WORKSPACE
    # workspace not 256-byte aligned
    code, msg = _code(gcn.train_step, g, d, P, X, X, 0.01, X,
                      _T(1, 1, ptr=FAKE + 16, nbytes=need), stream=0)
    assert code == gcn.E_INVALID_ARG and "aligned" in msg
    # features NULL, then not 16-byte aligned
    ws = _T(1, 1, nbytes=need)
    code, msg = _code(gcn.train_step, g, d, P, _T(100, 50, 52, ptr=0), X, 0.01, X, ws,
                      stream=0)
    assert code == gcn.E_INVALID_ARG
    code, msg = _code(gcn.train_step, g, d, P, _T(100, 50, 52, ptr=FAKE + 4), X, 0.01, X,
                      ws, stream=0)
    assert code == gcn.E_INVALID_ARG


def test_aggregate_checks_before_launch():
    g = _Graph()
    X, Y = _T(100, 16), _T(100, 16, ptr=FAKE + 65536)
    ws = _T(1, 1, nbytes=1 << 20)
    code, _ = _code(gcn.aggregate, g, 5, X, Y, ws, stream=0)          # unknown mode
    assert code == gcn.E_INVALID_ARG
    code, _ = _code(gcn.aggregate, g, gcn.AGG_MEAN, X, X, ws, stream=0)   # in place
    assert code == gcn.E_INVALID_ARG
    code, _ = _code(gcn.aggregate, g, gcn.AGG_MEAN, _T(100, 16, 18), Y, ws, stream=0)
    assert code == gcn.E_INVALID_ARG                                       # ld % 4
