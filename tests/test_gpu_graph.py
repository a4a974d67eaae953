"""The library allocates nothing and never synchronises, so its calls can be
captured into a HIP graph.  A captured training-step fragment (forward,
backward-data, backward-weight with its split reduction and overflow flag)
over a dense NHWC layer, an NCHW layer (transposes through the workspace),
a depthwise layer and a small-group layer is replayed several times, with
the outputs clobbered and eager library work run between replays; every
replay must reproduce the eager results bit for bit, and the eager results
must match the oracle."""
import numpy as np
import pytest

from gpu_util import Case, full_parity, to_dev, torch
from paper_2102_06725_amd import inputs as I
from paper_2102_06725_amd import nnconv as nc

pytestmark = pytest.mark.gpu

L = I.Layer

CASES = [
    Case(L("g_dense", 2, 64, 14, 13, 128, 3, 3, 1, 1)),
    Case(L("g_nchw", 2, 32, 11, 12, 48, 3, 3, 2, 1), layout="nchw"),
    Case(L("g_dw", 2, 96, 15, 14, 96, 5, 5, 2, 2, groups=96)),
    Case(L("g_sg", 2, 128, 9, 10, 128, 3, 3, 1, 1, groups=32), loss_scale=1024.0),
]


@pytest.fixture(scope="module", autouse=True)
def _setup(nnlib, oracle_lib):
    if not torch().cuda.is_available():
        pytest.skip("no GPU")
    yield


class Step:
    """Device buffers of one layer and the three passes queued on a stream."""

    def __init__(self, case):
        t = torch()
        self.case = case
        Ly = case.layer
        tens = case.tensors()
        self.d = case.desc()
        self.x, self.w, self.dy = to_dev(tens["x"]), to_dev(tens["w"]), to_dev(tens["dy"])
        self.y = t.empty(Ly.n * Ly.k * Ly.p * Ly.q, dtype=t.int16, device="cuda")
        self.dx = t.empty(Ly.n * Ly.c * Ly.h * Ly.w, dtype=t.int16, device="cuda")
        self.dw = t.empty(Ly.k * Ly.r * Ly.s * (Ly.c // Ly.groups), dtype=t.float32,
                          device="cuda")
        self.ws = {}
        for p in (nc.NNCONV_FWD, nc.NNCONV_DGRAD, nc.NNCONV_WGRAD):
            st, nb = nc.nnconv_workspace_size(self.d, p)
            nc.check(st, "workspace_size")
            self.ws[p] = (t.empty(max(nb, 1), dtype=t.uint8, device="cuda"), nb)

    def queue(self, stream, flag):
        c = self.case
        ws, nb = self.ws[nc.NNCONV_FWD]
        nc.check(nc.nnconv_fwd(self.d, self.x.data_ptr(), self.w.data_ptr(), self.y.data_ptr(),
                               1.0, ws.data_ptr(), nb, stream), "fwd")
        ws, nb = self.ws[nc.NNCONV_DGRAD]
        nc.check(nc.nnconv_dgrad(self.d, self.dy.data_ptr(), self.w.data_ptr(),
                                 self.dx.data_ptr(), 1.0, ws.data_ptr(), nb, stream), "dgrad")
        ws, nb = self.ws[nc.NNCONV_WGRAD]
        nc.check(nc.nnconv_wgrad(self.d, self.x.data_ptr(), self.dy.data_ptr(),
                                 self.dw.data_ptr(), nc.NNCONV_F32, 1.0 / c.loss_scale, 0,
                                 flag.data_ptr(), ws.data_ptr(), nb, stream), "wgrad")

    def outputs(self):
        return [self.y.clone(), self.dx.clone(), self.dw.clone()]

    def clobber(self):
        self.y.fill_(0x7BCD)
        self.dx.fill_(0x7BCD)
        self.dw.fill_(7.0)


def test_graph_replays_match_eager():
    t = torch()
    flag = t.zeros(1, dtype=t.int32, device="cuda")
    steps = [Step(c) for c in CASES]

    def run_all(stream_ptr):
        flag.zero_()  # a fill kernel, not a memset node
        for s in steps:
            s.queue(stream_ptr, flag)

    cur = t.cuda.current_stream()
    run_all(cur.cuda_stream)
    t.cuda.synchronize()
    eager = [s.outputs() for s in steps]
    assert int(flag.item()) == 0

    side = t.cuda.Stream()
    side.wait_stream(cur)
    with t.cuda.stream(side):
        run_all(side.cuda_stream)  # warm-up on the capture stream
    t.cuda.synchronize()
    g = t.cuda.CUDAGraph()
    with t.cuda.graph(g):
        run_all(t.cuda.current_stream().cuda_stream)
    t.cuda.synchronize()

    for rep in range(4):
        for s in steps:
            s.clobber()
        flag.fill_(1)
        t.cuda.synchronize()
        g.replay()
        t.cuda.synchronize()
        assert int(flag.item()) == 0, "replay %d: the captured flag clear did not run" % rep
        for s, ref in zip(steps, eager):
            for name, got, want in zip(("y", "dx", "dw"), s.outputs(), ref):
                assert t.equal(got, want), "replay %d, %s %s differs from eager" % (
                    rep, s.case.layer.name, name)
        # eager library work between replays, on the same buffers
        run_all(cur.cuda_stream)
        t.cuda.synchronize()


@pytest.mark.parametrize("case", CASES, ids=[c.layer.name for c in CASES])
def test_graph_cases_match_oracle(case):
    """The captured layers themselves are correct (eager, against the oracle)."""
    full_parity(case)
