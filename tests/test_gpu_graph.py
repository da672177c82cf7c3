"""The layer calls under HIP graph capture and on concurrent streams.

- The forward (NVFP4 weight amax computed, packed W_hat saved) and the backward from the saved
  operand, captured once into a graph and replayed several times with eager work between the
  replays (new inputs copied in), every replay bit-identical to the eager calls on the same
  inputs: the reduction slots of the amax pass clear themselves between replays, and no call
  records a memset node.
- The forward without a workspace (the static scratch) captured and replayed the same way.
- amax passes issued alternately on two streams: each returns its own tensor's amax.
"""
import numpy as np
import pytest

import oracle
import workloads
from tests.helpers import empty_bf16, from_dev, to_dev

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


@pytest.fixture(scope="module")
def qf():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2609_39223_amd as qf
    qf.lib()
    return qf


def _draw(seed, M, N, K):
    rng = np.random.default_rng(seed)
    return (workloads.normal_bf16(rng, (M, K), 1.0), workloads.normal_bf16(rng, (N, K), 0.02 * (1 + seed % 3)),
            workloads.normal_bf16(rng, (M, N), 1.0))


@pytest.mark.parametrize("wfmt,afmt", [("nvfp4", "none"), ("mxfp4", "mxfp4")])
def test_layer_captured_in_a_graph_replays_like_eager_calls(qf, wfmt, afmt):
    M, N, K = 512, 264, 768
    d = qf.qlinear_desc(M, N, K, wfmt, afmt)
    ws, sv = qf.workspace(d), qf.saved_buffer(d)
    X = torch.empty(M, K, dtype=torch.int16, device="cuda")
    W = torch.empty(N, K, dtype=torch.int16, device="cuda")
    dY = torch.empty(M, N, dtype=torch.int16, device="cuda")
    Y, dX = empty_bf16((M, N)), empty_bf16((M, K))
    dW = torch.empty(N, K, dtype=torch.float32, device="cuda")

    def calls():
        qf.qlinear_fwd(d, X, W, Y, ws, saved=sv)
        qf.qlinear_bwd_ste(d, dY, X, W, dX, dW, ws, saved=sv)

    def load(seed):
        for t, a in zip((X, W, dY), _draw(seed, M, N, K)):
            t.copy_(to_dev(a))

    def snap():
        return (from_dev(Y).view(np.uint16).copy(), from_dev(dX).view(np.uint16).copy(),
                from_dev(dW).view(np.uint32).copy())

    load(0)
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        calls()                                    # warm-up on the capturing stream kind
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        calls()
    for seed in (1, 2, 3, 1):
        load(seed)
        calls()                                    # eager reference on these inputs
        torch.cuda.synchronize()
        ref = snap()
        Y.fill_(0)
        dX.fill_(0)
        dW.fill_(0)
        g.replay()
        torch.cuda.synchronize()
        got = snap()
        for name, a, b in zip(("Y", "dX", "dW"), got, ref):
            assert np.array_equal(a, b), (name, seed)
    # and the replayed forward is the oracle's on the last inputs
    Xh, Wh, _ = _draw(1, M, N, K)
    want = oracle.linear_fwd(oracle.fakequant(Xh, afmt), oracle.fakequant(Wh, wfmt))
    from tests.helpers import assert_close, bf16_to_f64
    assert_close(bf16_to_f64(from_dev(Y)), want, "Y (graph)")


def test_noalloc_forward_captured_in_a_graph(qf):
    M, N, K = 256, 520, 512
    d = qf.qlinear_desc(M, N, K, "nvfp4", "none")
    X = torch.empty(M, K, dtype=torch.int16, device="cuda")
    W = torch.empty(N, K, dtype=torch.int16, device="cuda")
    Y = empty_bf16((M, N))
    Xh, Wh, _ = _draw(5, M, N, K)
    X.copy_(to_dev(Xh))
    W.copy_(to_dev(Wh))
    qf.qlinear_fwd_noalloc(d, X, W, Y)             # first call on the device: the scratch lookup
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        qf.qlinear_fwd_noalloc(d, X, W, Y)
    ws = qf.workspace(d)
    for seed in (6, 7, 6):
        Xh, Wh, _ = _draw(seed, M, N, K)
        X.copy_(to_dev(Xh))
        W.copy_(to_dev(Wh))
        Yref = empty_bf16((M, N))
        qf.qlinear_fwd(d, X, W, Yref, ws)
        Y.fill_(0)
        g.replay()
        torch.cuda.synchronize()
        assert np.array_equal(from_dev(Y).view(np.uint16), from_dev(Yref).view(np.uint16)), seed


def test_amax_on_two_streams(qf):
    rng = np.random.default_rng(31)
    a = workloads.normal_bf16(rng, (2048, 4096), 0.5)
    b = workloads.normal_bf16(rng, (1024, 3072), 0.01)
    A, B = to_dev(a), to_dev(b)
    s1, s2 = torch.cuda.Stream(), torch.cuda.Stream()
    oa = torch.zeros(200, dtype=torch.float32, device="cuda")
    ob = torch.zeros(200, dtype=torch.float32, device="cuda")
    torch.cuda.synchronize()
    for i in range(200):
        with torch.cuda.stream(s1):
            qf.amax(A, oa[i:i + 1])
        with torch.cuda.stream(s2):
            qf.amax(B, ob[i:i + 1])
    torch.cuda.synchronize()
    assert np.all(from_dev(oa) == oracle.amax(a))
    assert np.all(from_dev(ob) == oracle.amax(b))
