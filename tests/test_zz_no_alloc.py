"""qf_qlinear_fwd_noalloc (the forward with the library's static device scratch) against
qf_qlinear_fwd with a caller workspace: bit-identical Y on two calls in a row, the second
with a smaller input, and a clear error for shapes beyond the scratch."""
import numpy as np
import pytest

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


def _inputs(seed, M, N, K):
    rng = np.random.default_rng(seed)
    return (workloads.normal_bf16(rng, (M, K), 1.0), workloads.normal_bf16(rng, (N, K), 0.02))


@pytest.mark.parametrize("wfmt,afmt", [("nvfp4", "none"), ("mxfp4", "mxfp4"), ("q4k", "none"),
                                       ("nvfp4", "mxfp4")])
def test_noalloc_forward_matches_workspace_forward(qf, wfmt, afmt):
    # second call smaller than the first: what the first left in the scratch must not leak
    for seed, (M, N, K) in enumerate([(1024, 2048, 4096), (264, 520, 512)]):
        Xh, Wh = _inputs(seed + 3, M, N, K)
        X, W = to_dev(Xh), to_dev(Wh)
        d = qf.qlinear_desc(M, N, K, wfmt, afmt)
        ws = qf.workspace(d)
        Y_ref = empty_bf16((M, N))
        qf.qlinear_fwd(d, X, W, Y_ref, ws)
        Y = torch.full((M, N), 0x7FC0, dtype=torch.int16, device="cuda")
        qf.qlinear_fwd_noalloc(d, X, W, Y)
        torch.cuda.synchronize()
        assert np.array_equal(from_dev(Y).view(np.uint16), from_dev(Y_ref).view(np.uint16)), \
            (wfmt, afmt, M, N, K)


def test_noalloc_forward_rejects_shapes_beyond_the_scratch(qf):
    # 2 N K bytes of W_hat alone exceed 64 MiB; nothing is launched
    M, N, K = 8, 8200, 4096
    d = qf.qlinear_desc(M, N, K, "mxfp4", "none")
    X = torch.zeros(M, K, dtype=torch.int16, device="cuda")
    W = torch.zeros(N, K, dtype=torch.int16, device="cuda")
    Y = torch.full((M, N), 5, dtype=torch.int16, device="cuda")
    with pytest.raises(qf.QFError, match="QF_ESHAPE"):
        qf.qlinear_fwd_noalloc(d, X, W, Y)
    torch.cuda.synchronize()
    assert int((Y != 5).sum().item()) == 0
