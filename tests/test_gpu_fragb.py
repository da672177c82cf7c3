"""GPU parity of the GEMM whose B operand is in the fragment-major layout (B's MFMA operands
straight from memory, only A staged in LDS): the packing against the layout's definition, and the
product bit for bit against the k-contiguous GEMM on the row-major B (same products, same k
order), bf16 and FP32 outputs, ragged M and N, the split last round of FP32 outputs."""
import numpy as np
import pytest

import oracle
import workloads
from tests.helpers import assert_close, bf16_to_f64, from_dev, to_dev

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


@pytest.fixture(scope="module")
def qf():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2609_39223_amd as qf
    qf.lib()
    return qf


def _layout_reference(B):
    """Element (n, k) at ((n // 32) (K / 16) + k // 16) 512 + ((n % 32) + 32 ((k // 8) % 2)) 8
    + k % 8; rows past N up to a multiple of 32 are zero."""
    N, K = B.shape
    Np = (N + 31) // 32 * 32
    out = np.zeros(Np * K, np.uint16)
    n = np.arange(N)[:, None]
    k = np.arange(K)[None, :]
    idx = ((n // 32) * (K // 16) + k // 16) * 512 + ((n % 32) + 32 * ((k // 8) % 2)) * 8 + k % 8
    out[idx.reshape(-1)] = B.reshape(-1)
    return out


@pytest.mark.parametrize("N,K", [(64, 64), (40, 128), (520, 512), (8, 16)])
def test_pack_fragments_matches_layout(qf, N, K):
    rng = np.random.default_rng(N + K)
    B = workloads.normal_bf16(rng, (N, K), 1.0)
    out = torch.full((qf.fragment_bytes(N, K) // 2,), 0x1234, dtype=torch.int16, device="cuda")
    qf.pack_fragments(to_dev(B), out)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(from_dev(out).view(np.uint16), _layout_reference(B))


@pytest.mark.parametrize("c32", [0, 1])
@pytest.mark.parametrize("M,N,K", [(264, 520, 512), (300, 1000, 1024), (8, 2056, 64), (1, 8, 128),
                                   (2048, 4096, 1024), (513, 264, 4096)])
def test_fragb_gemm_equals_kcontiguous(qf, M, N, K, c32):
    rng = np.random.default_rng(M * 3 + N + K)
    A, B = workloads.normal_bf16(rng, (M, K), 1.0), workloads.normal_bf16(rng, (N, K), 1.0)
    Ad, Bd = to_dev(A), to_dev(B)
    Bf = torch.empty(qf.fragment_bytes(N, K) // 2, dtype=torch.int16, device="cuda")
    qf.pack_fragments(Bd, Bf)
    dt = torch.float32 if c32 else torch.int16
    ws = qf.gemm_workspace(M, N, 1) if c32 else None
    C1 = torch.full((M, N), 3, dtype=dt, device="cuda")
    C2 = torch.full((M, N), 5, dtype=dt, device="cuda")
    qf.gemm_bf16_fragb(M, N, K, Ad, K, Bf, C1, N, c32, ws=ws)
    qf.gemm_bf16(M, N, K, Ad, K, 1, Bd, K, 1, C2, N, c32, ws=ws)
    torch.cuda.synchronize()
    c1, c2 = from_dev(C1), from_dev(C2)
    view = np.uint32 if c32 else np.uint16
    assert np.array_equal(c1.view(view), c2.view(view))
    got = c1.astype(np.float64) if c32 else bf16_to_f64(c1)
    assert_close(got, oracle.linear_fwd(A, B), "fragb gemm")
