"""GPU parity of the engine-native export (Sec. 3.5; Sec. 3.2.3 "Engine-specific scale
sharing") and the weight-sync payload against the oracle: codes, block scales, the tied amax,
weight_scale_2 and input_scale bit for bit; the payload parsed back by the oracle's reader."""
import numpy as np
import pytest

import oracle
import workloads
from tests.helpers import from_dev, to_dev

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


@pytest.fixture(scope="module")
def qf():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2609_39223_amd as qf
    qf.lib()
    return qf


def _members(seed, K=512):
    rng = np.random.default_rng(seed)
    # a 9B-class fused QKV at 1/32 width: Q 128 rows, K 32, V 32 (different magnitudes)
    return [workloads.normal_bf16(rng, (n, K), s) for n, s in ((128, 0.02), (32, 0.06), (32, 0.01))]


def _dev_members(ms, pad=False):
    out = []
    for m in ms:
        if pad:   # a member inside a wider buffer (row stride K + 64), NaN padding never read
            buf = np.full((m.shape[0], m.shape[1] + 64), 0x7FC0, np.uint16)
            buf[:, :m.shape[1]] = m
            out.append(to_dev(buf)[:, :m.shape[1]])
        else:
            out.append(to_dev(m))
    return out


@pytest.mark.parametrize("pad", [False, True])
def test_nvfp4_fused_export(qf, pad):
    ms = _members(1)
    K, N = 512, sum(m.shape[0] for m in ms)
    X = workloads.normal_bf16(np.random.default_rng(2), (64, K))
    a_run = np.float32(2.5 * oracle.amax(X))
    codes = torch.empty(N, K // 2, dtype=torch.uint8, device="cuda")
    scales = torch.empty(N, K // 16, dtype=torch.uint8, device="cuda")
    f = lambda v: torch.full((1,), v, dtype=torch.float32, device="cuda")
    w_amax, ws2, a_amax, isc = f(-1.0), f(-1.0), f(float(a_run)), f(-1.0)
    dm = _dev_members(ms, pad)
    qf.export_fused(dm, "nvfp4", codes, scales, w_amax=w_amax, weight_scale_2=ws2, a_amax=a_amax,
                    input_scale=isc)
    torch.cuda.synchronize()
    ref = oracle.export_fused(ms, "nvfp4", a_amax=float(a_run))
    assert np.array_equal(from_dev(codes), ref["codes"])
    assert np.array_equal(from_dev(scales), ref["scales"])
    assert from_dev(w_amax)[0] == np.float32(ref["amax"])
    assert from_dev(ws2)[0] == np.float32(ref["weight_scale_2"])
    assert from_dev(isc)[0] == np.float32(ref["input_scale"])


def test_mxfp4_fused_export(qf):
    ms = _members(3, K=256)
    N = sum(m.shape[0] for m in ms)
    codes = torch.empty(N, 128, dtype=torch.uint8, device="cuda")
    scales = torch.empty(N, 8, dtype=torch.uint8, device="cuda")
    qf.export_fused(_dev_members(ms), "mxfp4", codes, scales)
    torch.cuda.synchronize()
    ref = oracle.export_fused(ms, "mxfp4")
    assert np.array_equal(from_dev(codes), ref["codes"])
    assert np.array_equal(from_dev(scales), ref["scales"])


@pytest.mark.parametrize("fmt", ["nvfp4", "mxfp4"])
def test_weight_sync_payload(qf, fmt):
    ms = _members(5)
    K, N = 512, sum(m.shape[0] for m in ms)
    lay = qf.payload_layout(fmt, N, K)
    ref_lay = oracle.payload_layout(fmt, N, K)
    assert (lay.codes, lay.scales, lay.scalars, lay.total) == \
        (ref_lay["codes"], ref_lay["scales"], ref_lay["scalars"], ref_lay["total"])
    payload = torch.full((lay.total,), 0xAB, dtype=torch.uint8, device="cuda")
    codes = payload[lay.codes:lay.codes + N * K // 2].view(N, K // 2)
    blk = 16 if fmt == "nvfp4" else 32
    scales = payload[lay.scales:lay.scales + N * K // blk].view(N, K // blk)
    scal = payload[lay.scalars:lay.scalars + 8].view(torch.float32)
    scal.zero_()
    kw = {}
    if fmt == "nvfp4":
        w_amax = torch.empty(1, dtype=torch.float32, device="cuda")
        a_amax = torch.full((1,), 12.0, dtype=torch.float32, device="cuda")
        kw = dict(w_amax=w_amax, weight_scale_2=scal[0:1], a_amax=a_amax, input_scale=scal[1:2])
    qf.export_fused(_dev_members(ms), fmt, codes, scales, **kw)
    qf.payload_write_header(fmt, N, K, payload)
    torch.cuda.synchronize()
    p = oracle.parse_payload(from_dev(payload))
    ref = oracle.export_fused(ms, fmt, a_amax=12.0 if fmt == "nvfp4" else None)
    assert p["magic"] == oracle.PAYLOAD_MAGIC and p["fmt"] == fmt
    assert (p["N"], p["K"], p["total"]) == (N, K, lay.total)
    assert np.array_equal(p["codes"], ref["codes"]) and np.array_equal(p["scales"], ref["scales"])
    if fmt == "nvfp4":
        assert p["scalars"][0] == np.float32(ref["weight_scale_2"])
        assert p["scalars"][1] == np.float32(ref["input_scale"])
    else:
        assert list(p["scalars"]) == [0.0, 0.0]
