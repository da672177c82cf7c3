"""Pins of the export oracle (Sec. 3.2.3 "Engine-specific scale sharing", NVFP4 paragraph;
Sec. 3.5): the tied tensor scale is the one of the concatenated weight, the fused codes decode
to the fake-quantized concatenation, the exported input scale is the decode scale the
activation quantizer uses for the same running amax, and the payload layout round-trips."""
import numpy as np

import oracle
import workloads


def _members(seed):
    rng = np.random.default_rng(seed)
    return [workloads.normal_bf16(rng, (n, 256), s) for n, s in ((96, 0.02), (32, 0.05), (32, 0.01))]


def test_tied_scale_is_the_concatenations():
    ms = _members(1)
    e = oracle.export_fused(ms, "nvfp4", a_amax=7.5)
    W = np.concatenate(ms)
    assert e["amax"] == max(oracle.amax(m) for m in ms)       # max over the members
    assert e["weight_scale_2"] == np.float32(e["amax"]) / np.float32(2688)
    dec = oracle.nvfp4_dequant(e["codes"], e["scales"], e["weight_scale_2"], 256)
    assert np.array_equal(dec, oracle.fakequant(W, "nvfp4"))
    # members quantized alone would use their own tensor scales: different codes
    own = oracle.nvfp4(ms[2])
    assert not np.array_equal(own["scales"], e["scales"][128:160])


def test_input_scale_matches_the_activation_quantizer():
    rng = np.random.default_rng(2)
    X = workloads.normal_bf16(rng, (64, 256), 1.0)
    running = 3.25 * oracle.amax(X)
    e = oracle.export_fused(_members(3), "nvfp4", a_amax=running)
    assert e["input_scale"] == oracle.nvfp4(X, running)["S"]


def test_mxfp4_fused_codes_are_row_blocks():
    ms = _members(4)
    e = oracle.export_fused(ms, "mxfp4")
    r0 = 0
    for m in ms:
        q = oracle.mxfp4(m)                  # no tensor scale: each member stands alone
        assert np.array_equal(e["codes"][r0:r0 + len(m)], q["codes"])
        assert np.array_equal(e["scales"][r0:r0 + len(m)], q["scales"])
        r0 += len(m)


def test_payload_layout_round_trip():
    N, K = 160, 256
    lay = oracle.payload_layout("nvfp4", N, K)
    assert lay["codes"] % 256 == 0 and lay["scales"] % 256 == 0 and lay["scalars"] % 256 == 0
    buf = np.zeros(lay["total"], np.uint8)
    hdr = np.zeros(64, np.uint8)
    hdr[0:8] = np.array([oracle.PAYLOAD_MAGIC, 1], "<u4").view(np.uint8)
    hdr[8:24] = np.array([N, K], "<i8").view(np.uint8)
    hdr[24:56] = np.array([lay["codes"], lay["scales"], lay["scalars"], lay["total"]], "<u8").view(np.uint8)
    buf[:64] = hdr
    rng = np.random.default_rng(5)
    codes = rng.integers(0, 256, (N, K // 2), dtype=np.uint8)
    scales = rng.integers(0, 127, (N, K // 16), dtype=np.uint8)
    buf[lay["codes"]:lay["codes"] + codes.size] = codes.ravel()
    buf[lay["scales"]:lay["scales"] + scales.size] = scales.ravel()
    buf[lay["scalars"]:lay["scalars"] + 8] = np.array([0.5, 0.25], "<f4").view(np.uint8)
    p = oracle.parse_payload(buf)
    assert p["magic"] == 0x31504651 and bytes(buf[:4]) == b"QFP1"
    assert (p["fmt"], p["N"], p["K"], p["total"]) == ("nvfp4", N, K, lay["total"])
    assert np.array_equal(p["codes"], codes) and np.array_equal(p["scales"], scales)
    assert list(p["scalars"]) == [0.5, 0.25]
