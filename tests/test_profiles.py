"""The committed rocprofv3 counter summaries against what the kernels must
move (CPU only: reads the text files under profiles/).

`bench.py` turns FETCH_SIZE and WRITE_SIZE per dispatch into HBM bytes with
the factor each counter shows on a plain 256 MiB device copy.  A wrong factor
(say, one taken from a copy of another size) would put the reported traffic
below the bytes the kernel cannot avoid, so the summaries are checked here:
the factors match their own copy probe and the gfx950 behaviour (the fetch
counter reads half of the bytes, the write counter all of them), and the input
transform's counted bytes equal its algorithmic bytes (read x, write Vq once),
while the tap GEMM's are at least its own (read Vq and Uq, write y)."""
import glob
import os

import pytest

import bench

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SUMMARIES = sorted(glob.glob(os.path.join(ROOT, "profiles", "*_hbm_counters.txt")))


def _parse(path):
    vals, kern = {}, {}
    for line in open(path):
        tok = line.split()
        if not tok or tok[0].startswith("#") or tok[0] == "source_sha256":
            continue
        if tok[0] == "kernel":
            kern[tok[1]] = (float(tok[3]), float(tok[5]))
        elif len(tok) == 2:
            vals[tok[0]] = float(tok[1])
    return vals, kern


def test_summaries_exist():
    assert any(p.endswith("C5_nhwc_hbm_counters.txt") for p in SUMMARIES)


@pytest.mark.parametrize("path", SUMMARIES, ids=[os.path.basename(p) for p in SUMMARIES])
def test_copy_probe_scales(path):
    vals, kern = _parse(path)
    probe = vals["copy_probe_bytes"]
    assert probe == 256 << 20
    assert vals["fetch_scale"] == pytest.approx(probe / 1024 / vals["copy_probe_FETCH_SIZE_KiB"], rel=1e-3)
    assert vals["write_scale"] == pytest.approx(probe / 1024 / vals["copy_probe_WRITE_SIZE_KiB"], rel=1e-3)
    assert 1.9 <= vals["fetch_scale"] <= 2.1
    assert 0.95 <= vals["write_scale"] <= 1.05
    assert kern


def test_c5_traffic_against_algorithmic_bytes():
    path = os.path.join(ROOT, "profiles", "C5_nhwc_hbm_counters.txt")
    vals, kern = _parse(path)
    n, cin, cout, h, w = 4, 256, 256, 160, 160
    t = n * ((h + 3) // 4) * ((w + 3) // 4)
    k1_alg = n * h * w * cin + 36 * t * cin
    k2_alg = 36 * t * cin + 36 * cin * cout + n * h * w * cout + 4 * cout

    def counted(prefix):
        (f, wr), = [v for k, v in kern.items() if k.startswith(prefix)]
        return f * 1024 * vals["fetch_scale"] + wr * 1024 * vals["write_scale"]

    assert 0.98 * k1_alg <= counted("wino_input_xform_nhwc<") <= 1.10 * k1_alg
    assert 1.0 * k2_alg <= counted("wino_tap_gemm_rows<") <= 2.0 * k2_alg
    # bench.py reads the same file; it reports null once the kernel source
    # differs from the one the counters were taken on
    got = bench.counter_traffic("C5", "nhwc", "wino_tap_gemm_rows")
    assert got is None or got == pytest.approx(counted("wino_tap_gemm_rows<"))
