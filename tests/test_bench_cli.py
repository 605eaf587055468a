"""Host-side pieces of bench.py: the one-GPU guard, the counter summary it reads for
`roofline.traffic`, and the source digest that ties that summary to the library it was taken on."""
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import bench  # noqa: E402


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr or "single MI355X" in r.stderr
    assert r.stdout == ""


def test_source_digest_is_stable_and_short():
    a, b = bench.source_digest(), bench.source_digest()
    assert a == b and len(a) == 16
    int(a, 16)


def _summary(tmp_path, kernel, workload, digest, value):
    d = tmp_path / "profiles"
    d.mkdir(exist_ok=True)
    (d / f"{kernel}_{workload}_hbm_traffic.txt").write_text(
        "# test summary\n"
        f"kernel: {kernel}\n"
        f"hbm_bytes_per_launch: {value}\n"
        f"source_digest: {digest}\n")


def test_traffic_read_only_for_matching_digest(tmp_path, monkeypatch):
    monkeypatch.setattr(bench, "ROOT", str(tmp_path))
    _summary(tmp_path, "conv2", "w", "0123456789abcdef", 1507518290)
    assert bench.load_traffic("conv2", "w", "0123456789abcdef") == 1507518290.0
    assert bench.load_traffic("conv2", "w", "fedcba9876543210") is None   # other source
    assert bench.load_traffic("conv3", "w", "0123456789abcdef") is None   # no summary


def test_committed_traffic_summary_parses():
    """The committed summary of the dominant kernel names a digest and a byte count that the bench
    can read (it reports them only when the digest matches the library's sources)."""
    path = os.path.join(ROOT, "profiles",
                        "conv2_xga768x1024_25scale_1200plane_batch16_hbm_traffic.txt")
    if not os.path.exists(path):
        pytest.skip("no committed traffic summary")
    vals = {}
    for line in open(path):
        if ":" in line and not line.startswith("#"):
            k, v = line.split(":", 1)
            vals[k.strip()] = v.strip()
    assert len(vals["source_digest"]) == 16
    assert float(vals["hbm_bytes_per_launch"]) > 0
    got = bench.load_traffic("conv2", "xga768x1024_25scale_1200plane_batch16", vals["source_digest"])
    assert got == float(vals["hbm_bytes_per_launch"])


def test_probe_library_exports_its_entry_point():
    """libprobe.so (the matrix-core rate probe behind `bench.py --ceilings`) loads without a GPU and
    exports its one entry point; argument checks run before any device call."""
    import ctypes
    path = os.path.join(ROOT, "paper_1404_1869_amd", "libprobe.so")
    if not os.path.exists(path):
        pytest.skip("libprobe.so not built")
    lib = ctypes.CDLL(path)
    fn = lib.densenet_probe_mfma_bf16
    fn.restype = ctypes.c_int
    fn.argtypes = [ctypes.c_int, ctypes.c_int, ctypes.c_void_p, ctypes.c_int64,
                   ctypes.POINTER(ctypes.c_double), ctypes.c_void_p]
    flop = ctypes.c_double()
    assert fn(3, 1, 1, 1 << 20, ctypes.byref(flop), None) == -1      # unknown mode
    assert fn(0, 0, 1, 1 << 20, ctypes.byref(flop), None) == -1      # no launches
    assert fn(0, 1, None, 1 << 20, ctypes.byref(flop), None) == -1   # no buffer


def test_cpu_model_names_the_host():
    s = bench.cpu_model()
    assert "logical CPUs usable" in s and s[0] != "("
