"""bench.py's host-side pieces, on the CPU: the kernel-source digest and the lookup of the
per-call HBM traffic in the committed rocprofv3 summary (the `traffic` field of the
bench line)."""
import os

import bench


def test_source_digest_is_stable_and_sensitive(tmp_path, monkeypatch):
    d = bench.kernel_source_digest()
    assert d == bench.kernel_source_digest() and len(d) == 16
    # a copy of the sources with one byte changed digests differently
    src = os.path.join(bench.ROOT, "paper_2606_13361_amd", "csrc")
    pkg = tmp_path / "paper_2606_13361_amd" / "csrc"
    pkg.mkdir(parents=True)
    for fn in os.listdir(src):
        if fn.endswith((".hip", ".hpp")):
            (pkg / fn).write_bytes(open(os.path.join(src, fn), "rb").read())
    monkeypatch.setattr(bench, "ROOT", str(tmp_path))
    assert bench.kernel_source_digest() == d
    first = sorted(p for p in os.listdir(pkg))[0]
    (pkg / first).write_bytes((pkg / first).read_bytes() + b"\n")
    assert bench.kernel_source_digest() != d


def test_traffic_lookup_parses_rows_and_checks_the_digest(tmp_path, monkeypatch):
    f = tmp_path / "t.md"
    f.write_text("# x\n\nsource digest: abc\n\n| call | kernels | n | fetch | write | bytes |\n|---|---|---|---|---|---|\n"
                 "| `prefill` | `k` | 3 | 1.0 | 2.0 | 12345 |\n| `readers` | `k` | 3 | 1.0 | 2.0 | 678.0 |\n")
    monkeypatch.setattr(bench, "TRAFFIC_FILE", str(f))
    assert bench.measured_traffic("abc") == {"prefill": 12345, "readers": 678}
    assert bench.measured_traffic("other") == {}
    monkeypatch.setattr(bench, "TRAFFIC_FILE", str(tmp_path / "missing.md"))
    assert bench.measured_traffic("abc") == {}


def test_committed_traffic_summary_matches_the_sources():
    """The committed profile was taken for the current kernel sources and covers every
    call of the bench step (otherwise the line's `traffic` would be null)."""
    t = bench.measured_traffic(bench.kernel_source_digest())
    for call in ("prefill", "continue32k", "continue16k", "readers", "decode_step"):
        assert t.get(call, 0) > 0, call
