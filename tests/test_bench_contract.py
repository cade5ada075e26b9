"""Host-side checks of the benchmark's reporting: the committed counter summary
that `roofline.traffic` comes from is readable and is tied to the kernel
source by its hash."""
import hashlib

import bench


def _summary_with_sha(tmp_path, sha):
    text = open(bench.TRAFFIC_SUMMARY).read()
    lines = [("- kernels.hip sha256: `%s`" % sha) if l.startswith("- kernels.hip sha256:") else l
             for l in text.splitlines()]
    p = tmp_path / "sweep_traffic.md"
    p.write_text("\n".join(lines) + "\n")
    return str(p)


def test_traffic_summary_parses_when_source_matches(tmp_path, monkeypatch):
    src = hashlib.sha256(open(bench.KERNEL_SOURCE, "rb").read()).hexdigest()
    monkeypatch.setattr(bench, "TRAFFIC_SUMMARY", _summary_with_sha(tmp_path, src))
    text = open(bench.TRAFFIC_SUMMARY).read()
    rows = [l for l in text.splitlines() if l.startswith("| `k_")]
    assert rows, "the summary lists no kernel"
    kernel = rows[0].split("|")[1].strip().strip("`")
    cells = [c.strip() for c in rows[0].strip().strip("|").split("|")]
    kv = {l[2:].split(":", 1)[0].strip(): l.split(":", 1)[1].strip().strip("`")
          for l in text.splitlines() if l.startswith("- ") and ":" in l}
    want = (float(cells[2]) * float(kv["fetch factor"]) + float(cells[3]) * float(kv["write factor"])) * 1024.0
    got = bench.measured_traffic(kernel)
    assert got is not None and abs(got - want) <= 1e-6 * want
    assert bench.measured_traffic("k_not_a_kernel<1>") is None
    assert bench.measured_traffic(kernel, int(cells[1])) == got
    assert bench.measured_traffic(kernel, int(cells[1]) + 1) is None


def test_traffic_summary_ignored_after_source_change(tmp_path, monkeypatch):
    monkeypatch.setattr(bench, "TRAFFIC_SUMMARY", _summary_with_sha(tmp_path, "0" * 64))
    text = open(bench.TRAFFIC_SUMMARY).read()
    kernel = [l for l in text.splitlines() if l.startswith("| `k_")][0].split("|")[1].strip().strip("`")
    assert bench.measured_traffic(kernel) is None

