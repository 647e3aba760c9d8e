"""Host logic of the profile summaries that bench.py reads (CPU only): the
traffic figure of a kernel comes from its traffic summary, never from a
counter summary of the same kernel and workload, and only while the kernel
sources are the ones the counters were taken on."""
import os

from paper_2605_19150_amd.profiling import read_traffic_summary, source_hash

W = "fsa-perm B16 L2048 H16 N64 K16"


def _write(d, name, kernel, workload, hash_, traffic=None):
    lines = ["# summary", "", "kernel: %s" % kernel, "workload: %s" % workload, "source-hash: %s" % hash_]
    if traffic is not None:
        lines.append("traffic-bytes-per-launch: %d" % traffic)
    with open(os.path.join(d, name), "w") as fh:
        fh.write("\n".join(lines) + "\n")


def test_traffic_ignores_counter_summaries(tmp_path):
    h = source_hash("k_bwd_fused")
    # sorts before the traffic summary and names the same kernel and workload
    _write(tmp_path, "k_bwd_fused_a_counters.md", "k_bwd_fused", W, h)
    _write(tmp_path, "k_bwd_fused_b_traffic.md", "k_bwd_fused", W, h, traffic=1650193603)
    assert read_traffic_summary(str(tmp_path), "k_bwd_fused", W) == 1650193603.0


def test_traffic_stale_sources_and_missing(tmp_path):
    _write(tmp_path, "k_bwd_fused_traffic.md", "k_bwd_fused", W, "0" * 16, traffic=5)
    assert read_traffic_summary(str(tmp_path), "k_bwd_fused", W) is None   # other sources
    assert read_traffic_summary(str(tmp_path), "k_fwd_fused", W) is None   # no summary
    assert read_traffic_summary(str(tmp_path), "k_bwd_fused", "other") is None


def test_committed_summaries_parse():
    """Every committed traffic summary gives a positive figure or None."""
    root = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "profiles")
    for name in sorted(os.listdir(root)):
        if not name.endswith("_traffic.md"):
            continue
        kv = {}
        with open(os.path.join(root, name)) as fh:
            for line in fh:
                if ": " in line and not line.startswith(("#", " ", "|")):
                    k, v = line.rstrip("\n").split(": ", 1)
                    kv[k] = v
        got = read_traffic_summary(root, kv["kernel"], kv["workload"])
        assert got is None or got > 0, name
