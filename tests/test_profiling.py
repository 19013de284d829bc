"""Host logic of the profile summaries: the traffic figure bench.py reports
is read back only for the kernel and the sources that were profiled."""
import os

from paper_2606_04238_amd import profiling


def _write(path, kernel, digest, traffic="1234"):
    with open(path, "w") as fh:
        fh.write("# x\n\n| a | b |\n\ntraffic_bytes_per_launch: %s\nkernel: %s\nsource_digest: %s\n"
                 % (traffic, kernel, digest))


def test_read_traffic_matches_digest_and_kernel(tmp_path):
    p = os.path.join(tmp_path, "k.md")
    _write(p, "fused_layer_kernel", profiling.source_digest())
    assert profiling.read_traffic(p, "fused_layer_kernel") == 1234.0
    assert profiling.read_traffic(p, "down_w4_kernel") is None


def test_read_traffic_stale_sources(tmp_path):
    p = os.path.join(tmp_path, "k.md")
    _write(p, "fused_layer_kernel", "0" * 16)
    assert profiling.read_traffic(p, "fused_layer_kernel") is None
    assert profiling.read_traffic(os.path.join(tmp_path, "missing.md"), "fused_layer_kernel") is None


def test_digest_is_stable():
    assert profiling.source_digest() == profiling.source_digest()
    assert len(profiling.source_digest()) == 16
