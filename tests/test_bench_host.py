"""Host-side pieces of bench.py (no GPU): the counter-derived HBM bytes are
read back from the committed profile only for the kernel and sources they
were taken with, and the per-shape kernel names are parsed from the
library's launch-table text."""

import bench


def test_traffic_read_back_for_current_sources():
    want = None
    with open(bench.TRAFFIC_PROFILE) as f:
        for line in f:
            if line.startswith("traffic:"):
                fields = dict(kv.split("=", 1) for kv in line.rstrip("\n").split("\t")[1:])
                want = fields
    assert want is not None
    got = bench.traffic_from_profile(want["kernel"])
    if want["kernel_source_sha256"] == bench.kernel_source_hash():
        assert got == int(want["hbm_bytes_per_launch"])
        assert 1.0 <= got / int(want["algorithmic_bytes_per_launch"]) < 1.2
    else:
        assert got is None                     # counters taken on other sources are not reported
    assert bench.traffic_from_profile("no_such_kernel<1>") is None


def test_kernel_names_from_launch_table():
    class FakeB:
        @staticmethod
        def qm_device_config():
            return ("arch=gfx950 cu=256 gemv_q4(3072->8192)=gemv_sub_kernel<1, 16, 8, false, 3> "
                    "gemv_q4(3072->128256)=gemv_kernel<1, 12, 8> gemm_tile(m=512,n=2048)=BM64 x 64")
    names = bench.gemv_kernel_names(FakeB)
    assert names == {"3072->8192": "gemv_sub_kernel<1, 16, 8, false, 3>",
                     "3072->128256": "gemv_kernel<1, 12, 8>"}
