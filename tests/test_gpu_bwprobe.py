"""The bandwidth probe reads its whole buffer: its figure is a plausible HBM
read rate (between 1 TB/s and the 8 TB/s of the spec sheet plus a margin
for timer resolution), and a buffer twice as large takes about twice as
long."""
import pytest
import torch

pytestmark = pytest.mark.gpu


def test_probe_reads_the_whole_buffer(gpu_lib):
    from paper_2502_15572_amd import bw_probe
    a = torch.ones((2 << 30) // 4, dtype=torch.float32, device="cuda:0")
    b = torch.ones((4 << 30) // 4, dtype=torch.float32, device="cuda:0")
    ga = bw_probe(a, reps=5)
    gb = bw_probe(b, reps=5)
    print("probe: 2 GiB %.0f GB/s, 4 GiB %.0f GB/s" % (ga, gb), flush=True)
    for g in (ga, gb):
        assert 1000.0 < g < 8800.0
    ta, tb = (2 << 30) / ga, (4 << 30) / gb
    assert 1.6 < tb / ta < 2.4
