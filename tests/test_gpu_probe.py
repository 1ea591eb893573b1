"""The measurement probes of libfqprobe.so on the GPU: the streaming read runs
and the XCD-placement probe reports valid XCD numbers."""

import pytest
import torch

pytestmark = pytest.mark.gpu


def test_stream_read_runs(gpu_lib):
    from paper_2608_15531_amd import probe
    buf = torch.ones(1 << 20, dtype=torch.int32, device="cuda")
    sink = torch.zeros(512, dtype=torch.int32, device="cuda")
    probe.fq_probe_stream_read(buf, buf.numel() * 4, 512, 4, 4, sink)
    torch.cuda.synchronize()


@pytest.mark.parametrize("workgroups,threads", [(8, 64), (512, 256), (4096, 1024)])
def test_workgroup_xcd_in_range(gpu_lib, workgroups, threads):
    """Every workgroup writes its XCD number, one of the eight of MI355X."""
    from paper_2608_15531_amd import probe
    out = torch.full((workgroups,), -1, dtype=torch.int32, device="cuda")
    probe.fq_probe_workgroup_xcd(out, workgroups, threads)
    torch.cuda.synchronize()
    ids = out.cpu()
    assert int(ids.min()) >= 0 and int(ids.max()) < 8
