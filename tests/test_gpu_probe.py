"""The HBM streaming probe's kernels move the bytes they are timed for: the
copy writes a to b, the in-place mix adds a to b once per launch (one
untimed, seven timed), the row sum writes each element's sum over the rows."""
import pytest
import torch

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("k,lds", [(1, 0), (2, 40960), (4, 65536)])
def test_stream_kernels_results(dev, k, lds):
    from paper_2102_02888_amd import hbm_probe
    n = 1 << 20
    s = torch.cuda.current_stream(dev)
    a = torch.arange(n, dtype=torch.float32, device=dev) % 97
    b = torch.full((n,), 3.0, dtype=torch.float32, device=dev)
    sink = torch.zeros(1, dtype=torch.float32, device=dev)
    ms, gbps = hbm_probe.stream_case("read", k, lds, a, None, sink, s)
    assert ms > 0 and gbps > 0
    torch.cuda.synchronize()
    assert sink.item() == 0.0
    hbm_probe.stream_case("copy", k, lds, a, b, sink, s)
    torch.cuda.synchronize()
    assert torch.equal(b, a)
    b0 = torch.full((n,), 3.0, dtype=torch.float32, device=dev)
    b.copy_(b0)
    hbm_probe.stream_case("mix", k, lds, a, b, sink, s)
    torch.cuda.synchronize()
    assert torch.equal(b, b0 + 8 * a)  # small integers: exact in fp32


@pytest.mark.parametrize("w,bb", [(16, 1), (16, 2), (8, 1), (4, 1)])
def test_rowsum_kernel_results(dev, w, bb):
    from paper_2102_02888_amd import hbm_probe
    R, D = 6, 1024 * 37  # 37 tiles: the last workgroup has spare waves
    s = torch.cuda.current_stream(dev)
    g = (torch.arange(R * D, dtype=torch.float32, device=dev) % 13).view(R, D)
    out = torch.zeros(D, dtype=torch.float32, device=dev)
    ms, gbps = hbm_probe.rowsum_case(w, bb, g, D, R, out, s)
    torch.cuda.synchronize()
    assert ms > 0 and torch.equal(out, g.sum(0))
