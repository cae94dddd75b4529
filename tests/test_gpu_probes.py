"""The peak probes on the GPU: the measured bf16 MFMA rate and HBM streaming
rates are positive and at most the published peaks (2.5 PFLOP/s, 8 TB/s)
with a margin, and the MFMA rate is a sizeable part of the peak (the probe
keeps every SIMD busy)."""
import pytest

from parity_util import say

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def ops():
    import torch
    assert torch.cuda.is_available()
    import paper_2608_13499_amd as P
    P.load()
    return P


def test_probe_mfma(ops):
    say("probe: bf16 MFMA")
    tf = ops.opscale_probe_mfma(iters=2048, reps=3)
    say(f"  {tf:.1f} TFLOP/s")
    assert 300.0 < tf < 2600.0


def test_probe_hbm(ops):
    import torch
    say("probe: HBM read and copy, 1 GiB")
    src = torch.ones(1 << 29, dtype=torch.int16, device="cuda")
    dst = torch.empty_like(src)
    rd = ops.opscale_probe_hbm(src, reps=3)
    cp = ops.opscale_probe_hbm(src, dst, reps=3)
    torch.cuda.synchronize()
    say(f"  read {rd:.0f} GB/s, copy {cp:.0f} GB/s")
    assert 1000.0 < rd < 8500.0 and 1000.0 < cp < 8500.0
    assert torch.equal(dst, src)  # the copy probe copies


@pytest.mark.parametrize("nvec", [1, 5, 196608 * 2 + 12345, 196608 * 5 + 1])
def test_probe_copy_ragged(ops, nvec):
    """Copies of 16-byte vectors that end inside a grid stride: every vector,
    the last included, lands once (196608 = lanes of the 768-workgroup grid)."""
    import torch
    say(f"probe: copy of {nvec} x 16 B")
    g = torch.Generator().manual_seed(nvec)
    src = torch.randint(-30000, 30000, (nvec * 8,), dtype=torch.int16, generator=g).cuda()
    dst = torch.zeros_like(src)
    ops.opscale_probe_hbm(src, dst, reps=1)
    torch.cuda.synchronize()
    assert torch.equal(dst, src)


def test_probe_rejects(ops):
    import torch
    with pytest.raises(ops.OpscaleError):
        ops.opscale_probe_mfma(iters=0)
    src = torch.ones(1024, dtype=torch.int16, device="cuda")
    with pytest.raises(ops.OpscaleError):
        ops.opscale_probe_hbm(src, torch.empty(8, dtype=torch.int16, device="cuda"))
    buf = torch.zeros(2048, dtype=torch.int16, device="cuda")
    with pytest.raises(ops.OpscaleError):  # the copy's source and destination overlap
        ops.opscale_probe_hbm(buf[:1024], buf[512:1536])
