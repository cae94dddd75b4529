"""The operator profiler on the GPU: sparse profiles of a few 8B-layer
operators over a reduced (B, L) domain, their prediction error on held-out
points, and the memory / payload fields of the measured samples."""
import numpy as np
import pytest

from parity_util import say

pytestmark = pytest.mark.gpu


def test_sparse_profiles_predict_heldout_points():
    import torch
    assert torch.cuda.is_available()
    import paper_2608_13499_amd as ops
    from paper_2608_13499_amd import profiler as pr
    from paper_2608_13499_amd.layer import LayerShape
    ops.load()
    shape = LayerShape(4096, 32, 8, 128, 14336)
    sigs = dict(pr.layer_operators(shape))
    meas = pr.Measurer(warmup=2, iters=7, flush_mib=256)
    pooled = []
    for name in ("prefill.input_norm", "prefill.qkv_proj", "prefill.attention", "decode.attention"):
        sig = sigs[name]
        dom = (pr.Domain(1, 16, 16, 4096, 16384) if sig.phase == pr.PREFILL else pr.Domain(1, 128, 16, 4096, 128 * 4096))
        pts = pr.sample_points(dom, 10, seed=1)
        prof = pr.OpProfile(sig, [meas(sig, B, L) for B, L in pts])
        ho = [meas(sig, B, L) for B, L in pr.sample_points(dom, 6, seed=2, with_corners=False) if (B, L) not in pts]
        r = pr.evaluate(prof, ho)
        say(f"  {name}: {len(pts)} samples, {len(ho)} held out: mean error {100 * r['mean_rel_err']:.1f}%, "
            f"p90 {100 * r['p90_rel_err']:.1f}%")
        pooled += list(pr.relative_errors(prof.time_model(), [(h.B, h.L) for h in ho], [h.us_median for h in ho]))
        s = prof.samples[-1]
        T = s.B * s.L if sig.phase == pr.PREFILL else s.B
        if sig.kind == "linear":
            assert s.weight_bytes == sig.p("N") * sig.p("K") * 2
            assert s.io_bytes == T * sig.p("N") * 2
        if sig.kind == "add_rmsnorm":
            assert s.weight_bytes == 4096 * 2 and s.io_bytes == 2 * T * 4096 * 2
        assert all(x.us_median > 0 for x in prof.samples)
    pooled = np.asarray(pooled)
    say(f"  pooled over {pooled.size} held-out points: mean {100 * pooled.mean():.1f}%, "
        f"p90 {100 * np.quantile(pooled, 0.9):.1f}%")
    assert pooled.mean() < 0.3
