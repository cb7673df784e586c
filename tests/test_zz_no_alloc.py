"""gefen_dp_codebook_static (the DP with the library's fixed per-GPU workspace, for
callers that cannot allocate) against gefen_dp_codebook, through the C ABI: two calls in
a row, the second smaller, each equal bit for bit to the allocating entry point on the
same histogram (codebook, cost and status), and to the oracle's DP; then a degenerate
histogram, and the size checks."""
import numpy as np
import pytest
import torch

import oracle

pytestmark = pytest.mark.gpu

gf = pytest.importorskip("paper_2606_13894_amd")


def _dev():
    if not torch.cuda.is_available():
        pytest.skip("no HIP device")
    return torch.device("cuda", 0)


def _hist(nbins, seed, heavy=False):
    rng = np.random.default_rng(seed)
    g = (rng.standard_t(3, 200_000) if heavy else rng.standard_normal(200_000)).astype(np.float32)
    return oracle.histogram_uniform(g, 500, nbins)


def _both(h, k, dev):
    ht = torch.from_numpy(h.view(np.int64).copy()).to(dev)
    cb_a, cost_a, st_a = gf.dp_codebook(ht, k)
    cb_s, cost_s, st_s = gf.dp_codebook_static(ht, k)
    torch.cuda.synchronize()
    return (cb_a.cpu().numpy(), cost_a, st_a), (cb_s.cpu().numpy(), cost_s.item(), st_s.item())


def test_static_dp_matches_the_allocating_dp_twice_then_smaller():
    dev = _dev()
    for nbins, k, seed in ((4096, 256, 1), (256, 16, 2)):
        h = _hist(nbins, seed, heavy=(k == 256))
        (cb_a, cost_a, st_a), (cb_s, cost_s, st_s) = _both(h, k, dev)
        np.testing.assert_array_equal(cb_s, cb_a)
        assert cost_s == cost_a and st_s == st_a == 0
        cb_ref, cost_ref, _, st_ref = oracle.dp_codebook(h, k)
        np.testing.assert_array_equal(cb_s, cb_ref)
        assert cost_s == cost_ref and st_ref == 0


def test_static_dp_degenerate_and_sizes():
    dev = _dev()
    h = np.zeros(4096, dtype=np.uint64)
    h[[0, 17, 2000, 4095]] = [5, 3, 9, 1]          # 4 non-empty bins, k = 256
    (cb_a, cost_a, st_a), (cb_s, cost_s, st_s) = _both(h, 256, dev)
    np.testing.assert_array_equal(cb_s, cb_a)
    assert cost_s == cost_a and st_s == st_a == 1
    ht = torch.zeros(4097, dtype=torch.int64, device=dev)
    with pytest.raises(gf.GefenError, match="EINVAL"):
        gf.dp_codebook_static(ht, 256)             # more bins than the largest DP
    with pytest.raises(gf.GefenError, match="EINVAL"):
        gf.dp_codebook_static(ht[:4096], 257)      # more entries than the largest DP
