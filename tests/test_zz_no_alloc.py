"""The allocation-free entry point dlmc_entropy_cdf_noalloc against the
allocating dlmc_entropy_cdf, through the C ABI: bit-identical entropies, row
maxima, g values and integer CDFs on two calls in a row (the second smaller,
so stale scratch contents from the first must not leak into it), and a clear
error beyond the static scratch."""
import numpy as np
import pytest

import workloads as wl
from oracle import cdf as OC
from oracle import schedule as OS

from gpu_common import log, shape

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

import paper_2608_11249_amd as dl  # noqa: E402


@pytest.mark.parametrize("V,P", [(126464, 24), (1001, 16)])
def test_noalloc_matches_allocating_entry_point(V, P):
    sh = shape(vocab=V, n_layers=0)
    with dl.Model(sh, max_chunk=8) as m, dl.Model(sh, max_chunk=8) as m2:
        for rows, seed in ((48, 1), (5, 2)):            # second call smaller
            log("no-alloc entropy/cdf", V, rows)
            lg = wl.random_logits(seed, rows, V, 7.0)
            lg[1] = 0.0                                   # uniform row
            dlg = torch.from_numpy(lg).cuda()
            ref = m.entropy_cdf(dlg, P)
            got = m.entropy_cdf_noalloc(dlg, P)
            for a, b in zip(ref, got):
                assert torch.equal(a, b)
            # another handle on the same GPU shares the scratch, one call at a time
            got2 = m2.entropy_cdf_noalloc(dlg, P)
            for a, b in zip(ref, got2):
                assert torch.equal(a, b)
            H = got[0].cpu().numpy()
            cdf = got[3].cpu().numpy().view(np.uint32).astype(np.int64)
            g = got[2].cpu().numpy().view(np.uint32).astype(np.int64)
            assert np.max(np.abs(H - OS.entropy_bits(lg.astype(np.float64)))) <= 1e-3
            for i in (0, 1, rows - 1):
                assert np.array_equal(cdf[i], OC.integer_cdf(g[i], P))
        H, mx, g, cdf = m.entropy_cdf_noalloc(dlg, P, want_cdf=False)
        assert torch.equal(H, ref[0]) and torch.equal(mx, ref[1])


def test_noalloc_rejects_requests_beyond_the_scratch():
    V = 126464
    per_row = 8 + 20 * -(-V // 4096)
    rows = (4 << 20) // per_row + 1
    with dl.Model(shape(vocab=V, n_layers=0), max_chunk=8) as m:
        lg = torch.zeros((rows, V), dtype=torch.float32, device="cuda")
        with pytest.raises(dl.DlmcError) as e:
            m.entropy_cdf_noalloc(lg, 24)
        assert e.value.code == -1 and "scratch" in str(e.value)
        H, mx, _, _ = m.entropy_cdf_noalloc(lg, 24, want_cdf=False)   # no CDF: no scratch
        assert torch.all(torch.isclose(H, torch.full_like(H, float(np.log2(V)))))
