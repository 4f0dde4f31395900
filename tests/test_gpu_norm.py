"""Normalize of Algorithm 1 on the device (mgn_norm_accumulate /
mgn_norm_apply) against the oracle: running statistics (fp64, summed in a
fixed order, so only the order of additions differs from the oracle's) and
the standardised rows (fp32, one rounding of the fp64 value)."""
import numpy as np
import pytest
import torch

import oracle
import paper_2307_13592_amd as mgn
from paper_2307_13592_amd.runner import Normalizer

pytestmark = pytest.mark.gpu


def _rows(seed, rows, cols):
    r = np.random.default_rng([seed, rows, cols])
    scale = np.linspace(0.01, 50.0, cols)
    return (r.normal(0.0, 1.0, (rows, cols)) * scale + np.linspace(-3.0, 7.0, cols)).astype(np.float32)


@pytest.mark.parametrize("cols", [1, 4, 11, 64])
@pytest.mark.parametrize("splits", [(0,), (1,), (1000, 0, 37), (4097, 3_000_001)])
def test_norm_against_oracle(cols, splits):
    print(f"[norm] cols={cols} splits={splits}", flush=True)
    nz = Normalizer(cols, "cuda:0")
    st = np.zeros(1 + 2 * cols)
    parts = [_rows(k, n, cols) for k, n in enumerate(splits)]
    for x in parts:
        nz.accumulate(torch.as_tensor(x).cuda())
        st = oracle.norm_accumulate(st, x)
    got = nz.stats.cpu().numpy()
    assert got[0] == st[0]
    assert np.allclose(got[1:], st[1:], rtol=1e-10, atol=1e-12 * max(1.0, float(np.abs(st[1:]).max())))
    x = parts[-1] if len(parts[-1]) else _rows(99, 300, cols)
    ref = oracle.norm_apply(st, x, eps=1e-8)
    xt = torch.as_tensor(x).cuda()
    out = nz.apply(xt).cpu().numpy().astype(np.float64)
    err = np.abs(out - ref)
    assert np.all(err <= 2.0 ** -23 * np.abs(ref) + 1e-9), float((err / (np.abs(ref) + 1e-30)).max())
    mgn.mgn_norm_apply(xt, nz.stats, xt)  # in place
    assert np.array_equal(xt.cpu().numpy().astype(np.float64), out)


def test_norm_reproducible_and_degenerate():
    """The same rows give the same statistics bits; a constant column keeps
    deviation eps (output 0); with no rows accumulated apply is the identity."""
    x = _rows(5, 200_003, 11)
    x[:, 4] = 2.5
    a, b = Normalizer(11, "cuda:0"), Normalizer(11, "cuda:0", eps=1e-3)
    for nz in (a, b):
        nz.accumulate(torch.as_tensor(x).cuda())
    assert torch.equal(a.stats, b.stats)
    y = b.apply(torch.as_tensor(x).cuda()).cpu().numpy()
    assert np.all(y[:, 4] == 0.0)
    fresh = Normalizer(11, "cuda:0")
    xt = torch.as_tensor(x[:100]).cuda()
    assert torch.equal(fresh.apply(xt), xt)
