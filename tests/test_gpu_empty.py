"""An empty batch (B = 0 positions) through every call of the Python binding and
the C ABI: nothing is launched and every output is empty.  Notation: p =
target, q = draft."""
import pytest
import torch

import paper_2410_18234_amd as mdss

pytestmark = pytest.mark.gpu
DEV = torch.device("cuda:0")
V = 1000


def _e(*shape, dtype=torch.float32):
    return torch.empty(shape, dtype=dtype, device=DEV)


def _all_empty(out):
    items = out.values() if isinstance(out, dict) else (out if isinstance(out, tuple) else (out,))
    for t in items:
        assert t is None or t.numel() == 0, t.shape


def test_empty_batch_every_call():
    p, q, q2 = _e(0, V), _e(0, V), _e(0, V)
    d2, d3 = _e(0, 2, dtype=torch.int32), _e(0, 3, dtype=torch.int32)
    u = _e(0, 3)
    _all_empty(mdss.induced_dist(p, q, 2))
    _all_empty(mdss.induced_dist(p, q, 3, s_max=64))
    _all_empty(mdss.select_intermediate(p, q, d2, u))
    _all_empty(mdss.accept_or_resample(p, q, _e(0, dtype=torch.int32), u, want_residual=True, want_mass=True))
    _all_empty(mdss.step(p, q, d2, u, want_residual=True))
    _all_empty(mdss.step(p, q, d3, None, s_max=64))
    _all_empty(mdss.induced_dist_pair(p, q, q2))
    _all_empty(mdss.step_pair(p, q, q2, d2, u, want_residual=True))
    for tail in (mdss.MDSS_TLP_SORTED, mdss.MDSS_TLP_HALF):
        _all_empty(mdss.truncated_lp(p, q, q2, 5, tail))
        _all_empty(mdss.step_truncated_lp(p, q, None, d2, s=5, tail=tail, u=u, want_residual=True))
    rs = mdss.induced_dist_successive(p, q, 4)
    assert rs.shape == (3, 0, V)
    _all_empty(mdss.select_successive(p, q, rs, _e(0, 4, dtype=torch.int32), _e(0, 3)))
    _all_empty(mdss.step_successive(p, q, d3, _e(0, 2), u, want_residual=True))
    _all_empty(mdss.optimal_acceptance(p, q, 3))
    _all_empty(mdss.acceptance(p, q))
    pt, mass = mdss.truncate_alphabet(p, 40)
    _all_empty((pt, mass))
    _all_empty(mdss.alphabet_post(p, pt, mass, _e(0, dtype=torch.int32), _e(0, 2)))
    _all_empty(mdss.step_alphabet(p, q, d2, 40, u=u))
    torch.cuda.synchronize()
    # parameters are still checked on an empty batch
    with pytest.raises(mdss.MdssError):
        mdss.induced_dist(p, q, 4)
    with pytest.raises(mdss.MdssError):
        mdss.truncated_lp(p, q, None, 17)
