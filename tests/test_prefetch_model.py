"""Eq. 6 (Section 5.3), tl_prefetch_degree, on the CPU: the degree it returns
keeps bandwidth x latency bytes in flight -- p (d + 1) > B L with d the
smallest such degree -- unless the K-iteration cap binds; the collision
factor scales the demand; arguments are validated."""
import math

import numpy as np
import pytest

import paper_2607_04031_amd as tl


def test_saturates_and_is_minimal():
    rng = np.random.default_rng(6)
    for _ in range(2000):
        B = float(rng.uniform(1e9, 1e13))          # bytes/s
        L = float(rng.uniform(0.0, 2e-5))          # s
        p = float(rng.uniform(1e4, 1e8))           # bytes per K iteration of all resident workgroups
        d = tl.tl_prefetch_degree(B, L, p, 1 << 40)
        assert p * (d + 1) > B * L * (1 - 1e-12)   # enough requests in flight
        assert d == 0 or p * d <= B * L * (1 + 1e-12)   # and no more than needed


def test_cap_is_the_k_iterations():
    assert tl.tl_prefetch_degree(1e12, 1e-5, 1e5, 7) == 7          # B L / p = 100, capped at 7
    assert tl.tl_prefetch_degree(1e12, 1e-5, 1e5, 1000) == 100


def test_collision_factor_and_hand_values():
    # 8 TB/s x 5 us = 40 MB in flight; 1024 workgroups x 16 KB per K iteration = 16 MiB
    p = 1024 * 16384
    assert tl.tl_prefetch_degree(8e12, 5e-6, p, 1 << 20) == math.floor(40e6 / p) == 2
    assert tl.tl_prefetch_degree(8e12, 5e-6, p, 1 << 20, 2.0) == math.floor(80e6 / p) == 4
    assert tl.tl_prefetch_degree(8e12, 0.0, p, 1 << 20) == 0        # no latency, no prefetch


@pytest.mark.parametrize("args", [(0.0, 1e-6, 1.0, 4, 1.0), (1e9, -1e-6, 1.0, 4, 1.0), (1e9, 1e-6, 0.0, 4, 1.0),
                                  (1e9, 1e-6, 1.0, -1, 1.0), (1e9, 1e-6, 1.0, 4, 0.0)])
def test_errors(args):
    with pytest.raises(tl.TLError) as e:
        tl.tl_prefetch_degree(*args)
    assert e.value.status == tl.TL_EINVAL


def test_lgms_argument_errors():
    d = tl.layout()
    for kw, status in ((dict(steps=3), tl.TL_EINVAL), (dict(lat=-1), tl.TL_EINVAL),
                       (dict(M=17), tl.TL_EUNSUPPORTED), (dict(layout=tl.layout(kind=tl.TL_LAYOUT_NK_ROW)), tl.TL_EUNSUPPORTED),
                       (dict(layout=tl.layout(G=16384, block_rows=64)), tl.TL_EUNSUPPORTED)):
        a = dict(M=8, steps=2, lat=1000, layout=d)
        a.update(kw)
        with pytest.raises(tl.TLError) as e:
            tl.tl_gemm_lgms(4096, 8192, 1 << 20, a["M"], 512, 1024, a["layout"], a["lat"], a["steps"], stream=0)
        assert e.value.status == status, kw
