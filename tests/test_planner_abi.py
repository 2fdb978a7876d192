"""The library's mesh planner (C ABI, host only) against the planner oracle.

Runs without a GPU: the planner calls enqueue nothing.
"""
import math
import random

import pytest

import paper_2301_08658_amd as atp
from oracle import planner as P

L, b, s, h = 24, 8, 2048, 4096
DIMS = dict(L=L, b=b, s=s, h=h)


def both(layers):
    """The same HCM for the library and for the oracle."""
    return atp.Hcm(layers), [P.Layer(r, g, p) for r, g, p in layers]


def same(x, y):
    if x is None:
        return y == 0.0
    if math.isinf(x) or math.isinf(y):
        return x == y
    return y == pytest.approx(x, rel=1e-12, abs=0.0)


def compare(layers):
    lib_h, orc_h = both(layers)
    dims = atp.model_dims(L, b, s, h)
    best, costs = atp.atp_plan_mesh(lib_h, dims)
    obest, ocosts = P.plan(orc_h, L, b, s, h)
    assert [(c["d1"], c["d2"]) for c in costs] == [(c["d1"], c["d2"]) for c in ocosts]
    for c, o in zip(costs, ocosts):
        for k in ("b1_eff", "b2_eff", "b1", "b2", "t_comm"):
            assert same(o[k], c[k]), (c["d1"], c["d2"], k, c[k], o[k])
        one = atp.atp_hcm_mesh_cost(lib_h, dims, c["d1"], c["d2"])
        assert one == c
    assert (best["d1"], best["d2"]) == obest


def test_paper_cluster_t7():
    p2p = [[0 if u == v else 200.0 for v in range(4)] for u in range(4)]
    lib_h, _ = both([(4, 25.0, None), (4, 600.0, p2p)])
    c = atp.atp_hcm_mesh_cost(lib_h, atp.model_dims(L, b, s, h), 8, 2)
    assert c["b1_eff"] == pytest.approx(12.5)
    assert c["b2_eff"] == pytest.approx(200.0)
    compare([(4, 25.0, None), (4, 600.0, p2p)])


def test_calibrated_t8():
    dims = atp.model_dims(L, b, s, h)
    t24 = atp.atp_tcomm(dims, 2, 4, 1.20, 4.95)
    t81 = atp.atp_tcomm(dims, 8, 1, 0.97, math.inf)
    assert t24 == pytest.approx(P.t_comm(L, b, s, h, 2, 4, 1.20, 4.95), rel=1e-14)
    assert 1 - t24 / t81 == pytest.approx(0.455, abs=5e-4)


@pytest.mark.parametrize("n", [1, 2, 4, 8, 16, 32, 64])
def test_switch_closed_form(n):
    G = 300.0
    lib_h, _ = both([(n, G, None)])
    dims = atp.model_dims(L, b, s, h)
    delta = 2.0 * L * b * s * h * 2 / (G * 1e9)
    best, costs = atp.atp_plan_mesh(lib_h, dims)
    for c in costs:
        d1, d2 = c["d1"], c["d2"]
        assert c["t_comm"] / delta == pytest.approx((14 * d2 + 4 * d1 - 18) / (d1 * d2))
    if n == 4:
        assert (best["d1"], best["d2"]) == (4, 1)
    if n == 16:
        assert (best["d1"], best["d2"]) == (8, 2)
    compare([(n, G, None)])


def test_mi355x_node_instance():
    # eight GPUs, one 153 GB/s xGMI link per pair: an axis group of k GPUs
    # gets (k - 1) links, so the direct all-reduce favours DeviceMesh(8, 1)
    hcm = atp.hcm_mi355x_xgmi()
    best, costs = atp.atp_plan_mesh(hcm, atp.model_dims(L, b, s, h))
    assert (best["d1"], best["d2"]) == (8, 1)
    by = {(c["d1"], c["d2"]): c for c in costs}
    assert by[(4, 2)]["b1_eff"] == pytest.approx(3 * 153.0)
    assert by[(4, 2)]["b2_eff"] == pytest.approx(153.0)
    assert by[(8, 1)]["b1_eff"] == pytest.approx(7 * 153.0)
    p2p = [[0.0 if u == v else 153.0 for v in range(8)] for u in range(8)]
    compare([(8, 7 * 153.0, p2p)])


@pytest.mark.parametrize("seed", range(40))
def test_random_hcm_matches_oracle(seed):
    rng = random.Random(1000 + seed)
    layers = []
    n_dev = 1
    for _ in range(rng.randint(1, 3)):
        r = rng.choice([1, 2, 2, 3, 4])
        if n_dev * r > 48:
            r = 1
        n_dev *= r
        g = rng.choice([10.0, 25.0, 50.0, 100.0, 600.0]) * rng.uniform(0.5, 2.0)
        if rng.random() < 0.3:
            p2p = None
        else:
            p2p = [[0.0 if u == v else (0.0 if rng.random() < 0.15 else rng.uniform(1, 300))
                    for v in range(r)] for u in range(r)]
        layers.append((r, g, p2p))
    compare(layers)


def test_tie_break_prefers_larger_d1():
    # two devices with no link: both meshes cost +inf; the larger d1 is kept
    lib_h, orc_h = both([(2, 10.0, [[0.0, 0.0], [0.0, 0.0]])])
    best, costs = atp.atp_plan_mesh(lib_h, atp.model_dims(L, b, s, h))
    assert [c["t_comm"] for c in costs] == [math.inf, math.inf]
    assert (best["d1"], best["d2"]) == (2, 1) == P.plan(orc_h, L, b, s, h)[0]
    # one device: the only mesh, no communication
    one, _ = both([(1, 10.0, None)])
    best, costs = atp.atp_plan_mesh(one, atp.model_dims(L, b, s, h))
    assert (best["d1"], best["d2"]) == (1, 1) and best["t_comm"] == 0.0 and len(costs) == 1


def status_of(fn):
    with pytest.raises(atp.AtpError) as ei:
        fn()
    return ei.value.status


def test_errors():
    dims = atp.model_dims(L, b, s, h)
    good, _ = both([(2, 10.0, None), (2, 20.0, None)])
    assert status_of(lambda: atp.atp_hcm_mesh_cost(good, dims, 3, 1)) == atp.ATP_ERR_SHAPE
    assert status_of(lambda: atp.atp_hcm_mesh_cost(good, dims, 0, 4)) == \
        atp.ATP_ERR_INVALID_ARGUMENT
    for bad in ([(0, 10.0, None)], [(2, 0.0, None)], [(2, float("nan"), None)],
                [(2, 10.0, [[0.0, -1.0], [1.0, 0.0]])],
                [(2, 10.0, [[0.0, float("inf")], [1.0, 0.0]])]):
        hb, _ = both(bad)
        assert status_of(lambda: atp.atp_plan_mesh(hb, dims)) == atp.ATP_ERR_INVALID_ARGUMENT
    big, _ = both([(256, 10.0, None), (512, 10.0, None)])
    assert status_of(lambda: atp.atp_plan_mesh(big, dims)) == atp.ATP_ERR_UNSUPPORTED
    assert status_of(lambda: atp.atp_plan_mesh(good, dims, max_costs=2)) == \
        atp.ATP_ERR_INVALID_ARGUMENT
    assert status_of(lambda: atp.atp_plan_mesh(good, atp.model_dims(0, b, s, h))) == \
        atp.ATP_ERR_INVALID_ARGUMENT
    assert status_of(lambda: atp.atp_tcomm(dims, 2, 2, 0.0, 1.0)) == atp.ATP_ERR_INVALID_ARGUMENT
    assert status_of(lambda: atp.atp_tcomm(dims, 2, 2, float("nan"), 1.0)) == \
        atp.ATP_ERR_INVALID_ARGUMENT
    too_many = atp.Hcm([(1, 1.0, None)] * 17)
    assert status_of(lambda: atp.atp_plan_mesh(too_many, dims)) == atp.ATP_ERR_INVALID_ARGUMENT
    assert "17" in atp.binding.last_error() or "n_layers" in atp.binding.last_error()
