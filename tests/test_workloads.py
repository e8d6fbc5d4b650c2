"""The synthetic workloads have the stated sizes and are seeded."""
import numpy as np
import pytest

import workloads


@pytest.mark.parametrize("name,count,numel", [
    ("c1", 1, 1048576), ("c2", 200, 123730176), ("c3", 254, 1543656960),
    ("c4", 290, 7504924672), ("c5", 1825, 7830919300)])
def test_sizes(name, count, numel):
    cfg = workloads.config(name)
    assert cfg.count == count and cfg.numel == numel


def test_c5_small_vectors():
    cfg = workloads.config("c5")
    assert sum(1 for s in cfg.specs if s.numel < 8192) == 1500


def test_inputs_seeded_and_settings():
    cfg = workloads.config("mini")
    a = workloads.make_inputs(cfg)
    b = workloads.make_inputs(cfg)
    for x, y in zip(a.theta + a.theta0 + a.grad_sim, b.theta + b.theta0 + b.grad_sim):
        assert x.equal(y)
    for spec, st in zip(cfg.specs, a.settings):
        assert (st.keep < 1.0) == (spec.kind == "linear")
        assert st.sigma > 0
    p0 = workloads.step_params(cfg, a.settings, 0)
    p1 = workloads.step_params(cfg, a.settings, 1)
    assert [p["s"] for p in p0] != [p["s"] for p in p1]
    assert all(0.3 <= p["s"] <= 1.0 for p in p0)


def test_c5_split_rule():
    cfg = workloads.config("c5")
    st = workloads.static_settings(cfg, [1e-4] * cfg.count)
    assert all(s.sigma == 0.0 and s.keep == np.float32(0.2) for s in st[0::2])
    assert all(s.keep == 1.0 and s.sigma > 0 for s in st[1::2])
