"""The seeded instance generator is deterministic and its fixtures are current."""
import pytest

from workloads import CONFIG_NAMES, dumps, fixture_path, make_instance, random_tiny


@pytest.mark.parametrize("name", CONFIG_NAMES)
def test_fixture_regenerates_byte_equal(name):
    with open(fixture_path(name)) as fh:
        assert fh.read() == dumps(make_instance(name)) + "\n"


@pytest.mark.parametrize("name", CONFIG_NAMES)
def test_instance_shape(name):
    inst = make_instance(name)
    L = len(inst["layers"]["fwd_flops"])
    K = len(inst["islands"]["n_gpus"])
    assert all(len(v) == L for v in inst["layers"].values())
    assert all(isinstance(x, int) and x >= 0 for v in inst["layers"].values() for x in v)
    assert all(sum(v) < 2 ** 62 for v in inst["layers"].values())
    assert sorted(inst["island_order"]) == list(range(K))
    assert len(inst["inter_bw"]) == K and all(len(r) == K for r in inst["inter_bw"])
    assert {8 * (n // 8) for n in inst["islands"]["n_gpus"]} <= set(inst["islands"]["n_gpus"]) \
        or name == "tiny"


def test_shapes_named_by_the_workloads():
    assert (len(make_instance("large")["islands"]["n_gpus"]),
            len(make_instance("large")["layers"]["fwd_flops"])) == (128, 128)
    assert len(make_instance("moe")["islands"]["n_gpus"]) == 32
    assert len(make_instance("dense70b")["islands"]["n_gpus"]) == 16
    fabric = {x for row in make_instance("large")["inter_bw"] for x in row}
    assert fabric == {0.0, 25e9, 100e9, 400e9}


def test_random_tiny_deterministic():
    assert dumps(random_tiny(5)) == dumps(random_tiny(5))
    assert dumps(random_tiny(5)) != dumps(random_tiny(6))
