"""The stored expected results are the oracle's: recomputing the small
instances' records with the committed oracle gives the committed files
(timings aside)."""
import pytest

from tests.golden import make_golden


@pytest.mark.parametrize("name", ["tiny", "dense8b"])
def test_stored_results_are_the_oracles(name):
    stored = make_golden.load(name)
    fresh = make_golden.golden(name)
    stored.pop("oracle_seconds")
    fresh.pop("oracle_seconds")
    import json
    assert json.loads(json.dumps(fresh, sort_keys=True)) == stored
