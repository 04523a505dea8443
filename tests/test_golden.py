"""Constants the paper prints, against the defaults of the oracle and the library.

The fixture ``tests/golden/paper_constants.json`` holds each value with its
citation. The paper prints no worked example of the path's arithmetic, so the
only printed values this repository uses are the scheduler's defaults.
"""
import json
import os

import paper_2512_04013_amd as aug
from oracle import former as of

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "paper_constants.json")


def _golden():
    with open(GOLDEN) as f:
        return json.load(f)


def test_every_golden_value_carries_a_citation():
    g = _golden()
    for name, entry in g.items():
        if name == "about":
            continue
        assert entry.get("cite"), name
        assert "value" in entry, name


def test_oracle_default_aging_factor_is_the_papers():
    g = _golden()
    assert of.Params().beta == g["beta_default"]["value"]
    assert g["beta_default"]["value"] in g["beta_sensitivity_grid"]["value"]


def test_library_default_aging_factor_is_the_papers():
    assert aug.former_params().beta == _golden()["beta_default"]["value"]
