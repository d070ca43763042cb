"""The skip sets the paper reports (Table 1) as fixtures: the configuration
map's sparsity ratio R_d = |S| / L (Domain-to-Configuration Mapping)
reproduces the table's sparsity column, and the sets load into a per-domain
map with the dense fallback for other domains."""
import json
import os

import pytest

from paper_2609_26100_amd.controller import ConfigMap, DomainConfig

FIX = os.path.join(os.path.dirname(__file__), "golden", "paper_table1_skip_sets.json")
ROWS = json.load(open(FIX))["rows"]


@pytest.mark.parametrize("row", ROWS, ids=[f"{r['model']}-{r['domain']}" for r in ROWS])
def test_sparsity_ratio_matches_table(row):
    phi = ConfigMap(row["n_layers"])
    phi.set(row["domain"], DomainConfig(row["skip"]))
    assert round(100 * phi.domains[row["domain"]].ratio, 1) == row["sparsity_percent"]


def test_per_model_maps_with_fallback():
    for model in {r["model"] for r in ROWS}:
        rows = [r for r in ROWS if r["model"] == model]
        phi = ConfigMap(rows[0]["n_layers"], {r["domain"]: {"skip": r["skip"]} for r in rows})
        for r in rows:
            assert phi.skip_set(r["domain"]) == tuple(sorted(r["skip"]))
            assert int(phi.mask(r["domain"]).sum()) == len(r["skip"])
        assert phi.skip_set("Code") == ()
