"""The plan-table tooling of the offline tuner (host only)."""
import os

from paper_1909_02765_amd import tune


def test_read_table_parses_the_shipped_table():
    table = tune.read_table()
    assert table, "the shipped plan table is empty"
    for key, (variant, splits) in table.items():
        assert len(key.split(",")) == 7
        assert variant and splits >= 1


def _entry(rows):
    return {"best": rows[0], "top": rows}


def test_choose_keeps_the_incumbent_within_the_margin():
    rows = [{"variant": "a", "splits": 1, "us": 10.0, "us_refined": 10.0},
            {"variant": "b", "splits": 2, "us": 10.1, "us_refined": 10.05}]
    assert tune.choose(_entry(rows), ("b", 2))["variant"] == "b"
    assert tune.choose(_entry(rows), None)["variant"] == "a"


def test_choose_replaces_a_slower_incumbent():
    rows = [{"variant": "a", "splits": 1, "us": 10.0, "us_refined": 10.0},
            {"variant": "b", "splits": 2, "us": 10.5, "us_refined": 10.5}]
    assert tune.choose(_entry(rows), ("b", 2))["variant"] == "a"
    # An incumbent that was not re-timed (not a finalist) never stays.
    rows[1].pop("us_refined")
    assert tune.choose(_entry(rows), ("b", 2))["variant"] == "a"


def test_emit_round_trips(tmp_path):
    path = os.path.join(tmp_path, "plans.inc")
    table = {"3,32,32,16,3,1,1": _entry([{"variant": "x", "path": 1, "splits": 1, "us": 4.0, "us_refined": 3.9}]),
             "64,56,56,64,3,1,1": _entry([{"variant": "y", "path": 1, "splits": 3, "us": 9.0}])}
    tune.emit(table, path)
    assert tune.read_table(path) == {"3,32,32,16,3,1,1": ("x", 1), "64,56,56,64,3,1,1": ("y", 3)}


def test_emit_merges_a_partial_sweep(tmp_path):
    """Shapes the sweep did not time keep their current line."""
    path = os.path.join(tmp_path, "plans.inc")
    tune.emit({"3,32,32,16,3,1,1": _entry([{"variant": "x", "path": 1, "splits": 1, "us": 4.0}]),
               "64,56,56,64,3,1,1": _entry([{"variant": "y", "path": 1, "splits": 3, "us": 9.0}])}, path)
    tune.emit({"64,56,56,64,3,1,1": _entry([{"variant": "z", "path": 1, "splits": 2, "us": 5.0,
                                            "us_refined": 5.0}])}, path)
    assert tune.read_table(path) == {"3,32,32,16,3,1,1": ("x", 1), "64,56,56,64,3,1,1": ("z", 2)}
