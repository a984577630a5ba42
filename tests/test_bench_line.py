"""The JSON line bench.py prints keeps its field contract (host only)."""
import copy
import os
import sys

import pytest

sys.path.insert(0, os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
import bench  # noqa: E402

GOOD = {"metric": "actions/s", "value": 281.0, "unit": "actions/s", "n_gpus": 1, "steps": 5, "warmup": 2,
        "ms_per_step": 227.8, "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "bf16",
        "data": "synthetic", "config": {"workload": "w"},
        "roofline": {"bound": "mfma", "achieved": 1350.0, "peak": 2500.0, "unit": "TFLOP/s", "frac": 0.54,
                     "traffic": None},
        "cpu_baseline": {"value": 0.027, "unit": "actions/s", "cores": 16, "kind": "oracle", "sample": "s"},
        "value_model": {"ms": 192.0}}


def test_good_line_passes():
    assert bench.check_line(copy.deepcopy(GOOD)) == GOOD


@pytest.mark.parametrize("path,bad", [(("value",), {"ms": 1.0}), (("value",), None), (("steps",), 5.0),
                                      (("higher_is_better",), 1), (("roofline", "frac"), None),
                                      (("cpu_baseline", "value"), "x"), (("config",), {})])
def test_malformed_line_is_rejected(path, bad):
    r = copy.deepcopy(GOOD)
    d = r
    for k in path[:-1]:
        d = d[k]
    d[path[-1]] = bad
    with pytest.raises(ValueError):
        bench.check_line(r)
