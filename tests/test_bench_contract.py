"""The one-line JSON contract of bench.py, checked without a GPU: the result dictionary has
unique keys (a second "steps" would silently replace the step count), carries every required
field, and a request for more than one GPU exits at once with a message."""
import ast
import json
import os
import subprocess
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
REQUIRED = {"metric", "value", "unit", "n_gpus", "steps", "warmup", "ms_per_step", "higher_is_better",
            "scaling", "vs_baseline", "dtype", "data", "config", "roofline"}


def _result_dict():
    tree = ast.parse(open(os.path.join(ROOT, "bench.py")).read())
    for node in ast.walk(tree):
        if isinstance(node, ast.Assign) and any(isinstance(t, ast.Name) and t.id == "result" for t in node.targets):
            if isinstance(node.value, ast.Dict):
                return node.value
    raise AssertionError("no `result = {...}` in bench.py")


def test_result_keys_unique_and_complete():
    d = _result_dict()
    keys = [k.value for k in d.keys if isinstance(k, ast.Constant)]
    dup = {k for k in keys if keys.count(k) > 1}
    assert not dup, f"duplicate keys in the bench result: {dup}"
    assert REQUIRED <= set(keys), REQUIRED - set(keys)
    # the step count is the integer argument, the roofline object names its four fields
    steps = d.values[keys.index("steps")]
    assert isinstance(steps, ast.Attribute) and steps.attr == "steps"
    roof = d.values[keys.index("roofline")]
    rkeys = {k.value for k in roof.keys}
    assert {"bound", "achieved", "peak", "unit", "frac", "traffic"} <= rkeys


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, timeout=120, cwd=ROOT)
    assert r.returncode == 2
    msg = json.loads(r.stdout.strip().splitlines()[-1])
    assert "one GPU" in msg["error"]
