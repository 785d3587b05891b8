"""Stored oracle digests (tests/golden/oracle_digests.json) for the GPU tests.

The digests were written by tests/golden/make_oracle_digests.py, which runs
only the oracle and the seeded input generators.  A test hashes its own output
the same way and compares; before that it checks that the stored entry was made
by the oracle sources as they are now and from the same inputs.
"""
import hashlib
import importlib.util
import json
import os

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
_SCRIPT = os.path.join(HERE, "golden", "make_oracle_digests.py")
_JSON = os.path.join(HERE, "golden", "oracle_digests.json")


def _script():
    spec = importlib.util.spec_from_file_location("make_oracle_digests", _SCRIPT)
    mod = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(mod)
    return mod


def sha256_of(a) -> str:
    a = np.ascontiguousarray(a, dtype=np.float32)
    return hashlib.sha256(a.astype("<f4", copy=False).tobytes()).hexdigest()


def entry(workload, inputs_used):
    """The stored digests of one workload, after checking that they belong to
    the current oracle sources and to these inputs (name -> host array)."""
    with open(_JSON) as fh:
        data = json.load(fh)
    assert workload in data, f"no stored digests for {workload}: run {_SCRIPT}"
    e = data[workload]
    assert e["oracle_sources_sha256"] == _script().oracle_source_sha256(), (
        f"the oracle sources changed since the {workload} digests were written: rerun {_SCRIPT}")
    for name, arr in inputs_used.items():
        assert e["inputs_sha256"][name] == sha256_of(arr), f"input {name} of {workload} differs"
    return e["outputs_sha256"]


def train_step_gradients(tokens, step_count=2):
    return _script().train_step_gradients(tokens, step_count)
