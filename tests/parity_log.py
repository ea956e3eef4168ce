"""Error log of the GPU parity tests.

Every comparison the GPU tests make against the oracle (relative Frobenius
errors per output, sampled entries, identity residuals) is recorded here with
its tolerance; at the end of the session conftest.py writes the records as
JSON lines to the file named by the environment variable GPPS_PARITY_LOG (when
it is set), so that the margins survive a quiet test run.
``tests/parity_summary.py`` turns such a file into a table.
"""
import json
import os

_RECORDS = []


def record(test, label, what, err, tol):
    _RECORDS.append({"test": test, "label": label, "what": what, "err": float(err),
                     "tol": None if tol is None else float(tol)})


def current_test():
    return os.environ.get("PYTEST_CURRENT_TEST", "").split(" ")[0]


def dump():
    path = os.environ.get("GPPS_PARITY_LOG")
    if not path or not _RECORDS:
        return
    os.makedirs(os.path.dirname(os.path.abspath(path)), exist_ok=True)
    with open(path, "a") as f:
        for r in _RECORDS:
            f.write(json.dumps(r) + "\n")
    _RECORDS.clear()
