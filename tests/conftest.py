import json
import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

# Parity reports of the session (units compared, near-ties, largest relative
# score error), printed in the terminal summary and, when VD_PARITY_LOG names
# a file, appended to it as JSON lines.
_REPORTS = []


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU and the built HIP library")


@pytest.fixture(scope="session")
def orc():
    from oracle.vdref import load
    return load()


@pytest.fixture(scope="session")
def parity_log():
    """parity_log(case, report, **extra) records one comparison's counts."""
    def add(case, rep, **extra):
        rec = {"case": case, "units": int(rep.units), "near_ties": int(rep.near_ties),
               "max_rel_score_err": float(rep.max_score_err), **extra}
        _REPORTS.append(rec)
        path = os.environ.get("VD_PARITY_LOG")
        if path:
            with open(path, "a") as fh:
                fh.write(json.dumps(rec) + "\n")
    return add


def pytest_terminal_summary(terminalreporter):
    if not _REPORTS:
        return
    tot_u = sum(r["units"] for r in _REPORTS)
    tot_t = sum(r["near_ties"] for r in _REPORTS)
    terminalreporter.write_sep("-", f"parity: {len(_REPORTS)} comparisons, {tot_u} units, "
                                    f"{tot_t} near-tie units")
    for r in _REPORTS:
        extra = " ".join(f"{k}={v}" for k, v in r.items()
                         if k not in ("case", "units", "near_ties", "max_rel_score_err"))
        terminalreporter.write_line(f"{r['case']}: units={r['units']} near_ties={r['near_ties']} "
                                    f"max_rel_err={r['max_rel_score_err']:.1e} {extra}".rstrip())
