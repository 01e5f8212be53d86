import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line(
        "markers", "gpu: needs an MI355X (gfx950) GPU; runs the HIP path")


def pytest_collection_modifyitems(config, items):
    # GPU tests fail loudly on a machine without a GPU rather than skipping,
    # unless they were deselected with -m "not gpu".
    pass


def pytest_terminal_summary(terminalreporter):
    """Parity summary of the GPU tests: per compared output, the normwise
    error and the arg-max near-tie exemptions (a flipped arg-max whose
    oracle top-2 gap is within twice the frame's max abs error)."""
    try:
        from harness import PARITY
    except ImportError:
        return
    if not PARITY:
        return
    tr = terminalreporter
    tr.write_sep("-", "parity against the oracle")
    ties = sum(r["near_ties"] for r in PARITY)
    vecs = sum(r["vectors"] for r in PARITY)
    bad = sum(r["mismatches"] for r in PARITY)
    untagged = [r for r in PARITY if not r["tag"]]
    if untagged:
        tr.write_line(f"layer-level outputs (untagged): {len(untagged)}, worst "
                      f"normwise {max(r['normwise'] for r in untagged):.3e}")
    for r in PARITY:
        if not r["tag"]:
            continue
        tr.write_line(
            f"{r['tag']:>22s} model {r['model']} output {r['output']}: "
            f"normwise {r['normwise']:.3e}"
            + (f"  argmax {r['vectors']} vectors, {r['near_ties']} near "
               f"ties, {r['mismatches']} mismatches" if r["vectors"] else ""))
    tr.write_line(f"outputs compared: {len(PARITY)}; worst normwise "
                  f"{max(r['normwise'] for r in PARITY):.3e}; argmax vectors "
                  f"{vecs}, near-tie exemptions {ties}, mismatches {bad}")
