import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU")
    config.addinivalue_line("markers", "slow: long-running CPU test")


@pytest.fixture(scope="session")
def hsa_gpu():
    """The HIP library binding; a GPU test fails loudly if the library is missing."""
    import torch
    if not torch.cuda.is_available():
        pytest.fail("GPU test collected on a machine without a GPU")
    import paper_2504_16795_amd as hsa
    hsa.load()          # raises if the built library is absent
    return hsa


@pytest.fixture
def kernel_path(hsa_gpu):
    """kernel_path(op, path): serve op with a kernel family for this test only
    (hsa_attn_set_path), restored to the default afterwards."""
    ops = []

    def setter(op, path):
        hsa_gpu.set_path(op, path)
        ops.append(op)

    yield setter
    for op in ops:
        hsa_gpu.set_path(op, hsa_gpu.HSA_PATH_AUTO)


def pytest_terminal_summary(terminalreporter):
    """Print the bf16 error ratios the parity tests recorded (max|err| / (2e-2 RMS(ref)) and
    max|err| / element bound), worst first; with HSA_PARITY_REPORT=<path>, also as JSON."""
    try:
        import parity
    except ImportError:
        return
    if not parity.RATIOS:
        return
    rows = sorted(parity.RATIOS, key=lambda r: -r[2])
    tr = terminalreporter
    tr.write_sep("-", "bf16 parity: contract ratio (beyond the output half-ulp), element-bound "
                      "ratio, raw ratio, rounded-oracle ratio")
    for test, name, rr, er, contract, raw, floor in rows[:40]:
        tr.write_line("%6.3f %6.3f %6.3f %6.3f %s %-4s %s" % (rr, er, raw, floor,
                                                             "C" if contract else "-", name, test))
    tr.write_line("%d comparisons; worst asserted contract ratio %.3f" % (
        len(rows), max((r[2] for r in rows if r[4]), default=0.0)))
    path = os.environ.get("HSA_PARITY_REPORT")
    if path:
        import json
        with open(path, "w") as f:
            json.dump([dict(test=t, tensor=n, contract_ratio=rr, element_ratio=er, asserted=c,
                            raw_ratio=raw, rounded_oracle_ratio=fl)
                       for t, n, rr, er, c, raw, fl in rows], f, indent=1)
