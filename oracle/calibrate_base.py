"""Fix the validity-margin bias of the calibrated synthetic workloads.

TEST INFRASTRUCTURE: calls only the oracle (and the input generator).

For a workload with a target invalid fraction p, the bias is
``-(float32) m_(floor(p*M))`` where m_(j) is the j-th smallest zero-bias
validity margin of the first M = 65536 candidates.  Only the bias of the
validity ensemble changes; trees and features are untouched.  The printed
values are the constants ``_BASE_V_MEDIUM`` / ``_BASE_V_SKEWED`` in
``gen/__init__.py``; ``tests/test_workloads.py`` recomputes them.

Run:  python -m oracle.calibrate_base
"""
from __future__ import annotations

import numpy as np

import gen
import oracle


def calibrated_base(workload: gen.Workload, threads: int | None = None) -> float:
    assert workload.calib_quantile is not None
    m_rows = min(workload.n, gen.CALIBRATION_ROWS)
    X = workload.features(rows=np.arange(m_rows, dtype=np.int64))
    v0 = workload.validity().with_base(0.0)
    _, margins = oracle.validity(v0, X, threads or gen.default_threads())
    order = np.sort(margins, kind="stable")
    q = order[int(np.floor(workload.calib_quantile * m_rows))]
    return float(-np.float32(q))


def main() -> None:
    for name in ("medium", "skewed"):
        w = gen.WORKLOADS[name]
        b = calibrated_base(w)
        print(f"{name}: base_v = {b!r}  (float32 bits 0x{np.float32(b).view(np.uint32):08x})")


if __name__ == "__main__":
    main()
