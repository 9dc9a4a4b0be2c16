"""fp64 CPU oracle for FPI / VMP / MMP.  Test infrastructure only: imported by
the tests, the smoke check and the benchmark's CPU-baseline leg, never by the
library itself."""
from .oracle import infer, infer_soft, predict, build, lib_path, default_threads  # noqa: F401
