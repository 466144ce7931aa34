"""fp64 CPU oracle of the TCL Mamba cost model (test infrastructure only).

Only the tests, the smoke check and the benchmark's CPU-baseline leg use
this package. It never imports the HIP library's package.
"""
from . import model  # noqa: F401
from . import kd  # noqa: F401
from . import select  # noqa: F401
from . import metric  # noqa: F401
from . import progressive  # noqa: F401
