"""CPU oracle for the spike-gated INT8 projection (test infrastructure only).

Only the test suite, the smoke check and the benchmark's CPU-baseline leg may
import this package.  The GPU library never uses it.
"""
from .spike_oracle import build, load, active_indices, spike_acc, spike_forward, dense_forward  # noqa: F401
from .quant_oracle import quantize_int8, export_column_major  # noqa: F401
from . import head_oracle  # noqa: F401
