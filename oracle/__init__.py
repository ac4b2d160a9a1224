"""fp64 CPU oracle for the DSTD-LIF layer (test infrastructure only).

Only the test suite, ``__graft_entry__.smoke()`` and the CPU-baseline leg of
``bench.py`` may import this package. It shares no code with the HIP library.
"""
from .oracle import (  # noqa: F401
    build_oracle,
    compile_oracle,
    use_library,
    kernel,
    kdstd,
    lambert_w0,
    dstd_events,
    dstd_forward,
    dstd_scan,
    dstd_backward,
    exact_forward,
    conv_out_hw,
    exact_backward,
    ms_forward,
    ms_backward,
    conv_forward,
    conv_backward,
    num_threads,
)
from .synfire import window, temporal_penalty, dead_neuron_penalty  # noqa: F401
