"""The native routing library's parity cases, collected again under the gpu marker.

The routing library is host code and its parity tests (test_routing_native)
run in the CPU suite.  This module re-collects the same cases with the gpu
marker so that a GPU-box run, which selects only gpu-marked tests, also loads
the shared library there and checks its routing against the oracle.
"""
import pytest

from tests import test_routing_native as _native

pytestmark = pytest.mark.gpu

calib = _native.calib
for _name in dir(_native):
    if _name.startswith("test_"):
        globals()[_name] = getattr(_native, _name)
del _name
