"""opfuse: optimizer fusion (arXiv 2104.00237) on AMD MI355X.

The compute path is the HIP library libopfuse.so (C ABI in include/opfuse.h);
`_lib` is its ctypes binding and `trainer` the host scheduler of the three
orderings (eager, forward-fusion, backward-fusion).
"""
from . import _lib  # noqa: F401
