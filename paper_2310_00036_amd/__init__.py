"""MI355X-native learner update of Cleanba's PPO / IMPALA: hand-written gfx950 HIP kernels
behind the C-ABI of include/cleanba_learner.h, with a thin ctypes binding of the same names.

``import paper_2310_00036_amd`` loads the in-tree ``libcleanba_learner.so`` and fails loudly
when it has not been built (``paper_2310_00036_amd.build.build()``).
"""
from . import _lib  # noqa: F401  (fails loudly without the library)
from ._lib import *  # noqa: F401,F403
