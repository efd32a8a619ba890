"""MI355X-native FL-GLM server stack: HIP kernels behind a C ABI
(include/flglm.h) with a thin ctypes binding.

The package fails loudly when its HIP library has not been built; there is
no CPU path.
"""

from . import flglm  # noqa: F401
from .flglm import BatchDesc, FlglmError, load  # noqa: F401
from .stack import ServerStack  # noqa: F401
from .optim import ParamArena, average  # noqa: F401
from .client import ClientHead, SplitModel  # noqa: F401
