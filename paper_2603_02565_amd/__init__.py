"""FlashEvaluator joint-evaluation forward pass on AMD MI355X (gfx950).

The compute path is libflasheval.so (HIP kernels behind the C ABI of include/flasheval.h);
`flasheval` is its ctypes binding.
"""
from . import flasheval  # noqa: F401
from .flasheval import Evaluator, load_library, param_names, pack_params  # noqa: F401
