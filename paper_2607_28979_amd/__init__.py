"""libmot: MI355X-native Mixture-of-Translators KV-cache translation.

The compute path is the C-ABI shared library ``csrc/libmot.so`` (HIP kernels
for gfx950).  ``binding`` is a thin ctypes layer over it; importing this
package does not load the library, the first call does, and it raises if the
library is missing.  There is no CPU fallback.
"""
from .configs import WORKLOADS, HEADLINE, Workload  # noqa: F401


def __getattr__(name):
    # lazy: the binding loads libmot.so on first use
    if name in ("translate", "translate_raw", "depth_ratio_map", "workspace_bytes",
                "abi_version", "status_string", "Shapes", "MotError", "lib_path",
                "load_library", "MOT_F32", "MOT_BF16"):
        from . import binding
        return getattr(binding, name)
    raise AttributeError(name)
