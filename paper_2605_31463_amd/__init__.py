"""MI355X-native MoE layer (forward and backward) behind the libmoe C ABI.

The binding (``paper_2605_31463_amd._lib``) and the buffer helper
(``paper_2605_31463_amd.layer``) are loaded on first use, so that the build
step can run before the library exists.  Loading fails loudly when libmoe.so
has not been built: there is no other implementation behind these names.
"""
import importlib

_LAZY = {"layer": "paper_2605_31463_amd.layer", "_lib": "paper_2605_31463_amd._lib"}


def __getattr__(name):
    if name in _LAZY:
        return importlib.import_module(_LAZY[name])
    lib = importlib.import_module("paper_2605_31463_amd._lib")
    if hasattr(lib, name):
        return getattr(lib, name)
    raise AttributeError(name)
