"""wsr: weight-streaming read kernels for MI355X (gfx950).

The product is libwsr.so (include/wsr.h); `paper_2608_12114_amd.wsr` is its Python binding.
Importing the package itself loads nothing, so that the build step (`paper_2608_12114_amd.build`)
runs on a tree where libwsr.so is not built yet.  Importing `paper_2608_12114_amd.wsr`, or reading
any entry point off the package, loads the library and fails loudly when it is missing.
"""
import os as _os

_HERE = _os.path.dirname(_os.path.abspath(__file__))


def __getattr__(name):
    # Submodule names (build, wsr) and dunders go to the import system, which asks for them here
    # first during `from package import submodule`.
    if name.startswith("__") or _os.path.exists(_os.path.join(_HERE, name + ".py")):
        raise AttributeError(name)
    from . import wsr
    return getattr(wsr, name)
