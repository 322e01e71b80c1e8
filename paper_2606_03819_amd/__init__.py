"""TreeFlash drafting on MI355X (gfx950): two-stage parallel AR approximation
and OPT-Tree selection as a C-ABI HIP library with a thin Python binding.

The binding (``paper_2606_03819_amd.binding``) loads ``libtreeflash.so`` on
first use; importing this package does not touch the GPU.
"""

__all__ = ["binding", "synth"]


def __getattr__(name):
    if name == "binding":
        from . import binding
        return binding
    if name == "synth":
        from . import synth
        return synth
    raise AttributeError(name)
