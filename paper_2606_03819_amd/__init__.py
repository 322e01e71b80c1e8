"""TreeFlash drafting on MI355X (gfx950): two-stage parallel AR approximation
and OPT-Tree selection as a C-ABI HIP library with a thin Python binding.

Submodules: ``binding`` (loads ``libtreeflash.so`` on first call),
``synth`` (seeded synthetic inputs), ``build`` (hipcc build).  Importing the
package itself touches neither the library nor the GPU.
"""
