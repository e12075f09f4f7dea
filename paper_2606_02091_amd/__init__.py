"""DFlare draft step on MI355X (gfx950): HIP kernels behind a C-ABI library.

The binding (``paper_2606_02091_amd.dflare``) loads ``_lib/libdflare.so`` on first
use and raises if it has not been built; nothing here falls back to the CPU.
"""
__all__ = ["synth"]
