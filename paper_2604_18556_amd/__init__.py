"""GSQ layer step on MI355X (gfx950): HIP kernels behind a C ABI, with a thin ctypes binding.

``paper_2604_18556_amd.binding`` loads ``libgsq.so`` (built in-tree by
``__graft_entry__.build()``) and fails loudly when it is missing; importing this
package itself loads nothing.
"""
__all__ = ["binding", "inputs"]
