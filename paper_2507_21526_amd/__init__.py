"""MI355X (gfx950) Triangle attention and dense causal attention.

The compute path is the HIP library ``libtriattn.so`` built from ``csrc/``;
``binding`` marshals torch tensors into its C interface.  Importing this
package loads nothing; ``binding.lib()`` loads the library and raises if it
has not been built.
"""
__all__ = ["binding", "inputs"]
