"""FastVLM self-speculative decoding on MI355X (gfx950).

  paper_2510_22641_amd.ssd       ctypes binding of libssd (include/ssd.h), same entry points
  paper_2510_22641_amd.runtime   device memory (weights, paged KV cache, workspace) for a context
  paper_2510_22641_amd.build     builds libssd.so in-tree with hipcc for gfx950

Importing the package loads nothing; ``paper_2510_22641_amd.ssd`` loads the library and raises
when it has not been built.
"""
