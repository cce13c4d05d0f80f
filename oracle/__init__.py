"""CPU oracle for the packed four-direction MDLSTM layer — TEST INFRASTRUCTURE ONLY.

Plain, slow, float64 NumPy definitions of what the GPU path computes:

* ``oracle.pack``   — example packing layout (Algorithm 1 of Appendix B and
  Section V-A), the binary mask, scatter into and gather out of the canvas,
  and the last-minute batch-padding layout of Section VI-B.
* ``oracle.mdlstm`` — the 2D MDLSTM cell (Section III), scanned in four
  directions (Section III), forward and backward, per example; plus a
  whole-canvas masked scan (Section V: masking blocks state from invalid
  predecessors).
* ``oracle.stack``  — the three-layer stack with block-strided convolutions
  and tensor-list chunking (Section V-B).
* ``oracle.head``   — the output layer shared by the four directions with the
  collapse of the rows (Section II), and the CTC loss with its gradient.

Only ``tests/``, ``__graft_entry__.smoke()`` and the CPU-baseline leg of
``bench.py`` may import this package. The product path (the HIP library and
its Python binding) never imports, calls or links anything here, and nothing
here imports the product path.

Parity unpinned: the block-convolution grouping convention of the three-layer
stack (one group per direction, outputs concatenated) is a reading, checked
only against its own definition and finite differences; so is the output
layer's collapse of the rows (a sum over the rows and the four directions),
while the CTC loss itself is pinned by hand-worked cases, brute force over
every frame path and PyTorch's float64 CTC loss.
"""
