"""CPU oracle for tile-sparse 3D attention -- test infrastructure, not product code.

A plain, slow, obviously correct float64 reference of what the GPU path
computes, written from the paper (Efficient-vDiT, arXiv 2502.06155):

* ``oracle.masks``: the k:(F-k) family of frame-tile masks (Sec. 3.3) and the
  128 x 128-block sparsity the paper reports (Sec. 4.2.1, tab:kernel_time).
* ``oracle.attention``: softmax attention restricted to the key frames a query
  frame's mask row keeps (Sec. 3.1, Sec. 3.3, App. B), and its log-sum-exp.
* ``oracle.backward``: the gradients of that attention with respect to q, k, v.
* ``oracle.mmdit``: the MM-DiT form, a dense text prefix before the tile-sparse video
  (Sec. 4.3, App. E).

Only ``tests/``, ``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of
``bench.py`` may import this package. The product path (the HIP library and
its Python binding) never imports it, and it imports nothing from the product.
"""
from . import attention, backward, masks, mmdit  # noqa: F401
