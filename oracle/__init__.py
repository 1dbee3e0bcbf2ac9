"""CPU oracle for block-structured pruned conv / FC inference.

TEST INFRASTRUCTURE ONLY.  Nothing in the product package may import, call,
link or execute anything here; only the tests, the smoke check and the CPU
baseline leg of the benchmark use it.  It shares no code with the HIP path.

What it computes (all in fp64, slow and plain on purpose):

* ``prune``  - the pruning regularity of Sec. 4.1 (block-based pruning: the
  GEMM-form weight matrix is cut into equal blocks and whole rows or whole
  columns are removed inside each block), with the group measure of Eqs. 2-3
  (squared Frobenius norm of a row / column of a block) and the one-shot
  magnitude selection of Sec. 5.1; block 1x1 = unstructured, whole matrix =
  structured (Sec. 4.4).  Also the canonical packing of kept indices and
  values (the storage idea of Sec. 4.3, in this library's own format).
* ``direct`` - plain direct convolution and matrix product on the masked
  dense weights, in C (gcc, OpenMP), the definition of what the pruned layer
  computes (layer i of Sec. 4.2 with weights W_i and bias b_i).
* ``brute``  - pure-Python loops for tiny shapes, used to pin ``direct``.
* ``glue``   - 2x2 max pooling between VGG stages.

Every function here has pins in ``tests/test_oracle_*.py``; see each module
header for the passage it follows and the pins that check it.
"""
