"""CPU oracle for the shard halo-convolution hot path.

TEST INFRASTRUCTURE. Only ``tests/``, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of ``bench.py`` may import or run anything in this
package. The product path (the HIP library and its Python binding) never
touches it, and this package never imports the product path: the two share no
code. Inputs come from the separate ``synth`` generator.

What it computes, from the paper (ShardTensor, section "ShardTensor" and its
subsection "PyTorch Dispatch"): a spatially sharded tensor is processed shard
by shard; a convolution on a shard first fetches the adjacent pixels from the
neighbouring shards (the "halo") so that the result is numerically consistent
with the unsharded operation, and a convolution that changes the global shape
produces uneven output chunks whose per-rank sizes are tracked as "sharding
shapes". The oracle is therefore the plain definition:

* ``geometry``  - which outputs a shard owns and which input rows (halo) it
                  needs, found by enumeration;
* ``conv``      - the full-domain zero-padded cross-correlation (PyTorch
                  semantics) restricted to any output box, its weight and input
                  gradients, and the zero-extended input box a shard's padded
                  tile holds;
* ``halo``      - the face slabs exchanged along each sharded axis;
* ``brute``     - scalar-loop and dense-matrix restatements used to pin the
                  above on tiny inputs;
* ``norm``      - group normalisation of a sharded tensor: per-shard sums, their
                  total over all shards, and the normalised interior;
* ``attention`` - one block step of ring attention: scaled dot-product
                  attention against one key/value block and the log-space merge
                  into the running result.

Everything is float64 NumPy (``numpy.tensordot`` and ``numpy.matmul`` are the
only library steps).

Parity status: every function here is pinned by tests marked ``not gpu``
(brute force, dense Toeplitz matrices, torch's float64 CPU convolution,
closed forms and invariants); none is "parity unpinned".
"""
from . import geometry, conv, halo, brute, norm, attention  # noqa: F401
