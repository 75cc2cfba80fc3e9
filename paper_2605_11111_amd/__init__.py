"""MI355X-native shard halo convolution (the per-shard hot path of ShardTensor-style
domain parallelism).

    from paper_2605_11111_amd import shardconv   # ctypes binding of libshardconv.so
    python -m paper_2605_11111_amd.build          # compile the HIP library in-tree

The binding module raises ImportError when the library has not been built.
"""
