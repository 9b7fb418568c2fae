"""ElasticKV mixed-fidelity paged KV attention for AMD MI355X (gfx950).

The compute path is the C-ABI library ``libekv.so`` built from ``csrc/``;
``ekv`` is its thin ctypes binding and ``workloads`` makes seeded synthetic
inputs.
"""
