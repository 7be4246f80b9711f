"""CPU oracle for the prefix-reuse prefill hot path.

TEST INFRASTRUCTURE. Only ``tests/``, ``__graft_entry__.smoke()`` and the CPU
baseline leg of ``bench.py`` may import anything from this package. The
product path (``paper_2603_23049_amd``) never does, and this package never
imports the product path.

Modules:
  datamove   plan, KV load, KV append and KV gather (integer / bit-copy steps)
  attention  fp64 causal GQA attention through the paged pool (C, OpenMP)
  tree       brute-force longest cached prefix (pins the host prefix tree)
  schedule   two-stage layer pipeline: brute-force event schedule
"""
