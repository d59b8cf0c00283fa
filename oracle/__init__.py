"""CPU oracle for mixed prefill/decode paged attention.

TEST INFRASTRUCTURE. Only tests/, __graft_entry__.smoke() and bench.py's
cpu_baseline leg import this package. It shares no code with the HIP library
(paper_2606_04415_amd), and the library never imports it.

* attention.py: fp64 paged attention (textbook definition, explicit page
  gather, two-pass softmax), brute-force scalar variant, split-K partials and
  their merge.
* plan.py: integer re-derivation of the host plan (validation, phase
  classification, split-K partition, prefill tiles).
"""
