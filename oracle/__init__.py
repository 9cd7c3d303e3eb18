"""fp64 CPU oracle for shared-prompt group attention.

TEST INFRASTRUCTURE ONLY. Nothing in the product path imports, calls or links
this package: only ``tests/``, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of ``bench.py`` may use it. It shares no code with the HIP
path; both only read the same seeded bf16 inputs.

What it computes (the plain definitions, in float64):

* ``attention.attend_fwd`` / ``attend_bwd``: masked softmax attention
  O = softmax(s * Q K^T + M) V (§2.2) and its gradients written out term by
  term.
* ``attention.flattened_fwd_bwd``: every branch as its own causal sequence
  [P; R_i] (the flattened view of the replay tree, §2.1), with the upstream
  gradient of the prompt rows split evenly over the G copies; prompt results
  are summed over the copies. This is the reference every GPU output is
  compared against.
* ``attention.shared_fwd_bwd``: the method's own decomposition (§3.2-§3.3):
  prompt prefill once, each branch as a prompt partial plus a branch-local
  causal partial merged by log-sum-exp, and the prompt-KV gradient as the
  prefill contribution plus the sum over branches (Eq. 2). Used only to check
  that the decomposition is exact against the flattened reference.
* ``attention.lse_merge``: the associative merge of partial softmax states
  (§3.3), in closed form.
* ``sampled``: the same definitions for single query rows or single key rows
  of full-size workloads, for parity at sizes the full oracle cannot reach.

Every function is pinned by ``tests/test_oracle.py`` against something other
than itself (closed forms, a library routine, finite differences, brute force
on tiny inputs, invariants of the method).
"""
from . import attention, sampled  # noqa: F401
