"""fp64 CPU oracle for PipeGCN's per-partition training step.

TEST INFRASTRUCTURE ONLY.  This package is the plain, slow, obviously correct
reference that the HIP path is checked against.  Only ``tests/``,
``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of ``bench.py`` may
import it.  It shares no code with the HIP path (``paper_2203_10428_amd``),
and it never imports that package.

Modules
-------
``partition``  inner / boundary / send sets and the local propagation matrix
               (Algorithm 1 set-up; Section 3.1; Appendix A.1 split of P).
``layers``     one GCN layer and one GraphSAGE (CONCAT) layer forward and
               backward, losses, moving average, SGD and Adam (Appendix A.1
               layer function and its gradients; Section 2; Section 3.4).
``philox``     Philox4x32-10 and the dropout mask drawn from it.
``pipegcn``    the multi-partition simulation of Algorithm 1 in pipelined
               (one-iteration-stale) and vanilla (synchronous) modes, with
               the GCN or GraphSAGE model, dropout, SGD or Adam.

Every quantity is computed in float64.  Parity status of each function is
stated in its docstring; all functions here are pinned by the CPU tests
(brute force, closed forms, finite differences, reductions to full-graph
GCN and GraphSAGE, published known-answer vectors, torch.optim.Adam), except
where a docstring says "parity unpinned".
"""
