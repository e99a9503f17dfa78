"""Oracle: a plain, slow, obviously correct CPU reference of the batched
dynamic-dataflow-graph forward pass (ED-Batch, arXiv 2302.03851).

TEST INFRASTRUCTURE ONLY.  Nothing in the product path imports, calls or
links this package; only the tests, the smoke check and the CPU-baseline leg
of the benchmark do.  It shares no code with the HIP path or its host
library.  It is written in numpy float64 (the paper fixes no precision).

Contents
  cells     the cell equations of the evaluated models (Section 5.1, Table 2)
  evaluate  node-at-a-time evaluation in topological order (the unbatched
            semantics that batching must not change, Section 2.1)
  schedule  Algorithm 1 (FSM-based dynamic batching) with table / agenda /
            depth policies and the sufficient-condition policy, the state
            encodings of Section 2.3, the lower
            bound of Appendix A.3, the Eq. 1 frontier ratio and a brute-force
            optimum (Appendix A.1)
  learn     the FSM policy learner (Section 2.3: Eq. 1 reward, tabular
            Q-learning with N-step bootstrapping) and its random source
  pqtree    a PQ tree (Booth and Lueker) with template reduction
  pqplan    the PQ-tree memory layout of Section 3.2 (construction,
            constraint broadcast, order decision by union-find, leaf order)
  plan      the batching-aware memory plan (Section 3.1 constraints; slot
            assignment by a reverse consumer-first pass) and its hazard check
  compare   the normwise relative error used by the parity tests
  mvrnn     the MV-RNN of Table 2 on binary trees (a vector and a matrix per
            node), evaluated on the tree itself
  latticegru  the lattice GRU of Table 2 (per-edge GRU proposals averaged per
            position), evaluated on the lattice itself
"""
