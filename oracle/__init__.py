"""CPU oracle for the batched, ragged Llama-2 greedy decode step.

TEST INFRASTRUCTURE ONLY.  Only tests/, __graft_entry__.smoke() and bench.py's
cpu_baseline leg may import, call, link or execute anything in this package.
The product path (paper_2403_12900_amd) never does, and the two share no code:
the oracle generates its own weights with its own implementation of the
counter-based generator (wgen.c) and computes everything in fp64 with plain
numpy operations.
"""
