"""CPU float64 oracle for the fused turn-KL path.

TEST INFRASTRUCTURE: only tests/, __graft_entry__.smoke() and bench.py's
cpu_baseline leg may import it.  The product path never does.
"""
