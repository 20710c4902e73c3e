"""CPU oracle for the encrypted scoring path -- TEST INFRASTRUCTURE ONLY.

Only tests/, __graft_entry__.smoke() and bench.py's CPU-baseline leg may
import this package; the product path never does.
"""
