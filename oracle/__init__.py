"""CPU oracle for ACDC / AFDF cascades -- test infrastructure only.

Only tests/, __graft_entry__.smoke() and bench.py's cpu_baseline leg may
import this package.
"""
