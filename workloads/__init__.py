"""Seeded synthetic workloads shared by the oracle and the GPU path.

Holds only input generation: decoder configurations, their tensor lists and
kernel access traces, and seeded initial contents.  None of the method's
arithmetic (cost model, roofline classification, planning, model math) is here.
"""
from . import format, configs, trace, init  # noqa: F401
