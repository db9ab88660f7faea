"""CPU oracle of the GNMR controller pass -- TEST INFRASTRUCTURE ONLY.

Only tests/, __graft_entry__.smoke() and the cpu_baseline leg of bench.py may
import, call or run anything under oracle/.  It shares no code with the HIP
library or its binding and imports neither.
"""
from .gnmr_oracle import (BF16, BUDGET_ACTIVE, BUDGET_ADMITTED, BUDGET_STATIC, F32,  # noqa: F401
                          Controller,
                          StepResult, sumsq, unit_norm, widen)
