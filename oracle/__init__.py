"""CPU oracle (test infrastructure only): plain float64 NumPy from the paper."""
from .asrkf_oracle import (SR, WR, FR, freeze_duration, duration_table, attention,  # noqa: F401
                           relevance, attend_rows, entropy, escalate, Instance, StepRecord,
                           recovery_schedule, run_instance)
