"""CPU oracle (test infrastructure only): plain float64 NumPy from the paper."""
from .asrkf_oracle import (SR, WR, FR, freeze_duration, duration_table, attention,  # noqa: F401
                           relevance, relevance_softmax, attend_rows, entropy, escalate,
                           TokenStates, LayerCache, Instance, GlobalInstance, StepRecord,
                           recovery_schedule, run_instance)
