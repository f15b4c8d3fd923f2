"""Float64 CPU oracle of the REAL-Q layer sweep.  Test infrastructure only: the
product library never imports it."""
from .realq_oracle import *  # noqa: F401,F403
from .realq_oracle import QParams, LayerResult, AdamState  # noqa: F401
