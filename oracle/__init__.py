"""CPU oracle (test infrastructure only; see domino_oracle's header)."""
from .domino_oracle import *  # noqa: F401,F403
from .domino_oracle import as_f64_weights  # noqa: F401
from . import sampling_oracle  # noqa: F401
from . import train_oracle  # noqa: F401
from . import target_oracle  # noqa: F401
