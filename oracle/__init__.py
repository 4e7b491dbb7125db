"""fp64 CPU oracle for block-sparse attention (test infrastructure only: the
product path never imports this package)."""
from .sparse_attention import *  # noqa: F401,F403
from .compensation import *  # noqa: F401,F403
from .fp8_linear import *  # noqa: F401,F403
from .causal_window import *  # noqa: F401,F403
from .backward import *  # noqa: F401,F403
