"""CPU oracle (test infrastructure only; see sq_oracle)."""
from .sq_oracle import *  # noqa: F401,F403
from .sq_oracle import RANGE_DYNAMIC, RANGE_STATIC, A4_GROUP, Q_MAX, W_QMAX  # noqa: F401
