"""Oracle package: test infrastructure only (see ref_attention)."""
from .ref_attention import *  # noqa: F401,F403
