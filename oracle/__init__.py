"""Oracle package: test infrastructure only (see ref_attention and ref_branches)."""
from .ref_attention import *  # noqa: F401,F403
from .ref_branches import *  # noqa: F401,F403
