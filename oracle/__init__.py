"""Oracle package: test infrastructure only (see ref_attention, ref_branches, ref_block)."""
from .ref_attention import *  # noqa: F401,F403
from .ref_branches import *  # noqa: F401,F403
from .ref_block import *  # noqa: F401,F403
