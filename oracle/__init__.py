"""CPU oracle of the BRISK-DLM decoding hot path (test infrastructure only)."""
from .brisk_oracle import *  # noqa: F401,F403
from .brisk_oracle import __all__ as _decode_all
from .profile_oracle import *  # noqa: F401,F403
from .profile_oracle import __all__ as _profile_all
from .spec_oracle import *  # noqa: F401,F403
from .spec_oracle import __all__ as _spec_all

__all__ = list(_decode_all) + list(_profile_all) + list(_spec_all)
