"""fp64 CPU oracle (test infrastructure only; never imported by the product path)."""
from .sparvar_oracle import *  # noqa: F401,F403
from .cs4a_oracle import *  # noqa: F401,F403
from .csla_oracle import *  # noqa: F401,F403
