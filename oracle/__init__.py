"""fp64 CPU oracle of the DiT denoising step (test infrastructure only; see
dit_oracle's header)."""
from .dit_oracle import *  # noqa: F401,F403
