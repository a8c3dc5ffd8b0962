"""CPU oracle (fp64 numpy) for the reward-coordinated compression hot path.

Test infrastructure: only the tests, the smoke check and the bench's CPU
baseline use it.  It shares no code with the HIP library."""
from .reco_oracle import *  # noqa: F401,F403
from .reco_oracle import score_cache, compress_cache, decode_cache  # noqa: F401
