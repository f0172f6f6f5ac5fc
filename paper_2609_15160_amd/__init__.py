"""T-LoopFormer routed prefill/decode on MI355X: binding of the libtlf HIP library."""
from . import tlf  # noqa: F401
