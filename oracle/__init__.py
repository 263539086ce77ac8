"""CPU oracle for the Kashin-DCT hot path (test infrastructure only; see kashin_ref)."""
from .kashin_ref import *  # noqa: F401,F403
