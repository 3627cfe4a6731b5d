"""fp64 CPU oracle for the BaKron solver (test infrastructure only; see oracle.py)."""
from .oracle import *  # noqa: F401,F403
from .oracle import build, babai, solve, ar1_diffusion, certificate, verdict, objective  # noqa: F401
from . import hessian  # noqa: F401,E402  (Kronecker-factor construction, App. A)
