"""CPU oracle for FP64 matrix multiplication through Ozaki schemes II and I on
base-13 E2M1 limbs (scheme II also with a two-term split of the converted
operands, and with the one-limb modulus 11 in the moduli list), and for FP32
matrix multiplication through scheme II.

TEST INFRASTRUCTURE ONLY. Nothing in the product path may import, call or
execute this package: only ``tests/``, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of ``bench.py`` use it. It shares no code, tables or
constants with the HIP library; every constant here is re-derived from the
paper's definitions.

Parity status: every function is pinned by ``tests/test_oracle_*.py`` against
values the paper prints, closed forms, invariants and brute force on tiny
inputs. No function is "parity unpinned".
"""

from .ozaki2_fp4 import *  # noqa: F401,F403
from .ozaki2_fp4 import __all__ as _all2
from .ozaki1_fp4 import *  # noqa: F401,F403
from .ozaki1_fp4 import __all__ as _all1
from .sgemm_fp4 import *  # noqa: F401,F403
from .sgemm_fp4 import __all__ as _all32
from .split2_fp4 import *  # noqa: F401,F403
from .split2_fp4 import __all__ as _alls
from .one_limb_fp4 import *  # noqa: F401,F403
from .one_limb_fp4 import __all__ as _all1l

__all__ = list(_all2) + list(_all1) + list(_all32) + list(_alls) + list(_all1l)
