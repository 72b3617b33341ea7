"""CPU oracle for the owner-local Muon / AdamW step (fp64, plain numpy).

TEST INFRASTRUCTURE ONLY. Nothing in the product path imports, calls or links this package:
only ``tests/``, ``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of ``bench.py`` use it.
It shares no code, table or helper with the HIP library, and it never reads anything the HIP
library produced except the outputs it is compared against.

What it computes follows the paper (MatrixFSDP, arxiv 2607.05895):

* Section 3: the owner of a whole 2D matrix applies the Newton-Schulz (NS) Muon update to the full
  matrix and updates its local parameter and Muon state; tail owners apply AdamW to non-matrix
  tensors.
* Section 2: NS steps are built from products such as X X^T of the whole matrix.
* Section 5.1 (Setup): Muon is ``torch.optim.Muon`` (momentum buffer, Nesterov, quintic NS with a
  fixed coefficient triple, shape-adjusted learning rate ``match_rms_adamw`` or the default
  ``original``, decoupled weight decay); AdamW is PyTorch AdamW with betas (0.9, 0.999), eps 1e-8.

Where the paper is silent, the readings used are the ones stated in each function's docstring.

* Section 5.7 (Generality beyond Muon): the owner runs Shampoo (full left/right preconditioners,
  inverse fourth root, ``shampoo.py``) and SOAP (Adam in the eigenbasis of Shampoo's statistics,
  ``soap.py``) on the same whole matrices.

Parity status: every function here is pinned by tests in ``tests/test_oracle_pins.py``,
``tests/test_planner_pins.py``, ``tests/test_shampoo_pins.py`` and ``tests/test_soap_pins.py``.
"""
from .muon import (  # noqa: F401
    bf16_widen,
    momentum_update,
    frobenius_normalize,
    ns_quintic_step,
    newton_schulz,
    lr_factor,
    apply_update,
    muon_step,
    reduce_gradients,
    step_coefficients,
)
from .adamw import adamw_step  # noqa: F401
from . import planner  # noqa: F401
from . import shampoo  # noqa: F401
from . import soap  # noqa: F401
