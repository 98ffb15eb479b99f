"""Plain fp64 CPU oracle of one transformer fine-tuning step.

TEST INFRASTRUCTURE ONLY.  Only ``tests/``, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of ``bench.py`` may import it.  The HIP library never
calls it and it never calls the HIP library: the two share no code.

What it computes is the work the Saturn paper (arXiv 2309.01226) schedules:
the fine-tuning of pre-trained transformers (GPT-2, GPT-J, ViT; Sec. 1 case
study and Table 3 / Sec. 5 "Workloads") with model selection over hyper-
parameters and over which layers are fine-tuned (Abstract, "layer-wise
finetuning"; Sec. 2 "Model selection").  The paper fixes no block details;
every reading of a silent point is listed in ``oracle.model`` and in the
repository's design notes.

Every function is the textbook definition written out in numpy float64 with
hand-written vector-Jacobian products.  Pins that tie it to something other
than itself (finite differences, torch library routines, closed forms,
invariants) live in ``tests/test_oracle_*.py``.
"""

from .model import (  # noqa: F401
    Config,
    param_spec,
    trainable_mask,
    init_params,
    forward,
    backward,
    adamw_update,
    train_step,
    eval_loss,
)
from . import layers  # noqa: F401
