"""fp64 CPU oracle for one GPipe pipeline partition.

TEST INFRASTRUCTURE ONLY.  Nothing in the product path may import, call or
execute this package; only the tests, the smoke entry point and the
benchmark's CPU-baseline leg use it.  It shares no code with the HIP path.

What it computes (GPipe, Sections 2.1-2.3): the partition's composite forward
function F_k (a stack of Transformer layers), its back-propagation function
B_k derived by hand, the loss head of the last partition, and the training
step in which a mini-batch of N examples is split into M equal micro-batches,
only the partition-boundary input of each micro-batch is kept during the
forward pass, each micro-batch's forward is recomputed (re-materialised)
inside its backward pass, and the M micro-batch gradients are accumulated
and applied in one synchronous update.

Modules:
  transformer -- layer forward/backward definitions (LayerNorm, attention,
                 encoder and decoder layers, loss heads);
  gpipe       -- the plain mini-batch definition and the micro-batched
                 re-materialising schedule, plus the update.
"""
from . import transformer, gpipe  # noqa: F401
