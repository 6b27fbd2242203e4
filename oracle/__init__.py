"""CPU oracle for sparse spiking BPTT (Perez-Nieves & Goodman, NeurIPS 2021).

TEST INFRASTRUCTURE ONLY. This package is the slow, plain reference that the
GPU path is checked against. Only the test suite, the package smoke check and
the benchmark's CPU-baseline leg may import it; the product path never calls
it and shares no code with it.

What it computes, and where the paper defines it:

* forward.py  -- discrete LIF layer, Eq. (lif) in Sec. 2.1 with V_rest = V_r = 0,
  V_th = 1, V[0] = 0; Heaviside spike Eq. (spike_fn); input trace of
  Eq. (lif_unrolled). float32, with a fixed summation order (ascending input
  index) so the GPU forward can be compared bit for bit.
* active.py   -- active set (Definition 1, Eq. (active)), truncated spike
  derivative (Definition 2) with the surrogate g(V) = 1/(beta|V - V_th| + 1)^2
  of Sec. 3 / App. E; CSR of the active set.
* loss.py     -- non-spiking readout (infinite threshold, Sec. 3) and the
  cross-entropy of App. E on max-over-time or sum-over-time logits.
* backward.py -- the gradient: dense BPTT with the surrogate truncated to zero
  outside the band (Eqs. (w_grad), (s_grad) with Definitions 1-2), which the
  sparse rule reaches exactly (Proposition 1, App. A; the sparse sums of
  Sec. 2.2 skip only terms multiplied by a zero derivative). Three variants:
  O1 literal sums, O2 memoised delta + BLAS (production), O3 event driven
  (Proposition 1 skip recurrence with the App. C schedule), plus operation
  counts (Table 1, App. B).
* regularize.py -- the activity penalties of App. E and their gradient w.r.t.
  spike counts.
* adam.py     -- the Adam update (App. E's optimiser; Kingma and Ba, Algorithm 1).
* train.py    -- a whole training step (loss with penalties, gradient, Adam) and
  the sparse vs full-surrogate gradient difference of App. H.
* conv.py     -- the convolutional spiking layer (3x3, padding 1) with 2x2 max
  pooling of its spikes into the readout (Sec. 3's convolutional experiment, App. E):
  forward through the layer's Toeplitz matrix, pooling, gradient routed back through
  the pooling, filter gradient.
* smooth.py   -- a smoothed-surrogate model whose exact gradient is the
  truncated-surrogate BPTT gradient; finite differences of it pin O2.

Parity status: every function here is pinned by tests in tests/test_oracle_*.py
(closed forms, finite differences, autograd, limits, the App. C example,
torch.optim.Adam, torch's conv2d and max_pool2d).
The paper's experimental numbers themselves are parity unpinned: they need the
datasets, trained weights or the authors' GPUs.
"""
from .forward import lif_forward, network_forward, summed_inputs, summed_inputs_loop  # noqa: F401
from .active import active_mask, active_csr, surrogate  # noqa: F401
from .loss import readout_logits, cross_entropy, readout_grad  # noqa: F401
from .backward import (  # noqa: F401
    delta_recurrence, layer_backward, network_backward, layer_backward_literal,
    layer_backward_events, skip_delta, csr_values,
)
from .regularize import spike_counts, activity_penalty, activity_grad  # noqa: F401
from .adam import adam_update  # noqa: F401
from .train import training_gradients, train_step, gradient_difference  # noqa: F401
