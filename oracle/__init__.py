"""CPU oracle for MPX's mixed-precision training step (test infrastructure).

This package is the plain, slow, obviously-correct reference that the HIP
path is checked against.  It is test infrastructure only: nothing outside
``tests/``, ``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of
``bench.py`` may import it.  It shares no code with the HIP path; the only
module both sides use is ``workloads`` (seeded random draws, no arithmetic of
the method).

What it computes (MPX, Gräfe & Trimpe, arXiv 2507.03312):

* §2 and §2.1: the mixed-precision recipe with dynamic loss scaling —
  forward in half precision, scale the loss, gradients of the scaled loss,
  convert them to float32, divide by the scale, update the scale (shrink and
  skip on overflow, grow after a long run of finite steps), update the model.
* §3.1: casting float leaves to float16 / bfloat16 (round to nearest even).
* §3.3: ``scale`` / ``unscale`` / ``adjust`` of the dynamic loss scaling state.
* §3.4: the transformed gradient function (cast inputs, run, scale, grad,
  unscale, check finiteness, adjust).
* §3.5: ``optimizer_update`` applying the optimizer only on finite steps; the
  optimizer is AdamW (decoupled weight decay).

Modules: ``numfmt`` (number formats), ``policy`` (per-op precision and the
GEMM definition), ``ops`` (layer forward/backward), ``scaling`` (unscale,
finite check, scale state machine), ``adamw`` (masked AdamW), ``models`` (MLP
and ViT), ``step`` (the whole training step).

Parity status: every function is pinned by tests under ``tests/`` marked
``not gpu`` (library cross-checks, closed forms, invariants, finite
differences).  Whole-network trajectories after several steps have no
independent value to pin against and are "parity unpinned" beyond the pins of
their parts.
"""
