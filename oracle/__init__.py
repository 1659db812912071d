"""fp64 CPU oracle of the group-batched step -- TEST INFRASTRUCTURE ONLY.

Only ``tests/``, ``__graft_entry__.smoke()`` and the CPU-baseline leg of
``bench.py`` may import this package.  The product path (the HIP library
and its Python binding) never imports, calls or links anything here, and
this package imports nothing from the product path.

What it computes (JoyNexus, Sec. 4.3 "Multi-Tenant Group Batching",
App. A.3 "Inference Queue Composition", Sec. 5.2 "Multi-Tenant
Group-Batched Execution"): grouping compatible tenant batches into one
physical batch only removes repeated base-model computation; every tenant
keeps its own loss, backward and update, and nothing is averaged across
tenants.  So the oracle never packs for compute: it runs every sample
through the frozen backbone *on its own*, pools it, and runs each tenant's
action head, loss and weight-gradient over that tenant's samples only.
The pack plan (the "slices" of App. A.3) is computed separately, with
plain loops, for bit-exact comparison.

Modules
  plan      -- pack plan and index maps (integer, plain loops)
  backbone  -- per-sample pre-RMSNorm transformer forward in fp64
  heads     -- per-tenant MLP head forward, MSE loss, hand-written backward
  expert    -- per-tenant action expert (config 4) forward, loss, gradients
  optim     -- per-tenant AdamW optimizer step
  step      -- the isolated-execution reference of the whole step
  batching  -- the inference queue's FIFO-compatible-prefix batching

Pins: every function here is checked in ``tests/test_oracle_pins.py``
against closed forms, invariants, special cases that reduce to library
routines, brute force on tiny inputs and finite differences.
"""
from . import plan, backbone, heads, step, expert, optim, batching  # noqa: F401
