"""CPU oracle for the packed causal-context DiT step -- TEST INFRASTRUCTURE ONLY.

Plain, slow, fp64 numpy code written from the paper ("Rethinking Streaming
Video Diffusion Model: Context, Execution, and Training").  It exists to check
the HIP path.  Only ``tests/``, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of ``bench.py`` may import or run anything in this package;
the product library never does, and this package never imports the product.

Modules
  policy     history selection, Sec. 3.2, Eq. 4-5 (selection table, visibility)
  plan       availability (Sec. 3.3 restrictions, Eq. 8) and page resolution
             over a model of the paged KV cache
  attention  softmax attention of each node over its selected states, Eq. 6
  rope       3D rotary position embedding (a reading: the paper does not define it)
  block      one DiT block: RMSNorm, QKV, RoPE, attention, out-projection, MLP
  pipeline   pipelined rounds, Eq. 7, with the sampler of Eq. 1

Parity status: functions whose result is not fixed by the paper or by
mathematics say "parity unpinned" in their docstrings.  The block composition,
the RoPE frequency split and the sampler form are readings of the workload
description, not statements of the paper.
"""
