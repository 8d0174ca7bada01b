"""Plain fp64 CPU oracle of Re-ttention's sparse attention and statistical reshape.

TEST INFRASTRUCTURE ONLY.  Only ``tests/``, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of ``bench.py`` may import anything from this package.  The
HIP library never calls it and shares no code, header, table or helper with it.

Modules
-------
attention    Eq.1-5 (dense and sparse softmax attention with row statistics),
             Eq.8 (denominator ratio rho), Eq.9 (reshape, with the lambda ramp of
             Sec.4.2), Eq.10 (residual), and the literal matrix forms of Eq.2-7
             and App. A.3 for tiny inputs.
block_index  The static block mask M / kept set S (Sec.3) as CSR lists of kept
             key blocks per query block, for the local-window patterns of App. A.4.
dynamic_mask The run-time block mask (future work of Sec.6 and App. A.2): per
             (batch, head), each query block keeps itself and the top-scoring
             key blocks of the block-pooled Q K^T described in Sec.2.
schedule     The denoising-step schedule of Sec.5 composed from the attention
             definitions, with the ramp of Sec.4.2.

Every function works on float64 copies of the inputs; bf16 tensors enter as the
exact values they hold.
"""

from . import attention, block_index, dynamic_mask  # noqa: F401
