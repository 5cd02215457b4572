"""CPU oracle for the Sparse-Reslim routed middle-block stack.

TEST INFRASTRUCTURE ONLY.  Only ``tests/``, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of ``bench.py`` may import anything from here.  The HIP
library never calls it, and it shares no code with the HIP path: it is a plain,
slow, fp64 (numpy) restatement of what the paper defines.

Modules
-------
``numerics``  bf16 <-> fp32 conversion (round-to-nearest-even) and storage -> fp64.
``select``    random K-subset selection (Sec. 3.2) and the top-k variant.
``routing``   gather and residual-delta scatter (Eq. scatter, Sec. 3.2).
``block``     pre-LN ViT block and the adaLN-modulated block, forward and
              hand-derived backward (Sec. 3.3 block equation), in fp64.
``stack``     the n2-block middle stack (Eq. sparse_forward), the routed step
              and the dense keep=100% mode (Sec. 3.4).

Parity status of each function is stated in its module header.
"""
