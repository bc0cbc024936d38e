"""CPU oracle for the GSQ layer step.  TEST INFRASTRUCTURE ONLY.

Only ``tests/``, ``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of
``bench.py`` may import anything from this package.  The product path (the HIP
library and its Python binding) never imports, links or calls it, and the two
share no code: the oracle is written from the paper, in plain numpy, in float64
wherever the paper does not fix a precision.

Modules
-------
philox      Philox4x32-10 counter-based generator (Salmon et al., SC'11) and the
            uniform / Gumbel / normal transforms drawn from it.
gsq         The method: initialisation (Eq. 4, App. A), Gumbel-Softmax sampling
            (Alg. 1), the layer reconstruction objective (Eq. 1), its gradient,
            the Adam update, hardening (Alg. 2's final argmax step).
pack        Bit-packing of hardened codes and scales (plain group-wise layout
            and the 256-weight super-block layout).

Parity status of each function is stated in its docstring ("pinned by ..." or
"parity unpinned").
"""
