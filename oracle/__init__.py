"""Plain, slow float64 CPU oracle for the WitCert hot path.

TEST INFRASTRUCTURE ONLY.  Only ``tests/``, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of ``bench.py`` may import this package.  It shares no code
with the HIP path (``paper_2607_28699_amd``) and neither imports the other; the
seeded input generators in ``synth`` are the only common dependency.

Every function follows one passage of the paper (cited by section, equation,
theorem or table) and is written for reading against it, not for speed:

* ``philox``     Philox4x32-10 (Salmon et al., SC'11), the counter-based dither
                 source named in Sec. 6.2 (research kernels) and Sec. 6.2
                 (storage side: slot-keyed counter).
* ``fpformats``  fp32 / fp16 / bf16 / fp8-e4m3 roundings used by the stored cache.
* ``quantizer``  subtractive-dither INT8 quantizer (Sec. 4.2), raw fp8 cast
                 (black-box scheme), band map and residual witness (Sec. 4.1,
                 Eq. witness, Lemma RoPE band unitarity).
* ``attention``  exact and compressed softmax attention, total variation (Sec. 3).
* ``meter``      per-token logit bound (Theorem black-box logit bound), e-form
                 TV bound (Theorem sound replacement), saturation reporting
                 (Sec. 4.3), the flawed certificate (Eq. flawed) and the
                 two-sided form (Proposition two-sided) for regression tests.
* ``tierb``      Tier-B sub-Gaussian certificate of the dithered cache (Sec. 4.2:
                 Lemma uniform sub-Gaussian proxy, radius, request-level budget).
* ``bypass``     fixed-channel outlier-pair bypass of the key cache with the
                 bypassed channels out of the amax (Sec. 4.2 outlier RoPE pairs;
                 Sec. 6.2 fixed-channel bypass, Tables 5 and 6).
* ``groupscale`` per-token scales over 32-channel groups (Sec. 6.2 storage
                 side, Table 4): one fp16 scale per token and group, the
                 quantizer with them, and the Tier-B radius it implies.
* ``value``      value side: the output bound of Sec. 3, the value meter and the
                 joint K+V gate (Sec. 4.2 value side and joint event).
* ``repair``     block-granular repair of gated heads (Sec. 6.3, block-level
                 paging): block shares of A - 1, the repair order, the repaired
                 state and the stop rule.
* ``gate``       threshold gate and exact fallback (the meter loop, Sec. 6).
* ``decode``     one metered decode of a batch over per-token caches, composed
                 from the above.

Parity status of each function is listed in its docstring; every function is
pinned by a CPU test in ``tests/test_oracle_*.py``.
"""
from . import (attention, bypass, decode, fpformats, gate, groupscale, meter, philox, quantizer,  # noqa: F401
               repair, tierb, value)
