"""CPU oracle for the 1-bit FQT layer backward (AGP + SCQ + binary products).

TEST INFRASTRUCTURE ONLY.  This package is a plain, slow, step-by-step
restatement of the method of "1-Bit FQT: Pushing the Limit of Fully Quantized
Training to 1-bit" (Gao et al., arXiv 2408.14267).  Only ``tests/``,
``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of ``bench.py`` may
import it.  It shares no code with the HIP library and never imports it; the
library must not route through it.

Modules
-------
philox : Philox4x32-10 counter-based generator (Salmon, Moraes, Dror, Shaw,
         "Parallel random numbers: as easy as 1, 2, 3", SC'11), written from that
         paper's definition.  The method's stochastic rounding and Bernoulli
         pruning draw their random words from it.
fqt    : the method itself -- group statistics, AGP probabilities and masks,
         SCQ stochastic rounding, bit-plane decomposition and packing, the two
         integer contractions and the per-group rescale (Sections 3.2, 5.2,
         5.3 and Appendix C of the paper).

Parity status of each function, and the reading taken where the paper is silent,
are stated in its docstring.
"""
