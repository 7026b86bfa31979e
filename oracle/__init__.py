"""CPU oracle for FP8 in-context-learning attention -- TEST INFRASTRUCTURE ONLY.

A plain, slow, obviously-correct fp64 (numpy) statement of what the GPU path
computes, written from "Attention Quantization for Tabular Foundation Models"
(Kuebler, Jaeger, Floege, Hollmann, Hutter):

* ``e4m3``      -- the OCP FP8 E4M3 ("e4m3fn") codec, the format that Sec. 3
                   (Method) quantizes Q, K, V and P to.
* ``quantize``  -- per-head dynamic absmax quantization, Eq. (2), with the
                   test queries reusing the train-query scale (Sec. 3, last
                   paragraph before Fig. 2), or on the per-call and joint
                   query scales the paper compares (Table 1; appendix).
* ``attention`` -- Eq. (1) in fp64 on exact inputs and on the dequantized
                   inputs, and a replay of the one-pass fused kernel of
                   Sec. 3 / Fig. 2 (Q and K scales folded into the softmax
                   scale, P lifted to 2^8 and rounded to e4m3 in-kernel, V
                   scale applied in the epilogue), with optional
                   grouped-query test rows (appendix).
* ``noise``     -- the per-head RMS-scaled Gaussian perturbation, Eq. (3).

Only ``tests/``, ``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of
``bench.py`` may import this package.  It imports nothing from the GPU
library and the GPU library never calls it: the two share no code.  Every
function is pinned by the ``-m "not gpu"`` tests against facts that do not
come from this package (a library FP8 cast, closed forms, brute force, the
paper's printed quantization error); there is no unpinned function.
"""
from . import e4m3, quantize, attention, noise  # noqa: F401
