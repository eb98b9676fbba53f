"""CPU oracle for the FP8-Flow-MoE expert-layer hot path.

TEST INFRASTRUCTURE ONLY.  Only ``tests/``, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of ``bench.py`` may import or call anything in this
package.  The product path (the HIP library and its Python binding) never
imports it, and this package imports nothing from the product path: the two
share no code, headers, tables or helpers.

The oracle is plain, slow and meant to be checked against the paper by eye:
numpy in float64 (the paper fixes no precision except where noted per
function), one step of the method per function, no blocking or fusion.

Modules
-------
codec   OCP FP8 E4M3 encode/decode and the bfloat16 rounding used for outputs.
quant   power-of-two tile scales, 1x128 row-wise and 128x128 block quantization,
        dequantization (paper section 3.1, scale / quantize / dequantize
        equations and the power-of-two constraint).
sat     the scaling-aware transpose (paper section 3.1, Algorithm 1 and the
        exponent-shift identity) and the naive dequantize-transpose-requantize
        conversion it replaces.
moe     fused permute+pad+quantize, grouped GEMMs (fprop/dgrad/wgrad), fused
        SwiGLU+quantize and its backward twin, unpermute (paper sections 3.2 and
        3.3).
layer   the whole expert layer forward+backward, stage by stage (section 3.2).

Parity status: every function is pinned by ``tests/test_oracle_*.py``; no
function is "parity unpinned".
"""

from . import codec, quant, sat, moe, layer  # noqa: F401
