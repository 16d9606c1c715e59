"""CPU oracle for the Fairy2i widely-linear layer -- test infrastructure only.

Only ``tests/``, ``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of
``bench.py`` may import this package.  It shares no code with the HIP library
or its binding and imports neither.
"""
from .fairy2i import *  # noqa: F401,F403
from .fairy2i import (CODEWORDS, axis_scales, code_planes, combine_accumulators,  # noqa: F401
                      dense_real_matrix, dequantize, dequantize_stage, exact_sum,
                      int8_accumulators, int8_as_complex, pack, project, quantize,
                      quantize_act_int8, quantize_with_residuals, realify_conj,
                      realify_lin, round_to_f32, stack_real, to_widely_linear,
                      to_widely_linear_f64, unpack, wl_matmul, wl_matmul_int8)
from . import block  # noqa: F401,E402
from . import groups  # noqa: F401,E402
from . import qat  # noqa: F401,E402
