"""The bf16 conversion instructions the step kernel rounds with agree with
the integer definitions of the two roundings on every fp32 input (GPU).

v_cvt_pk_bf16_f32 must equal round-to-nearest-even and v_cvt_sr_bf16_f32,
given the 16-bit draw in the high half of its random operand, the
stochastic rule (u + r16) >> 16, on all 2^32 bit patterns other than NaN;
the canonical quiet NaN must give the canonical bf16 NaN under both.  The
oracle defines both roundings from the value grid; this pins the hardware
to the same definitions.
"""
import ctypes

import pytest
import torch

from paper_2607_10611_amd import _build
from paper_2607_10611_amd import binding as B

pytestmark = pytest.mark.gpu


def test_bf16_conversion_instructions_match_the_definitions_exhaustively():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    B.lib()
    L = ctypes.CDLL(_build.PROBE_LIB)
    L.madd_probe_bf16_rounding.argtypes = [ctypes.c_void_p, ctypes.c_void_p]
    L.madd_probe_bf16_rounding.restype = ctypes.c_int32
    c = torch.zeros(4, dtype=torch.int64, device="cuda")
    assert L.madd_probe_bf16_rounding(c.data_ptr(), torch.cuda.current_stream().cuda_stream) == 0
    torch.cuda.synchronize()
    rne_bad, sr_bad, nan_bad, seen = c.tolist()
    assert seen == 2**32
    assert (rne_bad, sr_bad, nan_bad) == (0, 0, 0)
