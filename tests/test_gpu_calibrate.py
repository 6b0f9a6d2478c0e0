"""The VALU issue-rate calibration library on the GPU (measurement support for
the benchmark's roofline): every instruction kind launches, reports the exact
instruction count of its launch, and a rate inside what the GPU can issue."""
import ctypes as C
import os

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.mark.gpu
def test_every_calibration_kind_runs():
    import torch
    assert torch.cuda.is_available()
    torch.cuda.init()
    lib = C.CDLL(os.path.join(ROOT, "paper_2301_04285_amd", "libtaps_calibrate.so"))
    lib.taps_calibrate_valu.restype = C.c_int
    lib.taps_calibrate_valu.argtypes = [C.c_int, C.c_uint32, C.POINTER(C.c_float),
                                        C.POINTER(C.c_double), C.POINTER(C.c_uint32)]
    lib.taps_calibrate_valu_name.restype = C.c_char_p
    cus = torch.cuda.get_device_properties(0).multi_processor_count
    iters = 200
    rates = {}
    for kind in range(lib.taps_calibrate_valu_kinds()):
        ms, n, simds = C.c_float(), C.c_double(), C.c_uint32()
        name = lib.taps_calibrate_valu_name(kind).decode()
        print(f"calibration kind {kind}: {name}", flush=True)
        assert lib.taps_calibrate_valu(kind, iters, C.byref(ms), C.byref(n), C.byref(simds)) == 0
        assert simds.value == 4 * cus
        # 8 wavefronts on each SIMD, 128 instructions per loop iteration
        assert n.value == 8 * simds.value * iters * 128
        assert ms.value > 0
        rate = n.value / (ms.value * 1e-3)
        # at most one wavefront instruction per SIMD per cycle at 2.4 GHz, and
        # at least a tenth of that
        assert 0.1 * simds.value * 2.4e9 < rate < simds.value * 2.4e9, (name, rate)
        rates[name] = rate
    # the fast class issues faster than the slow one
    assert rates["v_and_b32"] > 1.3 * rates["v_bcnt_u32_b32"]
