"""ctypes binding of libdycl.so: the same names as include/dycl.h.

Argument marshalling only.  The library is loaded from this package's
directory; if it is missing, importing the binding raises at once (there is
no fallback path).
"""

from __future__ import annotations

import ctypes as C
import os

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libdycl.so")

DYCL_OK = 0
STATUS = {0: "DYCL_OK", -1: "DYCL_E_INVALID", -2: "DYCL_E_SPEC", -3: "DYCL_E_WEIGHTS", -4: "DYCL_E_BATCH",
          -5: "DYCL_E_OOM", -6: "DYCL_E_HIP"}

# every symbol include/dycl.h declares
EXPORTS = ["dycl_plan_create", "dycl_run", "dycl_run_seq", "dycl_plan_set_host_mode", "dycl_last_counts", "dycl_plan_info", "dycl_profile_enable",
           "dycl_profile_read", "dycl_profile_launches", "dycl_profile_launch_label", "dycl_profile_class", "dycl_spec_check", "dycl_plan_destroy", "dycl_last_error"]
# every symbol include/dycl_ops.h declares
OPS_EXPORTS = ["dycl_op_compact_workspace", "dycl_op_compact", "dycl_op_compact_noalloc", "dycl_op_move_rows", "dycl_op_conv_packed_bytes",
               "dycl_op_conv_pack", "dycl_op_conv_workspace_bytes", "dycl_op_conv", "dycl_op_conv_maxpool",
               "dycl_op_conv_pair"]


class DyclError(RuntimeError):
    def __init__(self, code: int, msg: str):
        super().__init__(f"{STATUS.get(code, code)}: {msg}")
        self.code = code


class Record(C.Structure):
    _fields_ = [("exit_index", C.c_int32), ("iterations", C.c_int32), ("skip_mask", C.c_uint64)]


def _load():
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is not built; run `python -m paper_2307_04963_amd.build` (needs hipcc)")
    # torch carries its own HIP runtime under the same soname
    # (libamdhip64.so.7); loading torch first makes libdycl.so bind to that
    # one, so the process has a single runtime and torch's device pointers
    # and streams are valid in the library.
    import torch  # noqa: F401
    lib = C.CDLL(LIB_PATH)
    vp, i32, i64p = C.c_void_p, C.c_int, C.POINTER(C.c_int64)
    lib.dycl_plan_create.argtypes = [C.c_char_p, vp, C.c_size_t, i32, i32, C.POINTER(vp)]
    lib.dycl_plan_create.restype = i32
    lib.dycl_run.argtypes = [vp, vp, i32, vp, vp, vp, vp]
    lib.dycl_run.restype = i32
    lib.dycl_run_seq.argtypes = [vp, vp, i32, vp, vp, vp, vp, vp]
    lib.dycl_run_seq.restype = i32
    lib.dycl_plan_set_host_mode.argtypes = [vp, i32]
    lib.dycl_plan_set_host_mode.restype = i32
    lib.dycl_last_counts.argtypes = [vp, C.POINTER(C.c_int32), i32]
    lib.dycl_last_counts.restype = i32
    lib.dycl_plan_info.argtypes = [vp, i64p, i32]
    lib.dycl_plan_info.restype = i32
    lib.dycl_profile_enable.argtypes = [vp, i32]
    lib.dycl_profile_enable.restype = i32
    lib.dycl_profile_read.argtypes = [vp, C.POINTER(C.c_double), i32]
    lib.dycl_profile_read.restype = i32
    lib.dycl_profile_launches.argtypes = [vp, C.POINTER(C.c_double), i32]
    lib.dycl_profile_launches.restype = i32
    lib.dycl_profile_launch_label.argtypes = [vp, i32]
    lib.dycl_profile_launch_label.restype = C.c_char_p
    lib.dycl_profile_class.argtypes = [i32]
    lib.dycl_profile_class.restype = C.c_char_p
    lib.dycl_spec_check.argtypes = [C.c_char_p, C.c_size_t, i32, C.c_char_p, C.c_size_t]
    lib.dycl_spec_check.restype = i32
    lib.dycl_plan_destroy.argtypes = [vp]
    lib.dycl_plan_destroy.restype = None
    lib.dycl_last_error.argtypes = []
    lib.dycl_last_error.restype = C.c_char_p
    lib.dycl_op_compact_workspace.argtypes = [C.c_int64]
    lib.dycl_op_compact_workspace.restype = C.c_size_t
    lib.dycl_op_compact.argtypes = [vp, vp, C.c_int64, vp, vp, vp, vp, vp, vp, C.c_size_t, vp]
    lib.dycl_op_compact.restype = i32
    lib.dycl_op_compact_noalloc.argtypes = [vp, vp, C.c_int64, vp, vp, vp, vp, vp, vp]
    lib.dycl_op_compact_noalloc.restype = i32
    lib.dycl_op_move_rows.argtypes = [vp, vp, vp, vp, C.c_size_t, C.c_int64, vp]
    lib.dycl_op_move_rows.restype = i32
    lib.dycl_op_conv_packed_bytes.argtypes = [i32, i32, i32]
    lib.dycl_op_conv_packed_bytes.restype = C.c_size_t
    lib.dycl_op_conv_pack.argtypes = [vp, i32, i32, i32, vp, C.c_size_t]
    lib.dycl_op_conv_pack.restype = i32
    lib.dycl_op_conv_workspace_bytes.argtypes = [i32] * 8
    lib.dycl_op_conv_workspace_bytes.restype = C.c_size_t
    lib.dycl_op_conv.argtypes = [vp, i32, i32, i32, i32, vp, i32, i32, i32, i32, vp, vp, vp, i32, vp, vp, C.c_size_t,
                                 vp]
    lib.dycl_op_conv.restype = i32
    lib.dycl_op_conv_maxpool.argtypes = [vp, i32, i32, i32, i32, vp, i32, i32, i32, i32, vp, vp, i32, vp, vp]
    lib.dycl_op_conv_maxpool.restype = i32
    lib.dycl_op_conv_pair.argtypes = [vp, i32, i32, i32, i32, vp, vp, vp, vp, i32, vp, vp, vp, vp, i32, vp, vp]
    lib.dycl_op_conv_pair.restype = i32
    return lib


lib = _load()


def check(rc: int) -> int:
    if rc < 0:
        raise DyclError(rc, lib.dycl_last_error().decode())
    return rc


def last_error() -> str:
    return lib.dycl_last_error().decode()
