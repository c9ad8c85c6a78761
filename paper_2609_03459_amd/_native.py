"""ctypes binding of libttemb.so (include/tt_emb.h).

Argument marshalling only: every step of the TT gather runs in the HIP
kernels of the library.  If the library has not been built this module
raises ImportError; there is no fallback path.
"""
from __future__ import annotations

import ctypes as C
import os
import re

HERE = os.path.dirname(os.path.abspath(__file__))
# TT_EMB_LIB names another build of the same library (the sanitizer test's host build)
LIB_PATH = os.environ.get("TT_EMB_LIB") or os.path.join(HERE, "libttemb.so")
HEADER = os.path.join(os.path.dirname(HERE), "include", "tt_emb.h")

TT_EMB_OK, TT_EMB_EINVAL, TT_EMB_ENOMEM, TT_EMB_EHIP, TT_EMB_ERANGE, TT_EMB_EUNSUPPORTED, TT_EMB_ESCRATCH = range(7)
NOALLOC_SCRATCH_BYTES = 64 << 20  # TT_EMB_NOALLOC_SCRATCH_BYTES
REUSE = {"prefix": 0, "unique": 1, "none": 2}
SCHED = {"steal": 0, "static": 1, "steal_ckpt": 2, "group": 3}
KERNELS = {"ingest": 1, "fwd_fused": 2, "pool": 3, "seg_sum": 4, "bwd_fused": 5, "merge": 6, "split": 7}


class tt_emb_desc(C.Structure):
    _fields_ = [
        ("num_tables", C.c_int32),
        ("num_rows", C.c_int64),
        ("row_factors", C.c_int32 * 3),
        ("dim_factors", C.c_int32 * 3),
        ("rank", C.c_int32),
        ("max_indices", C.c_int64),
        ("max_bags", C.c_int64),
    ]


MAX_CORES = 8


class tt_emb_desc_n(C.Structure):
    _fields_ = [
        ("num_tables", C.c_int32),
        ("num_rows", C.c_int64),
        ("num_cores", C.c_int32),
        ("row_factors", C.c_int32 * MAX_CORES),
        ("dim_factors", C.c_int32 * MAX_CORES),
        ("rank", C.c_int32),
        ("max_indices", C.c_int64),
        ("max_bags", C.c_int64),
    ]


if not os.path.exists(LIB_PATH):
    raise ImportError(f"{LIB_PATH} is missing: build it with `python paper_2609_03459_amd/build.py`")

lib = C.CDLL(LIB_PATH)

_P = C.c_void_p
_I64 = C.c_int64
_SIG = {
    "tt_emb_create": ([C.POINTER(tt_emb_desc), C.POINTER(_P)], C.c_int),
    "tt_emb_destroy": ([_P], C.c_int),
    "tt_emb_workspace_size": ([_P, _I64, _I64, C.POINTER(C.c_size_t)], C.c_int),
    "tt_emb_group": ([_P, _P, _I64, _P, _I64, _P, C.c_size_t, _P], C.c_int),
    "tt_emb_forward": ([_P, _P, _P, _P, _P, _I64, _P, _I64, _P, C.c_int, _P, C.c_size_t, _P], C.c_int),
    "tt_emb_backward": ([_P, _P, _P, _P, _P, _I64, _P, _I64, _P, _P, _P, _P, C.c_int, _P, C.c_size_t, _P],
                        C.c_int),
    "tt_emb_sgd": ([_P, _P, _P, _P, _P, _P, _P, C.c_float, _P], C.c_int),
    "tt_emb_backward_sgd": ([_P, _P, _P, _P, _P, _I64, _P, _I64, _P, C.c_float, C.c_int, _P, C.c_size_t, _P],
                            C.c_int),
    "tt_emb_check_errors": ([_P, _P, _P], C.c_int),
    "tt_emb_debug_grouping": ([_P, _P, _P, _P, _P, _P, _P, _P, _P, _P, _P], C.c_int),
    "tt_emb_status_string": ([C.c_int], C.c_char_p),
    "tt_emb_profile": ([_P, C.c_int, _P, _P], C.c_int),
    "tt_emb_kernel_uses_mfma": ([_P, C.c_int, C.c_int64, C.POINTER(C.c_int)], C.c_int),
    "tt_emb_set_reuse": ([_P, C.c_int], C.c_int),
    "tt_emb_set_schedule": ([_P, C.c_int], C.c_int),
    "tt_emb_create_n": ([C.POINTER(tt_emb_desc_n), C.POINTER(_P)], C.c_int),
    "tt_emb_forward_n": ([_P, _P, _P, _I64, _P, _I64, _P, C.c_int, _P, C.c_size_t, _P], C.c_int),
    "tt_emb_backward_n": ([_P, _P, _P, _I64, _P, _I64, _P, _P, C.c_int, _P, C.c_size_t, _P], C.c_int),
    "tt_emb_sgd_n": ([_P, _P, _P, C.c_float, _P], C.c_int),
    "tt_emb_forward_noalloc": ([_P, _P, _P, _P, _P, _I64, _P, _I64, _P, _P], C.c_int),
}
for _name, (_args, _res) in _SIG.items():
    _f = getattr(lib, _name)
    _f.argtypes = _args
    _f.restype = _res


def header_symbols() -> list[str]:
    """Names of the functions declared in include/tt_emb.h."""
    txt = open(HEADER).read()
    return sorted(set(re.findall(r"^\S.*?\b(tt_emb_[a-z_]+)\s*\(", txt, flags=re.M)))


def status_string(code: int) -> str:
    return lib.tt_emb_status_string(int(code)).decode()


class TTEmbError(RuntimeError):
    def __init__(self, where: str, code: int):
        super().__init__(f"{where}: {status_string(code)} ({code})")
        self.code = code


def check(where: str, code: int) -> None:
    if code != TT_EMB_OK:
        raise TTEmbError(where, code)


# thin wrappers with the C names (pointers are plain ints, stream a hipStream_t as int)
def tt_emb_create(desc: tt_emb_desc) -> int:
    h = _P()
    check("tt_emb_create", lib.tt_emb_create(C.byref(desc), C.byref(h)))
    return h.value


def tt_emb_create_n(desc: tt_emb_desc_n) -> int:
    h = _P()
    check("tt_emb_create_n", lib.tt_emb_create_n(C.byref(desc), C.byref(h)))
    return h.value


def ptr_array(ptrs):
    """Host array of device pointers (cores / grads of the L-core calls)."""
    arr = (_P * len(ptrs))(*ptrs)
    return arr


def tt_emb_forward_n(h, cores, idx, m, off, nb, out, reuse, ws, ws_bytes, stream) -> None:
    check("tt_emb_forward_n",
          lib.tt_emb_forward_n(h, ptr_array(cores), idx, m, off, nb, out, int(reuse), ws, ws_bytes, stream))


def tt_emb_backward_n(h, cores, idx, m, off, nb, dv, grads, reuse, ws, ws_bytes, stream) -> None:
    check("tt_emb_backward_n",
          lib.tt_emb_backward_n(h, ptr_array(cores), idx, m, off, nb, dv, ptr_array(grads), int(reuse), ws,
                                ws_bytes, stream))


def tt_emb_sgd_n(h, cores, grads, lr, stream) -> None:
    check("tt_emb_sgd_n", lib.tt_emb_sgd_n(h, ptr_array(cores), ptr_array(grads), float(lr), stream))


def tt_emb_destroy(h: int) -> None:
    check("tt_emb_destroy", lib.tt_emb_destroy(h))


def tt_emb_workspace_size(h: int, num_indices: int, num_bags: int) -> int:
    n = C.c_size_t()
    check("tt_emb_workspace_size", lib.tt_emb_workspace_size(h, int(num_indices), int(num_bags), C.byref(n)))
    return int(n.value)


def tt_emb_group(h, idx, m, off, nb, ws, ws_bytes, stream) -> None:
    check("tt_emb_group", lib.tt_emb_group(h, idx, m, off, nb, ws, ws_bytes, stream))


def tt_emb_forward(h, g1, g2, g3, idx, m, off, nb, out, reuse, ws, ws_bytes, stream) -> None:
    check("tt_emb_forward", lib.tt_emb_forward(h, g1, g2, g3, idx, m, off, nb, out, int(reuse), ws, ws_bytes, stream))


def tt_emb_backward(h, g1, g2, g3, idx, m, off, nb, dv, dg1, dg2, dg3, reuse, ws, ws_bytes, stream) -> None:
    check("tt_emb_backward",
          lib.tt_emb_backward(h, g1, g2, g3, idx, m, off, nb, dv, dg1, dg2, dg3, int(reuse), ws, ws_bytes, stream))


def tt_emb_sgd(h, g1, g2, g3, dg1, dg2, dg3, lr, stream) -> None:
    check("tt_emb_sgd", lib.tt_emb_sgd(h, g1, g2, g3, dg1, dg2, dg3, float(lr), stream))


def tt_emb_backward_sgd(h, g1, g2, g3, idx, m, off, nb, dv, lr, reuse, ws, wsb, stream) -> None:
    check("tt_emb_backward_sgd",
          lib.tt_emb_backward_sgd(h, g1, g2, g3, idx, m, off, nb, dv, float(lr), int(reuse), ws, wsb, stream))


def tt_emb_check_errors(h, ws, stream) -> int:
    return int(lib.tt_emb_check_errors(h, ws, stream))


def tt_emb_set_reuse(h, level: int) -> None:
    check("tt_emb_set_reuse", lib.tt_emb_set_reuse(h, int(level)))


def tt_emb_set_schedule(h, mode: int) -> None:
    check("tt_emb_set_schedule", lib.tt_emb_set_schedule(h, int(mode)))


def tt_emb_profile(h, kernel: int, ev_begin, ev_end) -> None:
    check("tt_emb_profile", lib.tt_emb_profile(h, int(kernel), ev_begin, ev_end))


def tt_emb_kernel_uses_mfma(h, kernel: int, num_indices: int) -> bool:
    flag = C.c_int(-1)
    check("tt_emb_kernel_uses_mfma", lib.tt_emb_kernel_uses_mfma(h, int(kernel), int(num_indices), C.byref(flag)))
    return bool(flag.value)


def tt_emb_forward_noalloc(h, g1, g2, g3, idx, m, off, nb, out, stream) -> None:
    check("tt_emb_forward_noalloc", lib.tt_emb_forward_noalloc(h, g1, g2, g3, idx, m, off, nb, out, stream))
