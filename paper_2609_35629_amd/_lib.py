"""ctypes declarations of libsantapp.so (the C ABI in include/santapp.h)."""
from __future__ import annotations

import ctypes
import os

PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(PKG, "libsantapp.so")

OK, EINVAL, EDTYPE, ENOMEM, EHIP, EWORKSPACE, ELIMIT = range(7)
BF16, FP32 = 0, 1

STATUS_NAMES = {OK: "OK", EINVAL: "EINVAL", EDTYPE: "EDTYPE", ENOMEM: "ENOMEM", EHIP: "EHIP",
                EWORKSPACE: "EWORKSPACE", ELIMIT: "ELIMIT"}

# every function include/santapp.h declares
EXPORTS = [
    "santapp_build_teams", "santapp_teams_info", "santapp_teams_destroy", "santapp_budget_to_K",
    "santapp_decode_workspace_bytes", "santapp_workspace_zero", "santapp_decode", "santapp_decode_static",
    "santapp_dense_workspace_bytes", "santapp_dense_decode", "santapp_last_error",
    "santapp_teams_set_route_keys", "santapp_routing_kl_workspace_bytes", "santapp_routing_kl",
    "santapp_kmeans_parents", "santapp_build_teams_from_labels", "santapp_decode_launch_info",
]

ROUTE_REPRESENTATIVE, ROUTE_CENTROID = 0, 1


class TeamsDesc(ctypes.Structure):
    _fields_ = [
        ("B", ctypes.c_int), ("Hkv", ctypes.c_int), ("N", ctypes.c_int), ("d", ctypes.c_int),
        ("dtype", ctypes.c_int), ("parent_size", ctypes.c_int), ("reps_per_parent", ctypes.c_int),
        ("M", ctypes.c_int),
        ("packed_K", ctypes.c_void_p), ("packed_V", ctypes.c_void_p), ("reps", ctypes.c_void_p),
        ("team_begin", ctypes.c_void_p), ("team_size", ctypes.c_void_p),
        ("log_n", ctypes.c_void_p), ("rep_token", ctypes.c_void_p), ("perm", ctypes.c_void_p),
        ("team_count", ctypes.c_void_p),
    ]


class KMeansSettings(ctypes.Structure):
    _fields_ = [
        ("batch_size", ctypes.c_int), ("max_iter", ctypes.c_int), ("max_no_improvement", ctypes.c_int),
        ("reassignment_ratio", ctypes.c_double), ("init_size", ctypes.c_int), ("seed", ctypes.c_uint64),
    ]


class DecodeDebug(ctypes.Structure):
    _fields_ = [
        ("phi", ctypes.c_void_p), ("Y", ctypes.c_void_p), ("sel", ctypes.c_void_p),
        ("logc", ctypes.c_void_p), ("tau", ctypes.c_void_p), ("union_teams", ctypes.c_void_p),
        ("union_rows", ctypes.c_void_p), ("events", ctypes.c_void_p * 4),
    ]


class SantappError(RuntimeError):
    def __init__(self, status: int, message: str):
        super().__init__(f"{STATUS_NAMES.get(status, status)}: {message}")
        self.status = status


_lib = None


def load(path: str = LIB_PATH) -> ctypes.CDLL:
    """Load the HIP library; raises if it has not been built."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise RuntimeError(
            f"{path} is missing: build the HIP library first "
            "(python -c 'import __graft_entry__ as g; g.build()')")
    L = ctypes.CDLL(path)
    vp, i, u64, sz = ctypes.c_void_p, ctypes.c_int, ctypes.c_uint64, ctypes.c_size_t
    L.santapp_build_teams.argtypes = [vp, vp, i, i, i, i, i, i, i, vp, ctypes.POINTER(vp)]
    L.santapp_teams_info.argtypes = [vp, ctypes.POINTER(TeamsDesc)]
    L.santapp_kmeans_parents.argtypes = [vp, i, i, i, i, i, i, ctypes.POINTER(KMeansSettings), vp,
                                         ctypes.POINTER(i), ctypes.POINTER(i), vp]
    L.santapp_build_teams_from_labels.argtypes = [vp, vp, i, i, i, i, i, vp, i, i, vp, ctypes.POINTER(vp)]
    L.santapp_teams_destroy.argtypes = [vp]
    L.santapp_teams_destroy.restype = None
    L.santapp_budget_to_K.argtypes = [i, i, i, i, ctypes.POINTER(i)]
    L.santapp_decode_workspace_bytes.argtypes = [vp, i, i, i, ctypes.POINTER(sz)]
    L.santapp_workspace_zero.argtypes = [vp, sz, vp]
    L.santapp_decode_launch_info.argtypes = [vp, i, i, i, ctypes.POINTER(i), ctypes.POINTER(i)]
    L.santapp_decode.argtypes = [vp, vp, vp, vp, i, i, i, i, u64, u64, ctypes.c_double, vp, vp, sz,
                                 ctypes.POINTER(DecodeDebug), vp]
    L.santapp_decode_static.argtypes = [vp, vp, vp, vp, i, i, i, i, u64, u64, ctypes.c_double, vp,
                                        ctypes.POINTER(DecodeDebug), vp]
    L.santapp_dense_workspace_bytes.argtypes = [i, i, i, i, i, i, ctypes.POINTER(sz)]
    L.santapp_dense_decode.argtypes = [vp, vp, vp, i, i, i, i, i, vp, vp, i, i, i, ctypes.c_double,
                                       vp, vp, sz, ctypes.POINTER(DecodeDebug), vp]
    L.santapp_teams_set_route_keys.argtypes = [vp, i, vp]
    L.santapp_routing_kl_workspace_bytes.argtypes = [vp, i, ctypes.POINTER(sz)]
    L.santapp_routing_kl.argtypes = [vp, vp, i, ctypes.c_double, vp, vp, sz, vp]
    L.santapp_last_error.argtypes = []
    L.santapp_last_error.restype = ctypes.c_char_p
    for name in EXPORTS:
        if name not in ("santapp_teams_destroy", "santapp_last_error"):
            getattr(L, name).restype = ctypes.c_int
    _lib = L
    return L


def check(status: int) -> None:
    if status != OK:
        msg = load().santapp_last_error().decode(errors="replace")
        raise SantappError(status, msg)
