"""Python binding of libhwsel.so (ctypes).

The functions carry the C ABI's names and only marshal arguments: torch
tensors in device memory become raw pointers, the current torch stream
becomes the hipStream_t.  Every step of the scored path runs in the HIP
library; there is no fallback of any kind -- if the library is missing the
call raises.
"""
from __future__ import annotations

import ctypes as C
import os

import numpy as np
import torch

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libhwsel.so")
HEADER = os.path.join(os.path.dirname(HERE), "include", "hwsel.h")

HWSEL_OK, HWSEL_EINVAL, HWSEL_EUNSUPPORTED, HWSEL_EHIP = 0, 1, 2, 3


class HwselError(RuntimeError):
    def __init__(self, fn: str, status: int, detail: str):
        super().__init__(f"{fn} -> {status} ({detail})")
        self.status = status


class hwsel_hw_t(C.Structure):
    _fields_ = [(n, C.c_int64) for n in (
        "n_sm", "smem_per_sm", "smem_per_block_max", "smem_reserved", "regs_per_sm",
        "max_regs_per_thread", "max_blocks_per_sm", "max_threads_per_sm", "arch_id",
        "llc_bytes", "hbm_bw_gbps")] + [("peak_gflops", C.c_int64 * 3)]


CAND_FIELDS = ("tile_m", "tile_n", "tile_k", "inst_n", "stages", "cluster_m", "cluster_n", "swizzle",
               "inst_m_div16", "inst_k", "kernel_sched", "epi_sched", "tile_sched")


class hwsel_cands_t(C.Structure):
    _fields_ = [(n, C.c_void_p) for n in CAND_FIELDS]


class hwsel_forest_t(C.Structure):
    _fields_ = [("n_trees", C.c_int32), ("depth", C.c_int32), ("n_features", C.c_int32),
                ("flags", C.c_uint32), ("base_score", C.c_float), ("node_feature", C.c_void_p),
                ("node_threshold", C.c_void_p), ("leaf_value", C.c_void_p)]


class hwsel_mlp_t(C.Structure):
    _fields_ = [("n_in", C.c_int32), ("h1", C.c_int32), ("h2", C.c_int32), ("h3", C.c_int32),
                ("mean", C.c_void_p), ("inv_std", C.c_void_p), ("W1", C.c_void_p), ("W2", C.c_void_p),
                ("W3", C.c_void_p), ("W4", C.c_void_p), ("b1", C.c_void_p), ("b2", C.c_void_p),
                ("b3", C.c_void_p), ("b4", C.c_void_p)]


class hwsel_cands_out_t(C.Structure):
    _fields_ = [(n, C.c_void_p) for n in CAND_FIELDS]


class hwsel_linear_t(C.Structure):
    _fields_ = [("n_features", C.c_int32), ("bias", C.c_float), ("mean", C.c_void_p), ("inv_std", C.c_void_p),
                ("w", C.c_void_p), ("w_onehot", C.c_void_p)]


_lib = None


def lib() -> C.CDLL:
    """Load the HIP library; raise if it has not been built."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it with "
                               "`python paper_2609_35587_amd/build.py` (there is no CPU fallback)")
        L = C.CDLL(LIB_PATH)
        L.hwsel_status_string.restype = C.c_char_p
        L.hwsel_last_error.restype = C.c_char_p
        vp, i32, i64 = C.c_void_p, C.c_int32, C.c_int64
        L.hwsel_features.argtypes = [hwsel_hw_t, vp, i32, vp, C.POINTER(hwsel_cands_t), i64, i32, vp, i64, vp]
        L.hwsel_forest_score.argtypes = [C.POINTER(hwsel_forest_t), vp, vp, i64, i64, vp, vp, C.c_size_t, vp]
        L.hwsel_forest_pack_bytes.argtypes = [C.POINTER(hwsel_forest_t), C.POINTER(C.c_size_t)]
        L.hwsel_forest_pack.argtypes = [C.POINTER(hwsel_forest_t), vp, C.c_size_t, vp]
        L.hwsel_forest_pack_host.argtypes = [C.POINTER(hwsel_forest_t), vp, C.c_size_t]
        L.hwsel_forest_workspace_bytes.argtypes = [C.POINTER(hwsel_forest_t), i64, C.POINTER(C.c_size_t)]
        L.hwsel_forest_score_checked.argtypes = [C.POINTER(hwsel_forest_t), vp, vp, i64, i64, vp, vp, C.c_size_t,
                                                 vp, vp, i64, i64, vp]
        L.hwsel_forest_leaves.argtypes = [C.POINTER(hwsel_forest_t), vp, i64, i64, vp, i64, vp, vp]
        L.hwsel_mlp_score.argtypes = [C.POINTER(hwsel_mlp_t), vp, vp, i64, i64, vp, vp]
        L.hwsel_mlp_pack_bytes.argtypes = [C.POINTER(hwsel_mlp_t), C.POINTER(C.c_size_t)]
        L.hwsel_mlp_pack.argtypes = [C.POINTER(hwsel_mlp_t), vp, C.c_size_t, vp]
        L.hwsel_topk_per_problem.argtypes = [vp, vp, i32, i32, vp, vp, vp]
        L.hwsel_regret.argtypes = [vp, vp, i32, vp, i32, vp, vp, vp, vp]
        L.hwsel_linear_score.argtypes = [C.POINTER(hwsel_linear_t), vp, i64, i64, vp, vp]
        sz = C.c_size_t
        L.hwsel_select_forest_workspace_bytes.argtypes = [C.POINTER(hwsel_forest_t), i64, C.POINTER(sz)]
        L.hwsel_select_forest.argtypes = [hwsel_hw_t, vp, i32, vp, C.POINTER(hwsel_cands_t), i64, i32,
                                          C.POINTER(hwsel_forest_t), vp, i32, vp, vp, vp, vp, sz, vp]
        L.hwsel_evaluate_workspace_bytes.argtypes = [i32, C.POINTER(sz)]
        L.hwsel_evaluate.argtypes = [vp, vp, i32, vp, i32, vp, vp, vp, vp, vp, sz, vp]
        L.hwsel_evaluate_noalloc.argtypes = [vp, vp, i32, vp, i32, vp, vp, vp, vp, vp]
        L.hwsel_static_config_workspace_bytes.argtypes = [i32, i32, C.POINTER(sz)]
        L.hwsel_static_config.argtypes = [vp, vp, i32, vp, i32, vp, vp, vp, sz, vp]
        L.hwsel_catalogue_mask.argtypes = [hwsel_hw_t, vp, i32, C.c_uint32, vp, vp, vp]
        L.hwsel_catalogue_compact.argtypes = [vp, vp, i32, vp, vp, i64, vp]
        L.hwsel_catalogue_candidates.argtypes = [vp, i32, vp, vp, i64, C.POINTER(hwsel_cands_out_t), vp]
        L.hwsel_sample_score.argtypes = [hwsel_hw_t, vp, i32, vp, C.POINTER(hwsel_cands_t), i64, vp, vp]
        _lib = L
    return _lib


def _check(fn: str, status: int) -> None:
    if status != HWSEL_OK:
        raise HwselError(fn, status, lib().hwsel_last_error().decode())


def _ptr(t) -> int | None:
    if t is None:
        return None
    if isinstance(t, int):
        return t
    return t.data_ptr()


def _stream(stream) -> int | None:
    if stream is None:
        return torch.cuda.current_stream().cuda_stream
    if isinstance(stream, int):
        return stream
    return stream.cuda_stream


def _dev(t: torch.Tensor, name: str) -> torch.Tensor:
    if not isinstance(t, torch.Tensor) or not t.is_cuda or not t.is_contiguous():
        raise ValueError(f"{name} must be a contiguous device tensor")
    return t


def _arg(t, name: str, dtypes, numel: int = 0, like: torch.Tensor | None = None) -> torch.Tensor:
    """A caller-supplied buffer the library reads or writes: a contiguous
    device tensor (on the same device as ``like``) of one of ``dtypes`` with
    at least ``numel`` elements.  Raises ValueError before anything runs."""
    t = _dev(t, name)
    if like is not None and t.device != like.device:
        raise ValueError(f"{name} is on {t.device}, the other operands on {like.device}")
    if t.dtype not in dtypes:
        raise ValueError(f"{name} has dtype {t.dtype}, expected one of {tuple(dtypes)}")
    if t.numel() < numel:
        raise ValueError(f"{name} holds {t.numel()} elements, {numel} needed")
    return t


def _matrix(X, name: str, cols: int, like: torch.Tensor | None = None) -> torch.Tensor:
    """A row-major fp32 matrix [R][ld] with ld >= cols (a column slice of a
    wider buffer is fine): rows are read or written ld apart."""
    if not isinstance(X, torch.Tensor) or not X.is_cuda or X.dim() != 2:
        raise ValueError(f"{name} must be a 2-D device tensor")
    if like is not None and X.device != like.device:
        raise ValueError(f"{name} is on {X.device}, the other operands on {like.device}")
    if X.dtype != torch.float32 or X.stride(1) != 1 or X.shape[1] < cols or X.stride(0) < cols:
        raise ValueError(f"{name} must be fp32 [R][>= {cols}] with unit column stride")
    return X


F32, I32, I64 = (torch.float32,), (torch.int32,), (torch.int64,)
U8 = (torch.uint8,)
U16 = (torch.int16, torch.uint16) if hasattr(torch, "uint16") else (torch.int16,)


# ----------------------------------------------------------------------------
# Marshalling helpers (numpy -> device tensors); no arithmetic of the path.
# ----------------------------------------------------------------------------
def to_device(a: np.ndarray, device="cuda") -> torch.Tensor:
    a = np.ascontiguousarray(a)
    if a.dtype == np.uint16:
        a = a.view(np.int16)
    elif a.dtype.fields is not None:
        a = a.view(np.uint8).reshape(len(a), -1)
    return torch.from_numpy(a).to(device)


def hw_struct(hw: dict) -> hwsel_hw_t:
    s = hwsel_hw_t()
    for n, _ in hwsel_hw_t._fields_[:-1]:
        setattr(s, n, int(hw[n]))
    for i, v in enumerate(hw["peak_gflops"]):
        s.peak_gflops[i] = int(v)
    return s


# ----------------------------------------------------------------------------
# Entry points
# ----------------------------------------------------------------------------
def hwsel_features(hw: dict, problems: torch.Tensor, seg_offsets: torch.Tensor, cands: dict,
                   n_features: int, X: torch.Tensor | None = None, stream=None) -> torch.Tensor:
    """problems: uint8 [P, 16] device records; seg_offsets int64 [P+1];
    cands: name -> device tensor of length R.  Returns X fp32 [R, ld]."""
    P = problems.shape[0]
    R = cands["tile_m"].shape[0]
    if X is None:
        X = torch.empty((R, n_features), dtype=torch.float32, device=problems.device)
    _matrix(X, "X", n_features, like=problems)
    if X.shape[0] < R:
        raise ValueError(f"X has {X.shape[0]} rows, {R} candidates")
    cs = _cands_struct(cands, R, problems)
    _check("hwsel_features", lib().hwsel_features(
        hw_struct(hw), _ptr(_dev(problems, "problems")), P, _ptr(_dev(seg_offsets, "seg_offsets")),
        C.byref(cs), R, n_features, _ptr(X), X.stride(0), _stream(stream)))
    return X


def _cands_struct(cands: dict, R: int, like: torch.Tensor) -> hwsel_cands_t:
    wide = ("tile_m", "tile_n", "tile_k", "inst_n")
    for n in CAND_FIELDS:
        _arg(cands[n], n, U16 if n in wide else U8, R, like)
    return hwsel_cands_t(*[_ptr(cands[n]) for n in CAND_FIELDS])


def hwsel_sample_score(hw: dict, problems: torch.Tensor, seg_offsets: torch.Tensor, cands: dict,
                       scores: torch.Tensor | None = None, stream=None) -> torch.Tensor:
    """The analytic sampling score per row (no feature matrix)."""
    P = problems.shape[0]
    R = cands["tile_m"].shape[0]
    if scores is None:
        scores = torch.empty(R, dtype=torch.float32, device=problems.device)
    _arg(scores, "scores", F32, R, problems)
    cs = _cands_struct(cands, R, problems)
    _check("hwsel_sample_score", lib().hwsel_sample_score(
        hw_struct(hw), _ptr(_dev(problems, "problems")), P, _ptr(_dev(seg_offsets, "seg_offsets")),
        C.byref(cs), R, _ptr(scores), _stream(stream)))
    return scores


def linear_struct(m: dict) -> hwsel_linear_t:
    return hwsel_linear_t(int(m["n_features"]), float(m["bias"]), _ptr(m["mean"]), _ptr(m["inv_std"]),
                          _ptr(m["w"]), _ptr(m["w_onehot"]))


def hwsel_linear_score(lin: dict, X: torch.Tensor, scores: torch.Tensor | None = None,
                       stream=None) -> torch.Tensor:
    R = X.shape[0]
    F = int(lin["n_features"])
    _matrix(X, "X", F)
    if scores is None:
        scores = torch.empty(R, dtype=torch.float32, device=X.device)
    _arg(scores, "scores", F32, R, X)
    for n in ("mean", "inv_std", "w"):
        _arg(lin[n], n, F32, F, X)
    _arg(lin["w_onehot"], "w_onehot", F32, 12, X)
    s = linear_struct(lin)
    _check("hwsel_linear_score", lib().hwsel_linear_score(C.byref(s), _ptr(X), R, X.stride(0), _ptr(scores),
                                                          _stream(stream)))
    return scores


def forest_struct(f: dict) -> hwsel_forest_t:
    return hwsel_forest_t(int(f["n_trees"]), int(f["depth"]), int(f["n_features"]), int(f["flags"]),
                          float(f["base_score"]), _ptr(f["node_feature"]), _ptr(f["node_threshold"]),
                          _ptr(f["leaf_value"]))


def hwsel_forest_pack_bytes(forest: dict) -> int:
    n = C.c_size_t(0)
    s = forest_struct(forest)
    _check("hwsel_forest_pack_bytes", lib().hwsel_forest_pack_bytes(C.byref(s), C.byref(n)))
    return int(n.value)


def hwsel_forest_pack(forest: dict, packed: torch.Tensor | None = None, stream=None) -> torch.Tensor:
    """Pack a device-resident forest once; returns the packed image (uint8)."""
    nbytes = hwsel_forest_pack_bytes(forest)
    _forest_arrays(forest)
    if packed is None:
        packed = torch.empty(nbytes, dtype=torch.uint8, device=forest["node_feature"].device)
    _arg(packed, "packed", U8, nbytes, forest["node_feature"])
    s = forest_struct(forest)
    _check("hwsel_forest_pack", lib().hwsel_forest_pack(C.byref(s), _ptr(packed), packed.numel(),
                                                        _stream(stream)))
    return packed


def _forest_arrays(forest: dict) -> None:
    T, d = int(forest["n_trees"]), int(forest["depth"])
    if not 1 <= d <= 12 or T < 1:
        return                                    # the library rejects the shape itself
    n_int = ((1 << d) - 1) * T
    ref = _arg(forest["node_feature"], "node_feature", U8, n_int)
    _arg(forest["node_threshold"], "node_threshold", F32, n_int, ref)
    _arg(forest["leaf_value"], "leaf_value", F32, (1 << d) * T, ref)


def _packed_image(forest: dict, packed: torch.Tensor, like: torch.Tensor) -> None:
    _arg(packed, "packed", U8, hwsel_forest_pack_bytes(forest), like)


def hwsel_forest_pack_host(forest: dict) -> np.ndarray:
    """The packed image of a forest given as host numpy arrays, built on the
    host (no GPU needed); returns it as uint8 numpy array."""
    arrays = {n: np.ascontiguousarray(forest[n], dt) for n, dt in
              (("node_feature", np.uint8), ("node_threshold", np.float32), ("leaf_value", np.float32))}
    f = dict(forest, **{n: a.ctypes.data for n, a in arrays.items()})
    n = C.c_size_t(0)
    s = forest_struct(f)
    _check("hwsel_forest_pack_bytes", lib().hwsel_forest_pack_bytes(C.byref(s), C.byref(n)))
    image = np.zeros(int(n.value), np.uint8)
    _check("hwsel_forest_pack_host", lib().hwsel_forest_pack_host(C.byref(s), image.ctypes.data, image.size))
    return image


def hwsel_forest_workspace_bytes(forest: dict, R: int) -> int:
    n = C.c_size_t(0)
    s = forest_struct(forest)
    _check("hwsel_forest_workspace_bytes", lib().hwsel_forest_workspace_bytes(C.byref(s), R, C.byref(n)))
    return int(n.value)


def hwsel_forest_score(forest: dict, X: torch.Tensor, scores: torch.Tensor | None = None,
                       packed: torch.Tensor | None = None, workspace: torch.Tensor | None = None,
                       stream=None) -> torch.Tensor:
    """Score rows of X.  With ``packed`` (from hwsel_forest_pack) the fast
    path runs and ``workspace`` (allocated here if None) holds its bins and
    partial sums."""
    R = X.shape[0]
    _matrix(X, "X", int(forest["n_features"]))
    _forest_arrays(forest)
    if scores is None:
        scores = torch.empty(R, dtype=torch.float32, device=X.device)
    _arg(scores, "scores", F32, R, X)
    ws_bytes = 0
    if packed is not None:
        _packed_image(forest, packed, X)
        if workspace is None:
            workspace = torch.empty(hwsel_forest_workspace_bytes(forest, R), dtype=torch.uint8, device=X.device)
        _arg(workspace, "workspace", U8, 0, X)
        ws_bytes = workspace.numel() * workspace.element_size()
    s = forest_struct(forest)
    _check("hwsel_forest_score", lib().hwsel_forest_score(
        C.byref(s), _ptr(packed), _ptr(X), R, X.stride(0), _ptr(scores), _ptr(workspace), ws_bytes,
        _stream(stream)))
    return scores


def hwsel_forest_score_checked(forest: dict, X: torch.Tensor, packed: torch.Tensor, with_hash: bool = True,
                               leaf_rows: tuple[int, int] | None = None, scores: torch.Tensor | None = None,
                               workspace: torch.Tensor | None = None, stream=None):
    """The packed traversal with its check outputs.  Returns (scores, leaf_hash
    uint64-as-int64 [R] or None, leaf_idx int16 [n][T] for the row range
    ``leaf_rows`` = (row0, n) or None)."""
    R = X.shape[0]
    _matrix(X, "X", int(forest["n_features"]))
    _forest_arrays(forest)
    _packed_image(forest, packed, X)
    if scores is None:
        scores = torch.empty(R, dtype=torch.float32, device=X.device)
    _arg(scores, "scores", F32, R, X)
    if workspace is None:
        workspace = torch.empty(hwsel_forest_workspace_bytes(forest, R), dtype=torch.uint8, device=X.device)
    _arg(workspace, "workspace", U8, 0, X)
    lh = torch.empty(R, dtype=torch.int64, device=X.device) if with_hash else None
    li, row0, n = None, 0, 0
    if leaf_rows is not None:
        row0, n = leaf_rows
        li = torch.empty((n, int(forest["n_trees"])), dtype=torch.int16, device=X.device)
    s = forest_struct(forest)
    _check("hwsel_forest_score_checked", lib().hwsel_forest_score_checked(
        C.byref(s), _ptr(packed), _ptr(X), R, X.stride(0), _ptr(scores), _ptr(workspace),
        workspace.numel() * workspace.element_size(), _ptr(lh), _ptr(li), row0, n, _stream(stream)))
    return scores, lh, li


def hwsel_forest_leaves(forest: dict, X: torch.Tensor, rows: torch.Tensor,
                        leaf_idx: torch.Tensor | None = None, stream=None) -> torch.Tensor:
    n = rows.shape[0]
    _matrix(X, "X", int(forest["n_features"]))
    _forest_arrays(forest)
    _arg(rows, "rows", I64, 0, X)
    if leaf_idx is None:
        leaf_idx = torch.empty((n, int(forest["n_trees"])), dtype=torch.int16, device=X.device)
    _arg(leaf_idx, "leaf_idx", U16, n * int(forest["n_trees"]), X)
    s = forest_struct(forest)
    _check("hwsel_forest_leaves", lib().hwsel_forest_leaves(
        C.byref(s), _ptr(X), X.shape[0], X.stride(0), _ptr(_dev(rows, "rows")), n, _ptr(leaf_idx),
        _stream(stream)))
    return leaf_idx


def mlp_struct(m: dict) -> hwsel_mlp_t:
    return hwsel_mlp_t(128, 512, 512, 256, *[_ptr(m[n]) for n in
                                             ("mean", "inv_std", "W1", "W2", "W3", "W4", "b1", "b2", "b3", "b4")])


def hwsel_mlp_pack(mlp: dict, packed: torch.Tensor | None = None, stream=None) -> torch.Tensor:
    """Arrange W1..W3 once for the matrix-core kernel; returns the image."""
    _mlp_arrays(mlp)
    s = mlp_struct(mlp)
    n = C.c_size_t(0)
    _check("hwsel_mlp_pack_bytes", lib().hwsel_mlp_pack_bytes(C.byref(s), C.byref(n)))
    if packed is None:
        packed = torch.empty(int(n.value), dtype=torch.uint8, device=mlp["W1"].device)
    _arg(packed, "packed", U8, int(n.value), mlp["W1"])
    _check("hwsel_mlp_pack", lib().hwsel_mlp_pack(C.byref(s), _ptr(packed), packed.numel(), _stream(stream)))
    return packed


def _mlp_arrays(mlp: dict) -> None:
    sizes = dict(mean=128, inv_std=128, W1=512 * 128, W2=512 * 512, W3=256 * 512, W4=256, b1=512, b2=512, b3=256,
                 b4=1)
    ref = mlp["W1"]
    for n, k in sizes.items():
        _arg(mlp[n], n, U16 if n.startswith("W") else F32, k, ref)


def hwsel_mlp_score(mlp: dict, X: torch.Tensor, scores: torch.Tensor | None = None,
                    packed: torch.Tensor | None = None, stream=None) -> torch.Tensor:
    R = X.shape[0]
    _matrix(X, "X", 128)
    _mlp_arrays(mlp)
    if scores is None:
        scores = torch.empty(R, dtype=torch.float32, device=X.device)
    _arg(scores, "scores", F32, R, X)
    if packed is not None:
        n = C.c_size_t(0)
        _check("hwsel_mlp_pack_bytes", lib().hwsel_mlp_pack_bytes(C.byref(mlp_struct(mlp)), C.byref(n)))
        _arg(packed, "packed", U8, int(n.value), X)
    s = mlp_struct(mlp)
    _check("hwsel_mlp_score", lib().hwsel_mlp_score(C.byref(s), _ptr(packed), _ptr(X), R, X.stride(0),
                                                    _ptr(scores), _stream(stream)))
    return scores


def hwsel_topk_per_problem(scores: torch.Tensor, seg_offsets: torch.Tensor, k: int,
                           idx: torch.Tensor | None = None, vals: torch.Tensor | None = None,
                           with_vals: bool = True, stream=None):
    P = seg_offsets.shape[0] - 1
    _arg(scores, "scores", F32)
    _arg(seg_offsets, "seg_offsets", I64, 1, scores)
    if idx is None:
        idx = torch.empty((P, k), dtype=torch.int32, device=scores.device)
    if vals is None and with_vals:
        vals = torch.empty((P, k), dtype=torch.float32, device=scores.device)
    _arg(idx, "idx", I32, P * k, scores)
    if vals is not None:
        _arg(vals, "vals", F32, P * k, scores)
    _check("hwsel_topk_per_problem", lib().hwsel_topk_per_problem(
        _ptr(_dev(scores, "scores")), _ptr(_dev(seg_offsets, "seg_offsets")), P, k, _ptr(idx), _ptr(vals),
        _stream(stream)))
    return idx, vals


def hwsel_regret(runtimes: torch.Tensor, seg_offsets: torch.Tensor, idx: torch.Tensor,
                 r1: torch.Tensor | None = None, rk: torch.Tensor | None = None,
                 best: torch.Tensor | None = None, stream=None):
    P, k = idx.shape
    dev = runtimes.device
    _arg(runtimes, "runtimes", F32)
    _arg(seg_offsets, "seg_offsets", I64, P + 1, runtimes)
    _arg(idx, "idx", I32, P * k, runtimes)
    r1 = torch.empty(P, dtype=torch.float32, device=dev) if r1 is None else r1
    rk = torch.empty(P, dtype=torch.float32, device=dev) if rk is None else rk
    best = torch.empty(P, dtype=torch.int32, device=dev) if best is None else best
    _arg(r1, "r1", F32, P, runtimes)
    _arg(rk, "rk", F32, P, runtimes)
    _arg(best, "best", I32, P, runtimes)
    _check("hwsel_regret", lib().hwsel_regret(
        _ptr(_dev(runtimes, "runtimes")), _ptr(_dev(seg_offsets, "seg_offsets")), P, _ptr(_dev(idx, "idx")), k,
        _ptr(r1), _ptr(rk), _ptr(best), _stream(stream)))
    return r1, rk, best


def hwsel_select_forest_workspace_bytes(forest: dict, R: int) -> int:
    n = C.c_size_t(0)
    s = forest_struct(forest)
    _check("hwsel_select_forest_workspace_bytes", lib().hwsel_select_forest_workspace_bytes(C.byref(s), R,
                                                                                            C.byref(n)))
    return int(n.value)


def hwsel_select_forest(hw: dict, problems: torch.Tensor, seg_offsets: torch.Tensor, cands: dict, n_features: int,
                        forest: dict, packed: torch.Tensor, k: int, workspace: torch.Tensor | None = None,
                        idx: torch.Tensor | None = None, vals: torch.Tensor | None = None,
                        scores: torch.Tensor | None = None, with_vals: bool = True, stream=None):
    """Fused features -> packed forest -> top-k; returns (idx, vals, scores)."""
    P = problems.shape[0]
    R = cands["tile_m"].shape[0]
    dev = problems.device
    _forest_arrays(forest)
    _packed_image(forest, packed, problems)
    if workspace is None:
        workspace = torch.empty(hwsel_select_forest_workspace_bytes(forest, R), dtype=torch.uint8, device=dev)
    _arg(workspace, "workspace", U8, 0, problems)
    if idx is None:
        idx = torch.empty((P, k), dtype=torch.int32, device=dev)
    if vals is None and with_vals:
        vals = torch.empty((P, k), dtype=torch.float32, device=dev)
    _arg(idx, "idx", I32, P * k, problems)
    if vals is not None:
        _arg(vals, "vals", F32, P * k, problems)
    if scores is not None:
        _arg(scores, "scores", F32, R, problems)
    cs = _cands_struct(cands, R, problems)
    f = forest_struct(forest)
    _check("hwsel_select_forest", lib().hwsel_select_forest(
        hw_struct(hw), _ptr(_dev(problems, "problems")), P, _ptr(_dev(seg_offsets, "seg_offsets")), C.byref(cs), R,
        n_features, C.byref(f), _ptr(packed), k, _ptr(idx), _ptr(vals), _ptr(scores), _ptr(workspace),
        workspace.numel(), _stream(stream)))
    return idx, vals, scores


HWSEL_EVAL_FIELDS = 9
HWSEL_CATALOGUE_SIZE = 534600


def hwsel_evaluate(runtimes: torch.Tensor, seg_offsets: torch.Tensor, idx: torch.Tensor,
                   workspace: torch.Tensor | None = None, per_group: bool = True, stream=None):
    """Returns (out fp64 [9], regret fp64 [P], rank int32 [P], ybar fp64 [P]);
    the per-group arrays are None unless per_group."""
    P, k = idx.shape
    dev = runtimes.device
    n = C.c_size_t(0)
    _check("hwsel_evaluate_workspace_bytes", lib().hwsel_evaluate_workspace_bytes(P, C.byref(n)))
    _arg(runtimes, "runtimes", F32)
    _arg(seg_offsets, "seg_offsets", I64, P + 1, runtimes)
    _arg(idx, "idx", I32, P * k, runtimes)
    if workspace is None:
        workspace = torch.empty(int(n.value), dtype=torch.uint8, device=dev)
    _arg(workspace, "workspace", U8, 0, runtimes)
    out = torch.empty(HWSEL_EVAL_FIELDS, dtype=torch.float64, device=dev)
    reg = rank = ybar = None
    if per_group:
        reg = torch.empty(P, dtype=torch.float64, device=dev)
        rank = torch.empty(P, dtype=torch.int32, device=dev)
        ybar = torch.empty(P, dtype=torch.float64, device=dev)
    _check("hwsel_evaluate", lib().hwsel_evaluate(
        _ptr(_dev(runtimes, "runtimes")), _ptr(_dev(seg_offsets, "seg_offsets")), P, _ptr(_dev(idx, "idx")), k,
        _ptr(out), _ptr(reg), _ptr(rank), _ptr(ybar), _ptr(workspace), workspace.numel(), _stream(stream)))
    return out, reg, rank, ybar


HWSEL_EVAL_NOALLOC_MAX_P = 65536


def hwsel_evaluate_noalloc(runtimes: torch.Tensor, seg_offsets: torch.Tensor, idx: torch.Tensor,
                           out: torch.Tensor | None = None, regret: torch.Tensor | None = None,
                           rank: torch.Tensor | None = None, ybar: torch.Tensor | None = None,
                           per_group: bool = True, stream=None):
    """hwsel_evaluate without a workspace (the library's own scratch array);
    outputs as for hwsel_evaluate.  Output tensors may be passed in."""
    P, k = idx.shape
    dev = runtimes.device
    _arg(runtimes, "runtimes", F32)
    _arg(seg_offsets, "seg_offsets", I64, P + 1, runtimes)
    _arg(idx, "idx", I32, P * k, runtimes)
    if out is None:
        out = torch.empty(HWSEL_EVAL_FIELDS, dtype=torch.float64, device=dev)
    _arg(out, "out", (torch.float64,), HWSEL_EVAL_FIELDS, runtimes)
    if per_group:
        regret = torch.empty(P, dtype=torch.float64, device=dev) if regret is None else regret
        rank = torch.empty(P, dtype=torch.int32, device=dev) if rank is None else rank
        ybar = torch.empty(P, dtype=torch.float64, device=dev) if ybar is None else ybar
    for n, t, dt in (("regret", regret, (torch.float64,)), ("rank", rank, I32), ("ybar", ybar, (torch.float64,))):
        if t is not None:
            _arg(t, n, dt, P, runtimes)
    _check("hwsel_evaluate_noalloc", lib().hwsel_evaluate_noalloc(
        _ptr(_dev(runtimes, "runtimes")), _ptr(_dev(seg_offsets, "seg_offsets")), P, _ptr(_dev(idx, "idx")), k,
        _ptr(out), _ptr(regret), _ptr(rank), _ptr(ybar), _stream(stream)))
    return out, regret, rank, ybar


def hwsel_static_config(runtimes: torch.Tensor, seg_offsets: torch.Tensor, config_id: torch.Tensor,
                        n_configs: int, workspace: torch.Tensor | None = None, stream=None):
    """Returns (best int32 [2] = (id, count), mean_y fp64 [1]) on the device."""
    P = seg_offsets.shape[0] - 1
    dev = runtimes.device
    n = C.c_size_t(0)
    _check("hwsel_static_config_workspace_bytes",
           lib().hwsel_static_config_workspace_bytes(P, n_configs, C.byref(n)))
    _arg(runtimes, "runtimes", F32)
    _arg(seg_offsets, "seg_offsets", I64, P + 1, runtimes)
    _arg(config_id, "config_id", I32, int(runtimes.numel()), runtimes)
    if workspace is None:
        workspace = torch.empty(int(n.value), dtype=torch.uint8, device=dev)
    _arg(workspace, "workspace", U8, 0, runtimes)
    best = torch.empty(2, dtype=torch.int32, device=dev)
    mean_y = torch.empty(1, dtype=torch.float64, device=dev)
    _check("hwsel_static_config", lib().hwsel_static_config(
        _ptr(_dev(runtimes, "runtimes")), _ptr(_dev(seg_offsets, "seg_offsets")), P,
        _ptr(_dev(config_id, "config_id")), n_configs, _ptr(best), _ptr(mean_y), _ptr(workspace),
        workspace.numel(), _stream(stream)))
    return best, mean_y


def hwsel_catalogue_mask(hw: dict, problems: torch.Tensor, flags: int = 0, mask: torch.Tensor | None = None,
                         stream=None):
    """Returns (mask uint8 [P, 534600], n_valid int64 [P])."""
    P = problems.shape[0]
    dev = problems.device
    if mask is None:
        mask = torch.empty((P, HWSEL_CATALOGUE_SIZE), dtype=torch.uint8, device=dev)
    _arg(mask, "mask", U8, P * HWSEL_CATALOGUE_SIZE, problems)
    n_valid = torch.empty(P, dtype=torch.int64, device=dev)
    _check("hwsel_catalogue_mask", lib().hwsel_catalogue_mask(
        hw_struct(hw), _ptr(_dev(problems, "problems")), P, flags, _ptr(mask), _ptr(n_valid), _stream(stream)))
    return mask, n_valid


def hwsel_catalogue_compact(mask: torch.Tensor, n_valid: torch.Tensor, capacity: int,
                            point: torch.Tensor | None = None, stream=None):
    """Returns (seg_offsets int64 [P+1], point int32 [capacity])."""
    P = mask.shape[0]
    dev = mask.device
    _arg(mask, "mask", U8, P * HWSEL_CATALOGUE_SIZE)
    _arg(n_valid, "n_valid", I64, P, mask)
    seg = torch.empty(P + 1, dtype=torch.int64, device=dev)
    if point is None:
        point = torch.empty(max(capacity, 1), dtype=torch.int32, device=dev)
    _arg(point, "point", I32, capacity, mask)
    _check("hwsel_catalogue_compact", lib().hwsel_catalogue_compact(
        _ptr(_dev(mask, "mask")), _ptr(_dev(n_valid, "n_valid")), P, _ptr(seg), _ptr(point), capacity,
        _stream(stream)))
    return seg, point


def hwsel_catalogue_candidates(problems: torch.Tensor, seg_offsets: torch.Tensor, R: int,
                               point: torch.Tensor | None = None, out: dict | None = None, stream=None) -> dict:
    """Candidate SoA (name -> device tensor of length R) of catalogue points;
    ``out`` may supply the field tensors (allocated here if None)."""
    P = problems.shape[0]
    dev = problems.device
    wide = ("tile_m", "tile_n", "tile_k", "inst_n")
    if out is None:
        out = {n: torch.empty(R, dtype=torch.int16 if n in wide else torch.uint8, device=dev) for n in CAND_FIELDS}
    _arg(seg_offsets, "seg_offsets", I64, P + 1, problems)
    if point is not None:
        _arg(point, "point", I32, R, problems)
    for n in CAND_FIELDS:
        t = _dev(out[n], n)
        if t.element_size() != (2 if n in wide else 1) or t.numel() < R or t.device != problems.device:
            raise ValueError(f"{n} must hold at least R elements of {2 if n in wide else 1} byte(s) on "
                             f"{problems.device}")
    s = hwsel_cands_out_t(*[_ptr(out[n]) for n in CAND_FIELDS])
    _check("hwsel_catalogue_candidates", lib().hwsel_catalogue_candidates(
        _ptr(_dev(problems, "problems")), P, _ptr(_dev(seg_offsets, "seg_offsets")), _ptr(point), R, C.byref(s),
        _stream(stream)))
    return out


def declared_functions() -> list[str]:
    """Names of the functions include/hwsel.h declares."""
    import re
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(hwsel_[a-z0-9_]+)\s*\(", text)))
