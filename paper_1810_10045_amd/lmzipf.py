"""Thin ctypes binding of ``liblmzipf.so`` (C ABI in ``include/lmzipf.h``).

Argument marshalling only: every step runs in the HIP kernels of the library.
Tensors are torch CUDA tensors (PyTorch supplies device memory and the
current stream); nothing here computes on the host. If the library has not
been built, importing this module raises — there is no fallback path.

Entry points have the C names without the ``lm_`` prefix: ``unique``,
``segsum``, ``map_ids``, ``fill_values``, ``sparse_apply``, the binary16
payload forms ``fill_values_f16`` and ``sparse_apply_f16``, and
``sample_ids``; ``unique_workspace_bytes`` is the workspace query that
``unique`` makes itself, for callers that size a workspace up front.
"""
from __future__ import annotations

import ctypes
import os
from typing import NamedTuple, Optional

import torch

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "liblmzipf.so")

OK, E_INVAL, E_WORKSPACE, E_HIP, E_UNSUPPORTED = 0, 1, 3, 4, 5
DEVERR_ID_RANGE, DEVERR_NOT_FOUND, DEVERR_CAPACITY, DEVERR_SPIN = 1, 2, 4, 8
DEVERR_NONFINITE = 16
I32, I64 = 0, 1
F32, BF16 = 0, 1
FILL_EXPAND, FILL_SCATTER, FILL_SCATTER_ADD = 0, 1, 2
OPT_SGD, OPT_ADAM = 0, 1
MAX_K = 1 << 30

EXPORTS = ("lm_status_string", "lm_abi_version", "lm_workspace_clear",
           "lm_unique_workspace_bytes", "lm_unique", "lm_segsum_workspace_bytes",
           "lm_segsum", "lm_map_ids", "lm_fill_values", "lm_sparse_apply",
           "lm_fill_values_f16", "lm_sparse_apply_f16", "lm_sample_ids")


class LmError(RuntimeError):
    pass


class DeviceError(RuntimeError):
    """Raised by :func:`check` when a kernel reported a data error."""


def _load():
    if not os.path.exists(LIB_PATH):
        raise ImportError(
            f"{LIB_PATH} is missing: build it with `python -c 'import __graft_entry__ as g; g.build()'`"
            " (the HIP library is the only implementation of these entry points)")
    L = ctypes.CDLL(LIB_PATH)
    P, I64_, SZ, I32_, F = (ctypes.c_void_p, ctypes.c_int64, ctypes.c_size_t,
                           ctypes.c_int32, ctypes.c_float)
    L.lm_status_string.argtypes = [ctypes.c_int]
    L.lm_status_string.restype = ctypes.c_char_p
    L.lm_abi_version.argtypes = []
    L.lm_workspace_clear.argtypes = [P, SZ, P]
    L.lm_unique_workspace_bytes.argtypes = [I64_, I32_, I64_]
    L.lm_unique_workspace_bytes.restype = SZ
    L.lm_unique.argtypes = [P, I32_, I64_, I64_, P, P, P, P, P, P, P, P, SZ, P]
    L.lm_unique_noalloc.argtypes = [P, I32_, I64_, I64_, P, P, P, P, P, P, P, P]
    L.lm_segsum_workspace_bytes.argtypes = [I64_, I64_]
    L.lm_segsum_workspace_bytes.restype = SZ
    L.lm_segsum.argtypes = [P, I32_, I64_, I64_, I64_, P, P, P, P, I64_, P, I64_, P, P, SZ, P]
    L.lm_segsum_rows.argtypes = [P, I32_, I64_, I64_, I64_, P, P, P, P, P, I32_, I64_, P, I64_, I64_,
                                 P, P, SZ, P]
    L.lm_segsum_sgd.argtypes = [P, I32_, I64_, I64_, I64_, P, P, P, P, P, I32_, I64_, P, I64_, I64_,
                                F, P, P, SZ, P]
    L.lm_segsum_adam.argtypes = [P, I32_, I64_, I64_, I64_, P, P, P, P, P, I32_, I64_, P, I64_, I64_,
                                 F, F, F, F, F, I64_, P, P, P, P, SZ, P]
    L.lm_map_ids.argtypes = [P, P, I64_, P, P, I64_, I32_, P, P, P]
    L.lm_fill_values.argtypes = [P, I64_, P, P, I64_, P, P, I32_, I64_, P, I64_, I64_, I32_, P, P]
    L.lm_sparse_apply.argtypes = [P, I64_, I64_, I64_, P, I32_, P, I64_, P, I64_, I32_,
                                  F, F, F, F, F, I64_, P, P, P, P]
    L.lm_fill_values_f16.argtypes = [P, I64_, P, P, I64_, P, P, I32_, I64_, P, I64_, I64_, I32_,
                                     F, P, P]
    L.lm_sparse_apply_f16.argtypes = [P, I64_, I64_, I64_, P, I32_, P, I64_, P, I64_, F, I32_,
                                      F, F, F, F, F, I64_, P, P, P, P]
    L.lm_sample_ids.argtypes = [P, I64_, I64_, P, I32_, P]
    L.lm_segsum_set_two_launches.argtypes = [I32_]
    L.lm_test_force_wait_failure.argtypes = [I32_, ctypes.c_uint32]
    for f in ("lm_abi_version", "lm_workspace_clear", "lm_unique", "lm_unique_noalloc",
              "lm_segsum", "lm_segsum_rows", "lm_segsum_sgd", "lm_segsum_adam", "lm_map_ids",
              "lm_fill_values", "lm_sparse_apply", "lm_fill_values_f16", "lm_sparse_apply_f16",
              "lm_sample_ids", "lm_segsum_set_two_launches", "lm_test_force_wait_failure"):
        getattr(L, f).restype = ctypes.c_int
    return L


_lib = _load()


def lib():
    return _lib


def status_string(rc: int) -> str:
    return _lib.lm_status_string(rc).decode()


def _call(rc: int, what: str):
    if rc != OK:
        raise LmError(f"{what}: {status_string(rc)}")


def _ptr(t: Optional[torch.Tensor]):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream(stream=None):
    s = stream if stream is not None else torch.cuda.current_stream()
    return ctypes.c_void_p(s.cuda_stream)


def _idtype(t: torch.Tensor) -> int:
    if t.dtype == torch.int32:
        return I32
    if t.dtype == torch.int64:
        return I64
    raise LmError(f"word ids must be int32 or int64, got {t.dtype}")


def _gtype(t: torch.Tensor) -> int:
    if t.dtype == torch.float32:
        return F32
    if t.dtype == torch.bfloat16:
        return BF16
    raise LmError(f"gradients must be float32 or bfloat16, got {t.dtype}")


def _rows(t: torch.Tensor, what: str):
    if t.dim() != 2 or t.stride(1) != 1:
        raise LmError(f"{what} must be a 2-D tensor with unit column stride")
    return t.stride(0)


def _dev(t: torch.Tensor, what: str):
    if not t.is_cuda:
        raise LmError(f"{what} must be a CUDA (HIP) tensor")


class Workspace:
    """A device scratch buffer that grows on demand (no entry point needs
    particular initial contents). Torch's allocator returns 512-byte aligned
    blocks, above the 256 bytes the library asks for."""

    def __init__(self, device=None):
        self.device = torch.device(device or "cuda")
        self.buf = torch.empty(0, dtype=torch.uint8, device=self.device)

    def get(self, nbytes: int) -> torch.Tensor:
        nbytes = max(int(nbytes), 256)
        if self.buf.numel() < nbytes:
            self.buf = torch.empty(nbytes, dtype=torch.uint8, device=self.device)
        return self.buf


_default_ws = {}


def default_workspace(device) -> Workspace:
    key = torch.device(device)
    if key not in _default_ws:
        _default_ws[key] = Workspace(key)
    return _default_ws[key]


def check(dev_err: torch.Tensor):
    """Synchronise on dev_err and raise DeviceError if any kernel set a bit."""
    v = int(dev_err.item())
    if v:
        names = [n for b, n in ((DEVERR_ID_RANGE, "id out of range"),
                                (DEVERR_NOT_FOUND, "id not found"),
                                (DEVERR_CAPACITY, "capacity exceeded"),
                                (DEVERR_SPIN, "inter-workgroup wait gave up"),
                                (DEVERR_NONFINITE, "compressed value not finite")) if v & b]
        raise DeviceError(f"device error 0x{v:x}: {', '.join(names)}")


class UniqueResult(NamedTuple):
    uniq: torch.Tensor
    counts: torch.Tensor
    offsets: torch.Tensor
    inverse: torch.Tensor
    perm: torch.Tensor
    num_unique: torch.Tensor
    dev_err: torch.Tensor


def unique_buffers(K: int, V: int, id_dtype, device) -> UniqueResult:
    cap = max(1, min(K, V))
    z = dict(device=device)
    return UniqueResult(
        torch.empty(cap, dtype=id_dtype, **z), torch.empty(cap, dtype=torch.int32, **z),
        torch.empty(cap + 1, dtype=torch.int32, **z), torch.empty(max(K, 1), dtype=torch.int32, **z),
        torch.empty(max(K, 1), dtype=torch.int32, **z), torch.zeros(1, dtype=torch.int64, **z),
        torch.zeros(1, dtype=torch.int32, **z))


def _check_unique_out(out: UniqueResult, ids: torch.Tensor, V: int):
    """The output buffers must hold what the kernels write: min(K, V) types,
    one offset more, K inverse and perm entries, on the ids' device."""
    K = ids.numel()
    cap = min(K, V)
    need = ((out.uniq, cap, ids.dtype), (out.counts, cap, torch.int32),
            (out.offsets, cap + 1, torch.int32), (out.inverse, K, torch.int32),
            (out.perm, K, torch.int32), (out.num_unique, 1, torch.int64),
            (out.dev_err, 1, torch.int32))
    for t, n, dt in need:
        if t.device != ids.device or t.dtype != dt or not t.is_contiguous() or t.numel() < n:
            raise LmError(f"unique output buffer: need {n} contiguous {dt} on {ids.device}")


def unique_workspace_bytes(K: int, V: int, id_dtype=torch.int32) -> int:
    """lm_unique_workspace_bytes: the workspace one lm_unique call of K ids
    of dtype id_dtype over [0, V) needs (0: the sizes are rejected)."""
    idt = I64 if id_dtype == torch.int64 else I32
    return int(_lib.lm_unique_workspace_bytes(K, idt, V))


def unique(ids: torch.Tensor, V: int, out: Optional[UniqueResult] = None,
           ws: Optional[Workspace] = None, stream=None) -> UniqueResult:
    """lm_unique: Sec. III-A steps 1/4. Returns device tensors; num_unique is
    a 1-element int64 tensor (no host sync)."""
    _dev(ids, "ids")
    K = ids.numel()
    idt = _idtype(ids)
    ids = ids.contiguous()
    if out is None:
        out = unique_buffers(K, V, ids.dtype, ids.device)
    _check_unique_out(out, ids, V)
    ws = ws or default_workspace(ids.device)
    need = _lib.lm_unique_workspace_bytes(K, idt, V)
    if need == 0 and K > 0:
        raise LmError("lm_unique_workspace_bytes rejected the sizes")
    buf = ws.get(need)
    _call(_lib.lm_unique(_ptr(ids), idt, K, V, _ptr(out.uniq), _ptr(out.counts), _ptr(out.offsets),
                         _ptr(out.inverse), _ptr(out.perm), _ptr(out.num_unique), _ptr(out.dev_err),
                         _ptr(buf), buf.numel(), _stream(stream)), "lm_unique")
    return out


UNIQUE_NOALLOC_MAX_K = 262144  # LM_UNIQUE_NOALLOC_MAX_K


def unique_noalloc(ids: torch.Tensor, V: int, out: UniqueResult, stream=None) -> UniqueResult:
    """lm_unique_noalloc: lm_unique with the library's own device workspace,
    for callers that cannot allocate. The outputs must be given (allocating
    them is the caller's business); at most UNIQUE_NOALLOC_MAX_K ids. Calls
    that overlap on one GPU share the workspace and race."""
    _dev(ids, "ids")
    if not ids.is_contiguous():
        raise LmError("ids must be contiguous (a copy would allocate)")
    K = ids.numel()
    _check_unique_out(out, ids, V)
    _call(_lib.lm_unique_noalloc(_ptr(ids), _idtype(ids), K, V, _ptr(out.uniq), _ptr(out.counts),
                                 _ptr(out.offsets), _ptr(out.inverse), _ptr(out.perm),
                                 _ptr(out.num_unique), _ptr(out.dev_err), _stream(stream)),
          "lm_unique_noalloc")
    return out


def segsum(grad: torch.Tensor, perm: torch.Tensor, inverse: torch.Tensor, offsets: torch.Tensor,
           num_unique: torch.Tensor, u_cap: Optional[int] = None,
           out: Optional[torch.Tensor] = None, dev_err: Optional[torch.Tensor] = None,
           ws: Optional[Workspace] = None, stream=None) -> torch.Tensor:
    """lm_segsum: Sec. III-A step 2. Returns the u_cap x D fp32 output (rows
    >= num_unique untouched)."""
    _dev(grad, "grad")
    K, D = grad.shape
    ld = _rows(grad, "grad")
    if u_cap is None:
        u_cap = offsets.numel() - 1
    if perm.numel() < K or inverse.numel() < K or offsets.numel() < 1:
        raise LmError("perm and inverse must hold K entries")
    if out is None:
        out = torch.empty((max(u_cap, 1), D), dtype=torch.float32, device=grad.device)
    if out.shape[0] < u_cap or out.shape[1] != D:
        raise LmError("out must be at least u_cap x D")
    ld_out = _rows(out, "out")
    if dev_err is None:
        dev_err = torch.zeros(1, dtype=torch.int32, device=grad.device)
    ws = ws or default_workspace(grad.device)
    buf = ws.get(_lib.lm_segsum_workspace_bytes(K, D))
    _call(_lib.lm_segsum(_ptr(grad), _gtype(grad), K, D, ld, _ptr(perm), _ptr(inverse), _ptr(offsets),
                         _ptr(num_unique), u_cap, _ptr(out), ld_out, _ptr(dev_err), _ptr(buf),
                         buf.numel(), _stream(stream)), "lm_segsum")
    return out


def segsum_rows(grad: torch.Tensor, perm: torch.Tensor, inverse: torch.Tensor,
                offsets: torch.Tensor, num_unique: torch.Tensor, row_ids: torch.Tensor,
                out: torch.Tensor, dev_err: Optional[torch.Tensor] = None,
                ws: Optional[Workspace] = None, stream=None) -> torch.Tensor:
    """lm_segsum_rows: Sec. III-A steps 2 and 5 in one pass: type u's sum goes
    to row row_ids[u] of `out` (e.g. the uniq ids into a dense V x D table);
    other rows of `out` are untouched. Returns `out`."""
    _dev(grad, "grad")
    _dev(row_ids, "row_ids")
    K, D = grad.shape
    ld = _rows(grad, "grad")
    if perm.numel() < K or inverse.numel() < K or offsets.numel() < 1:
        raise LmError("perm and inverse must hold K entries")
    if out.dim() != 2 or out.shape[1] != D or out.dtype != torch.float32:
        raise LmError("out must be an fp32 matrix with D columns")
    if not row_ids.is_contiguous():
        raise LmError("row_ids must be contiguous")
    ld_out = _rows(out, "out")
    if dev_err is None:
        dev_err = torch.zeros(1, dtype=torch.int32, device=grad.device)
    ws = ws or default_workspace(grad.device)
    buf = ws.get(_lib.lm_segsum_workspace_bytes(K, D))
    _call(_lib.lm_segsum_rows(_ptr(grad), _gtype(grad), K, D, ld, _ptr(perm), _ptr(inverse),
                              _ptr(offsets), _ptr(num_unique), _ptr(row_ids), _idtype(row_ids),
                              row_ids.numel(), _ptr(out), out.shape[0], ld_out, _ptr(dev_err),
                              _ptr(buf), buf.numel(), _stream(stream)), "lm_segsum_rows")
    return out


def segsum_sgd(grad: torch.Tensor, perm: torch.Tensor, inverse: torch.Tensor,
               offsets: torch.Tensor, num_unique: torch.Tensor, row_ids: torch.Tensor,
               table: torch.Tensor, lr: float, dev_err: Optional[torch.Tensor] = None,
               ws: Optional[Workspace] = None, stream=None) -> torch.Tensor:
    """lm_segsum_sgd: Sec. III-A steps 2 and 7 in one pass on one GPU:
    table[row_ids[u]] -= lr * (type u's sum), in place; other rows are
    untouched. Returns `table`."""
    _dev(grad, "grad")
    _dev(row_ids, "row_ids")
    K, D = grad.shape
    ld = _rows(grad, "grad")
    if perm.numel() < K or inverse.numel() < K or offsets.numel() < 1:
        raise LmError("perm and inverse must hold K entries")
    if table.dim() != 2 or table.shape[1] != D or table.dtype != torch.float32:
        raise LmError("table must be an fp32 matrix with D columns")
    if not row_ids.is_contiguous():
        raise LmError("row_ids must be contiguous")
    ld_t = _rows(table, "table")
    if dev_err is None:
        dev_err = torch.zeros(1, dtype=torch.int32, device=grad.device)
    ws = ws or default_workspace(grad.device)
    buf = ws.get(_lib.lm_segsum_workspace_bytes(K, D))
    _call(_lib.lm_segsum_sgd(_ptr(grad), _gtype(grad), K, D, ld, _ptr(perm), _ptr(inverse),
                             _ptr(offsets), _ptr(num_unique), _ptr(row_ids), _idtype(row_ids),
                             row_ids.numel(), _ptr(table), table.shape[0], ld_t, float(lr),
                             _ptr(dev_err), _ptr(buf), buf.numel(), _stream(stream)),
          "lm_segsum_sgd")
    return table


def segsum_adam(grad: torch.Tensor, perm: torch.Tensor, inverse: torch.Tensor,
                offsets: torch.Tensor, num_unique: torch.Tensor, row_ids: torch.Tensor,
                table: torch.Tensor, m: torch.Tensor, v: torch.Tensor, lr: float = 1e-3,
                beta1: float = 0.9, beta2: float = 0.999, eps: float = 1e-8,
                weight_decay: float = 0.0, step: int = 1, dev_err: Optional[torch.Tensor] = None,
                ws: Optional[Workspace] = None, stream=None) -> torch.Tensor:
    """lm_segsum_adam: Sec. III-A steps 2 and 7 in one pass on one GPU: the
    lazy-Adam step of table[row_ids[u]] (and of its m and v rows) with type
    u's sum as the gradient, in place; other rows are untouched. Returns
    `table`."""
    _dev(grad, "grad")
    _dev(row_ids, "row_ids")
    K, D = grad.shape
    ld = _rows(grad, "grad")
    if perm.numel() < K or inverse.numel() < K or offsets.numel() < 1:
        raise LmError("perm and inverse must hold K entries")
    if table.dim() != 2 or table.shape[1] != D or table.dtype != torch.float32:
        raise LmError("table must be an fp32 matrix with D columns")
    for t, n in ((m, "m"), (v, "v")):
        if t is None or t.shape != table.shape or t.stride() != table.stride() or t.dtype != table.dtype:
            raise LmError(f"{n} must have the table's shape, strides and dtype")
    if not row_ids.is_contiguous():
        raise LmError("row_ids must be contiguous")
    ld_t = _rows(table, "table")
    if dev_err is None:
        dev_err = torch.zeros(1, dtype=torch.int32, device=grad.device)
    ws = ws or default_workspace(grad.device)
    buf = ws.get(_lib.lm_segsum_workspace_bytes(K, D))
    _call(_lib.lm_segsum_adam(_ptr(grad), _gtype(grad), K, D, ld, _ptr(perm), _ptr(inverse),
                              _ptr(offsets), _ptr(num_unique), _ptr(row_ids), _idtype(row_ids),
                              row_ids.numel(), _ptr(table), table.shape[0], ld_t, float(lr),
                              float(beta1), float(beta2), float(eps), float(weight_decay),
                              int(step), _ptr(m), _ptr(v), _ptr(dev_err), _ptr(buf), buf.numel(),
                              _stream(stream)),
          "lm_segsum_adam")
    return table


def map_ids(sub_ids: torch.Tensor, n_sub: torch.Tensor, sup_ids: torch.Tensor,
            n_sup: torch.Tensor, out: Optional[torch.Tensor] = None,
            dev_err: Optional[torch.Tensor] = None, stream=None) -> torch.Tensor:
    """lm_map_ids: Sec. III-A step 4, the map J^ -> I^."""
    if sub_ids.dtype != sup_ids.dtype:
        raise LmError("sub_ids and sup_ids must share a dtype")
    cap = sub_ids.numel()
    if out is None:
        out = torch.empty(max(cap, 1), dtype=torch.int32, device=sub_ids.device)
    if dev_err is None:
        dev_err = torch.zeros(1, dtype=torch.int32, device=sub_ids.device)
    if out.numel() < cap:
        raise LmError("map output shorter than sub_ids")
    _call(_lib.lm_map_ids(_ptr(sub_ids), _ptr(n_sub), cap, _ptr(sup_ids), _ptr(n_sup),
                          sup_ids.numel(), _idtype(sub_ids), _ptr(out), _ptr(dev_err),
                          _stream(stream)), "lm_map_ids")
    return out


_MODES = {"expand": FILL_EXPAND, "scatter": FILL_SCATTER, "scatter_add": FILL_SCATTER_ADD}


def fill_values(src: torch.Tensor, src_ids: torch.Tensor, n_src: torch.Tensor,
                dst: torch.Tensor, dst_ids: Optional[torch.Tensor] = None,
                n_dst: Optional[torch.Tensor] = None, mode: str = "expand",
                dev_err: Optional[torch.Tensor] = None, stream=None) -> torch.Tensor:
    """lm_fill_values: Sec. III-A step 5 (expand) or a row scatter."""
    D = src.shape[1]
    if dst.shape[1] != D:
        raise LmError("src and dst widths differ")
    if dst_ids is not None and dst_ids.dtype != src_ids.dtype:
        raise LmError("src_ids and dst_ids must share a dtype")
    if dev_err is None:
        dev_err = torch.zeros(1, dtype=torch.int32, device=src.device)
    # capacities: rows of src that have an id, rows of dst that have an id
    src_cap = min(src.shape[0], src_ids.numel())
    dst_rows = dst.shape[0] if dst_ids is None else min(dst.shape[0], dst_ids.numel())
    _call(_lib.lm_fill_values(_ptr(src), _rows(src, "src"), _ptr(src_ids), _ptr(n_src),
                              src_cap, _ptr(dst_ids), _ptr(n_dst), _idtype(src_ids), D,
                              _ptr(dst), dst_rows, _rows(dst, "dst"), _MODES[mode],
                              _ptr(dev_err), _stream(stream)), "lm_fill_values")
    return dst


def sparse_apply(table: torch.Tensor, rows: torch.Tensor, n_rows: torch.Tensor,
                 vals: torch.Tensor, opt: str = "sgd", lr: float = 0.1, beta1: float = 0.9,
                 beta2: float = 0.999, eps: float = 1e-8, weight_decay: float = 0.0,
                 step: int = 1, m: Optional[torch.Tensor] = None, v: Optional[torch.Tensor] = None,
                 dev_err: Optional[torch.Tensor] = None, stream=None) -> torch.Tensor:
    """lm_sparse_apply: Sec. III-A step 7, in place on ``table`` (and m, v)."""
    V, D = table.shape
    if vals.shape[1] != D:
        raise LmError("vals and table widths differ")
    kind = {"sgd": OPT_SGD, "adam": OPT_ADAM}[opt]
    if kind == OPT_ADAM:
        for t, n in ((m, "m"), (v, "v")):
            if t is None or t.shape != table.shape or t.stride() != table.stride():
                raise LmError(f"Adam needs {n} shaped and strided like the table")
    if dev_err is None:
        dev_err = torch.zeros(1, dtype=torch.int32, device=table.device)
    rows_cap = min(rows.numel(), vals.shape[0])
    _call(_lib.lm_sparse_apply(_ptr(table), V, D, _rows(table, "table"), _ptr(rows),
                               _idtype(rows), _ptr(n_rows), rows_cap, _ptr(vals),
                               _rows(vals, "vals"), kind, lr, beta1, beta2, eps, weight_decay,
                               step, _ptr(m), _ptr(v), _ptr(dev_err), _stream(stream)),
          "lm_sparse_apply")
    return table


def _payload(t: torch.Tensor, what: str):
    if t.dtype not in (torch.float16, torch.int16, torch.uint16):
        raise LmError(f"{what} must hold binary16 (float16, or its bits as int16/uint16)")


def fill_values_f16(src: torch.Tensor, src_ids: torch.Tensor, n_src: torch.Tensor,
                    dst: torch.Tensor, dst_ids: Optional[torch.Tensor] = None,
                    n_dst: Optional[torch.Tensor] = None, mode: str = "expand",
                    scale: float = 1.0, dev_err: Optional[torch.Tensor] = None,
                    stream=None) -> torch.Tensor:
    """lm_fill_values_f16: Sec. III-C, EXPAND / SCATTER into a binary16 payload
    dst = binary16(src * scale)."""
    D = src.shape[1]
    _payload(dst, "dst")
    if dst.shape[1] != D:
        raise LmError("src and dst widths differ")
    if dst_ids is not None and dst_ids.dtype != src_ids.dtype:
        raise LmError("src_ids and dst_ids must share a dtype")
    if dev_err is None:
        dev_err = torch.zeros(1, dtype=torch.int32, device=src.device)
    src_cap = min(src.shape[0], src_ids.numel())
    dst_rows = dst.shape[0] if dst_ids is None else min(dst.shape[0], dst_ids.numel())
    _call(_lib.lm_fill_values_f16(_ptr(src), _rows(src, "src"), _ptr(src_ids), _ptr(n_src),
                                  src_cap, _ptr(dst_ids), _ptr(n_dst), _idtype(src_ids), D,
                                  _ptr(dst), dst_rows, _rows(dst, "dst"), _MODES[mode], scale,
                                  _ptr(dev_err), _stream(stream)), "lm_fill_values_f16")
    return dst


def sparse_apply_f16(table: torch.Tensor, rows: torch.Tensor, n_rows: torch.Tensor,
                     vals: torch.Tensor, inv_scale: float = 1.0, opt: str = "sgd",
                     lr: float = 0.1, beta1: float = 0.9, beta2: float = 0.999, eps: float = 1e-8,
                     weight_decay: float = 0.0, step: int = 1, m: Optional[torch.Tensor] = None,
                     v: Optional[torch.Tensor] = None, dev_err: Optional[torch.Tensor] = None,
                     stream=None) -> torch.Tensor:
    """lm_sparse_apply_f16: step 7 from a binary16 payload, g = fp32(vals) * inv_scale."""
    V, D = table.shape
    _payload(vals, "vals")
    if vals.shape[1] != D:
        raise LmError("vals and table widths differ")
    kind = {"sgd": OPT_SGD, "adam": OPT_ADAM}[opt]
    if kind == OPT_ADAM:
        for t, n in ((m, "m"), (v, "v")):
            if t is None or t.shape != table.shape or t.stride() != table.stride():
                raise LmError(f"Adam needs {n} shaped and strided like the table")
    if dev_err is None:
        dev_err = torch.zeros(1, dtype=torch.int32, device=table.device)
    rows_cap = min(rows.numel(), vals.shape[0])
    _call(_lib.lm_sparse_apply_f16(_ptr(table), V, D, _rows(table, "table"), _ptr(rows),
                                   _idtype(rows), _ptr(n_rows), rows_cap, _ptr(vals),
                                   _rows(vals, "vals"), inv_scale, kind, lr, beta1, beta2, eps,
                                   weight_decay, step, _ptr(m), _ptr(v), _ptr(dev_err),
                                   _stream(stream)), "lm_sparse_apply_f16")
    return table


def segsum_two_launches(enable: bool) -> bool:
    """lm_segsum_set_two_launches: every later lm_segsum call in the process
    takes the two-launch form (walk, then a separate fix-up kernel) while
    enabled. Returns the previous setting."""
    return bool(_lib.lm_segsum_set_two_launches(1 if enable else 0))


def force_wait_failure(enable: bool, spin_limit: int = 64):
    """lm_test_force_wait_failure: test hook for the failure path of the
    one-launch Seg-Sum's bounded waits (see include/lmzipf.h)."""
    _call(_lib.lm_test_force_wait_failure(1 if enable else 0, int(spin_limit)),
          "lm_test_force_wait_failure")


def sample_ids(r: torch.Tensor, V: int, out: Optional[torch.Tensor] = None,
               id_dtype=torch.int32, stream=None) -> torch.Tensor:
    """lm_sample_ids: Sec. III-B candidate sampler, ids = floor(r * V / 2^64)
    of caller-drawn 64-bit random words (``r`` int64 or uint64 bits)."""
    _dev(r, "r")
    if r.dtype not in (torch.int64, torch.uint64):
        raise LmError("random words must be 64-bit")
    if out is None:
        out = torch.empty(r.numel(), dtype=id_dtype, device=r.device)
    if out.numel() < r.numel():
        raise LmError("ids shorter than r")
    _call(_lib.lm_sample_ids(_ptr(r), r.numel(), V, _ptr(out), _idtype(out), _stream(stream)),
          "lm_sample_ids")
    return out
