"""Python binding of libvp: the VarioPath demand -> plan -> pack hot path on MI355X.

Argument marshalling only: every step runs in the HIP library's kernels
(``libvp.so`` next to this file, built by ``paper_2609_34340_amd.build``).
Torch supplies device memory and streams; tensors are passed as raw device
pointers and the current HIP stream.  If the library is missing this module
raises instead of falling back to anything else.
"""
from __future__ import annotations

import ctypes as C
import os
from typing import Optional

import numpy as np
import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libvp.so")

OK, INVALID_ARGUMENT, INVALID_DEMAND, NO_PROGRESS, CAPACITY, UNSUPPORTED, HIP_ERROR = range(7)
RESTRICT_NEAREST_PATH = 1
PATH_PIX, PATH_PXB, PATH_NIC, PATH_SYS = 0, 1, 2, 3
TOPO_SYS_P2P = 1
ROTATION_DYNAMIC_PATH, ROTATION_NEAREST_PATH = 0, 1
PIX, PXB, NIC = 0, 1, 2
STATUS_NAMES = {0: "ok", 1: "invalid argument", 2: "invalid demand", 3: "no progress",
                4: "capacity exceeded", 5: "unsupported", 6: "HIP error"}


class VPError(RuntimeError):
    def __init__(self, status: int, what: str):
        super().__init__("%s: %s" % (what, STATUS_NAMES.get(status, status)))
        self.status = status


class _Topology(C.Structure):
    _fields_ = [("n_nodes", C.c_int32), ("sockets_per_node", C.c_int32),
                ("switches_per_socket", C.c_int32), ("gpus_per_switch", C.c_int32),
                ("nics_per_switch", C.c_int32), ("flags", C.c_int32),
                ("pcie_bytes_per_ns", C.c_int64), ("nic_bytes_per_ns", C.c_int64)]


class PlanParams(C.Structure):
    _fields_ = [("k_target", C.c_int64), ("lambda_ns", C.c_int64), ("unit_bytes", C.c_int64),
                ("n_start", C.c_int32), ("i_aa", C.c_int32), ("seed", C.c_uint64),
                ("k_max", C.c_int32), ("reserved", C.c_int32)]


_lib = None


def lib():
    """Load libvp.so; raises if it has not been built."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise RuntimeError("libvp.so is not built (run paper_2609_34340_amd.build.build())")
    L = C.CDLL(LIB_PATH)
    vp, i32, i64, sz = C.c_void_p, C.c_int32, C.c_int64, C.c_size_t
    L.vp_build_catalog.argtypes = [C.POINTER(_Topology), C.POINTER(vp)]
    L.vp_catalog_info.argtypes = [vp, vp]
    L.vp_catalog_instances.argtypes = [vp] * 6
    L.vp_catalog_shapes.argtypes = [vp] * 6
    L.vp_catalog_families.argtypes = [vp] * 4
    L.vp_catalog_upload.argtypes = [vp, vp]
    L.vp_catalog_save.argtypes = [vp, vp, sz, C.POINTER(sz)]
    L.vp_catalog_restrict.argtypes = [vp, i32, C.POINTER(vp)]
    L.vp_rotation_time.argtypes = [vp, vp, i32, i64, vp, vp]
    L.vp_catalog_load.argtypes = [vp, sz, C.POINTER(vp)]
    L.vp_catalog_free.argtypes = [vp]
    L.vp_catalog_free.restype = None
    L.vp_demand_workspace.argtypes = [i32, i64, i32, i32]
    L.vp_demand_workspace.restype = sz
    L.vp_demand.argtypes = [vp, i32, i64, i32, i32, i32, i32, i32, i64, vp, vp, vp, vp, vp, vp, vp, sz, vp]
    L.vp_demand_heads.argtypes = [i64, vp, i64, i32, i32, i32, vp, vp, vp]
    L.vp_control_words.argtypes = [vp, i32, i32, i32, i32, vp, vp, vp]
    L.vp_receive_counts.argtypes = [vp, i64, vp, i32, i32, vp, vp]
    L.vp_plan_params_default.argtypes = [i32, i64, C.POINTER(PlanParams)]
    L.vp_plan_params_default.restype = None
    L.vp_plan_workspace.argtypes = [vp, C.POINTER(PlanParams)]
    L.vp_plan_workspace.restype = sz
    L.vp_plan.argtypes = [vp, vp, C.POINTER(PlanParams), vp, vp, vp, vp, vp, vp, vp, vp, vp, vp, vp, sz, vp]
    L.vp_plan_noalloc.argtypes = [vp, vp, C.POINTER(PlanParams), vp, vp, vp, vp, vp, vp, vp, vp, vp, vp, vp]
    L.vp_plan_batch_workspace.argtypes = [vp, C.POINTER(PlanParams), i32]
    L.vp_plan_batch_workspace.restype = sz
    L.vp_plan_batch.argtypes = [vp, i32, vp, C.POINTER(PlanParams), vp, vp, vp, vp, vp, vp, vp, vp, vp, vp, vp, sz,
                                vp]
    L.vp_pack_workspace.argtypes = [i32, i64, i64, i64, i32]
    L.vp_pack_workspace.restype = sz
    L.vp_pack_rows.argtypes = [vp, i64, i32, i64, vp, vp, vp, i32, i32, vp, vp, vp, vp, vp, i32, vp, i64, vp, vp,
                               vp, sz, vp]
    L.vp_pack_heads.argtypes = [vp, i64, i64, vp, i64, i32, i32, vp, vp, vp, vp, vp, i32, vp, i64, vp, vp, vp,
                                sz, vp]
    L.vp_pack_prepare_rows.argtypes = [vp, i64, i32, i64, vp, vp, vp, i32, i32, vp, vp, vp, vp, vp, i32, i64, vp,
                                       vp, vp, sz, vp]
    L.vp_pack_prepare_heads.argtypes = [vp, i64, i64, vp, i64, i32, i32, vp, vp, vp, vp, vp, i32, i64, vp, vp,
                                        vp, sz, vp]
    L.vp_pack_gather.argtypes = [vp, i64, i64, i32, vp, vp, i32, vp, i64, vp, vp, sz, vp]
    L.vp_slot_bytes.argtypes = [i64]
    L.vp_slot_bytes.restype = i64
    L.vp_unpack_workspace.argtypes = [i64]
    L.vp_unpack_workspace.restype = sz
    L.vp_demand_transpose.argtypes = [vp, i32, vp, vp]
    L.vp_unpack_rows.argtypes = [vp, i64, i64, vp, i32, i32, i32, vp, vp, vp, vp, i32, vp, i64, vp, vp, sz, vp]
    L.vp_pack_combine.argtypes = [vp, i64, i64, vp, i32, i32, i32, vp, vp, vp, i32, vp, i64, vp, vp, vp, sz, vp]
    L.vp_unpack_combine.argtypes = [vp, i64, i64, i64, i32, vp, vp, vp, i32, i32, vp, vp, vp, vp, i32, vp, vp, vp,
                                    sz, vp]
    L.vp_modeled_time.argtypes = [vp, i32, vp, vp, i64, vp, vp]
    L.vp_status_string.argtypes = [C.c_int]
    L.vp_status_string.restype = C.c_char_p
    L.vp_last_error.argtypes = []
    L.vp_last_error.restype = C.c_char_p
    _lib = L
    return L


def _check(st: int, what: str):
    if st != OK:
        raise VPError(st, "%s (%s)" % (what, lib().vp_last_error().decode()))


def _np(a: np.ndarray):
    return a.ctypes.data_as(C.c_void_p)


def _ptr(t: Optional[torch.Tensor]):
    return None if t is None else C.c_void_p(t.data_ptr())


def _dev(t: torch.Tensor, dtype, name: str):
    if not t.is_cuda or t.dtype != dtype or not t.is_contiguous():
        raise ValueError("%s must be a contiguous %s tensor on the GPU" % (name, dtype))
    return t


def _stream(stream=None):
    s = torch.cuda.current_stream() if stream is None else stream
    return C.c_void_p(s.cuda_stream)


def topology(topo) -> _Topology:
    """vp_topology from any object with the vpgen.Topology fields."""
    return _Topology(topo.n_nodes, topo.sockets_per_node, topo.switches_per_socket,
                     topo.gpus_per_switch, topo.nics_per_switch, getattr(topo, "flags", 0),
                     topo.pcie_bytes_per_ns, topo.nic_bytes_per_ns)


class Catalog:
    """Offline channel-family catalog (host build, one upload per device)."""

    def __init__(self, topo=None, *, payload: Optional[bytes] = None, restrict_of=None, rule: int = 0):
        """Build the catalog of topology `topo` (Alg. 1), load it from a
        payload written by save(), or restrict catalog `restrict_of` by `rule`."""
        h = C.c_void_p()
        if restrict_of is not None:
            _check(lib().vp_catalog_restrict(restrict_of.handle, rule, C.byref(h)), "vp_catalog_restrict")
            topo = restrict_of.topo
        elif payload is not None:
            buf = C.create_string_buffer(bytes(payload), len(payload))
            _check(lib().vp_catalog_load(buf, len(payload), C.byref(h)), "vp_catalog_load")
        else:
            t = topology(topo)
            _check(lib().vp_build_catalog(C.byref(t), C.byref(h)), "vp_build_catalog")
        self._h = h
        self.topo = topo
        info = np.zeros(8, np.int64)
        _check(lib().vp_catalog_info(self._h, _np(info)), "vp_catalog_info")
        (self.N, self.G, self.g, self.Q, self.n_nodes, self.n_shapes, self.n_families,
         self.n_instances) = (int(x) for x in info)

    @property
    def handle(self):
        return self._h

    def __del__(self):
        h = getattr(self, "_h", None)
        if h is not None and _lib is not None:
            _lib.vp_catalog_free(h)
            self._h = None

    def instances(self):
        n = self.n_instances
        cls, src, dst, copy = (np.zeros(n, np.int32) for _ in range(4))
        bw = np.zeros(n, np.int64)
        _check(lib().vp_catalog_instances(self._h, _np(cls), _np(src), _np(dst), _np(copy), _np(bw)),
               "vp_catalog_instances")
        return dict(cls=cls, src=src, dst=dst, copy=copy, bw=bw)

    def shapes(self):
        J, Q = self.n_shapes, self.Q
        k, fb, fe = (np.zeros(J, np.int32) for _ in range(3))
        L, R = np.zeros((J, Q, Q), np.int32), np.zeros((J, Q, Q), np.int32)
        _check(lib().vp_catalog_shapes(self._h, _np(k), _np(fb), _np(fe), _np(L), _np(R)),
               "vp_catalog_shapes")
        return dict(k=k, fam_begin=fb, fam_end=fe, L=L, R=R)

    def families(self):
        F = self.n_families
        shape, k = np.zeros(F, np.int32), np.zeros(F, np.int32)
        ids = np.zeros((F, self.Q * self.g), np.int32)
        _check(lib().vp_catalog_families(self._h, _np(shape), _np(k), _np(ids)), "vp_catalog_families")
        return dict(shape=shape, k=k, ids=ids)

    def save(self) -> bytes:
        """vp_catalog_save: the compact serialized catalog."""
        n = C.c_size_t(0)
        _check(lib().vp_catalog_save(self._h, None, 0, C.byref(n)), "vp_catalog_save")
        buf = C.create_string_buffer(n.value)
        _check(lib().vp_catalog_save(self._h, buf, n.value, C.byref(n)), "vp_catalog_save")
        return buf.raw[:n.value]

    @classmethod
    def load(cls, payload: bytes) -> "Catalog":
        return cls(payload=payload)

    def restrict(self, rule: int = 1) -> "Catalog":
        """vp_catalog_restrict: 1 = families on nearest paths only."""
        return Catalog(restrict_of=self, rule=rule)

    def rotation_time(self, D: np.ndarray, path_rule: int, lambda_ns: int = 10_000):
        """vp_rotation_time: (num, den) ns of the fixed cyclic rotation on D (host int64 [N, N])."""
        D = np.ascontiguousarray(D, np.int64)
        if D.shape != (self.N, self.N):
            raise ValueError("demand must be [%d, %d]" % (self.N, self.N))
        num, den = np.zeros(1, np.int64), np.zeros(1, np.int64)
        _check(lib().vp_rotation_time(self._h, _np(D), path_rule, lambda_ns, _np(num), _np(den)),
               "vp_rotation_time")
        return int(num[0]), int(den[0])

    def upload(self, stream=None):
        _check(lib().vp_catalog_upload(self._h, _stream(stream)), "vp_catalog_upload")

    def modeled_time(self, K: int, inst: np.ndarray, nbytes: np.ndarray, lambda_ns: int = 10_000):
        """Eq. (2) of a schedule as the exact fraction (num, den) in ns."""
        inst = np.ascontiguousarray(inst[:K], np.int32)
        nbytes = np.ascontiguousarray(nbytes[:K], np.int64)
        num, den = np.zeros(1, np.int64), np.zeros(1, np.int64)
        _check(lib().vp_modeled_time(self._h, K, _np(inst), _np(nbytes), lambda_ns, _np(num), _np(den)),
               "vp_modeled_time")
        return int(num[0]), int(den[0])


def plan_params(n_ranks: int, unit_bytes: int, **kw) -> PlanParams:
    p = PlanParams()
    lib().vp_plan_params_default(n_ranks, unit_bytes, C.byref(p))
    for key, v in kw.items():
        if v is not None:
            setattr(p, key, v)
    return p


def new_status(device="cuda") -> torch.Tensor:
    return torch.zeros(1, dtype=torch.int32, device=device)


def read_status(status: torch.Tensor) -> int:
    return int(status.item())


# ---------------------------------------------------------------- demand

def demand_workspace_bytes(R: int, T: int, k: int, E: int) -> int:
    return int(lib().vp_demand_workspace(R, T, k, E))


def demand(routing: torch.Tensor, n_ranks: int, n_experts: int, unit: int, first_rank: int = 0,
           sort_row: int = 0, status: Optional[torch.Tensor] = None, out: Optional[dict] = None,
           ws: Optional[torch.Tensor] = None, stream=None) -> dict:
    """vp_demand over routing [R, T, k] (int32, GPU).  Returns counts, demand rows,
    and for row `sort_row` the (expert, token) order (token and routing slot of
    each assignment) and destination offsets."""
    _dev(routing, torch.int32, "routing")
    R, T, k = routing.shape
    dev = routing.device
    if out is None:
        out = dict(counts=torch.empty((R, n_experts), dtype=torch.int32, device=dev),
                   demand=torch.empty((R, n_ranks), dtype=torch.int64, device=dev),
                   sorted_tok=torch.empty(max(T * k, 1), dtype=torch.int32, device=dev),
                   sorted_slot=torch.empty(max(T * k, 1), dtype=torch.uint8, device=dev),
                   dest_off=torch.empty(n_ranks + 1, dtype=torch.int64, device=dev))
    if status is None:
        status = new_status(dev)
    wsb = demand_workspace_bytes(R, T, k, n_experts)
    if ws is None:
        ws = torch.zeros(max(wsb, 1), dtype=torch.uint8, device=dev)
    _check(lib().vp_demand(_ptr(routing), R, T, k, n_experts, n_ranks, first_rank, sort_row, unit,
                           _ptr(out["counts"]), _ptr(out["demand"]), _ptr(out["sorted_tok"]),
                           _ptr(out.get("sorted_slot")), _ptr(out["dest_off"]), _ptr(status), _ptr(ws),
                           ws.numel(), _stream(stream)), "vp_demand")
    out["status"] = status
    return out


def demand_heads(T: int, head_lo: torch.Tensor, head_bytes: int, first_rank: int = 0, R: int = 1,
                 status: Optional[torch.Tensor] = None, out: Optional[torch.Tensor] = None,
                 stream=None) -> torch.Tensor:
    _dev(head_lo, torch.int64, "head_lo")
    N = head_lo.numel() - 1
    if out is None:
        out = torch.empty((R, N), dtype=torch.int64, device=head_lo.device)
    if status is None:
        status = new_status(head_lo.device)
    _check(lib().vp_demand_heads(T, _ptr(head_lo), head_bytes, N, first_rank, R, _ptr(out), _ptr(status),
                                 _stream(stream)), "vp_demand_heads")
    return out


def control_words(counts: torch.Tensor, n_ranks: int, first_rank: int = 0,
                  status: Optional[torch.Tensor] = None, out: Optional[torch.Tensor] = None,
                  stream=None) -> torch.Tensor:
    """vp_control_words over counts [R, E] (int32, GPU).  Returns the words
    [R, N] as int32 holding the uint32 bit patterns."""
    _dev(counts, torch.int32, "counts")
    R, E = counts.shape
    if out is None:
        out = torch.empty((R, n_ranks), dtype=torch.int32, device=counts.device)
    if status is None:
        status = new_status(counts.device)
    _check(lib().vp_control_words(_ptr(counts), R, E, n_ranks, first_rank, _ptr(out), _ptr(status),
                                  _stream(stream)), "vp_control_words")
    return out


def receive_counts(words: torch.Tensor, word_stride: int, signal: torch.Tensor, n_local: int,
                   offset: int = 0, out: Optional[torch.Tensor] = None, stream=None) -> torch.Tensor:
    """vp_receive_counts: a receiver's rows per (source, local expert), int32
    [N, L], from the words at flat positions offset + i * word_stride of the
    contiguous int32 tensor `words` and the signal counts [N, L]."""
    _dev(signal, torch.int32, "signal")
    _dev(words, torch.int32, "words")
    N = signal.shape[0]
    if signal.dim() != 2 or signal.shape[1] != n_local:
        raise ValueError("signal must be [N, n_local]")
    if offset < 0 or word_stride < 1 or offset + (N - 1) * word_stride >= words.numel():
        raise ValueError("words too short for N sources at this offset and stride")
    if out is None:
        out = torch.empty((N, n_local), dtype=torch.int32, device=signal.device)
    _check(lib().vp_receive_counts(C.c_void_p(words.data_ptr() + 4 * offset), word_stride, _ptr(signal), N,
                                   n_local, _ptr(out), _stream(stream)), "vp_receive_counts")
    return out


# ------------------------------------------------------------------ plan

def plan_workspace_bytes(cat: Catalog, p: PlanParams) -> int:
    return int(lib().vp_plan_workspace(cat.handle, C.byref(p)))


def alloc_schedule(N: int, k_max: int, device="cuda", layout: bool = False) -> dict:
    """Schedule buffers; with `layout` also the planner's per-rank send and
    stream offsets (the buffer layout the pack can use directly) and its
    receive view (the rank whose lane lands at each rank, for the unpack)."""
    s = dict(K=torch.zeros(1, dtype=torch.int32, device=device),
             family=torch.empty(k_max, dtype=torch.int32, device=device),
             dst=torch.empty((k_max, N), dtype=torch.int32, device=device),
             inst=torch.empty((k_max, N), dtype=torch.int32, device=device),
             bytes=torch.empty((k_max, N), dtype=torch.int64, device=device),
             tau=torch.zeros(1, dtype=torch.int64, device=device))
    if layout:
        s["send_off"] = torch.empty((k_max, N), dtype=torch.int64, device=device)
        s["stream_off"] = torch.empty((k_max, N), dtype=torch.int64, device=device)
        s["recv_src"] = torch.empty((k_max, N), dtype=torch.int32, device=device)
    return s


def plan(cat: Catalog, D: torch.Tensor, p: PlanParams, status: Optional[torch.Tensor] = None,
         out: Optional[dict] = None, ws: Optional[torch.Tensor] = None, stream=None) -> dict:
    """vp_plan on demand D [N, N] (int64, GPU): Alg. 2 in one device kernel."""
    _dev(D, torch.int64, "demand")
    N = cat.N
    if tuple(D.shape) != (N, N):
        raise ValueError("demand must be [%d, %d]" % (N, N))
    if out is None:
        out = alloc_schedule(N, p.k_max, D.device)
    if status is None:
        status = new_status(D.device)
    if ws is None:
        ws = torch.empty(plan_workspace_bytes(cat, p), dtype=torch.uint8, device=D.device)
    _check(lib().vp_plan(cat.handle, _ptr(D), C.byref(p), _ptr(out["K"]), _ptr(out["family"]),
                         _ptr(out["dst"]), _ptr(out["inst"]), _ptr(out["bytes"]), _ptr(out.get("send_off")),
                         _ptr(out.get("stream_off")), _ptr(out.get("recv_src")), _ptr(out["tau"]), _ptr(status),
                         _ptr(ws), ws.numel(),
                         _stream(stream)), "vp_plan")
    out["status"] = status
    return out


def plan_noalloc(cat: Catalog, D: torch.Tensor, p: PlanParams, status: Optional[torch.Tensor] = None,
                 out: Optional[dict] = None, stream=None) -> dict:
    """vp_plan_noalloc: vp_plan with the residual in the library's own device
    array (no workspace; at most 256 ranks)."""
    _dev(D, torch.int64, "demand")
    N = cat.N
    if tuple(D.shape) != (N, N):
        raise ValueError("demand must be [%d, %d]" % (N, N))
    if out is None:
        out = alloc_schedule(N, p.k_max, D.device)
    if status is None:
        status = new_status(D.device)
    _check(lib().vp_plan_noalloc(cat.handle, _ptr(D), C.byref(p), _ptr(out["K"]), _ptr(out["family"]),
                                 _ptr(out["dst"]), _ptr(out["inst"]), _ptr(out["bytes"]), _ptr(out.get("send_off")),
                                 _ptr(out.get("stream_off")), _ptr(out.get("recv_src")), _ptr(out["tau"]),
                                 _ptr(status), _stream(stream)), "vp_plan_noalloc")
    out["status"] = status
    return out


def plan_batch_workspace_bytes(cat: Catalog, p: PlanParams, B: int) -> int:
    return int(lib().vp_plan_batch_workspace(cat.handle, C.byref(p), B))


def alloc_schedule_batch(B: int, N: int, k_max: int, device="cuda", layout: bool = False) -> dict:
    """Schedule buffers of B matrices (leading dimension B)."""
    s = dict(K=torch.zeros(B, dtype=torch.int32, device=device),
             family=torch.empty((B, k_max), dtype=torch.int32, device=device),
             dst=torch.empty((B, k_max, N), dtype=torch.int32, device=device),
             inst=torch.empty((B, k_max, N), dtype=torch.int32, device=device),
             bytes=torch.empty((B, k_max, N), dtype=torch.int64, device=device),
             tau=torch.zeros(B, dtype=torch.int64, device=device))
    if layout:
        for key, dt in (("send_off", torch.int64), ("stream_off", torch.int64), ("recv_src", torch.int32)):
            s[key] = torch.empty((B, k_max, N), dtype=dt, device=device)
    return s


def plan_batch(cat: Catalog, D: torch.Tensor, p: PlanParams, status: Optional[torch.Tensor] = None,
               out: Optional[dict] = None, ws: Optional[torch.Tensor] = None, stream=None) -> dict:
    """vp_plan_batch on demands D [B, N, N] (int64, GPU), one workgroup per matrix;
    status is int32 [B] (matrix b's device errors)."""
    _dev(D, torch.int64, "demand")
    N = cat.N
    if D.dim() != 3 or tuple(D.shape[1:]) != (N, N):
        raise ValueError("demand must be [B, %d, %d]" % (N, N))
    B = D.shape[0]
    if out is None:
        out = alloc_schedule_batch(B, N, p.k_max, D.device)
    if out["K"].numel() != B or tuple(out["dst"].shape) != (B, p.k_max, N):
        raise ValueError("schedule buffers do not hold B = %d schedules of k_max = %d" % (B, p.k_max))
    if status is None:
        status = torch.zeros(B, dtype=torch.int32, device=D.device)
    if status.numel() != B:
        raise ValueError("status must hold B entries")
    need = plan_batch_workspace_bytes(cat, p, B)
    if ws is None:
        ws = torch.empty(need, dtype=torch.uint8, device=D.device)
    _check(lib().vp_plan_batch(cat.handle, B, _ptr(D), C.byref(p), _ptr(out["K"]), _ptr(out["family"]),
                               _ptr(out["dst"]), _ptr(out["inst"]), _ptr(out["bytes"]), _ptr(out.get("send_off")),
                               _ptr(out.get("stream_off")), _ptr(out.get("recv_src")), _ptr(out["tau"]),
                               _ptr(status), _ptr(ws), ws.numel(), _stream(stream)), "vp_plan_batch")
    out["status"] = status
    return out


def schedule_to_host(s: dict) -> dict:
    K = int(s["K"].item())
    return dict(K=K, family=s["family"][:K].cpu().numpy(), dst=s["dst"][:K].cpu().numpy(),
                inst=s["inst"][:K].cpu().numpy(), bytes=s["bytes"][:K].cpu().numpy(),
                tau=int(s["tau"].item()))


# ------------------------------------------------------------------ pack

def pack_workspace_bytes(k_max: int, send_capacity: int, unit: int, T: int = 0, k: int = 0) -> int:
    """Rows: T tokens, top-k k.  Heads: k = 0."""
    return int(lib().vp_pack_workspace(k_max, send_capacity, unit, T, k))


def pack_rows(tokens: torch.Tensor, row_bytes: int, sorted_tok: torch.Tensor, sorted_slot: torch.Tensor,
              dest_off: torch.Tensor,
              self_rank: int, sched: dict, send: torch.Tensor, step_off: torch.Tensor,
              status: torch.Tensor, ws: Optional[torch.Tensor] = None, stream=None):
    """vp_pack_rows: this rank's token rows into the send buffer in step order.
    sorted_tok holds T*k entries (T tokens, top-k k)."""
    if not tokens.is_cuda or not tokens.is_contiguous():
        raise ValueError("tokens must be a contiguous GPU tensor")
    T = tokens.numel() * tokens.element_size() // row_bytes
    if T == 0 or sorted_tok.numel() % T != 0:
        raise ValueError("sorted_tok must hold T*k entries")
    k = sorted_tok.numel() // T
    k_max = sched["dst"].shape[0]
    N = sched["dst"].shape[1]
    cap = send.numel() * send.element_size()
    if ws is None:
        ws = torch.zeros(pack_workspace_bytes(k_max, cap, row_bytes, T, k), dtype=torch.uint8,
                         device=send.device)
    _check(lib().vp_pack_rows(_ptr(tokens), T, k, row_bytes, _ptr(sorted_tok), _ptr(sorted_slot), _ptr(dest_off),
                              self_rank, N,
                              _ptr(sched["K"]), _ptr(sched["dst"]), _ptr(sched["bytes"]),
                              _ptr(sched.get("send_off")), _ptr(sched.get("stream_off")), k_max, _ptr(send),
                              cap, _ptr(step_off), _ptr(status), _ptr(ws), ws.numel(), _stream(stream)),
           "vp_pack_rows")


def pack_heads(act: torch.Tensor, token_stride: int, head_lo: torch.Tensor, head_bytes: int,
               self_rank: int, sched: dict, send: torch.Tensor, step_off: torch.Tensor,
               status: torch.Tensor, ws: Optional[torch.Tensor] = None, stream=None):
    """vp_pack_heads: this rank's head blocks into the send buffer in step order."""
    if not act.is_cuda or not act.is_contiguous():
        raise ValueError("activations must be a contiguous GPU tensor")
    T = act.numel() * act.element_size() // token_stride
    k_max = sched["dst"].shape[0]
    N = sched["dst"].shape[1]
    cap = send.numel() * send.element_size()
    if ws is None:
        ws = torch.zeros(pack_workspace_bytes(k_max, cap, head_bytes), dtype=torch.uint8, device=send.device)
    _check(lib().vp_pack_heads(_ptr(act), T, token_stride, _ptr(head_lo), head_bytes, self_rank, N,
                               _ptr(sched["K"]), _ptr(sched["dst"]), _ptr(sched["bytes"]),
                               _ptr(sched.get("send_off")), _ptr(sched.get("stream_off")), k_max,
                               _ptr(send), cap, _ptr(step_off), _ptr(status), _ptr(ws), ws.numel(),
                               _stream(stream)), "vp_pack_heads")


# ------------------------------------------------ receive side, combine

def slot_bytes(row_bytes: int) -> int:
    """Receive-slot stride: the row rounded up to 128 bytes."""
    return int(lib().vp_slot_bytes(row_bytes))


def unpack_workspace_bytes(buffer_rows: int) -> int:
    return int(lib().vp_unpack_workspace(buffer_rows))


def demand_transpose(D: torch.Tensor, out: Optional[torch.Tensor] = None, stream=None) -> torch.Tensor:
    """vp_demand_transpose: the combine's demand D^T."""
    _dev(D, torch.int64, "demand")
    N = D.shape[0]
    if out is None:
        out = torch.empty_like(D)
    _check(lib().vp_demand_transpose(_ptr(D), N, _ptr(out), _stream(stream)), "vp_demand_transpose")
    return out


def _nbytes(t: torch.Tensor) -> int:
    return t.numel() * t.element_size()


def unpack_rows(recv: torch.Tensor, row_bytes: int, counts: torch.Tensor, self_rank: int, sched: dict,
                out: torch.Tensor, status: torch.Tensor, ws: Optional[torch.Tensor] = None, stream=None):
    """vp_unpack_rows: rank self_rank's receive slots into its expert-major output."""
    _dev(counts, torch.int32, "counts")
    N, E = counts.shape
    k_max = sched["dst"].shape[0]
    cap = _nbytes(recv)
    if ws is None:
        ws = torch.empty(unpack_workspace_bytes(cap // slot_bytes(row_bytes)), dtype=torch.uint8, device=recv.device)
    _check(lib().vp_unpack_rows(_ptr(recv), cap, row_bytes, _ptr(counts), E, self_rank, N, _ptr(sched["K"]),
                                _ptr(sched["dst"]), _ptr(sched["bytes"]), _ptr(sched["recv_src"]), k_max,
                                _ptr(out), _nbytes(out), _ptr(status), _ptr(ws), ws.numel(), _stream(stream)),
           "vp_unpack_rows")


def pack_combine(out: torch.Tensor, row_bytes: int, counts: torch.Tensor, self_rank: int, sched: dict,
                 send: torch.Tensor, step_off: torch.Tensor, status: torch.Tensor, ws: Optional[torch.Tensor] = None,
                 stream=None):
    """vp_pack_combine: expert-major rows back to their sources in the combine schedule's order."""
    _dev(counts, torch.int32, "counts")
    N, E = counts.shape
    k_max = sched["dst"].shape[0]
    cap = _nbytes(send)
    if ws is None:
        ws = torch.empty(unpack_workspace_bytes(cap // row_bytes), dtype=torch.uint8, device=send.device)
    _check(lib().vp_pack_combine(_ptr(out), _nbytes(out), row_bytes, _ptr(counts), E, self_rank, N,
                                 _ptr(sched["K"]), _ptr(sched["dst"]), _ptr(sched["bytes"]), k_max, _ptr(send), cap,
                                 _ptr(step_off), _ptr(status), _ptr(ws), ws.numel(), _stream(stream)),
           "vp_pack_combine")


def unpack_combine(recv: torch.Tensor, row_bytes: int, T: int, k: int, sorted_tok: torch.Tensor,
                   sorted_slot: torch.Tensor, dest_off: torch.Tensor, self_rank: int, sched: dict,
                   combined: torch.Tensor, status: torch.Tensor, ws: Optional[torch.Tensor] = None, stream=None):
    """vp_unpack_combine: returned rows into combined [T * k, slot] at (token, routing slot)."""
    N = sched["dst"].shape[1]
    k_max = sched["dst"].shape[0]
    if _nbytes(combined) < T * k * slot_bytes(row_bytes):
        raise ValueError("combined must hold T * k slots")
    cap = _nbytes(recv)
    if ws is None:
        ws = torch.empty(unpack_workspace_bytes(cap // slot_bytes(row_bytes)), dtype=torch.uint8, device=recv.device)
    _check(lib().vp_unpack_combine(_ptr(recv), cap, row_bytes, T, k, _ptr(sorted_tok), _ptr(sorted_slot),
                                   _ptr(dest_off), self_rank, N, _ptr(sched["K"]), _ptr(sched["dst"]),
                                   _ptr(sched["bytes"]), _ptr(sched["recv_src"]), k_max, _ptr(combined),
                                   _ptr(status), _ptr(ws), ws.numel(), _stream(stream)), "vp_unpack_combine")


# -------------------------------------------------------------- pipeline

class Pipeline:
    """Preallocated demand -> plan -> pack for one workload on one GPU.

    ``step()`` enqueues the whole hot path on the current stream with no host
    synchronisation: vp_demand (or vp_demand_heads) over every rank's routing
    and, for MoE, vp_control_words of every pair; vp_plan on the resulting
    N x N matrix; and vp_pack of rank ``self_rank``.
    """

    def __init__(self, topo, mode: str, unit: int, *, n_experts: int = 0, tokens: int = 0,
                 top_k: int = 0, token_stride: int = 0, self_rank: int = 0, params: Optional[dict] = None,
                 device="cuda"):
        self.cat = Catalog(topo)
        self.cat.upload()
        self.mode, self.unit, self.self_rank = mode, unit, self_rank
        self.N = N = self.cat.N
        self.E, self.T, self.k = n_experts, tokens, top_k
        self.token_stride = token_stride or unit
        self.params = plan_params(N, unit, **(params or {}))
        kmax = self.params.k_max
        dev = device
        self.status = new_status(dev)
        self.sched = alloc_schedule(N, kmax, dev, layout=True)
        self.plan_ws = torch.empty(plan_workspace_bytes(self.cat, self.params), dtype=torch.uint8, device=dev)
        if mode == "moe":
            self.dem = dict(counts=torch.empty((N, n_experts), dtype=torch.int32, device=dev),
                            demand=torch.empty((N, N), dtype=torch.int64, device=dev),
                            sorted_tok=torch.empty(max(tokens * top_k, 1), dtype=torch.int32, device=dev),
                            sorted_slot=torch.empty(max(tokens * top_k, 1), dtype=torch.uint8, device=dev),
                            dest_off=torch.empty(N + 1, dtype=torch.int64, device=dev))
            self.dem_ws = torch.zeros(max(demand_workspace_bytes(N, tokens, top_k, n_experts), 1),
                                      dtype=torch.uint8, device=dev)
            self.words = torch.empty((N, N), dtype=torch.int32, device=dev)
            cap = tokens * top_k * unit
            ws_T, ws_k = tokens, top_k
        else:
            self.dem = dict(demand=torch.empty((N, N), dtype=torch.int64, device=dev))
            cap = tokens * (self.token_stride // unit) * unit
            ws_T, ws_k = tokens, 0
        self.send_capacity = cap
        self.send = torch.empty(max(cap, 16), dtype=torch.uint8, device=dev)
        self.step_off = torch.empty(kmax + 1, dtype=torch.int64, device=dev)
        self.pack_ws = torch.zeros(pack_workspace_bytes(kmax, cap, unit, ws_T, ws_k), dtype=torch.uint8,
                                   device=dev)

    # The hot path in stages (all enqueued on one stream, no host sync).
    def demand_stage(self, routing: Optional[torch.Tensor] = None, head_lo: Optional[torch.Tensor] = None,
                     stream=None):
        L, s = lib(), _stream(stream)
        if self.mode == "moe":
            R, T, k = routing.shape
            _check(L.vp_demand(_ptr(routing), R, T, k, self.E, self.N, 0, self.self_rank, self.unit,
                               _ptr(self.dem["counts"]), _ptr(self.dem["demand"]),
                               _ptr(self.dem["sorted_tok"]), _ptr(self.dem["sorted_slot"]),
                               _ptr(self.dem["dest_off"]), _ptr(self.status),
                               _ptr(self.dem_ws), self.dem_ws.numel(), s), "vp_demand")
        else:
            _check(L.vp_demand_heads(self.T, _ptr(head_lo), self.unit, self.N, 0, self.N,
                                     _ptr(self.dem["demand"]), _ptr(self.status), s), "vp_demand_heads")

    def words_stage(self, stream=None):
        """vp_control_words of every rank's pairs (MoE only; uint32 bit patterns in self.words)."""
        if self.mode == "moe":
            _check(lib().vp_control_words(_ptr(self.dem["counts"]), self.N, self.E, self.N, 0, _ptr(self.words),
                                          _ptr(self.status), _stream(stream)), "vp_control_words")

    def plan_stage(self, stream=None):
        p = self.params
        _check(lib().vp_plan(self.cat.handle, _ptr(self.dem["demand"]), C.byref(p), _ptr(self.sched["K"]),
                             _ptr(self.sched["family"]), _ptr(self.sched["dst"]), _ptr(self.sched["inst"]),
                             _ptr(self.sched["bytes"]), _ptr(self.sched["send_off"]),
                             _ptr(self.sched["stream_off"]), _ptr(self.sched["recv_src"]), _ptr(self.sched["tau"]),
                             _ptr(self.status),
                             _ptr(self.plan_ws), self.plan_ws.numel(), _stream(stream)), "vp_plan")

    def pack_prepare_stage(self, tokens: torch.Tensor, head_lo: Optional[torch.Tensor] = None, stream=None):
        L, s, p = lib(), _stream(stream), self.params
        if self.mode == "moe":
            T = tokens.numel() * tokens.element_size() // self.unit
            _check(L.vp_pack_prepare_rows(_ptr(tokens), T, self.k, self.unit, _ptr(self.dem["sorted_tok"]),
                                          _ptr(self.dem["sorted_slot"]), _ptr(self.dem["dest_off"]),
                                          self.self_rank, self.N,
                                          _ptr(self.sched["K"]), _ptr(self.sched["dst"]),
                                          _ptr(self.sched["bytes"]), _ptr(self.sched["send_off"]),
                                          _ptr(self.sched["stream_off"]), p.k_max, self.send_capacity,
                                          _ptr(self.step_off), _ptr(self.status), _ptr(self.pack_ws),
                                          self.pack_ws.numel(), s), "vp_pack_prepare_rows")
        else:
            T = tokens.numel() * tokens.element_size() // self.token_stride
            _check(L.vp_pack_prepare_heads(_ptr(tokens), T, self.token_stride, _ptr(head_lo), self.unit,
                                           self.self_rank, self.N, _ptr(self.sched["K"]),
                                           _ptr(self.sched["dst"]), _ptr(self.sched["bytes"]),
                                           _ptr(self.sched["send_off"]), _ptr(self.sched["stream_off"]), p.k_max,
                                           self.send_capacity, _ptr(self.step_off), _ptr(self.status),
                                           _ptr(self.pack_ws), self.pack_ws.numel(), s), "vp_pack_prepare_heads")

    def pack_gather_stage(self, tokens: torch.Tensor, send: Optional[torch.Tensor] = None, stream=None):
        send = self.send if send is None else send
        if send.numel() < self.send_capacity:
            raise ValueError("send buffer smaller than the pipeline's capacity")
        if self.mode == "moe":
            T, k = tokens.numel() * tokens.element_size() // self.unit, self.k
        else:
            T, k = tokens.numel() * tokens.element_size() // self.token_stride, 0
        _check(lib().vp_pack_gather(_ptr(tokens), self.unit, T, k, _ptr(self.sched["K"]), _ptr(self.step_off),
                                    self.params.k_max, _ptr(send), self.send_capacity, _ptr(self.status),
                                    _ptr(self.pack_ws), self.pack_ws.numel(), _stream(stream)),
               "vp_pack_gather")
        return send

    def pack_stage(self, tokens: torch.Tensor, head_lo: Optional[torch.Tensor] = None,
                   send: Optional[torch.Tensor] = None, stream=None):
        """The pack in one call (vp_pack_rows / vp_pack_heads): both halves,
        or for heads with a short schedule one kernel that does both."""
        send = self.send if send is None else send
        if send.numel() < self.send_capacity:
            raise ValueError("send buffer smaller than the pipeline's capacity")
        L, s, p = lib(), _stream(stream), self.params
        if self.mode == "moe":
            T = tokens.numel() * tokens.element_size() // self.unit
            _check(L.vp_pack_rows(_ptr(tokens), T, self.k, self.unit, _ptr(self.dem["sorted_tok"]),
                                  _ptr(self.dem["sorted_slot"]), _ptr(self.dem["dest_off"]), self.self_rank, self.N,
                                  _ptr(self.sched["K"]), _ptr(self.sched["dst"]), _ptr(self.sched["bytes"]),
                                  _ptr(self.sched["send_off"]), _ptr(self.sched["stream_off"]), p.k_max, _ptr(send),
                                  self.send_capacity, _ptr(self.step_off), _ptr(self.status), _ptr(self.pack_ws),
                                  self.pack_ws.numel(), s), "vp_pack_rows")
        else:
            T = tokens.numel() * tokens.element_size() // self.token_stride
            _check(L.vp_pack_heads(_ptr(tokens), T, self.token_stride, _ptr(head_lo), self.unit, self.self_rank,
                                   self.N, _ptr(self.sched["K"]), _ptr(self.sched["dst"]), _ptr(self.sched["bytes"]),
                                   _ptr(self.sched["send_off"]), _ptr(self.sched["stream_off"]), p.k_max, _ptr(send),
                                   self.send_capacity, _ptr(self.step_off), _ptr(self.status), _ptr(self.pack_ws),
                                   self.pack_ws.numel(), s), "vp_pack_heads")
        return send

    def step(self, routing: Optional[torch.Tensor] = None, tokens: Optional[torch.Tensor] = None,
             head_lo: Optional[torch.Tensor] = None, send: Optional[torch.Tensor] = None, stream=None):
        """demand (+ control words) -> plan -> pack for one matrix; returns the send buffer."""
        self.demand_stage(routing, head_lo, stream)
        self.words_stage(stream)
        self.plan_stage(stream)
        return self.pack_stage(tokens, head_lo, send, stream)
