"""Oracle: plain CPU reference of the demand -> plan -> pack path.

TEST INFRASTRUCTURE ONLY.  Only ``tests/``, ``__graft_entry__.smoke()`` and
the CPU-baseline leg of ``bench.py`` may import this package.  It shares no
code with the HIP library (``paper_2609_34340_amd``) and never imports it.

The C++ source ``vp_oracle.cpp`` is compiled with g++ into
``liboracle.so`` next to it; :func:`build` (re)compiles it.
"""
from __future__ import annotations

import ctypes as C
import os
import subprocess
from typing import Optional

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "vp_oracle.cpp")
_LIB = os.path.join(_HERE, "liboracle.so")

OK, INVALID_ARGUMENT, INVALID_DEMAND, NO_PROGRESS, CAPACITY, UNSUPPORTED = range(6)
PIX, PXB, NIC, SYS = 0, 1, 2, 3
TOPO_SYS_P2P = 1

DEFAULT_LAMBDA_NS = 10_000
DEFAULT_N_START = 4
DEFAULT_I_AA = 8


def build(force: bool = True) -> str:
    """Compile the oracle (single-threaded, -O2, no intrinsics)."""
    if force or not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
        tmp = _LIB + ".tmp%d" % os.getpid()
        subprocess.check_call(["g++", "-O2", "-std=c++17", "-shared", "-fPIC", "-o", tmp, _SRC])
        os.replace(tmp, _LIB)
    return _LIB


class _Topo(C.Structure):
    _fields_ = [("n_nodes", C.c_int32), ("sockets_per_node", C.c_int32),
                ("switches_per_socket", C.c_int32), ("gpus_per_switch", C.c_int32),
                ("nics_per_switch", C.c_int32), ("flags", C.c_int32),
                ("pcie_bytes_per_ns", C.c_int64), ("nic_bytes_per_ns", C.c_int64)]


def _topo(topo) -> "_Topo":
    return _Topo(topo.n_nodes, topo.sockets_per_node, topo.switches_per_socket, topo.gpus_per_switch,
                 topo.nics_per_switch, getattr(topo, "flags", 0), topo.pcie_bytes_per_ns, topo.nic_bytes_per_ns)


class _Params(C.Structure):
    _fields_ = [("k_target", C.c_int64), ("lambda_ns", C.c_int64), ("unit_bytes", C.c_int64),
                ("n_start", C.c_int32), ("i_aa", C.c_int32), ("seed", C.c_uint64)]


_lib = None


def lib():
    global _lib
    if _lib is None:
        build(force=False)
        L = C.CDLL(_LIB)
        vp = C.c_void_p
        L.orc_catalog_build.argtypes = [C.POINTER(_Topo), C.c_int, C.POINTER(vp)]
        L.orc_catalog_free.argtypes = [vp]
        L.orc_catalog_info.argtypes = [vp, vp]
        L.orc_catalog_table.argtypes = [vp] + [vp] * 6
        L.orc_catalog_shapes.argtypes = [vp] + [vp] * 5
        L.orc_catalog_families.argtypes = [vp, vp, vp, vp]
        L.orc_catalog_cluster_family.argtypes = [vp, C.c_int32, vp, vp, vp, vp]
        L.orc_demand.argtypes = [vp, C.c_int64, C.c_int32, C.c_int32, C.c_int32, C.c_int32,
                                 C.c_int64, vp, vp, vp, vp, vp]
        L.orc_demand_heads.argtypes = [C.c_int64, vp, C.c_int64, C.c_int32, C.c_int32, vp]
        L.orc_control_words.argtypes = [vp, C.c_int32, C.c_int32, C.c_int32, vp]
        L.orc_rotation_time.argtypes = [C.POINTER(_Topo), vp, C.c_int32, C.c_int64, vp, vp]
        L.orc_receive_counts.argtypes = [vp, vp, C.c_int32, C.c_int32, vp]
        L.orc_plan.argtypes = [vp, vp, C.POINTER(_Params), C.c_int32, vp, vp, vp, vp, vp, vp,
                               vp, C.c_int64, vp]
        L.orc_plan_candidates.argtypes = [vp, vp, C.POINTER(_Params), C.c_int32, vp, vp, vp, vp, vp, vp,
                                          C.c_int64, vp]
        L.orc_start_binding.argtypes = [vp, vp, C.POINTER(_Params), C.c_int64, C.c_int32, C.c_int32, vp, vp]
        L.orc_shape_candidates.argtypes = [vp, vp, C.POINTER(_Params), C.c_int64, C.c_int32, vp, C.c_int64, vp,
                                           vp]
        L.orc_splitmix_stream.argtypes = [C.c_uint64, vp, C.c_int32, vp]
        L.orc_utility_greater.argtypes = [C.c_int64] * 7
        L.orc_modeled_time.argtypes = [vp, C.c_int32, C.c_int32, vp, vp, C.c_int64, vp, vp]
        L.orc_pack_rows.argtypes = [vp, C.c_int64, C.c_int64, vp, vp, C.c_int32, C.c_int32,
                                    C.c_int32, vp, vp, vp, vp]
        L.orc_pack_heads.argtypes = [vp, C.c_int64, C.c_int64, vp, C.c_int64, C.c_int32,
                                     C.c_int32, C.c_int32, vp, vp, vp, vp]
        L.orc_layout.argtypes = [C.c_int32, C.c_int32, vp, vp, vp, vp, vp]
        L.orc_receive.argtypes = [C.c_int32, C.c_int32, C.c_int32, vp, vp, C.c_int64, C.c_int64, vp, vp, vp, vp]
        L.orc_unpack_rows.argtypes = [vp, C.c_int32, C.c_int32, C.c_int32, vp, vp, C.c_int64, C.c_int64, vp,
                                      C.c_int32, vp]
        L.orc_pack_combine.argtypes = [vp, C.c_int32, C.c_int32, C.c_int32, vp, vp, C.c_int64, C.c_int64, vp,
                                       C.c_int32, vp, vp]
        L.orc_unpack_combine.argtypes = [vp, C.c_int32, C.c_int32, C.c_int32, vp, vp, C.c_int64, C.c_int64,
                                         C.c_int64, C.c_int32, vp, vp, vp, vp]
        _lib = L
    return _lib


def _p(a: np.ndarray):
    return a.ctypes.data_as(C.c_void_p)


class OracleError(RuntimeError):
    def __init__(self, status: int, what: str):
        super().__init__("%s failed with status %d" % (what, status))
        self.status = status


class Catalog:
    """Oracle catalog (node-circulant, or the full Alg. 1 catalog with full=True);
    nearest=True keeps only families whose lanes all take their group pair's
    nearest path (the "fixed nearest path" ablation of Sec. 6.3)."""

    def __init__(self, topo, full: bool = False, nearest: bool = False):
        t = _topo(topo)
        h = C.c_void_p()
        st = lib().orc_catalog_build(C.byref(t), (1 if full else 0) | (2 if nearest else 0), C.byref(h))
        if st != OK:
            raise OracleError(st, "orc_catalog_build")
        self._h = h
        self.topo = topo
        self.full = full
        self.nearest = nearest
        info = np.zeros(8, np.int64)
        lib().orc_catalog_info(self._h, _p(info))
        (self.N, self.G, self.g, self.Q, self.n_nodes, self.n_shapes, self.n_families,
         self.n_table) = (int(x) for x in info)

    def __del__(self):
        h = getattr(self, "_h", None)
        if h is not None and _lib is not None:
            _lib.orc_catalog_free(h)
            self._h = None

    def table(self):
        n = self.n_table
        cls, src, dst, copy = (np.zeros(n, np.int32) for _ in range(4))
        bw = np.zeros(n, np.int64)
        res = np.zeros((n, 2), np.int32)
        lib().orc_catalog_table(self._h, _p(cls), _p(src), _p(dst), _p(copy), _p(bw), _p(res))
        return dict(cls=cls, src=src, dst=dst, copy=copy, bw=bw, res=res)

    def shapes(self):
        J = self.n_shapes
        k, fb, fe = (np.zeros(J, np.int32) for _ in range(3))
        if self.full:
            Lm = np.zeros((J, self.G, self.G), np.int32)
            Rm = np.zeros((J, 1), np.int32)
        else:
            Lm = np.zeros((J, self.Q, self.Q), np.int32)
            Rm = np.zeros((J, self.Q, self.Q), np.int32)
        lib().orc_catalog_shapes(self._h, _p(k), _p(fb), _p(fe), _p(Lm), _p(Rm))
        return dict(k=k, fam_begin=fb, fam_end=fe, L=Lm, R=Rm)

    def families(self):
        F = self.n_families
        w = self.N if self.full else self.Q * self.g
        shape, k = np.zeros(F, np.int32), np.zeros(F, np.int32)
        ids = np.zeros((F, w), np.int32)
        lib().orc_catalog_families(self._h, _p(shape), _p(k), _p(ids))
        return dict(shape=shape, k=k, ids=ids)

    def cluster_family(self, f: int):
        n = self.N
        cls, a, d, ids = (np.zeros(n, np.int32) for _ in range(4))
        st = lib().orc_catalog_cluster_family(self._h, f, _p(cls), _p(a), _p(d), _p(ids))
        if st != OK:
            raise OracleError(st, "orc_catalog_cluster_family")
        return dict(cls=cls, a=a, d=d, id=ids)

    def plan(self, D: np.ndarray, unit: int, k_target: Optional[int] = None,
             lambda_ns: int = DEFAULT_LAMBDA_NS, n_start: int = DEFAULT_N_START,
             i_aa: int = DEFAULT_I_AA, seed: int = 0, k_max: Optional[int] = None,
             trace_cap: int = 0, check: bool = True):
        """Alg. 2 on demand D (int64 [N, N] bytes).  Returns a dict schedule."""
        N = self.N
        D = np.ascontiguousarray(D, dtype=np.int64)
        assert D.shape == (N, N)
        k_target = 2 * N if k_target is None else k_target
        k_max = 8 * N if k_max is None else k_max
        P = _Params(k_target, lambda_ns, unit, n_start, i_aa, seed)
        K = np.zeros(1, np.int32)
        cap = max(k_max, 1)
        fam = np.full(cap, -1, np.int32)
        dst = np.full((cap, N), -1, np.int32)
        inst = np.full((cap, N), -1, np.int32)
        nbytes = np.zeros((cap, N), np.int64)
        tau = np.zeros(1, np.int64)
        trace = np.zeros((max(trace_cap, 1), 5), np.int64)
        tn = np.zeros(1, np.int64)
        st = lib().orc_plan(self._h, _p(D), C.byref(P), k_max, _p(K), _p(fam), _p(dst),
                            _p(inst), _p(nbytes), _p(tau), _p(trace) if trace_cap else None,
                            trace_cap, _p(tn))
        if check and st != OK:
            raise OracleError(st, "orc_plan")
        k = int(K[0])
        out = dict(status=st, K=k, family=fam[:k].copy(), dst=dst[:k].copy(),
                   inst=inst[:k].copy(), bytes=nbytes[:k].copy(), tau=int(tau[0]))
        if trace_cap:
            out["trace"] = trace[: int(tn[0])].copy()
        return out

    def plan_candidates(self, D: np.ndarray, unit: int, k_target: Optional[int] = None,
                        lambda_ns: int = DEFAULT_LAMBDA_NS, n_start: int = DEFAULT_N_START,
                        i_aa: int = DEFAULT_I_AA, seed: int = 0, k_max: Optional[int] = None,
                        log_cap: int = 100000):
        """The plan of D together with every candidate it evaluated: a list of
        dicts (iteration, family, S, xm, bm, and per instance in family order
        src, dst and the volume x)."""
        N = self.N
        D = np.ascontiguousarray(D, dtype=np.int64)
        k_target = 2 * N if k_target is None else k_target
        k_max = 8 * N if k_max is None else k_max
        P = _Params(k_target, lambda_ns, unit, n_start, i_aa, seed)
        K = np.zeros(1, np.int32)
        cap = max(k_max, 1)
        fam = np.full(cap, -1, np.int32)
        dst = np.full((cap, N), -1, np.int32)
        inst = np.full((cap, N), -1, np.int32)
        nbytes = np.zeros((cap, N), np.int64)
        w = 5 + 3 * N
        log = np.zeros((log_cap, w), np.int64)
        ln = np.zeros(1, np.int64)
        st = lib().orc_plan_candidates(self._h, _p(D), C.byref(P), k_max, _p(K), _p(fam), _p(dst), _p(inst),
                                       _p(nbytes), _p(log), log_cap, _p(ln))
        if st != OK:
            raise OracleError(st, "orc_plan_candidates")
        k = int(K[0])
        n = int(ln[0])
        assert n < log_cap, "candidate log full"
        cands = []
        for r in log[:n]:
            lanes = r[5:].reshape(N, 3)
            cands.append(dict(iter=int(r[0]), family=int(r[1]), S=int(r[2]), xm=int(r[3]), bm=int(r[4]),
                              src=lanes[:, 0].copy(), dst=lanes[:, 1].copy(), x=lanes[:, 2].copy()))
        sched = dict(status=st, K=k, family=fam[:k].copy(), dst=dst[:k].copy(), inst=inst[:k].copy(),
                     bytes=nbytes[:k].copy())
        return sched, cands

    def shape_candidates(self, D: np.ndarray, unit: int, shape: int, iteration: int = 0,
                         k_target: Optional[int] = None, lambda_ns: int = DEFAULT_LAMBDA_NS,
                         n_start: int = DEFAULT_N_START, i_aa: int = DEFAULT_I_AA, seed: int = 0):
        """Steps 2-3 of the planner on `shape` with D as the residual: the
        candidates of every family of the bucket (as plan_candidates lists
        them) and the family the planner keeps."""
        N = self.N
        D = np.ascontiguousarray(D, dtype=np.int64)
        k_target = 2 * N if k_target is None else k_target
        P = _Params(k_target, lambda_ns, unit, n_start, i_aa, seed)
        cap = 4096
        log = np.zeros((cap, 5 + 3 * N), np.int64)
        ln = np.zeros(1, np.int64)
        chosen = np.zeros(1, np.int32)
        st = lib().orc_shape_candidates(self._h, _p(D), C.byref(P), iteration, shape, _p(log), cap, _p(ln),
                                        _p(chosen))
        if st != OK:
            raise OracleError(st, "orc_shape_candidates")
        n = int(ln[0])
        assert n < cap
        cands = []
        for r in log[:n]:
            lanes = r[5:].reshape(N, 3)
            cands.append(dict(iter=int(r[0]), family=int(r[1]), S=int(r[2]), xm=int(r[3]), bm=int(r[4]),
                              src=lanes[:, 0].copy(), dst=lanes[:, 1].copy(), x=lanes[:, 2].copy()))
        return cands, int(chosen[0])

    def start_binding(self, D: np.ndarray, unit: int, family: int, start: int, iteration: int = 0,
                      k_target: Optional[int] = None, seed: int = 0):
        """MultiStartAA's start binding `start` of `family` on residual D
        (before any sweep): (src, dst) rank per instance in family order."""
        N = self.N
        D = np.ascontiguousarray(D, dtype=np.int64)
        k_target = 2 * N if k_target is None else k_target
        P = _Params(k_target, DEFAULT_LAMBDA_NS, unit, DEFAULT_N_START, DEFAULT_I_AA, seed)
        src = np.zeros(N, np.int32)
        dst = np.zeros(N, np.int32)
        st = lib().orc_start_binding(self._h, _p(D), C.byref(P), iteration, family, start, _p(src), _p(dst))
        if st != OK:
            raise OracleError(st, "orc_start_binding")
        return src, dst

    def modeled_time(self, sched, lambda_ns: int = DEFAULT_LAMBDA_NS):
        """Eq. (2) as an exact fraction (numerator, denominator) in ns."""
        K = int(sched["K"])
        inst = np.ascontiguousarray(sched["inst"], np.int32)
        nb = np.ascontiguousarray(sched["bytes"], np.int64)
        num, den = np.zeros(1, np.int64), np.zeros(1, np.int64)
        lib().orc_modeled_time(self._h, K, self.N, _p(inst), _p(nb), lambda_ns, _p(num), _p(den))
        return int(num[0]), int(den[0])


def splitmix_stream(n: int, state: int = 0, key=None) -> np.ndarray:
    """SplitMix64 outputs from a raw state, or from the keyed state of the
    random AA starts when key = (seed, iteration, family, start, group, side)."""
    out = np.zeros(n, np.uint64)
    f = None if key is None else np.asarray(key, np.uint64)
    lib().orc_splitmix_stream(state, None if f is None else _p(f), n, _p(out))
    return out


def utility_greater(S1, x1, b1, S2, x2, b2, lambda_ns) -> bool:
    """The planner's exact comparison of two Eq. (10) utilities."""
    return bool(lib().orc_utility_greater(S1, x1, b1, S2, x2, b2, lambda_ns))


def demand(routing: np.ndarray, n_ranks: int, n_experts: int, self_rank: int, unit: int):
    """One source rank's demand row, expert counts, (expert, token) order (the
    token and routing slot of every assignment) and offsets."""
    r = np.ascontiguousarray(routing, dtype=np.int32)
    T, k = r.shape
    row = np.zeros(n_ranks, np.int64)
    counts = np.zeros(n_experts, np.int32)
    order = np.zeros(T * k, np.int32)
    slot = np.zeros(T * k, np.uint8)
    off = np.zeros(n_ranks + 1, np.int64)
    st = lib().orc_demand(_p(r), T, k, n_experts, n_ranks, self_rank, unit, _p(row), _p(counts),
                          _p(order), _p(slot), _p(off))
    if st != OK:
        raise OracleError(st, "orc_demand")
    return dict(row=row, counts=counts, sorted_tok=order, sorted_slot=slot, dest_off=off)


def control_words(counts: np.ndarray, n_ranks: int, self_rank: int) -> np.ndarray:
    """One source rank's sparse-EP control words (uint32 [N]) from its expert
    counts (int32 [E])."""
    c = np.ascontiguousarray(counts, dtype=np.int32)
    words = np.zeros(n_ranks, np.uint32)
    st = lib().orc_control_words(_p(c), c.shape[0], n_ranks, self_rank, _p(words))
    if st != OK:
        raise OracleError(st, "orc_control_words")
    return words


def receive_counts(words: np.ndarray, signal: np.ndarray, n_local: int) -> np.ndarray:
    """A receiver's rows per (source, local expert) (int32 [N, L]) from the
    control words it received (uint32 [N]) and the per-expert signal counts
    (int32 [N, L]; read only for active, non-designated experts)."""
    w = np.ascontiguousarray(words, dtype=np.uint32)
    sg = np.ascontiguousarray(signal, dtype=np.int32)
    N = w.shape[0]
    out = np.zeros((N, n_local), np.int32)
    st = lib().orc_receive_counts(_p(w), _p(sg), N, n_local, _p(out))
    if st != OK:
        raise OracleError(st, "orc_receive_counts")
    return out


def rotation_time(topo, D: np.ndarray, nearest: bool, lambda_ns: int = DEFAULT_LAMBDA_NS):
    """Exact (num, den) ns of the fixed cyclic peer rotation on D (Sec. 6.3)."""
    t = _topo(topo)
    Dc = np.ascontiguousarray(D, np.int64)
    num, den = np.zeros(1, np.int64), np.zeros(1, np.int64)
    st = lib().orc_rotation_time(C.byref(t), _p(Dc), 1 if nearest else 0, lambda_ns, _p(num), _p(den))
    if st != OK:
        raise OracleError(st, "orc_rotation_time")
    return int(num[0]), int(den[0])


def demand_heads(tokens: int, head_lo: np.ndarray, head_bytes: int, self_rank: int):
    hl = np.ascontiguousarray(head_lo, dtype=np.int64)
    N = hl.shape[0] - 1
    row = np.zeros(N, np.int64)
    st = lib().orc_demand_heads(tokens, _p(hl), head_bytes, N, self_rank, _p(row))
    if st != OK:
        raise OracleError(st, "orc_demand_heads")
    return row


def demand_matrix(rows) -> np.ndarray:
    return np.stack(list(rows)).astype(np.int64)


def pack_rows(tokens: np.ndarray, row_bytes: int, sorted_tok, dest_off, self_rank: int, sched):
    tok = np.ascontiguousarray(tokens).view(np.uint8).reshape(-1)
    T = tok.size // row_bytes
    N = sched["dst"].shape[1] if sched["K"] else len(dest_off) - 1
    K = int(sched["K"])
    dst = np.ascontiguousarray(sched["dst"], np.int32)
    nb = np.ascontiguousarray(sched["bytes"], np.int64)
    total = int(nb[:, self_rank].sum()) if K else 0
    send = np.zeros(total, np.uint8)
    step_off = np.zeros(K + 1, np.int64)
    st = lib().orc_pack_rows(_p(tok), T, row_bytes, _p(np.ascontiguousarray(sorted_tok, np.int32)),
                             _p(np.ascontiguousarray(dest_off, np.int64)), self_rank, N, K,
                             _p(dst), _p(nb), _p(send), _p(step_off))
    if st != OK:
        raise OracleError(st, "orc_pack_rows")
    return send, step_off


def pack_heads(act: np.ndarray, token_stride: int, head_lo, head_bytes: int, self_rank: int, sched):
    a = np.ascontiguousarray(act).view(np.uint8).reshape(-1)
    T = a.size // token_stride
    hl = np.ascontiguousarray(head_lo, np.int64)
    N = hl.shape[0] - 1
    K = int(sched["K"])
    dst = np.ascontiguousarray(sched["dst"], np.int32)
    nb = np.ascontiguousarray(sched["bytes"], np.int64)
    total = int(nb[:, self_rank].sum()) if K else 0
    send = np.zeros(total, np.uint8)
    step_off = np.zeros(K + 1, np.int64)
    st = lib().orc_pack_heads(_p(a), T, token_stride, _p(hl), head_bytes, self_rank, N, K,
                              _p(dst), _p(nb), _p(send), _p(step_off))
    if st != OK:
        raise OracleError(st, "orc_pack_heads")
    return send, step_off


# ------------------------------------------------------- receive / combine

def slot_bytes(row_bytes: int) -> int:
    """Receive slot of one row: rounded up to 128 bytes (Sec. 5 low-latency protocol)."""
    return (row_bytes + 127) // 128 * 128


def _sched(s):
    dst = np.ascontiguousarray(s["dst"], dtype=np.int32)
    nb = np.ascontiguousarray(s["bytes"], dtype=np.int64)
    return int(s["K"]), dst, nb


def layout(s, N: int):
    """Sec. 5 buffer layout of a schedule: send, stream and receive offsets per step and lane."""
    K, dst, nb = _sched(s)
    so, co, ro = (np.zeros((K, N), np.int64) for _ in range(3))
    st = lib().orc_layout(K, N, _p(dst), _p(nb), _p(so), _p(co), _p(ro))
    if st != OK:
        raise OracleError(st, "orc_layout")
    return dict(send_off=so, stream_off=co, recv_off=ro)


def received_rows(s, N: int, r: int, row_bytes: int) -> int:
    K, dst, nb = _sched(s)
    return int(nb[dst == r].sum()) // row_bytes


def receive(r: int, N: int, s, row_bytes: int, sends, step_offs):
    """Transfer emulation (test infrastructure): rank r's receive buffer from
    every rank's send buffer and step offsets, one row per 128-B slot."""
    K, dst, nb = _sched(s)
    base = np.zeros(N, np.int64)
    base[1:] = np.cumsum([x.size for x in sends])[:-1]
    allsend = np.ascontiguousarray(np.concatenate(sends)) if sends else np.zeros(1, np.uint8)
    offs = np.ascontiguousarray(np.stack([np.asarray(o, np.int64)[:K + 1] for o in step_offs]))
    sb = slot_bytes(row_bytes)
    recv = np.zeros(max(received_rows(s, N, r, row_bytes), 1) * sb, np.uint8)
    st = lib().orc_receive(r, N, K, _p(dst), _p(nb), row_bytes, sb, _p(allsend), _p(base), _p(offs), _p(recv))
    if st != OK:
        raise OracleError(st, "orc_receive")
    return recv


def expert_rows(counts: np.ndarray, r: int, N: int) -> int:
    E = counts.shape[1]
    eloc = E // N
    return int(counts[:, r * eloc:(r + 1) * eloc].sum())


def unpack_rows(recv: np.ndarray, r: int, N: int, s, row_bytes: int, counts: np.ndarray):
    """Dispatch receive of rank r into its expert-major output (128-B slots)."""
    K, dst, nb = _sched(s)
    c = np.ascontiguousarray(counts, dtype=np.int32)
    sb = slot_bytes(row_bytes)
    out = np.zeros(max(expert_rows(c, r, N), 1) * sb, np.uint8)
    st = lib().orc_unpack_rows(_p(np.ascontiguousarray(recv)), r, N, K, _p(dst), _p(nb), row_bytes, sb, _p(c),
                               c.shape[1], _p(out))
    if st != OK:
        raise OracleError(st, "orc_unpack_rows")
    return out


def pack_combine(out: np.ndarray, r: int, N: int, s, row_bytes: int, counts: np.ndarray):
    """Combine send of rank r (schedule planned on the transposed demand)."""
    K, dst, nb = _sched(s)
    c = np.ascontiguousarray(counts, dtype=np.int32)
    send = np.zeros(max(int(nb[:, r].sum()), 1), np.uint8)
    step_off = np.zeros(K + 1, np.int64)
    st = lib().orc_pack_combine(_p(np.ascontiguousarray(out)), r, N, K, _p(dst), _p(nb), row_bytes,
                                slot_bytes(row_bytes), _p(c), c.shape[1], _p(send), _p(step_off))
    if st != OK:
        raise OracleError(st, "orc_pack_combine")
    return send, step_off


def unpack_combine(recv: np.ndarray, self_rank: int, N: int, s, row_bytes: int, T: int, k: int,
                   sorted_tok: np.ndarray, sorted_slot: np.ndarray, dest_off: np.ndarray,
                   combined: np.ndarray = None):
    """Combine receive at its source rank: every returned row into its
    (token, routing slot) slot of combined [T, k] (128-B slots)."""
    K, dst, nb = _sched(s)
    sb = slot_bytes(row_bytes)
    if combined is None:
        combined = np.zeros(T * k * sb, np.uint8)
    st = lib().orc_unpack_combine(_p(np.ascontiguousarray(recv)), self_rank, N, K, _p(dst), _p(nb), row_bytes,
                                  sb, T, k, _p(np.ascontiguousarray(sorted_tok, dtype=np.int32)),
                                  _p(np.ascontiguousarray(sorted_slot, dtype=np.uint8)),
                                  _p(np.ascontiguousarray(dest_off, dtype=np.int64)), _p(combined))
    if st != OK:
        raise OracleError(st, "orc_unpack_combine")
    return combined
