"""Thin ctypes binding of libasap.so (the C ABI declared in include/asap.h).

Functions carry the C names and only marshal arguments: host arrays become
pointers, torch CUDA tensors become device pointers, the stream defaults to
torch's current stream.  Every non-OK status raises AsapError with the
library's message.  All compute runs in the HIP kernels of libasap.so; if the
library is missing this module raises instead of falling back to anything.

`Session` bundles one context with torch-allocated device memory (workspace
and the two model buffers): PyTorch provides memory and streams only.
"""
from __future__ import annotations

import ctypes as C
import os

import numpy as np

_LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libasap.so")

OK, E_INVALID_ARG, E_GRAPH, E_STATE, E_DEVICE, E_EPOCH = range(6)
STATUS_NAMES = {0: "ASAP_OK", 1: "ASAP_E_INVALID_ARG", 2: "ASAP_E_GRAPH", 3: "ASAP_E_STATE",
                4: "ASAP_E_DEVICE", 5: "ASAP_E_EPOCH"}
LOSS = {"logistic": 0, "hinge": 1}
LR = {"const": 0, "inv_sqrt": 1}
ALLOW_NON_DS = 1

# Every symbol include/asap.h declares.
EXPORTS = (
    "asap_graph_ring", "asap_graph_root_expander", "asap_graph_chain", "asap_graph_complete",
    "asap_graph_random_regular",
    "asap_metropolis_weights", "asap_schedule", "asap_create", "asap_workspace_size",
    "asap_bind_workspace", "asap_bind_models", "asap_bind_dense", "asap_bind_csr", "asap_set_csr_members",
    "asap_get_csr_members",
    "asap_local_sgd", "asap_prepare_sgd", "asap_stochastic_reduce", "asap_round", "asap_run_rounds",
    "asap_current",
    "asap_set_round", "asap_drop_workers", "asap_get_graph", "asap_schedule_device", "asap_metrics", "asap_check",
    "asap_metrics_noalloc", "asap_rounds_plan_size", "asap_bind_rounds_plan",
    "asap_debug_set_tag", "asap_last_error", "asap_destroy",
)


class AsapError(RuntimeError):
    def __init__(self, status: int, message: str):
        super().__init__(f"{STATUS_NAMES.get(status, status)}: {message}")
        self.status = status


class SgdParams(C.Structure):
    _fields_ = [("loss", C.c_int32), ("lr_kind", C.c_int32), ("lr0", C.c_float),
                ("l2", C.c_float), ("batch", C.c_int32), ("local_steps", C.c_int32),
                ("seed", C.c_uint64)]


_lib = None


def lib():
    """Load libasap.so once; raise loudly if it has not been built."""
    global _lib
    if _lib is not None:
        return _lib
    # torch first when it is there: the library then binds to the HIP runtime
    # torch has loaded instead of loading a second one beside it
    try:
        import torch  # noqa: F401
    except ImportError:
        pass
    if not os.path.exists(_LIB_PATH):
        raise RuntimeError(f"{_LIB_PATH} is missing: build it with `python -m paper_1612_08608_amd.build`")
    L = C.CDLL(_LIB_PATH)
    p, i32, i64, u32, u64, sz = C.c_void_p, C.c_int32, C.c_int64, C.c_uint32, C.c_uint64, C.c_size_t
    sigs = {
        "asap_graph_ring": [i32, p, p],
        "asap_graph_root_expander": [i32, p, p],
        "asap_graph_chain": [i32, p, p],
        "asap_graph_complete": [i32, p, p],
        "asap_graph_random_regular": [i32, i32, u64, p, p],
        "asap_metropolis_weights": [i32, p, p, p],
        "asap_schedule": [i64, u64, i32, i64, p],
        "asap_create": [i32, i64, p, p, p, u32, C.POINTER(p)],
        "asap_workspace_size": [p, C.POINTER(sz)],
        "asap_bind_workspace": [p, p, sz, p],
        "asap_bind_models": [p, p, p, i64, p],
        "asap_bind_dense": [p, p, p, i64, i64],
        "asap_bind_csr": [p, p, p, p, p, i64, i64, p],
        "asap_set_csr_members": [p, i32],
        "asap_get_csr_members": [p, C.POINTER(i32)],
        "asap_local_sgd": [p, C.POINTER(SgdParams), p],
        "asap_prepare_sgd": [p, C.POINTER(SgdParams), p],
        "asap_stochastic_reduce": [p, p],
        "asap_round": [p, C.POINTER(SgdParams), p],
        "asap_run_rounds": [p, C.POINTER(SgdParams), i64, i32, p],
        "asap_current": [p, C.POINTER(i32), C.POINTER(i64), C.POINTER(i32)],
        "asap_set_round": [p, i64, i32, p],
        "asap_drop_workers": [p, i32, p, p, p, p, u32, p],
        "asap_get_graph": [p, C.POINTER(i32), C.POINTER(i64), p, p, p],
        "asap_schedule_device": [p, u64, i64, p, p],
        "asap_metrics": [p, i32, C.c_float, p, p],
        "asap_metrics_noalloc": [p, i32, C.c_float, p, p],
        "asap_rounds_plan_size": [p, i64, C.POINTER(sz)],
        "asap_bind_rounds_plan": [p, p, sz, p],
        "asap_check": [p, p, C.POINTER(i32)],
        "asap_debug_set_tag": [p, i32, i32, i64, p],
    }
    for name, args in sigs.items():
        f = getattr(L, name)
        f.argtypes = args
        f.restype = C.c_int
    L.asap_last_error.argtypes = [p]
    L.asap_last_error.restype = C.c_char_p
    L.asap_destroy.argtypes = [p]
    L.asap_destroy.restype = None
    _lib = L
    return L


def _check(status: int, ctx=None):
    if status != OK:
        msg = lib().asap_last_error(ctx)
        raise AsapError(status, msg.decode() if msg else "")


def _host(a, dtype):
    a = np.ascontiguousarray(a, dtype=dtype)
    return a, a.ctypes.data_as(C.c_void_p)


def _dev(t):
    """Device pointer of a torch CUDA tensor (or a raw integer address)."""
    if t is None:
        return None
    if isinstance(t, int):
        return C.c_void_p(t)
    if not t.is_cuda:
        raise ValueError("expected a device tensor")
    if not t.is_contiguous():
        raise ValueError("expected a contiguous tensor")
    return C.c_void_p(t.data_ptr())


def _stream(stream):
    if stream is None:
        import torch
        return C.c_void_p(torch.cuda.current_stream().cuda_stream)
    if isinstance(stream, int):
        return C.c_void_p(stream)
    return C.c_void_p(stream.cuda_stream)


# ---------------------------------------------------------------------------
# host-only builders
# ---------------------------------------------------------------------------
def asap_graph_ring(n: int):
    ptr = np.zeros(n + 1, np.int32)
    idx = np.zeros(3 * max(n, 0), np.int32)
    _check(lib().asap_graph_ring(n, ptr.ctypes.data_as(C.c_void_p), idx.ctypes.data_as(C.c_void_p)))
    return ptr, idx


def asap_graph_root_expander(n: int):
    ptr = np.zeros(n + 1, np.int32)
    idx = np.zeros(3 * max(n, 0), np.int32)
    _check(lib().asap_graph_root_expander(n, ptr.ctypes.data_as(C.c_void_p), idx.ctypes.data_as(C.c_void_p)))
    return ptr, idx


def asap_graph_chain(n: int):
    ptr = np.zeros(n + 1, np.int32)
    idx = np.zeros(2 * max(n, 0), np.int32)
    _check(lib().asap_graph_chain(n, ptr.ctypes.data_as(C.c_void_p), idx.ctypes.data_as(C.c_void_p)))
    return ptr, idx


def asap_graph_complete(n: int):
    ptr = np.zeros(n + 1, np.int32)
    idx = np.zeros(max(n, 0) * max(n, 0), np.int32)
    _check(lib().asap_graph_complete(n, ptr.ctypes.data_as(C.c_void_p), idx.ctypes.data_as(C.c_void_p)))
    return ptr, idx


def asap_graph_random_regular(n: int, d: int, seed: int):
    ptr = np.zeros(max(n, 0) + 1, np.int32)
    idx = np.zeros(max(n, 0) * (max(d, 0) + 1), np.int32)
    _check(lib().asap_graph_random_regular(n, d, seed, ptr.ctypes.data_as(C.c_void_p),
                                           idx.ctypes.data_as(C.c_void_p)))
    return ptr, idx


def asap_metropolis_weights(ptr, idx):
    ptr, pp = _host(ptr, np.int32)
    idx, ip = _host(idx, np.int32)
    w = np.zeros(idx.size, np.float32)
    _check(lib().asap_metropolis_weights(ptr.size - 1, pp, ip, w.ctypes.data_as(C.c_void_p)))
    return w


def asap_schedule(samples: int, seed: int, worker: int, round_: int):
    out = np.zeros(max(samples, 0), np.int32)
    _check(lib().asap_schedule(samples, seed, worker, round_, out.ctypes.data_as(C.c_void_p)))
    return out


# ---------------------------------------------------------------------------
# context calls (ctx is a ctypes c_void_p)
# ---------------------------------------------------------------------------
def asap_create(n: int, dim: int, ptr, idx, w, flags: int = 0):
    ptr, pp = _host(ptr, np.int32)
    idx, ip = _host(idx, np.int32)
    w, wp = _host(w, np.float32)
    ctx = C.c_void_p()
    _check(lib().asap_create(n, dim, pp, ip, wp, flags, C.byref(ctx)))
    return ctx


def asap_workspace_size(ctx) -> int:
    out = C.c_size_t()
    _check(lib().asap_workspace_size(ctx, C.byref(out)), ctx)
    return out.value


def asap_bind_workspace(ctx, dev, nbytes: int, stream=None):
    _check(lib().asap_bind_workspace(ctx, _dev(dev), nbytes, _stream(stream)), ctx)


def asap_bind_models(ctx, buf0, buf1, ld: int, stream=None):
    _check(lib().asap_bind_models(ctx, _dev(buf0), _dev(buf1), ld, _stream(stream)), ctx)


def asap_bind_dense(ctx, X, y, samples: int, ldx: int):
    _check(lib().asap_bind_dense(ctx, _dev(X), _dev(y), samples, ldx), ctx)


def asap_set_csr_members(ctx, members: int):
    _check(lib().asap_set_csr_members(ctx, int(members)), ctx)


def asap_get_csr_members(ctx) -> int:
    m = C.c_int32(0)
    _check(lib().asap_get_csr_members(ctx, C.byref(m)), ctx)
    return m.value


def asap_bind_csr(ctx, row_ptr, col, val, y, samples: int, nnz: int, stream=None):
    _check(lib().asap_bind_csr(ctx, _dev(row_ptr), _dev(col), _dev(val), _dev(y), samples, nnz,
                               _stream(stream)), ctx)


def sgd_params(loss="logistic", lr_kind="const", lr0=0.1, l2=0.0, batch=1, seed=0, local_steps=0) -> SgdParams:
    return SgdParams(LOSS.get(loss, loss), LR.get(lr_kind, lr_kind), lr0, l2, batch, local_steps, seed)


def asap_local_sgd(ctx, params: SgdParams, stream=None):
    _check(lib().asap_local_sgd(ctx, C.byref(params), _stream(stream)), ctx)


def asap_prepare_sgd(ctx, params: SgdParams, stream=None):
    _check(lib().asap_prepare_sgd(ctx, C.byref(params), _stream(stream)), ctx)


def asap_stochastic_reduce(ctx, stream=None):
    _check(lib().asap_stochastic_reduce(ctx, _stream(stream)), ctx)


def asap_round(ctx, params: SgdParams, stream=None):
    _check(lib().asap_round(ctx, C.byref(params), _stream(stream)), ctx)


def asap_run_rounds(ctx, params: SgdParams, rounds: int, wait_ms: int = 0, stream=None):
    _check(lib().asap_run_rounds(ctx, C.byref(params), int(rounds), int(wait_ms), _stream(stream)), ctx)


def asap_current(ctx):
    b, r, h = C.c_int32(), C.c_int64(), C.c_int32()
    _check(lib().asap_current(ctx, C.byref(b), C.byref(r), C.byref(h)), ctx)
    return b.value, r.value, h.value


def asap_set_round(ctx, round_: int, buffer: int, stream=None):
    _check(lib().asap_set_round(ctx, round_, buffer, _stream(stream)), ctx)


def asap_drop_workers(ctx, dropped, ptr, idx, w, flags: int = 0, stream=None):
    d, dp = _host(dropped, np.int32)
    ptr, pp = _host(ptr, np.int32)
    idx, ip = _host(idx, np.int32)
    w, wp = _host(w, np.float32)
    _check(lib().asap_drop_workers(ctx, int(d.size), dp, pp, ip, wp, flags, _stream(stream)), ctx)


def asap_get_graph(ctx):
    """(nbr_ptr, nbr_idx, nbr_w) of the graph the context runs on (host copies)."""
    n, m = C.c_int32(), C.c_int64()
    _check(lib().asap_get_graph(ctx, C.byref(n), C.byref(m), None, None, None), ctx)
    ptr = np.empty(n.value + 1, np.int32)
    idx = np.empty(m.value, np.int32)
    w = np.empty(m.value, np.float32)
    _check(lib().asap_get_graph(ctx, C.byref(n), C.byref(m), ptr.ctypes.data, idx.ctypes.data, w.ctypes.data), ctx)
    return ptr, idx, w


def asap_schedule_device(ctx, seed: int, round_: int, out, stream=None):
    _check(lib().asap_schedule_device(ctx, seed, round_, _dev(out), _stream(stream)), ctx)


def asap_metrics(ctx, loss="logistic", l2=0.0, stream=None):
    out = np.zeros(4, np.float64)
    _check(lib().asap_metrics(ctx, LOSS.get(loss, loss), l2, out.ctypes.data_as(C.c_void_p),
                              _stream(stream)), ctx)
    return out


def asap_metrics_noalloc(ctx, loss="logistic", l2=0.0, stream=None):
    out = np.zeros(4, np.float64)
    _check(lib().asap_metrics_noalloc(ctx, LOSS.get(loss, loss), l2, out.ctypes.data_as(C.c_void_p),
                                      _stream(stream)), ctx)
    return out


def asap_rounds_plan_size(ctx, passes: int) -> int:
    out = C.c_size_t(0)
    _check(lib().asap_rounds_plan_size(ctx, int(passes), C.byref(out)), ctx)
    return out.value


def asap_bind_rounds_plan(ctx, dev, nbytes: int, stream=None):
    _check(lib().asap_bind_rounds_plan(ctx, _dev(dev), int(nbytes), _stream(stream)), ctx)


def asap_check(ctx, stream=None):
    """Returns (status, bad_worker) without raising, so callers can inspect E_EPOCH."""
    bad = C.c_int32(-1)
    st = lib().asap_check(ctx, _stream(stream), C.byref(bad))
    return st, bad.value


def asap_debug_set_tag(ctx, buffer: int, worker: int, value: int, stream=None):
    _check(lib().asap_debug_set_tag(ctx, buffer, worker, value, _stream(stream)), ctx)


def asap_last_error(ctx=None) -> str:
    m = lib().asap_last_error(ctx)
    return m.decode() if m else ""


def asap_destroy(ctx):
    if ctx:
        lib().asap_destroy(ctx)


def model_ld(dim: int) -> int:
    """Row stride (floats) for the model buffers: dim rounded up to 64, plus
    128 when that is a multiple of 1024.  Rows a multiple of 4 KiB apart all
    start in the same DRAM channel and bank, which costs the reduce, whose
    loads touch every row at the same column, up to a third of its rate."""
    ld = (int(dim) + 63) // 64 * 64
    return ld + 128 if ld % 1024 == 0 else ld


# ---------------------------------------------------------------------------
# Session: one context plus its torch-owned device memory
# ---------------------------------------------------------------------------
class Session:
    """A context with torch-allocated workspace and model buffers on `device`.

    Data tensors passed to bind_dense / bind_csr are kept referenced here so
    that they outlive the context, as the C ABI requires.
    """

    def __init__(self, n, dim, ptr, idx, w, flags=0, device="cuda:0"):
        import torch
        self.torch = torch
        self.device = torch.device(device)
        self.n, self.dim = int(n), int(dim)
        self.ld = model_ld(self.dim)
        self.ctx = asap_create(self.n, self.dim, ptr, idx, w, flags)
        self.bufs = [torch.zeros((self.n, self.ld), dtype=torch.float32, device=self.device) for _ in range(2)]
        self._keep = []
        self._data = None
        self.ws = None
        asap_bind_models(self.ctx, self.bufs[0], self.bufs[1], self.ld)

    # binds --------------------------------------------------------------
    def set_models(self, W, stream=None):
        """Copy W [n, dim] into buffer 0 and restart at round 0."""
        t = self.torch
        W = t.as_tensor(W, dtype=t.float32)
        self.bufs[0].zero_()
        self.bufs[0][:self.n, :self.dim].copy_(W.to(self.device))
        asap_bind_models(self.ctx, self.bufs[0], self.bufs[1], self.ld, stream)
        self.ws = None

    def bind_dense(self, X, y):
        t = self.torch
        X = t.as_tensor(X, dtype=t.float32)
        n, S, D = X.shape
        ldx = (D + 3) // 4 * 4
        if ldx != D:
            X = t.nn.functional.pad(X, (0, ldx - D))
        X = X.to(self.device).contiguous()
        y = t.as_tensor(y, dtype=t.float32).to(self.device).contiguous()
        self._keep += [X, y]
        asap_bind_dense(self.ctx, X, y, S, ldx)
        self._data = ("dense", X, y, S)
        self.ws = None

    def bind_csr(self, row_ptr, col, val, y, samples):
        t = self.torch
        rp = t.as_tensor(np.asarray(row_ptr, np.int64)).to(self.device)
        cl = t.as_tensor(np.asarray(col, np.int32)).to(self.device)
        vl = t.as_tensor(np.asarray(val, np.float32)).to(self.device)
        yy = t.as_tensor(np.asarray(y, np.float32)).to(self.device)
        self._keep += [rp, cl, vl, yy]
        asap_bind_csr(self.ctx, rp, cl, vl, yy, samples, int(cl.numel()))
        self._data = ("csr", rp, cl, vl, yy, int(samples))
        self.ws = None

    def set_csr_members(self, members):
        """Workgroups per worker of the planned CSR pass (0: the library's choice)."""
        asap_set_csr_members(self.ctx, members)
        self.ws = None

    def csr_members(self):
        return asap_get_csr_members(self.ctx)

    def ready(self, stream=None):
        """(Re)bind a workspace of the size the current bindings need."""
        if self.ws is None:
            nbytes = asap_workspace_size(self.ctx)
            self.ws = self.torch.empty(max(nbytes, 256), dtype=self.torch.uint8, device=self.device)
            asap_bind_workspace(self.ctx, self.ws, self.ws.numel(), stream)
        return self

    # hot path -----------------------------------------------------------
    def local_sgd(self, params, stream=None):
        asap_local_sgd(self.ready().ctx, params, stream)

    def prepare_sgd(self, params, stream=None):
        asap_prepare_sgd(self.ready().ctx, params, stream)

    def stochastic_reduce(self, stream=None):
        asap_stochastic_reduce(self.ready().ctx, stream)

    def round(self, params, stream=None):
        asap_round(self.ready().ctx, params, stream)

    def run_rounds(self, params, rounds, wait_ms=0, stream=None):
        """`rounds` rounds in one launch with per-worker NOTIFY-ACK."""
        asap_run_rounds(self.ready().ctx, params, rounds, wait_ms, stream)

    def bind_rounds_plan(self, passes, stream=None):
        """Device memory for the plans of `passes` passes, so that a
        multi-round launch over CSR shards runs the planned pass."""
        nbytes = asap_rounds_plan_size(self.ready().ctx, passes)
        self.ring = self.torch.empty(nbytes, dtype=self.torch.uint8, device=self.device)
        asap_bind_rounds_plan(self.ctx, self.ring, nbytes, stream)

    def drop_workers(self, dropped, ptr, idx, w, flags=0, stream=None):
        """Workers `dropped` leave (asap_drop_workers); the survivors keep
        their models, renumbered in order, run on the graph (ptr, idx, w) and
        have their shards bound again (device-side gathers of the bound
        tensors)."""
        t = self.torch
        dropped = sorted(int(k) for k in dropped)
        keep = [k for k in range(self.n) if k not in set(dropped)]
        asap_drop_workers(self.ctx, dropped, ptr, idx, w, flags, stream)
        self.n = len(keep)
        self.ws = None
        data, self._data = self._data, None
        if data is None:
            return
        if data[0] == "dense":
            _, X, y, S = data
            sel = t.as_tensor(keep, dtype=t.long, device=self.device)
            X2 = X.index_select(0, sel).contiguous()
            y2 = y.index_select(0, sel).contiguous()
            self._keep += [X2, y2]
            asap_bind_dense(self.ctx, X2, y2, S, int(X2.shape[2]))
            self._data = ("dense", X2, y2, S)
        else:
            _, rp, cl, vl, yy, S = data
            rph = rp.cpu().numpy()
            segs = [(int(rph[k * S]), int(rph[(k + 1) * S])) for k in keep]
            cols = t.cat([cl[a:b] for a, b in segs]) if segs else cl[:0]
            vals = t.cat([vl[a:b] for a, b in segs]) if segs else vl[:0]
            yys = t.cat([yy[k * S:(k + 1) * S] for k in keep])
            rp2 = np.concatenate([[0]] + [rph[k * S + 1:(k + 1) * S + 1] - rph[k * S] for k in keep])
            off = np.concatenate([[0], np.cumsum([b - a for a, b in segs])])
            for q in range(len(keep)):  # rows of survivor q start after the earlier survivors' nonzeros
                rp2[q * S + 1:(q + 1) * S + 1] += off[q]
            rp2 = t.as_tensor(rp2.astype(np.int64)).to(self.device)
            cols, vals, yys = cols.contiguous(), vals.contiguous(), yys.contiguous()
            self._keep += [rp2, cols, vals, yys]
            asap_bind_csr(self.ctx, rp2, cols, vals, yys, S, int(cols.numel()))
            self._data = ("csr", rp2, cols, vals, yys, S)

    # inspection ---------------------------------------------------------
    def current(self):
        return asap_current(self.ctx)

    # checkpoints ----------------------------------------------------------
    def save(self, path):
        """Write the models and the round counter between two rounds (npz).

        The models are those every worker holds at the start of the next
        round, so a session that loads the file continues bit for bit as this
        one would (same data, graph and parameters)."""
        b, rnd, half = self.current()
        if half:
            raise RuntimeError("a checkpoint is taken between rounds, not after a half-step")
        W = self.bufs[b][:self.n, :self.dim].cpu().numpy()
        with open(path, "wb") as f:
            np.savez(f, models=W, round=np.int64(rnd), n=np.int64(self.n), dim=np.int64(self.dim))

    def load(self, path, stream=None):
        """Resume from a file written by save(): models into buffer 0, round
        counter and epoch tags as at that round's start (asap_set_round)."""
        with np.load(path, allow_pickle=False) as z:
            W, rnd = z["models"], int(z["round"])
            if int(z["n"]) != self.n or int(z["dim"]) != self.dim:
                raise ValueError(f"checkpoint is {int(z['n'])} x {int(z['dim'])}, session is {self.n} x {self.dim}")
        self.set_models(W, stream)
        asap_set_round(self.ready(stream).ctx, rnd, 0, stream)

    def models(self):
        """Current models [n, dim] as a device view (no copy)."""
        b, _, _ = self.current()
        return self.bufs[b][:self.n, :self.dim]

    def metrics(self, loss="logistic", l2=0.0):
        return asap_metrics(self.ready().ctx, loss, l2)

    def check(self):
        return asap_check(self.ctx)

    def close(self):
        """Ordered teardown: wait for the device, destroy the context (which
        waits for its look-ahead stream and releases its stream and events),
        then drop the device memory the context used."""
        if self.ctx:
            self.torch.cuda.synchronize(self.device)
            asap_destroy(self.ctx)
            self.ctx = None
        self.bufs, self.ws, self._keep, self._data, self.ring = [], None, [], None, None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass
