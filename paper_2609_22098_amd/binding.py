"""ctypes binding of libtreespark.so (the C ABI in include/treespark.h).

Argument marshalling only: every step of the draft-tree path runs in the HIP
kernels behind the C ABI.  PyTorch provides device memory and the stream.
The binding raises if the shared library is missing; there is no fallback.
"""
from __future__ import annotations

import atexit
import ctypes
import os
from dataclasses import dataclass

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libtreespark.so")

TS_OK, TS_EINVAL, TS_EUNSUPPORTED, TS_EHIP, TS_ENOSPACE, TS_EINTERNAL = 0, -1, -2, -3, -4, -5
TS_F32, TS_BF16 = 0, 1
TS_MAX_K, TS_MAX_D = 16, 16

# Every symbol include/treespark.h declares.
SAMPLERS = {"gumbel": 0, "sequential": 1}  # ts_sampler
EXPORTED = ("ts_ladder_lookup", "ts_ladder_default", "ts_tree_mask_words", "ts_tree_mask",
            "ts_expand_workspace_size", "ts_expand", "ts_build_tree_workspace_size", "ts_build_tree",
            "ts_verify_workspace_size", "ts_verify", "ts_calib_labels_workspace_size", "ts_calib_labels",
            "ts_calib_fit", "ts_last_error", "ts_version", "ts_release_thread_state", "ts_expand_noalloc",
            "ts_verify_level_counts", "ts_verify_set_mode")
TS_NOALLOC_SCRATCH_BYTES = 32 << 20


class TreeSparkError(RuntimeError):
    def __init__(self, code, msg):
        super().__init__(f"treespark error {code}: {msg}")
        self.code = code


class Drafter(ctypes.Structure):
    _fields_ = [("U", ctypes.c_void_p), ("E", ctypes.c_void_p), ("W2", ctypes.c_void_p),
                ("R", ctypes.c_int32), ("D", ctypes.c_int32), ("V", ctypes.c_int32),
                ("r", ctypes.c_int32), ("dtype", ctypes.c_int32)]


class Calib(ctypes.Structure):
    _fields_ = [("a", ctypes.c_float), ("b", ctypes.c_float)]


class ExpandOut(ctypes.Structure):
    _fields_ = [(name, ctypes.c_void_p) for name in
                ("child_token", "child_log_q0", "child_log_qT", "child_log_surv", "slot_key",
                 "rank_token", "rank_log_q0", "lse0", "lseT", "diag", "events")]


class Tree(ctypes.Structure):
    _fields_ = [("R", ctypes.c_int32), ("cap", ctypes.c_int32)] + [
        (name, ctypes.c_void_p) for name in
        ("n", "token", "parent", "depth", "rank", "path", "log_surv", "log_q0", "log_qT", "key", "evals")]


# ts_parent: 24 bytes
PARENT_DTYPE = np.dtype([("token", "<i4"), ("depth", "<i4"), ("request", "<i4"),
                         ("log_surv", "<f4"), ("path", "<u8")])
assert PARENT_DTYPE.itemsize == 24

_lib = None


def lib():
    """Load the HIP library; raises if it has not been built."""
    global _lib
    if _lib is None:
        try:
            # Bind to the HIP runtime torch already loaded (same soname), so that
            # torch's streams and events are this library's streams and events.
            import torch  # noqa: F401
        except ImportError:
            pass
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it first (__graft_entry__.build())")
        L = ctypes.CDLL(LIB_PATH)
        P, I32, U64, SZ, F = ctypes.c_void_p, ctypes.c_int32, ctypes.c_uint64, ctypes.c_size_t, ctypes.c_float
        L.ts_expand_workspace_size.argtypes = [P, I32, I32, F]
        L.ts_expand_workspace_size.restype = SZ
        L.ts_expand.argtypes = [P, P, I32, Calib, I32, F, U64, I32, P, P, SZ, P]
        L.ts_expand.restype = I32
        L.ts_expand_noalloc.argtypes = [P, P, I32, Calib, I32, F, U64, I32, P, P]
        L.ts_expand_noalloc.restype = I32
        L.ts_build_tree_workspace_size.argtypes = [P, I32, I32, F]
        L.ts_build_tree_workspace_size.restype = SZ
        L.ts_build_tree.argtypes = [P, P, P, I32, I32, I32, Calib, F, U64, I32, P, P, P, SZ, P]
        L.ts_build_tree.restype = I32
        L.ts_verify_workspace_size.argtypes = [P, I32, F]
        L.ts_verify_workspace_size.restype = SZ
        L.ts_verify.argtypes = [P, P, P, I32, F, U64, P, P, P, P, SZ, P]
        L.ts_verify.restype = I32
        L.ts_calib_labels_workspace_size.argtypes = [I32, I32]
        L.ts_calib_labels_workspace_size.restype = SZ
        L.ts_calib_labels.argtypes = [P, P, I32, I32, P, P, P, P, SZ, P]
        L.ts_calib_labels.restype = I32
        L.ts_calib_fit.argtypes = [P, P, P, I32, I32, ctypes.c_double, P, P]
        L.ts_calib_fit.restype = I32
        L.ts_ladder_lookup.argtypes = [P, I32, I32, F, I32, I32, I32, P]
        L.ts_ladder_lookup.restype = I32
        L.ts_ladder_default.argtypes = [P, I32]
        L.ts_ladder_default.restype = I32
        L.ts_tree_mask_words.argtypes = [I32]
        L.ts_tree_mask_words.restype = I32
        L.ts_tree_mask.argtypes = [P, P, I32, I32, P, P, P, P]
        L.ts_tree_mask.restype = I32
        L.ts_last_error.restype = ctypes.c_char_p
        L.ts_version.restype = ctypes.c_char_p
        L.ts_release_thread_state.argtypes = []
        L.ts_release_thread_state.restype = I32
        L.ts_verify_level_counts.argtypes = [P, P, P]
        L.ts_verify_level_counts.restype = I32
        L.ts_verify_set_mode.argtypes = [I32]
        L.ts_verify_set_mode.restype = I32
        _lib = L
        # atexit runs its handlers last-registered first: this one (registered
        # after torch's import) frees the library's pinned buffer
        # while torch and the HIP runtime are still up
        atexit.register(release_thread_state)
    return _lib


VERIFY_MODES = {"auto": 0, "staged": 1}  # TS_VERIFY_AUTO, TS_VERIFY_STAGED


def verify_set_mode(mode):
    """ts_verify_set_mode for the calling thread: "auto" or "staged"."""
    _check(lib().ts_verify_set_mode(VERIFY_MODES[mode]))


def verify_level_counts():
    """ts_verify_level_counts for the calling thread: (fused, fallbacks, staged) T > 0 levels."""
    out = [ctypes.c_int64(0) for _ in range(3)]
    _check(lib().ts_verify_level_counts(*(ctypes.byref(x) for x in out)))
    return tuple(int(x.value) for x in out)


def release_thread_state():
    """ts_release_thread_state for the calling thread (a no-op before the library is loaded)."""
    if _lib is None:
        return
    _check(_lib.ts_release_thread_state())


def _check(rc):
    if rc != TS_OK:
        raise TreeSparkError(rc, lib().ts_last_error().decode())


def _torch():
    import torch
    return torch


# Host output arrays reused from call to call: their checked addresses.  An
# entry holds its array, so the array's id is not reused (and numpy does not
# resize it) while it is cached; taking an array's address costs about a
# microsecond.
_addr_cache = {}


def _int32_out_addr(a, shape):
    e = _addr_cache.get(id(a))
    if e is not None and e[0] is a and e[2] == shape:
        return e[1]
    assert a.shape == shape and a.dtype == np.int32 and a.flags.c_contiguous
    if len(_addr_cache) >= 64:
        _addr_cache.clear()
    addr = a.ctypes.data
    _addr_cache[id(a)] = (a, addr, shape)
    return addr


def _stream(stream):
    torch = _torch()
    if stream is None:
        stream = torch.cuda.current_stream()
    return ctypes.c_void_p(stream.cuda_stream)


def torch_empty_bytes(n, device="cuda"):
    """A device byte buffer of at least one byte (for the workspace arguments)."""
    return _torch().empty((max(int(n), 1),), dtype=_torch().uint8, device=device)


def _dtype_code(t):
    torch = _torch()
    dt = t.dtype
    if dt is torch.bfloat16:
        return TS_BF16
    if dt is torch.float32:
        return TS_F32
    raise TypeError(f"unsupported dtype {t.dtype}")


@dataclass
class DeviceDrafter:
    """Device tensors U [R][D][V], E [V][r], W2 [V][r] (same dtype, contiguous)."""
    U: object
    E: object
    W2: object

    def __post_init__(self):
        R, D, V = self.U.shape
        r = self.E.shape[1]
        assert self.E.shape == (V, r) and self.W2.shape == (V, r)
        assert self.U.is_contiguous() and self.E.is_contiguous() and self.W2.is_contiguous()
        assert self.U.dtype == self.E.dtype == self.W2.dtype
        self.struct = Drafter(self.U.data_ptr(), self.E.data_ptr(), self.W2.data_ptr(), R, D, V, r,
                              _dtype_code(self.U))

    @property
    def R(self):
        return self.struct.R

    @property
    def D(self):
        return self.struct.D

    @property
    def V(self):
        return self.struct.V

    @property
    def r(self):
        return self.struct.r

    def ref(self):
        return ctypes.byref(self.struct)


def drafter_from_host(dr, device="cuda"):
    """Copy a synth.Drafter to the device."""
    torch = _torch()

    def dev(a):
        t = torch.from_numpy(np.ascontiguousarray(a))
        if a.dtype == np.uint16:
            t = t.view(torch.bfloat16)
        return t.to(device)

    return DeviceDrafter(dev(dr.U), dev(dr.E), dev(dr.W2))


def parents_to_device(token, depth, request, log_surv, path, device="cuda"):
    """Pack frontier parents into a device byte tensor of ts_parent records."""
    torch = _torch()
    a = np.zeros(len(token), dtype=PARENT_DTYPE)
    a["token"], a["depth"], a["request"] = token, depth, request
    a["log_surv"], a["path"] = log_surv, path
    return torch.from_numpy(a.view(np.uint8).copy()).to(device)


def expand_workspace_size(d: DeviceDrafter, P, k, T):
    return lib().ts_expand_workspace_size(d.ref(), P, k, float(T))


_EXPAND_OUT_NAMES = tuple(name for name, _ in ExpandOut._fields_[:-1])
# Output dicts reused from call to call: their ExpandOut, rebuilt whenever a
# tensor's address differs from the cached one (the events field is set on
# every call).  An entry holds its dict, so the dict's id is not reused while
# it is cached.
_expand_out_cache = {}


def _expand_out(outputs, events):
    ptrs = tuple(outputs[name].data_ptr() if outputs.get(name) is not None else None
                 for name in _EXPAND_OUT_NAMES)
    e = _expand_out_cache.get(id(outputs))
    if e is not None and e[0] is outputs and e[1] == ptrs:
        out = e[2]
        out.events = events
        return out
    out = ExpandOut(*ptrs, events)
    if len(_expand_out_cache) >= 64:
        _expand_out_cache.clear()
    _expand_out_cache[id(outputs)] = (outputs, ptrs, out)
    return out


def expand(d: DeviceDrafter, parents, P, k, T, seed, calib=(0.67, -0.46), workspace=None,
           stream=None, outputs=None, events=None, sampler="gumbel"):
    """ts_expand.  parents: device uint8 tensor of P ts_parent records.  Returns a dict of
    device tensors (asynchronous on the stream).  events: optional ctypes array of three
    hipEvent_t handles recorded around the two kernels, given by address.  sampler:
    "gumbel" or "sequential" (the realisation of the draws at T > 0)."""
    torch = _torch()
    dev = parents.device
    if outputs is None:
        outputs = dict(
            child_token=torch.empty((P, k), dtype=torch.int32, device=dev),
            child_log_q0=torch.empty((P, k), dtype=torch.float32, device=dev),
            child_log_qT=torch.empty((P, k), dtype=torch.float32, device=dev),
            child_log_surv=torch.empty((P, k), dtype=torch.float32, device=dev),
            slot_key=torch.empty((P, k), dtype=torch.float32, device=dev),
            rank_token=torch.empty((P, k), dtype=torch.int32, device=dev),
            rank_log_q0=torch.empty((P, k), dtype=torch.float32, device=dev),
            lse0=torch.empty((P,), dtype=torch.float32, device=dev),
            lseT=torch.empty((P,), dtype=torch.float32, device=dev),
            diag=torch.empty((P,), dtype=torch.int32, device=dev))
    if workspace is None:
        n = expand_workspace_size(d, P, k, T)
        workspace = torch.empty((max(n, 1),), dtype=torch.uint8, device=dev)
    out = _expand_out(outputs, events)
    rc = lib().ts_expand(d.ref(), ctypes.c_void_p(parents.data_ptr()), P, Calib(*calib), k, float(T),
                         ctypes.c_uint64(seed), SAMPLERS[sampler], ctypes.byref(out), ctypes.c_void_p(workspace.data_ptr()),
                         workspace.numel(), _stream(stream))
    _check(rc)
    outputs["_workspace"] = workspace
    return outputs


def expand_noalloc(d: DeviceDrafter, parents, P, k, T, seed, outputs, calib=(0.67, -0.46), stream=None,
                   sampler="gumbel"):
    """ts_expand_noalloc: ts_expand in the library's per-GPU scratch array, with no workspace and
    no allocation in the call.  outputs: a dict of preallocated device tensors, as expand returns
    (rank_token, rank_log_q0, lse0, lseT, diag and child_log_qT may be absent)."""
    out = ExpandOut(*[outputs[name].data_ptr() if outputs.get(name) is not None else None
                      for name, _ in ExpandOut._fields_[:-1]], None)
    rc = lib().ts_expand_noalloc(d.ref(), ctypes.c_void_p(parents.data_ptr()), P, Calib(*calib), k, float(T),
                                 ctypes.c_uint64(seed), SAMPLERS[sampler], ctypes.byref(out), _stream(stream))
    _check(rc)
    return outputs


@dataclass
class HostTree:
    n: np.ndarray
    token: np.ndarray
    parent: np.ndarray
    depth: np.ndarray
    rank: np.ndarray
    path: np.ndarray
    log_surv: np.ndarray
    log_q0: np.ndarray
    log_qT: np.ndarray
    key: np.ndarray
    evals: np.ndarray

    @classmethod
    def empty(cls, R, cap):
        z = lambda dt: np.zeros((R, cap), dtype=dt)
        return cls(np.zeros(R, np.int32), z(np.int32), z(np.int32), z(np.int32), z(np.int32),
                   z(np.uint64), z(np.float32), z(np.float32), z(np.float32), z(np.float32),
                   np.zeros(R, np.int32))

    @property
    def R(self):
        return self.token.shape[0]

    @property
    def cap(self):
        return self.token.shape[1]

    def struct(self):
        """The ts_tree view of the arrays.  Built once and reused while the same array
        objects are attached (taking an array's address costs microseconds)."""
        arrs = tuple(getattr(self, f) for f, _ in Tree._fields_[2:])
        cached = self.__dict__.get("_struct")
        if cached is not None and len(cached[0]) == len(arrs) and all(a is b for a, b in zip(cached[0], arrs)):
            return cached[1]
        st = Tree(self.R, self.cap, *[a.ctypes.data for a in arrs])
        self.__dict__["_struct"] = (arrs, st)
        return st


class DeviceTree:
    """A tree in the ts_tree layout held in device memory (torch tensors; path as int64)."""

    _INT = ("token", "parent", "depth", "rank")
    _FLT = ("log_surv", "log_q0", "log_qT", "key")

    def __init__(self, R, cap, device="cuda"):
        torch = _torch()
        self.R, self.cap = R, cap
        self.n = torch.zeros(R, dtype=torch.int32, device=device)
        self.evals = torch.zeros(R, dtype=torch.int32, device=device)
        for f in self._INT:
            setattr(self, f, torch.zeros((R, cap), dtype=torch.int32, device=device))
        self.path = torch.zeros((R, cap), dtype=torch.int64, device=device)
        for f in self._FLT:
            setattr(self, f, torch.zeros((R, cap), dtype=torch.float32, device=device))

    def struct(self):
        return Tree(self.R, self.cap, *[getattr(self, f).data_ptr() for f, _ in Tree._fields_[2:]])


def build_tree_workspace_size(d: DeviceDrafter, N, K, T):
    return lib().ts_build_tree_workspace_size(d.ref(), N, K, float(T))


def build_tree(d: DeviceDrafter, anchor, theta, N, K, T, seed, calib=(0.67, -0.46), workspace=None,
               stream=None, tree=None, sampler="gumbel", budget=0, device_tree=None) -> HostTree:
    """ts_build_tree: one tree per request; budget > 0 shares one node budget across requests.
    device_tree (a DeviceTree of the same R and cap) also receives the tree in device memory."""
    torch = _torch()
    anchor = np.ascontiguousarray(anchor, dtype=np.int32)
    theta = np.ascontiguousarray(theta, dtype=np.float32)
    if tree is None:
        tree = HostTree.empty(d.R, N + 1)
    if workspace is None:
        n = build_tree_workspace_size(d, N, K, T)
        workspace = torch.empty((max(n, 1),), dtype=torch.uint8, device=d.U.device)
    s = tree.struct()
    ds = None
    if device_tree is not None:
        assert (device_tree.R, device_tree.cap) == (tree.R, tree.cap)
        ds = device_tree.struct()
    rc = lib().ts_build_tree(d.ref(), anchor.ctypes.data, theta.ctypes.data, N, int(budget), K, Calib(*calib),
                             float(T), ctypes.c_uint64(seed), SAMPLERS[sampler], ctypes.byref(s),
                             ctypes.byref(ds) if ds is not None else None,
                             ctypes.c_void_p(workspace.data_ptr()), workspace.numel(), _stream(stream))
    _check(rc)
    return tree


def verify_workspace_size(d: DeviceDrafter, cap, T):
    return lib().ts_verify_workspace_size(d.ref(), cap, float(T))


def verify(d: DeviceDrafter, tree: HostTree, target, T, seed, workspace=None, stream=None, out=None):
    """ts_verify.  target: device tensor [R][cap][V] (float32 or bfloat16).
    Returns (path_nodes [R][16], path_len [R], bonus [R]) as numpy arrays; out = (path_nodes,
    path_len, bonus) reuses given int32 arrays of those shapes."""
    torch = _torch()
    R, cap = tree.R, tree.cap
    assert tuple(target.shape) == (R, cap, d.V) and target.is_contiguous()
    if out is None:
        path = np.zeros((R, TS_MAX_D), np.int32)
        plen = np.zeros(R, np.int32)
        bonus = np.zeros(R, np.int32)
    else:
        path, plen, bonus = out
    a_path = _int32_out_addr(path, (R, TS_MAX_D))
    a_plen = _int32_out_addr(plen, (R,))
    a_bonus = _int32_out_addr(bonus, (R,))
    if workspace is None:
        n = verify_workspace_size(d, cap, T)
        workspace = torch.empty((max(n, 1),), dtype=torch.uint8, device=target.device)
    s = tree.struct()
    rc = lib().ts_verify(d.ref(), ctypes.byref(s), ctypes.c_void_p(target.data_ptr()), _dtype_code(target),
                         float(T), ctypes.c_uint64(seed), a_path, a_plen, a_bonus,
                         ctypes.c_void_p(workspace.data_ptr()), workspace.numel(), _stream(stream))
    _check(rc)
    return path, plen, bonus


def tree_mask(parent, n, cap, pos_offset=None, stream=None, out=None):
    """ts_tree_mask.  parent [R][cap] and n [R] int32 DEVICE tensors (ts_tree layout),
    pos_offset optional [R] int32 device tensor.  Returns (mask [R][cap][W] int32 tensor holding
    the uint32 words, pos [R][cap] int32), asynchronous on the stream; out = (mask, pos) reuses
    given output tensors."""
    torch = _torch()
    R = parent.shape[0]
    assert tuple(parent.shape) == (R, cap) and parent.dtype == torch.int32 and parent.is_contiguous()
    assert tuple(n.shape) == (R,) and n.dtype == torch.int32
    if out is None:
        W = lib().ts_tree_mask_words(cap)
        mask = torch.empty((R, cap, W), dtype=torch.int32, device=parent.device)
        pos = torch.empty((R, cap), dtype=torch.int32, device=parent.device)
    else:
        mask, pos = out
        assert tuple(mask.shape) == (R, cap, (cap + 31) // 32) and tuple(pos.shape) == (R, cap)
    off = ctypes.c_void_p(pos_offset.data_ptr()) if pos_offset is not None else None
    rc = lib().ts_tree_mask(ctypes.c_void_p(parent.data_ptr()), ctypes.c_void_p(n.data_ptr()), R, cap, off,
                            ctypes.c_void_p(mask.data_ptr()), ctypes.c_void_p(pos.data_ptr()), _stream(stream))
    _check(rc)
    return mask, pos


class TreeMaskBuffers:
    """Reusable page-locked staging and device buffers for masks of HostTrees of one shape."""

    def __init__(self, R, cap, device="cuda"):
        torch = _torch()
        self.R, self.cap = R, cap
        self.host = torch.empty((R * (cap + 1),), dtype=torch.int32, pin_memory=True)
        self.dev = torch.empty((R * (cap + 1),), dtype=torch.int32, device=device)
        W = (cap + 31) // 32
        self.out = (torch.empty((R, cap, W), dtype=torch.int32, device=device),
                    torch.empty((R, cap), dtype=torch.int32, device=device))
        self.copied = torch.cuda.Event()  # recorded after each copy out of the staging buffer
        self.pending = False

    def upload(self, tree: HostTree, stream=None):
        torch = _torch()
        if self.pending:
            self.copied.synchronize()  # the previous copy has left the staging buffer
        h = self.host.numpy()
        h[: self.R * self.cap] = tree.parent.reshape(-1)
        h[self.R * self.cap:] = tree.n
        s = torch.cuda.current_stream() if stream is None else stream
        with torch.cuda.stream(s):
            self.dev.copy_(self.host, non_blocking=True)
            self.copied.record(s)
        self.pending = True
        return self.dev[: self.R * self.cap].view(self.R, self.cap), self.dev[self.R * self.cap:]


def tree_mask_from_host(tree: HostTree, pos_offset=None, device="cuda", stream=None, buffers=None):
    """Upload a HostTree's parents and sizes (through page-locked staging), then ts_tree_mask."""
    torch = _torch()
    buf = buffers or TreeMaskBuffers(tree.R, tree.cap, device)
    parent, n = buf.upload(tree, stream)
    off = None if pos_offset is None else torch.from_numpy(np.ascontiguousarray(pos_offset, np.int32)).to(device)
    return tree_mask(parent, n, tree.cap, off, stream, out=buf.out)


def calib_labels(tree: HostTree, target, workspace=None, stream=None):
    """ts_calib_labels: greedy labels of a round's trees.  target: device tensor [R][cap][V]
    (float32 or bfloat16).  Returns device tensors (x [R][cap] float32 = logit q0,
    y [R][cap] int32, sel [R][cap] int32)."""
    torch = _torch()
    R, cap = tree.R, tree.cap
    assert target.dim() == 3 and tuple(target.shape[:2]) == (R, cap) and target.is_contiguous()
    dev = target.device
    x = torch.empty((R, cap), dtype=torch.float32, device=dev)
    y = torch.empty((R, cap), dtype=torch.int32, device=dev)
    sel = torch.empty((R, cap), dtype=torch.int32, device=dev)
    if workspace is None:
        workspace = torch.empty((lib().ts_calib_labels_workspace_size(R, cap),), dtype=torch.uint8, device=dev)
    s = tree.struct()
    rc = lib().ts_calib_labels(ctypes.byref(s), ctypes.c_void_p(target.data_ptr()), _dtype_code(target),
                               int(target.shape[2]), ctypes.c_void_p(x.data_ptr()), ctypes.c_void_p(y.data_ptr()),
                               ctypes.c_void_p(sel.data_ptr()), ctypes.c_void_p(workspace.data_ptr()),
                               workspace.numel(), _stream(stream))
    _check(rc)
    return x, y, sel


def calib_fit(x, y, sel, max_iter=100, tol=1e-10, stream=None):
    """ts_calib_fit over device tensors x (float32), y, sel (int32) of equal size.
    Returns (a, b, mean negative log-likelihood, steps) as Python numbers."""
    torch = _torch()
    n = x.numel()
    assert y.numel() == n and sel.numel() == n
    assert x.dtype == torch.float32 and y.dtype == torch.int32 and sel.dtype == torch.int32
    assert x.is_contiguous() and y.is_contiguous() and sel.is_contiguous()
    out = torch.empty(4, dtype=torch.float32, device=x.device)
    rc = lib().ts_calib_fit(ctypes.c_void_p(x.data_ptr()), ctypes.c_void_p(y.data_ptr()),
                            ctypes.c_void_p(sel.data_ptr()), n, int(max_iter), float(tol),
                            ctypes.c_void_p(out.data_ptr()), _stream(stream))
    _check(rc)
    a, b, nll, steps = out.cpu().tolist()
    return a, b, nll, int(steps)


class LadderRung(ctypes.Structure):
    _fields_ = [("bs_max", ctypes.c_int32), ("T", ctypes.c_float), ("theta", ctypes.c_float)]


class RoundPolicy(ctypes.Structure):
    _fields_ = [("theta", ctypes.c_float), ("K", ctypes.c_int32), ("N", ctypes.c_int32),
                ("chain", ctypes.c_int32)]


def ladder_default():
    """The paper's measured A100 ladder: a list of (bs_max, T, theta) with theta < 0 = chain."""
    n = lib().ts_ladder_default(None, 0)
    arr = (LadderRung * n)()
    lib().ts_ladder_default(arr, n)
    return [(r.bs_max, r.T, r.theta) for r in arr]


def ladder_lookup(rungs, bs, T, K, N, block_len):
    """ts_ladder_lookup over a list of (bs_max, T, theta); returns (theta, K, N, chain)."""
    arr = (LadderRung * len(rungs))(*[LadderRung(int(b), float(t), float(th)) for b, t, th in rungs])
    out = RoundPolicy()
    _check(lib().ts_ladder_lookup(arr, len(rungs), int(bs), float(T), int(K), int(N), int(block_len),
                                  ctypes.byref(out)))
    return out.theta, out.K, out.N, bool(out.chain)
