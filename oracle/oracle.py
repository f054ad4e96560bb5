"""ctypes wrapper of the TreeSpark CPU oracle (liboracle.so).

TEST INFRASTRUCTURE ONLY: tests/, __graft_entry__.smoke() and bench.py's
cpu_baseline leg may import this module.  It shares no code with the HIP path.

Every function works on numpy arrays in host memory.  Float inputs are the
exact values the GPU path sees (bf16 inputs are passed as the float32 values
they represent); the arithmetic is fp64.  The calibration functions (greedy
labels and the two-scalar Platt fit of §3.4 Eq. 3) are written here in numpy.
"""
from __future__ import annotations

import ctypes
import os
import subprocess
from dataclasses import dataclass

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "treespark_oracle.c")
_LIB = os.path.join(_HERE, "liboracle.so")

TAG_EXPAND, TAG_ACCEPT, TAG_BONUS = 1, 2, 3


def build(force: bool = False) -> str:
    """Compile the oracle with gcc (plain -O2, no OpenMP, no BLAS)."""
    if force or not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
        tmp = _LIB + ".tmp"
        subprocess.check_call(["gcc", "-O2", "-std=c99", "-fPIC", "-shared", "-o", tmp, _SRC, "-lm"])
        os.replace(tmp, _LIB)
    return _LIB


_lib = None


def lib():
    global _lib
    if _lib is None:
        _lib = ctypes.CDLL(build())
        _declare(_lib)
    return _lib


class _Model(ctypes.Structure):
    _fields_ = [("R", ctypes.c_int), ("D", ctypes.c_int), ("V", ctypes.c_int), ("r", ctypes.c_int),
                ("U", ctypes.c_void_p), ("E", ctypes.c_void_p), ("W2", ctypes.c_void_p)]


class _Tree(ctypes.Structure):
    _fields_ = [("n", ctypes.c_int), ("evals", ctypes.c_int)] + [
        (name, ctypes.c_void_p) for name in
        ("token", "parent", "depth", "rank", "path", "log_surv", "log_q0", "log_qT", "key",
         "margin", "eval_gap", "draw_gap")] + [("stop_key", ctypes.c_double)]


_P = ctypes.c_void_p
_D = ctypes.c_double
_I = ctypes.c_int
_U64 = ctypes.c_uint64


def _declare(L):
    L.tso_philox4x32_10.argtypes = [_P, _P, _P]
    L.tso_u_token.argtypes = [_U64, _I, _I, _U64, _I, _I]
    L.tso_u_token.restype = _D
    L.tso_u_stage.argtypes = [_U64, _I, _I, _U64, _I, _I]
    L.tso_u_stage.restype = _D
    L.tso_log_phat.argtypes = [_D, _D, _D]
    L.tso_log_phat.restype = _D
    L.tso_eval.argtypes = [ctypes.POINTER(_Model), _I, _I, _I, _U64, _D, _U64, _I, _I,
                           _P, _P, _P, _P, _P, _P, _P, _P]
    L.tso_eval.restype = _I
    L.tso_expand_tree.argtypes = [ctypes.POINTER(_Model), _I, _I, _D, _I, _I, _D, _D, _D, _U64, _I,
                                  _I, ctypes.POINTER(_Tree)]
    L.tso_draw_sequential.argtypes = [_P, _I, _D, _U64, _I, _I, _U64, _I, _P, _P]
    L.tso_draw_sequential.restype = None
    L.tso_expand_forest.argtypes = [ctypes.POINTER(_Model), _I, _P, _P, _I, _I, _I, _D, _D, _D, _U64, _I, _P]
    L.tso_expand_forest.restype = _I
    L.tso_tree_mask.argtypes = [_P, _I, _I, _I, _P, _P]
    L.tso_tree_mask.restype = _I
    L.tso_expand_tree.restype = _I
    L.tso_verify_greedy.argtypes = [ctypes.POINTER(_Tree), _P, _I, _P, _P, _P, _P]
    L.tso_verify_greedy.restype = _I
    L.tso_residual_stages.argtypes = [_I, _P, _P, _I, _P, _P, _P, _P]
    L.tso_residual_stages.restype = _I
    L.tso_verify_sample.argtypes = [ctypes.POINTER(_Model), _I, ctypes.POINTER(_Tree), _P, _D, _U64,
                                    _P, _P, _P, _P]
    L.tso_verify_sample.restype = _I


def _ptr(a: np.ndarray | None):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


class Model:
    """Host copies of U [R][D][V], E [V][r], W2 [V][r] as float32 (exact input values)."""

    def __init__(self, U, E, W2):
        self.U = np.ascontiguousarray(U, dtype=np.float32)
        self.E = np.ascontiguousarray(E, dtype=np.float32)
        self.W2 = np.ascontiguousarray(W2, dtype=np.float32)
        R, D, V = self.U.shape
        r = self.E.shape[1]
        assert self.E.shape == (V, r) and self.W2.shape == (V, r)
        self.R, self.D, self.V, self.r = R, D, V, r
        self._s = _Model(R, D, V, r, self.U.ctypes.data, self.E.ctypes.data, self.W2.ctypes.data)

    @property
    def struct(self):
        return ctypes.byref(self._s)


def philox4x32_10(counter, key):
    c = np.ascontiguousarray(counter, dtype=np.uint32)
    k = np.ascontiguousarray(key, dtype=np.uint32)
    out = np.zeros(4, dtype=np.uint32)
    lib().tso_philox4x32_10(_ptr(c), _ptr(k), _ptr(out))
    return out


def u_token(seed, request, depth, path, tag, y):
    return lib().tso_u_token(seed, request, depth, path, tag, y)


def u_stage(seed, request, depth, path, tag, j):
    return lib().tso_u_stage(seed, request, depth, path, tag, j)


def log_phat(lq, a=0.67, b=-0.46):
    return lib().tso_log_phat(float(lq), float(a), float(b))


@dataclass
class Eval:
    z: np.ndarray
    lse0: float
    lseT: float
    pi: np.ndarray        # [K]
    pi_z: np.ndarray      # [K+1]
    sigma: np.ndarray     # [K]  (T > 0)
    sigma_g: np.ndarray   # [K+1]
    sigma_z: np.ndarray   # [K]


SAMPLERS = {"gumbel": 0, "sequential": 1}


def eval_node(model: Model, request, token, depth, path, T, seed, K, want_z=True,
              sampler="gumbel") -> Eval:
    z = np.zeros(model.V, dtype=np.float64) if want_z else None
    lse0 = np.zeros(1); lseT = np.zeros(1)
    pi = np.zeros(K, dtype=np.int32); pi_z = np.zeros(K + 1)
    sigma = np.zeros(K, dtype=np.int32); sigma_g = np.zeros(K + 1); sigma_z = np.zeros(K)
    rc = lib().tso_eval(model.struct, request, token, depth, path, float(T), seed, SAMPLERS[sampler], K,
                        _ptr(z),
                        _ptr(lse0), _ptr(lseT), _ptr(pi), _ptr(pi_z), _ptr(sigma), _ptr(sigma_g),
                        _ptr(sigma_z))
    if rc != 0:
        raise ValueError("tso_eval: invalid arguments")
    return Eval(z, float(lse0[0]), float(lseT[0]), pi, pi_z, sigma, sigma_g, sigma_z)


@dataclass
class Tree:
    n: int
    evals: int
    token: np.ndarray
    parent: np.ndarray
    depth: np.ndarray
    rank: np.ndarray
    path: np.ndarray
    log_surv: np.ndarray
    log_q0: np.ndarray
    log_qT: np.ndarray
    key: np.ndarray
    margin: np.ndarray
    eval_gap: np.ndarray
    draw_gap: np.ndarray
    stop_key: float
    _keep: tuple = ()

    def struct(self):
        s = _Tree(self.n, self.evals, *[a.ctypes.data for a in (
            self.token, self.parent, self.depth, self.rank, self.path, self.log_surv, self.log_q0,
            self.log_qT, self.key, self.margin, self.eval_gap, self.draw_gap)], self.stop_key)
        return s


def expand_tree(model: Model, request, anchor, theta, N, K, T, seed, a=0.67, b=-0.46,
                control_topk=False, sampler="gumbel") -> Tree:
    cap = N + 1
    arr = dict(token=np.zeros(cap, np.int32), parent=np.zeros(cap, np.int32),
               depth=np.zeros(cap, np.int32), rank=np.zeros(cap, np.int32),
               path=np.zeros(cap, np.uint64), log_surv=np.zeros(cap), log_q0=np.zeros(cap),
               log_qT=np.zeros(cap), key=np.zeros(cap), margin=np.zeros(cap),
               eval_gap=np.zeros(cap), draw_gap=np.zeros(cap))
    t = Tree(0, 0, stop_key=float("nan"), **arr)
    s = t.struct()
    rc = lib().tso_expand_tree(model.struct, request, anchor, float(theta), N, K, float(a), float(b),
                               float(T), seed, SAMPLERS[sampler], int(control_topk), ctypes.byref(s))
    if rc != 0:
        raise ValueError("tso_expand_tree: invalid arguments")
    t.n, t.evals, t.stop_key = s.n, s.evals, s.stop_key
    n1 = t.n + 1
    for name in arr:
        setattr(t, name, getattr(t, name)[:n1].copy())
    return t


def draw_sequential(z, T, seed, request, depth, path, K):
    """K sequential draws without replacement from softmax(z / T) (sampler 1).
    Returns (tokens in draw order, smallest relative gap of all the picks)."""
    z = np.ascontiguousarray(z, dtype=np.float64)
    sigma = np.zeros(K, np.int32)
    gap = np.zeros(K)
    lib().tso_draw_sequential(_ptr(z), len(z), float(T), seed, request, depth, path, K, _ptr(sigma),
                              _ptr(gap))
    return sigma, float(gap.min()) if K else float("inf")


def _tree_struct(t: Tree):
    return t.struct()


def verify_greedy(tree: Tree, target: np.ndarray):
    target = np.ascontiguousarray(target, dtype=np.float32)
    V = target.shape[-1]
    assert target.shape[0] >= tree.n + 1
    path = np.zeros(max(1, tree.n), np.int32)
    plen = np.zeros(1, np.int32); bonus = np.zeros(1, np.int32); gap = np.zeros(tree.n + 1)
    s = _tree_struct(tree)
    rc = lib().tso_verify_greedy(ctypes.byref(s), _ptr(target), V, _ptr(path), _ptr(plen), _ptr(bonus),
                                 _ptr(gap))
    if rc != 0:
        raise ValueError("tso_verify_greedy: invalid arguments")
    return path[:plen[0]].copy(), int(bonus[0]), gap[:plen[0] + 1].copy()


def verify_sample(model: Model, request, tree: Tree, target: np.ndarray, T, seed):
    target = np.ascontiguousarray(target, dtype=np.float32)
    assert target.shape[-1] == model.V and target.shape[0] >= tree.n + 1
    path = np.zeros(max(1, tree.n), np.int32)
    plen = np.zeros(1, np.int32); bonus = np.zeros(1, np.int32); margin = np.zeros(tree.n + 1)
    s = _tree_struct(tree)
    rc = lib().tso_verify_sample(model.struct, request, ctypes.byref(s), _ptr(target), float(T), seed,
                                 _ptr(path), _ptr(plen), _ptr(bonus), _ptr(margin))
    if rc != 0:
        raise ValueError("tso_verify_sample: invalid arguments")
    return path[:plen[0]].copy(), int(bonus[0]), margin[:plen[0] + 1].copy()


def residual_stages(p, qT, x):
    p = np.ascontiguousarray(p, dtype=np.float64)
    qT = np.ascontiguousarray(qT, dtype=np.float64)
    x = np.ascontiguousarray(x, dtype=np.int32)
    m = len(x)
    ratio = np.zeros(m); Z = np.zeros(m); pf = np.zeros(len(p))
    lib().tso_residual_stages(len(p), _ptr(p), _ptr(qT), m, _ptr(x), _ptr(ratio), _ptr(Z), _ptr(pf))
    return ratio, Z, pf


def tree_mask(parent, n, cap, offset=0):
    """Ancestor bitmask [cap][ceil(cap/32)] (uint32) and position ids [cap] of one tree."""
    parent = np.ascontiguousarray(parent, dtype=np.int32)
    W = (cap + 31) // 32
    mask = np.zeros((cap, W), np.uint32)
    pos = np.zeros(cap, np.int32)
    rc = lib().tso_tree_mask(_ptr(parent), int(n), int(cap), int(offset), _ptr(mask), _ptr(pos))
    if rc != 0:
        raise ValueError("tso_tree_mask: malformed tree")
    return mask, pos


def expand_forest(model: Model, anchors, thetas, N, budget, K, T, seed, a=0.67, b=-0.46, sampler="gumbel"):
    """Trees of requests 0..R-1 (R = len(anchors)) under one global node budget (budget <= 0: none)."""
    R = len(anchors)
    cap = N + 1
    trees = []
    for _ in range(R):
        arr = dict(token=np.zeros(cap, np.int32), parent=np.zeros(cap, np.int32),
                   depth=np.zeros(cap, np.int32), rank=np.zeros(cap, np.int32),
                   path=np.zeros(cap, np.uint64), log_surv=np.zeros(cap), log_q0=np.zeros(cap),
                   log_qT=np.zeros(cap), key=np.zeros(cap), margin=np.zeros(cap),
                   eval_gap=np.zeros(cap), draw_gap=np.zeros(cap))
        trees.append(Tree(0, 0, stop_key=float("nan"), **arr))
    structs = (_Tree * R)(*[t.struct() for t in trees])
    anc = np.ascontiguousarray(anchors, np.int32)
    th = np.ascontiguousarray(thetas, np.float64)
    rc = lib().tso_expand_forest(model.struct, R, _ptr(anc), _ptr(th), N, int(budget), K, float(a), float(b),
                                 float(T), seed, SAMPLERS[sampler], structs)
    if rc != 0:
        raise ValueError("tso_expand_forest: invalid arguments")
    for t, s in zip(trees, structs):
        t.n, t.evals, t.stop_key = s.n, s.evals, s.stop_key
        n1 = t.n + 1
        for name in ("token", "parent", "depth", "rank", "path", "log_surv", "log_q0", "log_qT", "key",
                     "margin", "eval_gap", "draw_gap"):
            setattr(t, name, getattr(t, name)[:n1].copy())
    return trees


# ---------------------------------------------------------------- calibration (§3.4 Eq. 3)

def logit_q0(log_q0):
    """logit q0 = log q0 - log(1 - q0) from log q0, fp64; +inf where q0 == 1."""
    lq = np.asarray(log_q0, dtype=np.float64)
    out = np.full(lq.shape, np.inf)
    m = lq < 0.0
    l = lq[m]
    # log(1 - q0) = log1mexp(log q0), two-branch form (Maechler 2012)
    l1m = np.where(l > -np.log(2.0), np.log(-np.expm1(np.minimum(l, -1e-300))), np.log1p(-np.exp(l)))
    out[m] = l - l1m
    return out


def calib_labels(parent, token, n, target):
    """The greedy labels of one tree (§3.4): the verifier shows, for every node, whether its token is
    the target's greedy choice at its parent.  y[i] = 1 iff token[i] is the argmax (smallest id on
    ties) of the target row of parent[i]; sel[i] = 1 iff every edge on the root path of parent[i]
    has y = 1 (the ancestors-accepted population the two scalars are fitted on).  Row 0 and rows
    past n: y = -1, sel = 0.  Parents precede their children."""
    cap = len(parent)
    y = np.full(cap, -1, np.int32)
    sel = np.zeros(cap, np.int32)
    greedy = [int(np.argmax(np.asarray(target[i], dtype=np.float64))) for i in range(n + 1)]
    path_ok = np.zeros(cap, bool)  # every edge on the root path of node i accepted
    path_ok[0] = True
    for i in range(1, n + 1):
        p = int(parent[i])
        y[i] = 1 if int(token[i]) == greedy[p] else 0
        sel[i] = 1 if path_ok[p] else 0
        path_ok[i] = path_ok[p] and y[i] == 1
    return y, sel


def _nll(a, b, x, y):
    z = a * x + b
    return float(np.sum(np.logaddexp(0.0, z) - y * z))


def platt_fit(x, y, max_iter=100, tol=1e-10):
    """Maximum-likelihood (a, b) of y ~ Bernoulli(sigmoid(a x + b)): the two-scalar map of Eq. 3.
    Newton's method on the log-likelihood from (0, 0); a step that raises the negative
    log-likelihood is halved until it does not.  fp64.  Returns (a, b, mean negative
    log-likelihood, Newton steps taken)."""
    x = np.asarray(x, dtype=np.float64)
    y = np.asarray(y, dtype=np.float64)
    a = b = 0.0
    f = _nll(a, b, x, y)
    steps = 0
    for steps in range(1, max_iter + 1):
        p = 1.0 / (1.0 + np.exp(-(a * x + b)))
        r = p - y
        w = p * (1.0 - p)
        g = np.array([np.sum(r * x), np.sum(r)])
        H = np.array([[np.sum(w * x * x), np.sum(w * x)], [np.sum(w * x), np.sum(w)]])
        da, db = np.linalg.solve(H, g)
        t = 1.0
        while True:
            fa, fb = a - t * da, b - t * db
            fc = _nll(fa, fb, x, y)
            if fc <= f or t < 2.0 ** -30:
                break
            t *= 0.5
        a, b, f = fa, fb, fc
        if max(abs(t * da), abs(t * db)) < tol:
            break
    return a, b, f / max(len(x), 1), steps
