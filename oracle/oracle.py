"""ctypes front end of the C oracle (agft_oracle.c).

Test infrastructure only: see the header of agft_oracle.c for what is
computed and which readings of the paper it takes.
"""
import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "agft_oracle.c")
_LIB = os.path.join(_HERE, "libagft_oracle.so")
_lib = None


def build_library(src=_SRC, out=_LIB, extra_flags=()):
    """Compile the oracle with gcc (fp64, OpenMP over instances)."""
    cmd = ["gcc", "-O2", "-std=c99", "-fopenmp", "-fPIC", "-shared", "-Wall",
           *extra_flags, src, "-o", out + ".tmp", "-lm"]
    subprocess.run(cmd, check=True)
    os.replace(out + ".tmp", out)
    return out


def _declare(lib):
    P, I, D, L = ctypes.c_void_p, ctypes.c_int, ctypes.c_double, ctypes.c_long
    lib.ora_create.restype = P
    lib.ora_create.argtypes = [I, I, I, D, D, I, I, I]
    lib.ora_destroy.argtypes = [P]
    lib.ora_decide.argtypes = [P, P, P, P, P, P, P]
    lib.ora_decide_ex.argtypes = [P, P, P, P, P, P, P, P]
    lib.ora_set_heuristics.argtypes = [P, I, I, D, I, I, D, I, I]
    lib.ora_get_rsum.argtypes = [P, I, P]
    lib.ora_set_exploit.argtypes = [P, I, D, D, I, I]
    lib.ora_get_ph.argtypes = [P, I, P, P, P, P]
    lib.ora_set_ph.argtypes = [P, I, P, D, L, L]
    lib.ora_set_refine.argtypes = [P, I, I, I, I, I, I]
    lib.ora_set_sticky.argtypes = [P, I]
    lib.ora_get_window.argtypes = [P, I, P, P, P]
    lib.ora_get_ph_all.argtypes = [P, P, P, P, P]
    lib.ora_get_window_all.argtypes = [P, P]
    lib.ora_set_window.argtypes = [P, I, I, I, I]
    lib.ora_commit.argtypes = [P, P, P, P]
    lib.ora_flush.argtypes = [P, P]
    lib.ora_get.argtypes = [P, I, P, P, P, P, P, P, P]
    lib.ora_alpha.restype = D
    lib.ora_alpha.argtypes = [P, L]
    lib.ora_t_now.restype = L
    lib.ora_t_now.argtypes = [P]
    lib.ora_threads.restype = I
    lib.ora_set_threads.argtypes = [I]
    return lib


def load_library(path=None):
    """Load the oracle library, building it first if it is not there."""
    global _lib
    if path is not None:
        return _declare(ctypes.CDLL(path))
    if _lib is None:
        if not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
            build_library()
        _lib = _declare(ctypes.CDLL(_LIB))
    return _lib


def _ptr(a):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


class Oracle:
    """B independent disjoint-LinUCB tuners in double precision (Eq. 1-5)."""

    def __init__(self, B, K, d, lam=1.0, alpha0=1.0, sched=0, prune=0, period=50,
                 lib=None):
        self.lib = lib if lib is not None else load_library()
        self.B, self.K, self.d = int(B), int(K), int(d)
        self.h = self.lib.ora_create(self.B, self.K, self.d, float(lam), float(alpha0),
                                     int(sched), int(prune), int(period))
        if not self.h:
            raise ValueError("oracle: invalid configuration")

    @classmethod
    def from_workload(cls, wl, B=None, lib=None):
        o = cls(wl.B if B is None else B, wl.K, wl.d, wl.lam, wl.alpha0,
                wl.alpha_sched, wl.prune, wl.period, lib=lib)
        if not wl.prune_sticky:
            o.set_sticky(False)
        if wl.prune & 14:
            o.set_heuristics(**wl.heuristics())
        if wl.exploit:
            o.set_exploit(True, **wl.page_hinkley())
        if wl.refine:
            o.set_refine(True, **wl.refinement())
        return o

    def set_sticky(self, sticky):
        """Rule 1 removes arms for good (True, the default) or is re-evaluated
        over the whole action space at each of its steps (False)."""
        self.lib.ora_set_sticky(self.h, int(bool(sticky)))

    def set_exploit(self, on, ph_delta, ph_lambda, ph_window, ph_min_rounds):
        """Page-Hinkley switch to greedy exploitation (Sec. 4.2, Eq. 2)."""
        self.lib.ora_set_exploit(self.h, int(bool(on)), float(ph_delta), float(ph_lambda),
                                 int(ph_window), int(ph_min_rounds))

    def page_hinkley(self, i):
        """(stats[6]: n, mean, m+, min m+, m-, min m-; last margin; last alarm
        round; mode) of instance i, in double precision."""
        stats = np.empty(6, dtype=np.float64)
        margin = ctypes.c_double(0.0)
        last = ctypes.c_long(0)
        mode = ctypes.c_long(0)
        self.lib.ora_get_ph(self.h, int(i), _ptr(stats), ctypes.byref(margin), ctypes.byref(last),
                            ctypes.byref(mode))
        return stats, margin.value, last.value, mode.value

    def set_refine(self, on, refine_period, refine_stride, refine_half, refine_mature,
                   refine_min_n):
        """Mixed-maturity refinement of the action space (Sec. 4.4)."""
        self.lib.ora_set_refine(self.h, int(bool(on)), int(refine_period), int(refine_stride),
                                int(refine_half), int(refine_mature), int(refine_min_n))

    def window(self, i):
        """(lo, hi, stride) of instance i's action space."""
        v = [ctypes.c_int(0) for _ in range(3)]
        self.lib.ora_get_window(self.h, int(i), *(ctypes.byref(q) for q in v))
        return tuple(q.value for q in v)

    def page_hinkley_all(self):
        """Every instance's (stats [B][6], margin [B], last alarm round [B],
        mode [B]), in double precision."""
        stats = np.empty((self.B, 6), dtype=np.float64)
        margin = np.empty(self.B, dtype=np.float64)
        last = np.empty(self.B, dtype=np.int64)
        mode = np.empty(self.B, dtype=np.int64)
        self.lib.ora_get_ph_all(self.h, _ptr(stats), _ptr(margin), _ptr(last), _ptr(mode))
        return stats, margin, last, mode

    def windows(self):
        """Every instance's action space, [B][3] = (lo, hi, stride)."""
        win = np.empty((self.B, 3), dtype=np.int32)
        self.lib.ora_get_window_all(self.h, _ptr(win))
        return win

    def set_window(self, i, lo, hi, stride):
        self.lib.ora_set_window(self.h, int(i), int(lo), int(hi), int(stride))

    def set_page_hinkley(self, i, stats, margin, last, mode):
        """Overwrite instance i's Page-Hinkley state and mode."""
        st = np.ascontiguousarray(stats, dtype=np.float64)
        self.lib.ora_set_ph(self.h, int(i), _ptr(st), float(margin), int(last), int(mode))

    def set_heuristics(self, ext_rounds, ext_min_n, ext_thr, hist_after, hist_min_n, hist_kappa,
                       hist_min_arms, cascade_k):
        """Parameters of the paper's pruning rules (bits 2, 4, 8 of the rule mask)."""
        self.lib.ora_set_heuristics(self.h, int(ext_rounds), int(ext_min_n), float(ext_thr),
                                    int(hist_after), int(hist_min_n), float(hist_kappa),
                                    int(hist_min_arms), int(cascade_k))

    def __del__(self):
        h = getattr(self, "h", None)
        if h:
            self.lib.ora_destroy(h)
            self.h = None

    @property
    def t(self):
        return int(self.lib.ora_t_now(self.h))

    def alpha(self, t=None):
        return float(self.lib.ora_alpha(self.h, self.t if t is None else int(t)))

    def decide(self, x, r=None, margins=False):
        """Apply the pending update, score x_t, prune, pick a_t.

        Returns (ucb [B][K], lcb [B][K], keep [B][K] bool, action [B]) and, with
        margins=True, also the per-arm distances of the rule-2/4 comparisons
        from their thresholds [B][K] (inf where no such rule applied)."""
        x = np.ascontiguousarray(x, dtype=np.float64).reshape(self.B, self.d)
        r = None if r is None else np.ascontiguousarray(r, dtype=np.float64).reshape(self.B)
        ucb = np.empty((self.B, self.K))
        lcb = np.empty((self.B, self.K))
        keep = np.empty((self.B, self.K), dtype=np.uint8)
        action = np.empty(self.B, dtype=np.int32)
        marg = np.empty((self.B, self.K)) if margins else None
        self.lib.ora_decide_ex(self.h, _ptr(x), _ptr(r), _ptr(ucb), _ptr(lcb), _ptr(keep),
                               _ptr(action), _ptr(marg))
        if margins:
            return ucb, lcb, keep.astype(bool), action, marg
        return ucb, lcb, keep.astype(bool), action

    def commit(self, x, action, keep):
        x = np.ascontiguousarray(x, dtype=np.float64).reshape(self.B, self.d)
        action = np.ascontiguousarray(action, dtype=np.int32).reshape(self.B)
        keep = np.ascontiguousarray(keep, dtype=np.uint8).reshape(self.B, self.K)
        self.lib.ora_commit(self.h, _ptr(x), _ptr(action), _ptr(keep))

    def step(self, x, r=None):
        """decide + commit of the oracle's own decision."""
        ucb, lcb, keep, action = self.decide(x, r)
        self.commit(x, action, keep)
        return ucb, lcb, keep, action

    def flush(self, r):
        r = np.ascontiguousarray(r, dtype=np.float64).reshape(self.B)
        self.lib.ora_flush(self.h, _ptr(r))

    def get(self, i):
        K, d = self.K, self.d
        out = dict(A=np.empty((K, d, d)), b=np.empty((K, d)), Ainv=np.empty((K, d, d)),
                   theta=np.empty((K, d)), active=np.empty(K, dtype=np.uint8),
                   nsel=np.empty(K, dtype=np.int32))
        bad = ctypes.c_int(0)
        self.lib.ora_get(self.h, int(i), _ptr(out["A"]), _ptr(out["b"]), _ptr(out["Ainv"]),
                         _ptr(out["theta"]), _ptr(out["active"]), _ptr(out["nsel"]),
                         ctypes.byref(bad))
        out["active"] = out["active"].astype(bool)
        out["bad"] = bad.value
        out["rsum"] = np.empty(K)
        self.lib.ora_get_rsum(self.h, int(i), _ptr(out["rsum"]))
        return out

    @staticmethod
    def threads():
        return int(load_library().ora_threads())

    @staticmethod
    def set_threads(n):
        load_library().ora_set_threads(int(n))
