"""Python front end of the batched tuner: torch supplies device memory and the
stream, every step of the method runs in the HIP kernels behind libagft.so."""
import ctypes

import torch

from . import _lib as L


def _ptr(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream_handle(stream):
    return ctypes.c_void_p(stream.cuda_stream)


def make_config(B, K, d, lam=1.0, alpha0=1.0, alpha_sched=0, prune_rule=0, prune_period=50,
                adopt=False, heuristics=None, exploit=None, refine=None, prune_sticky=1):
    """The agft_config of a tuner (no device work)."""
    cfg = L.agft_config(int(B), int(K), int(d), float(lam), float(alpha0), int(alpha_sched),
                        int(prune_rule), int(prune_period), int(prune_sticky),
                        L.AGFT_ADOPT_STATE if adopt else 0)
    for name, value in (heuristics or {}).items():
        setattr(cfg, name, value)
    if exploit:
        cfg.exploit = 1
        for name, value in exploit.items():
            setattr(cfg, name, value)
    if refine:
        cfg.refine = 1
        for name, value in refine.items():
            setattr(cfg, name, value)
    return cfg


def workload_config(wl, B=None):
    """The agft_config of a workload from agft_workloads."""
    return make_config(wl.B if B is None else B, wl.K, wl.d, wl.lam, wl.alpha0, wl.alpha_sched,
                       wl.prune, wl.period, heuristics=wl.heuristics(),
                       exploit=wl.page_hinkley() if wl.exploit else None,
                       refine=wl.refinement() if wl.refine else None, prune_sticky=wl.prune_sticky)


def launch_shape(cfg):
    """How agft_step launches the step kernel for cfg: dict(waves,
    simd_waves, tail_floats, early_update, cu_workgroups)."""
    code, shape = L.agft_launch_shape_for(cfg)
    L.check("agft_launch_shape_for", code)
    return {name: int(getattr(shape, name)) for name, _ in shape._fields_}


class Tuner:
    """B independent AGFT frequency tuners (disjoint LinUCB over K arms, Sec. 4.2)."""

    def __init__(self, B, K, d, lam=1.0, alpha0=1.0, alpha_sched=0, prune_rule=0,
                 prune_period=50, device="cuda", stream=None, state=None, adopt=False,
                 heuristics=None, exploit=None, refine=None, prune_sticky=1):
        self.device = torch.device(device)
        if self.device.type == "cuda" and self.device.index is None:
            self.device = torch.device("cuda", torch.cuda.current_device())
        self.cfg = make_config(B, K, d, lam, alpha0, alpha_sched, prune_rule, prune_period, adopt,
                               heuristics, exploit, refine, prune_sticky)
        self.nbytes = L.agft_state_bytes(self.cfg)
        if self.nbytes == 0:
            raise ValueError("invalid tuner configuration")
        if state is None:
            if adopt:
                raise ValueError("adopt=True needs an existing state buffer")
            # zeroed so that the alignment gaps between regions are deterministic
            state = torch.zeros(self.nbytes, dtype=torch.uint8, device=self.device)
        if state.dtype != torch.uint8 or state.dim() != 1 or not state.is_contiguous():
            raise ValueError("state must be a contiguous 1-D uint8 tensor")
        if state.data_ptr() % 256 != 0:
            raise ValueError("state buffer must be 256-byte aligned")
        self.state = state
        self.stream = stream if stream is not None else torch.cuda.current_stream(self.device)
        self.B, self.K, self.d = int(B), int(K), int(d)
        code, h = L.agft_create(self.cfg, _ptr(state), state.numel(), _stream_handle(self.stream))
        L.check("agft_create", code)
        self.h = h

    @classmethod
    def from_workload(cls, wl, B=None, **kw):
        return cls(wl.B if B is None else B, wl.K, wl.d, wl.lam, wl.alpha0, wl.alpha_sched,
                   wl.prune, wl.period, heuristics=wl.heuristics(),
                   exploit=wl.page_hinkley() if wl.exploit else None,
                   refine=wl.refinement() if wl.refine else None, prune_sticky=wl.prune_sticky, **kw)

    def close(self):
        if getattr(self, "h", None):
            try:
                L.agft_destroy(self.h)
            except TypeError:      # interpreter shutdown: ctypes already torn down
                pass
            self.h = None

    def __del__(self):
        self.close()

    def _check(self, t, shape, dtype):
        if t is None:
            return
        if t.device != self.device or t.dtype != dtype or not t.is_contiguous():
            raise ValueError(f"expected a contiguous {dtype} tensor on {self.device}")
        if tuple(t.shape) != tuple(shape):
            raise ValueError(f"expected shape {tuple(shape)}, got {tuple(t.shape)}")

    def step(self, ctx, reward=None, action=None, scores=None):
        """Fold `reward` (of the previous decision) in, decide on `ctx`.

        ctx [B][d] fp32, reward [B] fp32 (None before the first decision),
        action [B] int32 out (allocated if None), scores [B][2][K] fp32 out or None.
        """
        self._check(ctx, (self.B, self.d), torch.float32)
        self._check(reward, (self.B,), torch.float32)
        if action is None:
            action = torch.empty(self.B, dtype=torch.int32, device=self.device)
        self._check(action, (self.B,), torch.int32)
        self._check(scores, (self.B, 2, self.K), torch.float32)
        L.check("agft_step", L.agft_step(self.h, _ptr(ctx), _ptr(reward), _ptr(action),
                                         _ptr(scores)))
        return action

    def flush(self, reward):
        """Fold the last decision's reward in without deciding."""
        self._check(reward, (self.B,), torch.float32)
        L.check("agft_step", L.agft_step(self.h, None, _ptr(reward), None, None))

    def set_stream(self, stream):
        self.stream = stream
        L.check("agft_set_stream", L.agft_set_stream(self.h, _stream_handle(stream)))

    def view(self):
        """Tensor views into the state buffer (no copies)."""
        code, v = L.agft_get_state(self.h)
        L.check("agft_get_state", code)
        base = self.state.data_ptr()

        def region(ptr, count, dtype, shape):
            off = ptr - base
            nb = count * torch.tensor([], dtype=dtype).element_size()
            return self.state[off:off + nb].view(dtype).view(shape)

        B, K, d, C, KW, IW = v.B, v.K, v.d, v.chunks, v.mask_words, v.inst_words
        NB = v.block_arms
        KB = (K + NB - 1) // NB
        inst = region(v.inst, B * IW, torch.int32, (B, IW))
        return dict(
            t=int(v.t), pending=int(v.pending),
            # [B][blocks][NB * chunks][4]: per block the NB main parts, then the NB tails
            arms=region(v.arms, B * KB * NB * C * 4, torch.float32, (B, KB, NB * C, 4)),
            mask=region(v.mask, B * KW, torch.int32, (B, KW)),
            inst=inst,
            aprev=inst[:, 0], kact=inst[:, 1], bad=inst[:, 2], mode=inst[:, 3], ph=inst[:, 3:12],
            window=inst[:, 12:15], gap=inst[:, 15].view(torch.float32),
            xprev=inst[:, 16:16 + d].view(torch.float32),
            stats=region(v.stats, B * K * 2, torch.int32, (B, K, 2)),
            theta=region(v.theta, B * K * d, torch.float32, (B, K, d)) if v.theta else None,
        )

    @property
    def t(self):
        code, v = L.agft_get_state(self.h)
        L.check("agft_get_state", code)
        return int(v.t)

    def active_mask(self, view=None):
        """[B][K] bool of the active arms (a device op on the mask words)."""
        v = self.view() if view is None else view
        words = v["mask"]
        k = torch.arange(self.K, device=self.device)
        return ((words[:, k // 32] >> (k % 32)) & 1).bool()

    def export(self, theta=True, ainv=False):
        th = torch.empty(self.B, self.K, self.d, device=self.device) if theta else None
        ai = torch.empty(self.B, self.K, self.d, self.d, device=self.device) if ainv else None
        L.check("agft_export", L.agft_export(self.h, _ptr(th), _ptr(ai)))
        return th, ai
