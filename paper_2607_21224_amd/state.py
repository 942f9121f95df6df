"""Device-resident CPDP state and the host cadence that drives it.

PyTorch only allocates the HBM buffers and supplies the stream; every update
goes through the C ABI (``cpdp.py``).  Layout: params / mom are (W, ld)
tensors whose first P columns are the replicas' coordinates (row stride ld);
slow_mom (u) and anchor (the reference model) are (P,) fp32 tensors.

Every method that launches takes ``stream``: a ``torch.cuda.Stream``, a raw
``hipStream_t`` integer, or None for torch's current stream, as torch's own
operations use (the C ABI itself reads a NULL stream as the null stream).
"""
from __future__ import annotations

from dataclasses import dataclass

import torch

from . import cpdp


def round_up(x: int, m: int) -> int:
    return (x + m - 1) // m * m


def check_exact(ref: torch.Tensor, src, name: str) -> None:
    """A checkpointed tensor must have exactly the shape and dtype of the state
    buffer it restores: never a broadcast or a conversion."""
    if not isinstance(src, torch.Tensor):
        raise ValueError(f"{name}: expected a tensor, got {type(src).__name__}")
    if tuple(src.shape) != tuple(ref.shape) or src.dtype != ref.dtype:
        raise ValueError(f"{name}: expected {tuple(ref.shape)} {ref.dtype}, "
                         f"got {tuple(src.shape)} {src.dtype}")


def load_exact(dst: torch.Tensor, src, name: str) -> None:
    check_exact(dst, src, name)
    dst.copy_(src)


# torch's raw handle of the current stream (no Stream object built per call)
_raw_current_stream = getattr(torch._C, "_cuda_getCurrentRawStream", None)
_has_gpu = None  # torch.cuda.is_available(), asked once per process


def _on(stream):
    """The stream a launch goes to: the one given, else torch's current
    stream, so work inside ``torch.cuda.stream(s)`` (or a graph capture on
    ``s``) stays ordered with the rest of that stream."""
    global _has_gpu
    if stream is not None:
        return stream
    if _has_gpu is None:
        _has_gpu = torch.cuda.is_available()
    if not _has_gpu:
        return None  # without a GPU the binding rejects the buffers itself
    if _raw_current_stream is not None:
        return _raw_current_stream(torch.cuda.current_device())
    return torch.cuda.current_stream()


@dataclass(frozen=True)
class Hyper:
    """Hyperparameters as the fp32 values the kernels use."""
    lr: float
    mu: float
    beta: float
    alpha: float

    @staticmethod
    def fp32(lr, mu, beta, alpha) -> "Hyper":
        f = lambda x: float(torch.tensor(x, dtype=torch.float32))  # noqa: E731
        return Hyper(f(lr), f(mu), f(beta), f(alpha))


@dataclass(frozen=True)
class Optimizer:
    """A per-replica optimizer (Table 3): "sgd" (momentum, coupled weight
    decay) or "adamw" (betas (momentum, beta2), eps, decoupled weight decay).
    Values are the fp32 numbers the kernels use."""
    kind: str
    lr: float
    momentum: float = 0.0
    beta2: float = 0.999
    eps: float = 1e-8
    weight_decay: float = 0.0

    def c_struct(self, step: int) -> "cpdp.cpdp_optimizer":
        k = {"sgd": cpdp.CPDP_OPT_SGD, "adamw": cpdp.CPDP_OPT_ADAMW}[self.kind]
        return cpdp.cpdp_optimizer(k, self.lr, self.momentum, self.beta2, self.eps,
                                   self.weight_decay, int(step))


class StepTable:
    """Per-step scalars of n consecutive steps in device memory (the C ABI's
    step table).  ``entries`` is a sequence of (Optimizer, step, beta, alpha):
    the optimizer of that step (its lr from any schedule), AdamW's 1-based
    step count, and the SlowMo coefficients of a CPDP sync at that step."""

    def __init__(self, entries, device="cuda"):
        entries = list(entries)
        self.n = len(entries)
        nbytes = cpdp.cpdp_step_table_bytes(self.n)
        if nbytes <= 0:
            raise ValueError("a step table needs at least one entry")
        self.buf = torch.empty(nbytes, dtype=torch.uint8, device=device)
        self.handle = cpdp.cpdp_step_table()
        self.handle.table = self.buf.data_ptr()
        cpdp.cpdp_step_table_fill(self.handle, nbytes, [o.c_struct(st) for o, st, _, _ in entries],
                                  [b for _, _, b, _ in entries], [a for _, _, _, a in entries])

    def set_position(self, position: int = 0, stream=None) -> None:
        cpdp.cpdp_step_table_set_position(self.handle, position, _on(stream))

    def position(self) -> int:
        """The entry the next table step uses (synchronous read)."""
        return cpdp.cpdp_step_table_position(self.handle)


class CpdpState:
    """W replicas of a P-coordinate model with per-replica momentum, SlowMo
    velocity u and the reference (anchor) model, all in HBM."""

    # Default row stride: rows rounded up to a multiple of 1 MiB.  On MI355X
    # the fused reconcile, which streams all W rows of three families at the
    # same offset, ran 3-7 % faster with such strides than with 256-byte ones
    # on the ResNet-50-sized states; the padding costs at most 1 MiB per row.
    ROW_ALIGN_BYTES = 1 << 20

    def __init__(self, W: int, P: int, ld: int | None = None, K: int = 1,
                 param_dt: str = "f32", device="cuda", grad_dt: str = "f32",
                 mom_dt: str = "f32", adamw: bool = False):
        """grad_dt / mom_dt: storage types of the gradient rows the steps take
        and of the momentum buffers, "f32", or "bf16" for the momentum-SGD
        path (init, local_step, reconcile, localsgd_sync, ddp_step, step());
        the general-optimizer and step-table paths take fp32 for both.
        adamw=True allocates AdamW's second-moment rows now, together with
        the other state buffers, rather than at init_opt (after whatever the
        caller allocated in between).  Where the rows land changes the AdamW
        local step's speed on MI355X by several percent either way; placed
        with the state it was never slower in the runs measured."""
        for name, dt in (("param_dt", param_dt), ("grad_dt", grad_dt), ("mom_dt", mom_dt)):
            if dt not in ("f32", "bf16"):
                raise ValueError(f"{name} must be 'f32' or 'bf16', got {dt!r}")
        self.grad_dt, self.mom_dt = grad_dt, mom_dt
        self.W, self.P, self.K = int(W), int(P), int(K)
        esize = 2 if param_dt == "bf16" else 4
        align = self.ROW_ALIGN_BYTES // esize
        self.ld = int(ld) if ld is not None else round_up(max(self.P, 1), align)
        self.param_dt = param_dt
        tdt = torch.bfloat16 if param_dt == "bf16" else torch.float32
        self.params = torch.empty((self.W, self.ld), dtype=tdt, device=device)
        mdt = torch.bfloat16 if mom_dt == "bf16" else torch.float32
        self.mom = torch.empty((self.W, self.ld), dtype=mdt, device=device)
        self.slow_mom = torch.empty(max(self.P, 1), dtype=torch.float32, device=device)
        self.anchor = torch.empty(max(self.P, 1), dtype=torch.float32, device=device)
        # AdamW second moments: allocated here when asked for, else by init_opt
        self.mom2 = torch.empty_like(self.mom) if adamw else None
        self.opt_step = 0         # optimizer updates applied (AdamW bias correction)
        self._count = None        # device word of count_unsynced

    @property
    def torch_param_dtype(self):
        return self.params.dtype

    def init(self, theta0: torch.Tensor, stream=None) -> None:
        """Algorithm 1 initialisation; theta0 is (P,) in the parameter dtype."""
        self._check_theta0(theta0)
        cpdp.cpdp_state_init(theta0, self.params, self.mom, self.slow_mom,
                             self.anchor, self.W, self.P, self.ld, self.K,
                             self.param_dt, self.mom_dt, _on(stream))

    def local_step(self, grads: torch.Tensor, h: Hyper, stream=None) -> None:
        self._check_grads(grads)
        cpdp.cpdp_local_step(self.params, self.mom, grads, self.W, self.P,
                             self.ld, self.K, h.lr, h.mu, self.param_dt, self.grad_dt,
                             self.mom_dt, _on(stream))

    def reconcile(self, grads: torch.Tensor, h: Hyper, stream=None) -> None:
        self._check_grads(grads)
        cpdp.cpdp_reconcile(self.params, self.mom, grads, self.slow_mom,
                            self.anchor, self.W, self.P, self.ld, self.K, h.lr,
                            h.mu, h.beta, h.alpha, self.param_dt, self.grad_dt, self.mom_dt,
                            _on(stream))

    def localsgd_sync(self, grads: torch.Tensor, h: Hyper, stream=None,
                      write_anchor: bool = True) -> None:
        """LocalSGD synchronisation (Sec. 5.3): local step, then parameter
        averaging; the average also goes to ``anchor`` unless told not to."""
        self._check_grads(grads)
        cpdp.cpdp_localsgd_sync(self.params, self.mom, grads,
                                self.anchor if write_anchor else None, self.W,
                                self.P, self.ld, self.K, h.lr, h.mu,
                                self.param_dt, self.grad_dt, self.mom_dt, _on(stream))

    def ddp_step(self, grads: torch.Tensor, h: Hyper, stream=None) -> None:
        """Synchronous DDP step (Sec. 3.1, Sec. 5.3)."""
        self._check_grads(grads)
        cpdp.cpdp_ddp_step(self.params, self.mom, grads, self.W, self.P,
                           self.ld, h.lr, h.mu, self.param_dt, self.grad_dt, self.mom_dt,
                           _on(stream))

    METHODS = ("cpdp", "localsgd", "ddp")

    # ---- general optimizers (SGD with weight decay, AdamW) -------------------

    def init_opt(self, theta0: torch.Tensor, opt: Optimizer, stream=None) -> None:
        """Initialisation for a general optimizer (second-moment buffers for
        AdamW are allocated and zeroed too)."""
        self._check_theta0(theta0)
        if self.mom_dt != "f32":
            raise ValueError("the general optimizers keep fp32 momentum; "
                             "this state was made with mom_dt='bf16'")
        if opt.kind == "adamw" and self.mom2 is None:
            self.mom2 = torch.empty_like(self.mom)
        cpdp.cpdp_state_init_opt(theta0, self.params, self.mom,
                                 self.mom2 if opt.kind == "adamw" else None,
                                 self.slow_mom, self.anchor, self.W, self.P, self.ld,
                                 self.K, self.param_dt, _on(stream))
        self.opt_step = 0

    def step_opt(self, t: int, grads: torch.Tensor, opt: Optimizer, beta: float = 0.0,
                 alpha: float = 1.0, T: int = 0, stream=None, method: str = "cpdp",
                 flags: int = 0) -> str:
        """One step of ``method`` with a general optimizer (see step()).
        ``flags`` selects sync-step variants (cpdp.CPDP_SYNC_WRITE_GRAD_MEAN,
        cpdp.CPDP_SYNC_AVERAGE_OPT_STATE)."""
        self._check_grads(grads, fp32_only=True)
        if method not in self.METHODS:
            raise ValueError(method)
        # the update counter advances only once the library has taken the step
        c = opt.c_struct(self.opt_step + 1)
        mom2 = self.mom2 if opt.kind == "adamw" else None
        if method == "ddp" or cpdp.cpdp_is_sync_step(t, self.K, T):
            cpdp.cpdp_sync_step_opt(method, self.params, self.mom, mom2, grads,
                                    self.slow_mom, self.anchor, self.W, self.P, self.ld,
                                    self.K, c, beta, alpha, flags, self.param_dt, _on(stream))
            kind = "reconcile"
        else:
            cpdp.cpdp_local_step_opt(self.params, self.mom, mom2, grads, self.W, self.P,
                                     self.ld, self.K, c, self.param_dt, _on(stream))
            kind = "local"
        self.opt_step += 1
        return kind

    def step(self, t: int, grads: torch.Tensor, h: Hyper, T: int = 0,
             stream=None, method: str = "cpdp") -> str:
        """Step t (1-based within the epoch) of a synchronisation strategy.

        cpdp / localsgd: a synchronisation step when the cadence of Sec. 3.2
        (with the epoch-end rule of Sec. 3.1) says so, else a local step.
        ddp: every step synchronises the gradient (the K = 1 schedule).
        Returns "reconcile" for a synchronisation step, "local" otherwise."""
        if method == "ddp":
            self.ddp_step(grads, h, stream)
            return "reconcile"
        if method not in self.METHODS:
            raise ValueError(method)
        if cpdp.cpdp_is_sync_step(t, self.K, T):
            if method == "cpdp":
                self.reconcile(grads, h, stream)
            else:
                self.localsgd_sync(grads, h, stream)
            return "reconcile"
        self.local_step(grads, h, stream)
        return "local"

    def step_table(self, t: int, grads: torch.Tensor, table: StepTable, T: int = 0,
                   stream=None, method: str = "cpdp", flags: int = 0) -> str:
        """Step t of ``method`` with the scalars of the table's current entry,
        then advance the table (both on ``stream``).  Same cadence and
        semantics as step_opt; the optimizer state must match the table's
        update rule (init_opt with an AdamW optimizer for an AdamW table)."""
        self._check_grads(grads, fp32_only=True)
        if method not in self.METHODS:
            raise ValueError(method)
        h = table.handle
        if h.update == 2 and self.mom2 is None:
            raise ValueError("an AdamW step table needs the state initialised by init_opt(adamw)")
        mom2 = self.mom2 if h.update == 2 else None
        if method == "ddp" or cpdp.cpdp_is_sync_step(t, self.K, T):
            cpdp.cpdp_sync_step_table(method, self.params, self.mom, mom2, grads, self.slow_mom,
                                      self.anchor, self.W, self.P, self.ld, self.K, h, flags,
                                      self.param_dt, _on(stream))
            kind = "reconcile"
        else:
            cpdp.cpdp_local_step_table(self.params, self.mom, mom2, grads, self.W, self.P,
                                       self.ld, self.K, h, self.param_dt, _on(stream))
            kind = "local"
        cpdp.cpdp_step_table_advance(h, _on(stream))
        return kind

    def capture_steps(self, grads: list, table: StepTable, T: int = 0, t0: int = 1,
                      method: str = "cpdp", flags: int = 0):
        """Capture steps t0 .. t0+len(grads)-1 (cadence decided now) as table
        steps into a HIP graph.  Every replay runs them with the table's next
        len(grads) entries, so a graph of one period replays successive
        periods of a schedule.  Returns (graph, kinds)."""
        for g in grads:
            self._check_grads(g, fp32_only=True)
        graph = torch.cuda.CUDAGraph()
        kinds = []
        side = torch.cuda.Stream()
        side.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(side):
            torch.cuda.synchronize()
            with torch.cuda.graph(graph, stream=side):
                cs = torch.cuda.current_stream()
                for j, g in enumerate(grads):
                    kinds.append(self.step_table(t0 + j, g, table, T, stream=cs, method=method,
                                                 flags=flags))
        torch.cuda.current_stream().wait_stream(side)
        return graph, kinds

    def count_unsynced(self, stream=None) -> int:
        """Coordinates at which some replica does not hold the reference model
        (bitwise, in the parameter storage type).  0 right after every CPDP or
        LocalSGD synchronisation; anything else is a missed or partial sync.
        Synchronises the stream to read the result."""
        if self._count is None:
            self._count = torch.zeros(1, dtype=torch.int64, device=self.params.device)
        cpdp.cpdp_count_unsynced(self.params, self.anchor, self.W, self.P, self.ld, self._count,
                                 self.param_dt, _on(stream))
        if isinstance(stream, torch.cuda.Stream):
            stream.synchronize()
        elif stream is None:
            torch.cuda.current_stream().synchronize()
        else:
            torch.cuda.synchronize(self.params.device)
        return int(self._count.item())

    # ---- HIP graph capture of a period --------------------------------------------

    def capture_period(self, grads: list, h: Hyper, method: str = "cpdp", T: int = 0,
                       t0: int = 1):
        """Capture steps t0 .. t0+len(grads)-1 (cadence decided now, from
        ``self.K``) into a HIP graph; replaying it runs those steps on the
        gradient buffers ``grads`` (refill them between replays).  For
        fixed-scalar steps only: the hyperparameters are baked into the graph.
        Returns (graph, kinds)."""
        for g in grads:
            self._check_grads(g)
        graph = torch.cuda.CUDAGraph()
        kinds = []
        side = torch.cuda.Stream()
        side.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(side):
            torch.cuda.synchronize()
            with torch.cuda.graph(graph, stream=side):
                cs = torch.cuda.current_stream()
                for j, g in enumerate(grads):
                    kinds.append(self.step(t0 + j, g, h, T, stream=cs, method=method))
        torch.cuda.current_stream().wait_stream(side)
        return graph, kinds

    # ---- checkpoint / resume ---------------------------------------------------

    def state_dict(self) -> dict:
        """Host copy of the whole CPDP state (replicas, optimizer state, SlowMo
        state, reference model, step counter), enough to resume bitwise.
        Waits for all work on the device first, so steps launched on any
        stream are included."""
        torch.cuda.synchronize(self.params.device)
        d = {"W": self.W, "P": self.P, "ld": self.ld, "K": self.K,
             "param_dt": self.param_dt, "grad_dt": self.grad_dt, "mom_dt": self.mom_dt,
             "opt_step": self.opt_step,
             "params": self.params.cpu(), "mom": self.mom.cpu(),
             "slow_mom": self.slow_mom.cpu(), "anchor": self.anchor.cpu()}
        if self.mom2 is not None:
            d["mom2"] = self.mom2.cpu()
        return d

    @classmethod
    def from_state_dict(cls, d: dict, device="cuda") -> "CpdpState":
        """A new state holding a state_dict's values.  Every buffer must have
        exactly the shape and type the layout (W, P, ld, param_dt) implies:
        the kernels trust the state's W and ld, so a mismatched buffer is
        rejected here rather than copied or broadcast."""
        st = cls(d["W"], d["P"], d["ld"], d["K"], d["param_dt"], device=device,
                 grad_dt=d.get("grad_dt", "f32"), mom_dt=d.get("mom_dt", "f32"),
                 adamw="mom2" in d)
        for name in ("params", "mom", "slow_mom", "anchor") + (("mom2",) if "mom2" in d else ()):
            load_exact(getattr(st, name), d[name], name)
        st.opt_step = int(d["opt_step"])
        return st

    # The ABI takes raw addresses, so these shape checks are what keeps a
    # kernel inside the caller's buffers: they raise, they are not asserts.
    def _check_grads(self, g: torch.Tensor, fp32_only: bool = False) -> None:
        if fp32_only and (self.grad_dt, self.mom_dt) != ("f32", "f32"):
            raise ValueError("the general-optimizer and step-table paths take fp32 gradients "
                             "and momentum; this state was made with "
                             f"grad_dt={self.grad_dt!r}, mom_dt={self.mom_dt!r}")
        want = torch.bfloat16 if self.grad_dt == "bf16" else torch.float32
        if g.dtype != want or not g.is_contiguous():
            raise ValueError(f"grads must be a contiguous {want} tensor")
        if tuple(g.shape) != (self.W, self.ld):
            raise ValueError(f"grads must have shape {(self.W, self.ld)}, got {tuple(g.shape)}")
        if g.device != self.params.device:
            raise ValueError(f"grads are on {g.device}, the state on {self.params.device}")

    def _check_theta0(self, theta0: torch.Tensor) -> None:
        if theta0.dtype != self.params.dtype or not theta0.is_contiguous():
            raise ValueError(f"theta0 must be a contiguous {self.params.dtype} tensor")
        if theta0.numel() < self.P:
            raise ValueError(f"theta0 has {theta0.numel()} elements, P = {self.P}")
        if theta0.device != self.params.device:
            raise ValueError(f"theta0 is on {theta0.device}, the state on {self.params.device}")
