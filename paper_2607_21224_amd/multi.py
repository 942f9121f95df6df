"""Multi-tensor CPDP state: the model as a list of separate tensors per
replica (as a framework holds it), driven through a device-resident plan so
each step is one launch over all tensors."""
from __future__ import annotations

import torch

from . import cpdp
from .state import Hyper, Optimizer, _on, check_exact, load_exact


class CpdpMultiState:
    """W replicas of a model given as tensor sizes ``numels``; every
    (replica, tensor) of params / mom (/ mom2) / grads is its own allocation;
    slow_mom and anchor are one tensor per model tensor."""

    def __init__(self, W: int, numels, K: int = 1, param_dt: str = "f32",
                 adamw: bool = False, device="cuda"):
        if param_dt not in ("f32", "bf16"):
            raise ValueError(f"param_dt must be 'f32' or 'bf16', got {param_dt!r}")
        self.W, self.K, self.param_dt = int(W), int(K), param_dt
        self.numels = [int(x) for x in numels]
        n = self.n = len(self.numels)
        tdt = torch.bfloat16 if param_dt == "bf16" else torch.float32
        mk = lambda dt: [[torch.empty(max(x, 1), dtype=dt, device=device)  # noqa: E731
                          for x in self.numels] for _ in range(W)]
        self.params, self.mom, self.grads = mk(tdt), mk(torch.float32), mk(torch.float32)
        self.mom2 = mk(torch.float32) if adamw else None
        self.slow_mom = [torch.empty(max(x, 1), device=device) for x in self.numels]
        self.anchor = [torch.empty(max(x, 1), device=device) for x in self.numels]
        nbytes = cpdp.cpdp_plan_bytes(W, n)
        self.table = torch.empty(nbytes, dtype=torch.uint8, device=device)
        self.plan = cpdp.cpdp_plan()
        self.plan.table = self.table.data_ptr()
        flat = lambda fam: [fam[i][t] for i in range(W) for t in range(n)]  # noqa: E731
        cpdp.cpdp_plan_build(self.plan, nbytes, W, n, self.numels, flat(self.params),
                             flat(self.mom), flat(self.mom2) if adamw else None,
                             flat(self.grads), self.slow_mom, self.anchor, param_dt)
        self.opt_step = 0

    def init(self, theta0_list, stream=None) -> None:
        """Algorithm 1 initialisation from per-tensor initial values.  The
        values are taken in the parameter storage type (rounded to nearest
        even if given wider), so the reference model starts equal to what
        every replica holds, as in the flat layout."""
        if len(theta0_list) != self.n:
            raise ValueError(f"expected {self.n} initial tensors, got {len(theta0_list)}")
        pdt = self.params[0][0].dtype
        for t, (a, th) in enumerate(zip(self.anchor, theta0_list)):
            if th.numel() != self.numels[t]:
                raise ValueError(f"tensor {t}: {th.numel()} elements, expected {self.numels[t]}")
            a[: th.numel()].copy_(th.reshape(-1).to(pdt).float())
        torch.cuda.synchronize()
        cpdp.cpdp_state_init_plan(self.plan, _on(stream))
        self.opt_step = 0

    def step(self, t: int, opt: Optimizer, beta: float = 0.0, alpha: float = 1.0, T: int = 0,
             stream=None, method: str = "cpdp", flags: int = 0) -> str:
        """Step t on the gradients currently in self.grads (see
        CpdpState.step_opt)."""
        # the update counter advances only once the library has taken the step
        c = opt.c_struct(self.opt_step + 1)
        if method == "ddp" or cpdp.cpdp_is_sync_step(t, self.K, T):
            cpdp.cpdp_sync_step_plan(method, self.plan, self.K, c, beta, alpha, flags, _on(stream))
            kind = "reconcile"
        else:
            cpdp.cpdp_local_step_plan(self.plan, self.K, c, _on(stream))
            kind = "local"
        self.opt_step += 1
        return kind

    def step_table(self, t: int, table, T: int = 0, stream=None, method: str = "cpdp",
                   flags: int = 0) -> str:
        """Step t on self.grads with the scalars of the step table's current
        entry, then advance the table (see CpdpState.step_table)."""
        h = table.handle
        if method == "ddp" or cpdp.cpdp_is_sync_step(t, self.K, T):
            cpdp.cpdp_sync_step_plan_table(method, self.plan, self.K, h, flags, _on(stream))
            kind = "reconcile"
        else:
            cpdp.cpdp_local_step_plan_table(self.plan, self.K, h, _on(stream))
            kind = "local"
        cpdp.cpdp_step_table_advance(h, _on(stream))
        return kind

    def capture_steps(self, n_steps: int, table, T: int = 0, t0: int = 1,
                      method: str = "cpdp", flags: int = 0):
        """Capture steps t0 .. t0+n_steps-1 (cadence decided now) as table
        steps on self.grads into a HIP graph; every replay runs them with the
        table's next n_steps entries.  Returns (graph, kinds)."""
        graph = torch.cuda.CUDAGraph()
        kinds = []
        side = torch.cuda.Stream()
        side.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(side):
            torch.cuda.synchronize()
            with torch.cuda.graph(graph, stream=side):
                cs = torch.cuda.current_stream()
                for j in range(n_steps):
                    kinds.append(self.step_table(t0 + j, table, T, stream=cs, method=method,
                                                 flags=flags))
        torch.cuda.current_stream().wait_stream(side)
        return graph, kinds

    # ---- checkpoint / resume ---------------------------------------------------

    FAMILIES = ("params", "mom", "mom2", "grads", "slow_mom", "anchor")

    def state_dict(self) -> dict:
        """Host copy of every tensor of the state (and the optimizer step
        count), enough to resume bitwise.  Waits for all device work first."""
        torch.cuda.synchronize()
        d = {"W": self.W, "numels": list(self.numels), "K": self.K, "param_dt": self.param_dt,
             "opt_step": self.opt_step}
        for fam in self.FAMILIES:
            src = getattr(self, fam)
            if src is None:
                continue
            if fam in ("slow_mom", "anchor"):
                d[fam] = [x.cpu() for x in src]
            else:
                d[fam] = [[x.cpu() for x in row] for row in src]
        return d

    def load_state_dict(self, d: dict) -> None:
        """Copy a state_dict into this state's tensors in place (the plan keeps
        pointing at them).  Shapes, replica count and types must match."""
        if (d["W"], list(d["numels"]), d["param_dt"]) != (self.W, self.numels, self.param_dt):
            raise ValueError("state_dict is for a different model layout")
        if ("mom2" in d) != (self.mom2 is not None):
            raise ValueError("state_dict and state differ in AdamW second moments")
        pairs = []
        for fam in self.FAMILIES:
            dst = getattr(self, fam)
            if dst is None:
                continue
            rows = [dst] if fam in ("slow_mom", "anchor") else dst
            src = [d[fam]] if fam in ("slow_mom", "anchor") else d[fam]
            if len(src) != len(rows) or any(len(a) != len(b) for a, b in zip(rows, src)):
                raise ValueError(f"{fam}: state_dict has a different number of tensors")
            for i, (row_x, row_y) in enumerate(zip(rows, src)):
                for t, (x, y) in enumerate(zip(row_x, row_y)):
                    pairs.append((x, y, f"{fam}[{i}][{t}]"))
        # every tensor is checked before any is overwritten
        for x, y, name in pairs:
            check_exact(x, y, name)
        for x, y, name in pairs:
            load_exact(x, y, name)
        self.opt_step = int(d["opt_step"])
        torch.cuda.synchronize()

    def sgd(self, h: Hyper) -> Optimizer:
        return Optimizer("sgd", h.lr, h.mu)

    def gather(self, fam: str, i: int | None = None) -> torch.Tensor:
        """Concatenate replica i's tensors of a family (or a per-model family
        when i is None) into one flat tensor, in model order."""
        src = getattr(self, fam)
        parts = src if i is None else src[i]
        return torch.cat([p[:x] for p, x in zip(parts, self.numels)])
