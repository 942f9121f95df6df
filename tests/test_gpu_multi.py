"""Multi-tensor plans on the GPU: a model held as separate tensors per replica
gives bitwise the same results as the flat layout, and matches the oracle on
ragged tensor lists (empty and non-multiple-of-4 tensors included)."""
import numpy as np
import pytest
import torch

import oracle
from gpu_harness import Case, GpuRun, compare, log, state_from_grads
from paper_2607_21224_amd.multi import CpdpMultiState
from paper_2607_21224_amd.state import Optimizer
from synth import WORKLOADS, gen

pytestmark = pytest.mark.gpu


ADAMW_VIT = dict(kind="adamw", lr=5e-4, momentum=0.9, beta2=0.999, eps=1e-8, weight_decay=0.05)


@pytest.mark.parametrize("name,opt", [("r50_100", None), ("vit_s", None), ("r50_200", None),
                                      ("r50_100", ADAMW_VIT)],
                         ids=["r50_100", "vit_s", "r50_200", "r50_100-adamw"])
def test_plan_equals_flat_model_layouts(name, opt):
    """The model's tensors (ResNet-50: 161, ViT-S: 146) x W replicas, each its
    own allocation, against the flat buffer on the same seeded inputs over two
    periods: bitwise equal after every step (momentum SGD, and AdamW with its
    second moments, whose local steps take another block order)."""
    w = WORKLOADS[name]
    numels = [x for _, x in w.tensors]
    offs = np.cumsum([0] + numels)
    c = Case(W=w.W, P=w.P, K=w.K, lr=w.lr, mu=w.mu, beta=w.beta, alpha=w.alpha,
             steps=2 * w.K, ld=w.ld, outlier_rate=w.outlier_rate, opt=opt)
    log(f"[multi] {name} layout: {len(numels)} tensors, W={c.W}, "
        f"{opt['kind'] if opt else 'sgd'}")
    flat = GpuRun(c)
    multi = CpdpMultiState(c.W, numels, c.K, adamw=opt is not None)
    multi.init([flat.st.anchor[offs[t]:offs[t + 1]] for t in range(len(numels))])
    opt = flat.opt if opt is not None else Optimizer("sgd", flat.h.lr, flat.h.mu)
    for s in range(1, c.steps + 1):
        kind = flat.step(s)
        for i in range(c.W):
            for t in range(len(numels)):
                multi.grads[i][t][:numels[t]].copy_(flat.grads[i, offs[t]:offs[t + 1]])
        assert multi.step(s, opt, flat.h.beta, flat.h.alpha) == kind
        torch.cuda.synchronize()
        for i in range(c.W):
            assert torch.equal(multi.gather("params", i), flat.st.params[i, :c.P]), (s, i)
            assert torch.equal(multi.gather("mom", i), flat.st.mom[i, :c.P]), (s, i)
            if flat.st.mom2 is not None:
                assert torch.equal(multi.gather("mom2", i), flat.st.mom2[i, :c.P]), (s, i)
        assert torch.equal(multi.gather("slow_mom"), flat.st.slow_mom[:c.P]), s
        assert torch.equal(multi.gather("anchor"), flat.st.anchor[:c.P]), s


NUMELS = [1, 3, 5, 0, 1024, 1025, 4099, 7, 64, 2]

CASES = []
for method in ("cpdp", "localsgd", "ddp"):
    for kind in ("sgd", "adamw"):
        for dt in ("f32", "bf16"):
            CASES.append((method, kind, dt, 0))
    CASES.append((method, "adamw", "f32", 3))


@pytest.mark.parametrize("method,kind,dt,flags", CASES,
                         ids=[f"{m}-{k}-{d}-flags{f}" for m, k, d, f in CASES])
def test_plan_ragged_matches_oracle(method, kind, dt, flags):
    W, K, steps, seed = 5, 3, 9, 11
    P = sum(NUMELS)
    idx = np.arange(P)
    f32 = lambda x: float(np.float32(x))  # noqa: E731
    if kind == "sgd":
        opt = Optimizer("sgd", f32(0.1), f32(0.9), weight_decay=f32(5e-4))
        mk = lambda s: oracle.sgd(opt.lr, opt.momentum, opt.weight_decay)  # noqa: E731
    elif dt == "f32":
        opt = Optimizer("adamw", f32(1e-2), f32(0.9), f32(0.99), f32(1e-6), f32(0.01))
        mk = lambda s: oracle.adamw(opt.lr, opt.momentum, opt.beta2, opt.eps,  # noqa: E731
                                    opt.weight_decay, s)
    else:
        # bf16 parameters with the paper's AdamW (Table 3): at lr 1e-2 every step
        # moves a parameter by ~1e-2, the size of its own bf16 ulp, so rounding-
        # boundary flips between two correct fp32 paths would dominate the test
        opt = Optimizer("adamw", f32(5e-4), f32(0.9), f32(0.999), f32(1e-8), f32(0.05))
        mk = lambda s: oracle.adamw(opt.lr, opt.momentum, opt.beta2, opt.eps,  # noqa: E731
                                    opt.weight_decay, s)
    beta, alpha = f32(0.5), f32(1.0)
    th0 = gen.theta0(seed, idx)
    if dt == "bf16":
        th0 = gen.bf16_round(th0)
    grads = [gen.grads(seed, s, W, idx) for s in range(1, steps + 1)]
    refs = {}
    oracle.run_opt(th0.astype(np.float64), lambda s, W_, P_: grads[s - 1].astype(np.float64), W,
                   K, steps, mk, beta, alpha, method=method, param_dt=dt, flags=flags,
                   callback=lambda s, k, st, m2: refs.__setitem__(s, (k, st.copy(), m2.copy())))

    offs = np.cumsum([0] + NUMELS)
    multi = CpdpMultiState(W, NUMELS, K, param_dt=dt, adamw=kind == "adamw")
    multi.init([torch.from_numpy(th0[offs[t]:offs[t + 1]]).cuda() for t in range(len(NUMELS))])
    for s in range(1, steps + 1):
        for i in range(W):
            for t in range(len(NUMELS)):
                if NUMELS[t]:
                    multi.grads[i][t][:NUMELS[t]].copy_(
                        torch.from_numpy(grads[s - 1][i, offs[t]:offs[t + 1]]))
        k = multi.step(s, opt, beta, alpha, method=method, flags=flags)
        torch.cuda.synchronize()
        rk, ref, m2 = refs[s]
        assert k == rk
        snap = {"params": np.stack([multi.gather("params", i).float().cpu().numpy()
                                    for i in range(W)]).astype(np.float64),
                "mom": np.stack([multi.gather("mom", i).cpu().numpy()
                                 for i in range(W)]).astype(np.float64),
                "slow_mom": multi.gather("slow_mom").cpu().numpy().astype(np.float64),
                "anchor": multi.gather("anchor").cpu().numpy().astype(np.float64)}
        if kind == "adamw":
            snap["mom2"] = np.stack([multi.gather("mom2", i).cpu().numpy()
                                     for i in range(W)]).astype(np.float64)
        compare(snap, ref, dt, f"{method} {kind} step {s}", mom2=m2 if kind == "adamw" else None,
                scaled=True, velocity_lr=opt.lr if kind == "adamw" else None, lr=opt.lr,
                fp32_state=state_from_grads({"kind": opt.kind,
                                             "weight_decay": opt.weight_decay}))


@pytest.mark.parametrize("method,flags", [("cpdp", 0), ("cpdp", 3), ("localsgd", 0), ("ddp", 1)])
def test_plan_with_step_table(method, flags):
    """Plan steps driven by a step table (AdamW, warmup + cosine lr) are
    bitwise the plan steps with the scalars passed directly; a HIP graph of one
    period of table steps, replayed for successive periods, is bitwise the
    eager loop."""
    from paper_2607_21224_amd import cpdp
    from paper_2607_21224_amd.state import StepTable
    from synth import device as sdev
    W, K, periods = 5, 3, 3
    n = K * periods
    beta, alpha = 0.5, 0.75
    opts = [Optimizer("adamw", cpdp.cpdp_lr_at(s, n, K, 5e-4, 5e-5), 0.9, 0.999, 1e-8, 0.05)
            for s in range(n)]
    log(f"[plan-table] {method} flags={flags} W={W} K={K} periods={periods}")
    states = [CpdpMultiState(W, NUMELS, K, adamw=True) for _ in range(3)]
    offs = np.cumsum([0] + NUMELS)
    th = torch.from_numpy(gen.theta0(13, np.arange(sum(NUMELS)))).cuda()
    for st in states:
        st.init([th[offs[t]:offs[t + 1]] for t in range(len(NUMELS))])
    direct, tabled, graphed = states
    t_eager = StepTable([(opts[s], s + 1, beta, alpha) for s in range(n)])
    t_graph = StepTable([(opts[s], s + 1, beta, alpha) for s in range(n)])
    graph, kinds = graphed.capture_steps(K, t_graph, method=method, flags=flags)
    g = torch.empty((W, max(sum(NUMELS), 1)), device="cuda")

    def load_grads(st):
        for i in range(W):
            for t in range(len(NUMELS)):
                if NUMELS[t]:
                    st.grads[i][t][:NUMELS[t]].copy_(g[i, offs[t]:offs[t + 1]])

    def same(a, b, tag):
        for fam in ("params", "mom", "mom2"):
            for i in range(W):
                x, y = a.gather(fam, i), b.gather(fam, i)
                assert torch.equal(x.view(torch.int32), y.view(torch.int32)), (tag, fam, i)
        for fam in ("slow_mom", "anchor"):
            assert torch.equal(a.gather(fam).view(torch.int32), b.gather(fam).view(torch.int32)), \
                (tag, fam)

    for r in range(periods):
        # one gradient set per period: the graph reads the same buffers at every step
        sdev.fill_grads(g, sum(NUMELS), 13, r + 1, 1e-3, 0.0)
        for st in states:
            load_grads(st)
        graph.replay()
        for j in range(K):
            s = r * K + j + 1
            ka = direct.step(s, opts[s - 1], beta, alpha, 0, method=method, flags=flags)
            kb = tabled.step_table(s, t_eager, method=method, flags=flags)
            assert ka == kb == kinds[j]
            torch.cuda.synchronize()
            same(direct, tabled, f"step {s}")
        # every state steps on its own copy of the period's gradients, which the
        # write-back variant overwrites with their mean at each sync, identically
        same(direct, graphed, f"period {r + 1}")
    assert t_eager.position() == n and t_graph.position() == n


def test_plan_checkpoint_resume_bitwise():
    """Two periods, save, load into a fresh state, two more periods: bitwise
    the four periods run straight (AdamW, so the step count is resumed too)."""
    W, K = 4, 3
    opt = Optimizer("adamw", 5e-4, 0.9, 0.999, 1e-8, 0.05)
    offs = np.cumsum([0] + NUMELS)
    th = torch.from_numpy(gen.theta0(21, np.arange(sum(NUMELS)))).cuda()
    a = CpdpMultiState(W, NUMELS, K, adamw=True)
    b = CpdpMultiState(W, NUMELS, K, adamw=True)
    for st in (a, b):
        st.init([th[offs[t]:offs[t + 1]] for t in range(len(NUMELS))])

    def run(st, steps):
        for s in steps:
            g = torch.from_numpy(gen.grads(21, s, W, np.arange(sum(NUMELS)))).cuda()
            for i in range(W):
                for t in range(len(NUMELS)):
                    if NUMELS[t]:
                        st.grads[i][t][:NUMELS[t]].copy_(g[i, offs[t]:offs[t + 1]])
            st.step(s, opt, 0.5, 1.0)
        torch.cuda.synchronize()

    run(a, range(1, 2 * K + 1))
    saved = a.state_dict()
    c = CpdpMultiState(W, NUMELS, K, adamw=True)
    c.load_state_dict(saved)
    run(c, range(2 * K + 1, 4 * K + 1))
    run(b, range(1, 4 * K + 1))
    for fam in ("params", "mom", "mom2"):
        for i in range(W):
            assert torch.equal(b.gather(fam, i).view(torch.int32), c.gather(fam, i).view(torch.int32)), (fam, i)
    for fam in ("slow_mom", "anchor"):
        assert torch.equal(b.gather(fam).view(torch.int32), c.gather(fam).view(torch.int32)), fam
    assert c.opt_step == b.opt_step == 4 * K

    # a checkpoint with one tensor of the wrong size is rejected before any
    # tensor of the state is overwritten
    bad = dict(saved, mom2=[list(row) for row in saved["mom2"]])
    bad["mom2"][1][2] = torch.zeros(bad["mom2"][1][2].numel() + 1)
    before = c.gather("params", 0).clone()
    with pytest.raises(ValueError, match=r"mom2\[1\]\[2\]"):
        c.load_state_dict(bad)
    assert torch.equal(c.gather("params", 0), before)


def test_bf16_plan_init_rounds_the_reference_model():
    """Initial values given wider than bf16 are taken rounded to the parameter
    type: the reference model starts bitwise equal to every replica (as the
    flat layout's initialisation from bf16 values does), and equal to the
    host's round-to-nearest-even of the inputs."""
    W = 3
    offs = np.cumsum([0] + NUMELS)
    th = gen.theta0(5, np.arange(sum(NUMELS)))
    st = CpdpMultiState(W, NUMELS, 2, param_dt="bf16")
    st.init([torch.from_numpy(th[offs[t]:offs[t + 1]]).cuda() for t in range(len(NUMELS))])
    torch.cuda.synchronize()
    anchor = st.gather("anchor")
    want = torch.from_numpy(gen.bf16_round(th)).cuda()
    assert torch.equal(anchor.view(torch.int32), want.view(torch.int32))
    for i in range(W):
        assert torch.equal(st.gather("params", i).float().view(torch.int32),
                           anchor.view(torch.int32)), i
