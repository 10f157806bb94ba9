"""The execute calls under HIP graph capture.

Plan executions only launch kernels (their tables are written at bind, and
every buffer they clear is cleared by a kernel, not by a memset), so one
training step, sparsify then the aggregate + momentum update, can be
captured once and replayed. The step is captured on fixed buffers; between
replays the program copies the next gradient and the other workers' lists
into them eagerly and synchronizes. Every replay is compared bit for bit with
the same step run eagerly (the update in deterministic mode, so that both
runs sum in the same order). The per-tensor and MSTopK selections and the
LARS step are captured and replayed the same way.
"""
import numpy as np
import pytest

import gen
import paper_2010_10458_amd as tk
from gpu_common import announce, assert_bitwise, need_gpu, to_dev, to_host

pytestmark = pytest.mark.gpu

STEPS, OTHERS, K_OTHER = 4, 3, 25_600


class Step:
    """Buffers and plans of one sparsify + update step on fixed storage."""

    def __init__(self, sizes, dev):
        import torch
        d = sum(sizes)
        self.sizes, self.d = sizes, d
        self.grads = [torch.empty(n, device=dev) for n in sizes]
        self.res = to_dev([np.zeros(n, np.float32) for n in sizes], dev)
        self.w = to_dev(gen.params_like(sizes, config=5), dev)
        self.b = to_dev([np.zeros(n, np.float32) for n in sizes], dev)
        self.sp = tk.SparsifyPlan(sizes, rho=0.001).bind(self.grads, self.res)
        self.k = self.sp.k_total
        self.stride = max(self.k, K_OTHER)
        self.up = tk.UpdatePlan(sizes, P=1 + OTHERS, stride=self.stride,
                                deterministic=True).bind(self.w, self.b)
        n = (1 + OTHERS) * self.stride
        self.idx = torch.zeros(n, dtype=torch.int32, device=dev)
        self.val = torch.zeros(n, dtype=torch.float32, device=dev)
        self.nnz = torch.tensor([self.k] + [K_OTHER] * OTHERS, dtype=torch.int32, device=dev)

    def load_inputs(self, s):
        """Eager: this step's gradient and the other workers' lists."""
        import torch
        for t, a in zip(self.grads, gen.resnet_grads(step=s)):
            t.copy_(torch.from_numpy(a))
        li, lv = gen.sparse_lists(self.d, OTHERS, K_OTHER, step=2000 + s)
        for p in range(OTHERS):
            lo = (1 + p) * self.stride
            self.idx[lo:lo + K_OTHER].copy_(torch.from_numpy(li[p]))
            self.val[lo:lo + K_OTHER].copy_(torch.from_numpy(lv[p]))

    def run(self):
        """The step's GPU work: the calls that are captured."""
        self.sp.execute(idx_out=self.idx[:self.k], val_out=self.val[:self.k])
        self.up.execute(self.idx, self.val, lr=0.1, mu=0.9, wd=5e-5, nnz=self.nnz)

    def state(self):
        return (gen.concat(to_host(self.res)), gen.concat(to_host(self.w)),
                gen.concat(to_host(self.b)), self.idx[:self.k].cpu().numpy().copy(),
                self.val[:self.k].cpu().numpy().copy())


def test_captured_step_replays_match_eager_steps():
    import torch
    dev = need_gpu()
    sizes = gen.numels(gen.resnet50_shapes())
    announce("graph: eager reference steps")
    eager = Step(sizes, dev)
    ref = []
    for s in range(STEPS):
        eager.load_inputs(s)
        eager.run()
        torch.cuda.synchronize()
        ref.append(eager.state())
    del eager

    announce("graph: capture one step")
    g = Step(sizes, dev)
    graph = torch.cuda.CUDAGraph()
    torch.cuda.synchronize()
    with torch.cuda.graph(graph):
        g.run()
    torch.cuda.synchronize()
    # capture records the kernels without running them: the state is untouched
    assert not torch.cat(g.res).any().item()
    for s in range(STEPS):
        announce(f"graph: replay {s}")
        g.load_inputs(s)
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        for name, a, b in zip(("residual", "w", "b", "idx", "val"), g.state(), ref[s]):
            assert_bitwise(a, b, f"{name} after replay {s}")


@pytest.mark.parametrize("mode", ["per_tensor", "approx"])
def test_captured_sparsify_modes_replay(mode):
    """Per-tensor selection and MSTopK: each mode's execution (its own
    kernels and zeroed scratch) captured once and replayed on changing
    gradients, every replay bitwise equal to eager execution."""
    import torch
    dev = need_gpu()
    sizes = [300_007, 8192, 1, 77_777, 4096 * 3]
    tmode = {"per_tensor": tk.PER_TENSOR, "approx": tk.APPROX}[mode]

    def make():
        g = [torch.empty(n, device=dev) for n in sizes]
        r = [torch.zeros(n, device=dev) for n in sizes]
        plan = tk.SparsifyPlan(sizes, rho=0.01, mode=tmode).bind(g, r)
        idx = torch.empty(plan.k_total, dtype=torch.int32, device=dev)
        val = torch.empty(plan.k_total, dtype=torch.float32, device=dev)
        return g, r, plan, idx, val

    def load(g, s):
        for t, n in zip(g, sizes):
            t.copy_(torch.from_numpy(gen.flat_normal(n, config=7, step=s)))

    announce(f"graph {mode}: eager")
    g, r, plan, idx, val = make()
    ref = []
    for s in range(3):
        load(g, s)
        plan.execute(idx, val)
        torch.cuda.synchronize()
        ref.append((idx.cpu().numpy().copy(), val.cpu().numpy().copy(),
                    gen.concat(to_host(r))))
    announce(f"graph {mode}: capture and replay")
    g, r, plan, idx, val = make()
    graph = torch.cuda.CUDAGraph()
    torch.cuda.synchronize()
    with torch.cuda.graph(graph):
        plan.execute(idx, val)
    torch.cuda.synchronize()
    for s in range(3):
        load(g, s)
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        got = (idx.cpu().numpy(), val.cpu().numpy(), gen.concat(to_host(r)))
        for name, a, b in zip(("idx", "val", "residual"), got, ref[s]):
            assert_bitwise(a, b, f"{mode} {name} after replay {s}")


def test_captured_lars_step_replays():
    """The LARS step fused with the aggregate (segment table, norm pass,
    rates, step pass) captured once and replayed on changing lists, with
    momentum: every replay's parameters, momentum and rates bitwise equal to
    the same step run eagerly (deterministic sums; the rates' double sums
    run in a fixed order)."""
    import torch
    dev = need_gpu()
    sizes = [300_007, 8192, 1, 77_777, 4096 * 3]
    d, P, K = sum(sizes), 6, 20_000
    gamma, eta, eps, mu = 1e-3, 0.1, 5e-5, 0.9

    def make():
        w = to_dev(gen.params_like(sizes, config=11), dev)
        b = to_dev([np.zeros(n, np.float32) for n in sizes], dev)
        plan = tk.UpdatePlan(sizes, P=P, stride=K, deterministic=True).bind(w, b)
        idx = torch.zeros((P, K), dtype=torch.int32, device=dev)
        val = torch.zeros((P, K), dtype=torch.float32, device=dev)
        rates = torch.zeros(len(sizes), dtype=torch.float64, device=dev)
        return w, b, plan, idx, val, rates

    def load(idx, val, s):
        li, lv = gen.sparse_lists(d, P, K, config=11, step=s)
        idx.copy_(torch.from_numpy(li))
        val.copy_(torch.from_numpy(lv))

    def state(w, b, rates):
        return (gen.concat(to_host(w)), gen.concat(to_host(b)), rates.cpu().numpy().copy())

    announce("graph lars: eager")
    w, b, plan, idx, val, rates = make()
    ref = []
    for s in range(3):
        load(idx, val, s)
        plan.lars_execute(idx, val, gamma, eta, eps, mu=mu, rates=rates)
        torch.cuda.synchronize()
        ref.append(state(w, b, rates))
    announce("graph lars: capture and replay")
    w, b, plan, idx, val, rates = make()
    graph = torch.cuda.CUDAGraph()
    torch.cuda.synchronize()
    with torch.cuda.graph(graph):
        plan.lars_execute(idx, val, gamma, eta, eps, mu=mu, rates=rates)
    torch.cuda.synchronize()
    for s in range(3):
        load(idx, val, s)
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        for name, a, r in zip(("w", "b", "rates"), state(w, b, rates), ref[s]):
            assert_bitwise(a, r, f"lars {name} after replay {s}")
