"""Checkpoint and resume: the library keeps no state between calls (the
residuals, parameters and momentum buffers are the caller's), so a run that
stops after a step, copies those buffers to the host and starts again from
the copies in fresh buffers and fresh plans continues exactly as the
uninterrupted run does. Ten steps of the ResNet-50-shaped workload
(sparsify with error feedback at rho = 0.001, then the momentum update
with the local list and three other workers' lists, summed in worker order
so that both runs are bitwise comparable), split after step 5.
"""
import numpy as np
import pytest

import gen
import paper_2010_10458_amd as tk
from gpu_common import announce, assert_bitwise, need_gpu, to_dev, to_host

pytestmark = pytest.mark.gpu

STEPS, SPLIT, OTHERS, K_OTHER = 10, 5, 3, 25_600


def _run(sizes, state, steps, dev):
    """state: host arrays (residuals, params, momentum); runs `steps` (a
    range of step numbers) in fresh buffers and returns the final state and
    every step's (idx, val)."""
    import torch
    d = sum(sizes)
    res, w, b = (to_dev(a, dev) for a in state)
    grads = [torch.empty(n, device=dev) for n in sizes]
    sp = tk.SparsifyPlan(sizes, rho=0.001).bind(grads, res)
    k = sp.k_total
    stride = max(k, K_OTHER)
    up = tk.UpdatePlan(sizes, P=1 + OTHERS, stride=stride, deterministic=True).bind(w, b)
    idx_all = torch.zeros((1 + OTHERS) * stride, dtype=torch.int32, device=dev)
    val_all = torch.zeros((1 + OTHERS) * stride, dtype=torch.float32, device=dev)
    nnz = torch.tensor([k] + [K_OTHER] * OTHERS, dtype=torch.int32, device=dev)
    outs = []
    for s in steps:
        for t, a in zip(grads, gen.resnet_grads(step=s)):
            t.copy_(torch.from_numpy(a))
        sp.execute(idx_out=idx_all[:k], val_out=val_all[:k])
        li, lv = gen.sparse_lists(d, OTHERS, K_OTHER, step=1000 + s)
        for p in range(OTHERS):
            lo = (1 + p) * stride
            idx_all[lo:lo + K_OTHER].copy_(torch.from_numpy(li[p]))
            val_all[lo:lo + K_OTHER].copy_(torch.from_numpy(lv[p]))
        up.execute(idx_all, val_all, lr=0.1, mu=0.9, wd=5e-5, nnz=nnz)
        torch.cuda.synchronize()
        outs.append((idx_all[:k].cpu().numpy().copy(), val_all[:k].cpu().numpy().copy()))
    return (to_host(res), to_host(w), to_host(b)), outs


def test_resume_after_host_copy_is_bitwise_identical():
    dev = need_gpu()
    sizes = gen.numels(gen.resnet50_shapes())
    start = ([np.zeros(n, np.float32) for n in sizes], gen.params_like(sizes, config=5),
             [np.zeros(n, np.float32) for n in sizes])
    announce(f"resume: {STEPS} steps uninterrupted")
    full_state, full_out = _run(sizes, start, range(STEPS), dev)
    announce(f"resume: {SPLIT} steps, host copy, {STEPS - SPLIT} more")
    mid_state, first_out = _run(sizes, start, range(SPLIT), dev)
    mid_state = tuple([a.copy() for a in arrs] for arrs in mid_state)   # the checkpoint
    end_state, second_out = _run(sizes, mid_state, range(SPLIT, STEPS), dev)
    for s, ((i1, v1), (i2, v2)) in enumerate(zip(full_out, first_out + second_out)):
        assert_bitwise(i2, i1, f"idx step {s}")
        assert_bitwise(v2, v1, f"val step {s}")
    for name, a, b in zip(("residual", "w", "b"), end_state, full_state):
        assert_bitwise(gen.concat(a), gen.concat(b), name)
