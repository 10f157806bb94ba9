"""The C ABI library on the CPU: it loads, exports every function that
include/tkef.h declares, and validates arguments on the host before any GPU
work (no call here reaches the GPU)."""
import ctypes
import os
import re

import pytest

import paper_2010_10458_amd as tk

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "tkef.h")


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(tkef_[a-z0-9_]+)\s*\(", text)))


def test_header_symbols_exported():
    names = declared_functions()
    assert len(names) >= 20
    L = tk.lib()
    for n in names:
        assert hasattr(L, n), f"{n} declared in tkef.h but not exported"


def test_version_and_strerror():
    L = tk.lib()
    assert L.tkef_version() == 10200
    for code in (0, -1, -2, -3, -4, -5, -6):
        assert L.tkef_strerror(code)
    assert b"unknown" in L.tkef_strerror(-99)


@pytest.mark.parametrize("d,rho,k", [(1_048_576, 0.001, 1049), (25_557_032, 0.001, 25_558),
                                     (109_708_544, 0.01, 1_097_086), (340_000_000, 0.001, 340_000),
                                     (0, 0.5, 0), (5, 1.0, 5), (3, 1e-9, 1)])
def test_k_from_rho(d, rho, k):
    assert tk.k_from_rho(d, rho) == k


@pytest.mark.parametrize("rho", [0.0, -0.1, 1.0000001, float("nan"), float("inf")])
def test_k_from_rho_rejects(rho):
    assert tk.k_from_rho(10, rho) == tk.ERANGE


def _create(numels, mode=tk.GLOBAL, rho=0.01, k=0, n=None):
    L = tk.lib()
    h = ctypes.c_void_p()
    arr = (ctypes.c_int64 * max(1, len(numels)))(*numels) if numels is not None else None
    rc = L.tkef_sparsify_plan_create(arr, len(numels) if n is None else n, mode, rho, k,
                                     ctypes.byref(h))
    if rc == 0:
        L.tkef_sparsify_plan_destroy(h)
    return rc


def test_sparsify_plan_validation():
    assert _create([10, 20]) == tk.OK
    assert _create(None, n=2) == tk.EINVAL
    assert _create([10], n=0) == tk.EINVAL
    assert _create([10, -1]) == tk.EINVAL
    assert _create([0, 0]) == tk.ERANGE
    assert _create([2**31 - 1]) == tk.OK
    assert _create([2**31]) == tk.ERANGE
    assert _create([2**30, 2**30]) == tk.ERANGE
    assert _create([10], mode=7) == tk.EINVAL
    assert _create([10], rho=0.0) == tk.ERANGE
    assert _create([10], rho=2.0) == tk.ERANGE
    assert _create([10], k=11, rho=0.0) == tk.ERANGE
    assert _create([10], k=10, rho=0.0) == tk.OK
    assert _create([10], k=-1) == tk.ERANGE
    # at most 2^18 tiles of 8,192 elements in a list, whatever the mode
    mixed = [4096] * 2**17 + [1] * 2**17  # exactly 2^18 tiles
    for mode in (tk.GLOBAL, tk.APPROX):
        assert _create(mixed, mode=mode) == tk.OK
    for mode in (tk.GLOBAL, tk.PER_TENSOR, tk.APPROX):
        assert _create(mixed + [1], mode=mode) == tk.ERANGE
    assert _create([2**31 - 8192, 8191], mode=tk.PER_TENSOR) == tk.OK
    assert _create([10, 5], mode=tk.PER_TENSOR, k=3) == tk.EINVAL
    L = tk.lib()
    assert L.tkef_sparsify_plan_create(None, 1, 0, 0.1, 0, None) == tk.EINVAL


def test_sparsify_plan_sizes():
    p = tk.SparsifyPlan([100, 8192 * 3 + 1, 0, 7], rho=0.01)
    assert p.k_total == tk.k_from_rho(100 + 8192 * 3 + 1 + 7, 0.01) and p.ngroups == 1
    assert p.ws_bytes % 256 == 0 and p.ws_bytes > 0
    q = tk.SparsifyPlan([100, 8192 * 3 + 1, 0, 7], mode=tk.PER_TENSOR, rho=0.01)
    assert q.group_k() == [1, 246, 0, 1] and q.k_total == 248


def test_bind_and_execute_validation_without_gpu():
    L = tk.lib()
    p = tk.SparsifyPlan([1000], rho=0.01)
    h = p._h
    P = ctypes.c_void_p
    ptrs = (P * 1)(P(0x1000))
    rptrs = (P * 1)(P(0x100000))
    # workspace missing / misaligned / too small
    assert L.tkef_sparsify_plan_bind(h, ptrs, rptrs, None, 10**9, None) == tk.EWORKSPACE
    assert L.tkef_sparsify_plan_bind(h, ptrs, rptrs, P(0x10010), 10**9, None) == tk.EWORKSPACE
    assert L.tkef_sparsify_plan_bind(h, ptrs, rptrs, P(0x10000), 1, None) == tk.EWORKSPACE
    # null tensor pointers, overlapping g and r
    nul = (P * 1)(None)
    assert L.tkef_sparsify_plan_bind(h, nul, rptrs, P(0x10000), 10**9, None) == tk.EINVAL
    same = (P * 1)(P(0x1000 + 64))
    assert L.tkef_sparsify_plan_bind(h, ptrs, same, P(0x10000), 10**9, None) == tk.EINVAL
    assert L.tkef_sparsify_plan_bind(None, ptrs, rptrs, P(0x10000), 10**9, None) == tk.EINVAL
    # execute before bind
    assert L.tkef_sparsify_execute(h, P(0x10000), 10**9, P(0x2000), P(0x3000), None,
                                   None) == tk.ESTATE
    assert L.tkef_sparsify_execute(h, None, 10**9, P(0x2000), P(0x3000), None,
                                   None) == tk.EWORKSPACE
    assert L.tkef_sparsify_plan_set_events(h, None, 0) == tk.OK
    assert L.tkef_sparsify_plan_set_events(h, None, -1) == tk.EINVAL
    assert L.tkef_sparsify_plan_launch_name(h, 99) is None


def test_update_plan_validation():
    L = tk.lib()

    def create(numels, P, stride):
        h = ctypes.c_void_p()
        arr = (ctypes.c_int64 * len(numels))(*numels)
        rc = L.tkef_update_plan_create(arr, len(numels), P, stride, ctypes.byref(h))
        if rc == 0:
            L.tkef_update_plan_destroy(h)
        return rc

    assert create([10, 20], 1, 5) == tk.OK
    assert create([10, 20], 0, 5) == tk.EINVAL
    assert create([10, 20], 65536, 5) == tk.EINVAL
    assert create([10, 20], 4, -1) == tk.ERANGE
    assert create([10, 20], 4, 2**31) == tk.ERANGE
    assert create([0], 4, 5) == tk.ERANGE
    u = tk.UpdatePlan([10, 20], P=3, stride=4)
    P = ctypes.c_void_p
    w = (P * 2)(P(0x1000), P(0x2000))
    b = (P * 2)(P(0x1000 + 8), P(0x3000))
    assert L.tkef_update_plan_bind(u._h, w, b, P(0x10000), 10**9, None) == tk.EINVAL
    assert L.tkef_update_plan_bind(u._h, None, None, P(0x10000), 10**9, None) == tk.EINVAL
    assert L.tkef_update_plan_bind(u._h, w, None, P(0x10001), 10**9, None) == tk.EWORKSPACE
    assert L.tkef_update_execute(u._h, P(0x10), P(0x20), None, 0.1, 0.0, 0.0, P(0x10000),
                                 10**9, None, None) == tk.ESTATE
    assert L.tkef_update_plan_set_deterministic(u._h, 1) == tk.OK
    assert L.tkef_update_plan_set_deterministic(u._h, 0) == tk.OK
    assert L.tkef_update_plan_set_deterministic(u._h, 2) == tk.EINVAL
    assert L.tkef_update_plan_set_deterministic(None, 1) == tk.EINVAL
    assert tk.UpdatePlan([10, 20], P=3, stride=4, deterministic=True).deterministic


def test_no_cpu_fallback_when_library_missing(tmp_path, monkeypatch):
    """The binding raises instead of computing anything itself."""
    monkeypatch.setattr(tk, "_lib", None)
    monkeypatch.setattr(tk, "LIB_PATH", str(tmp_path / "missing.so"))
    with pytest.raises(RuntimeError):
        tk.lib()


def test_per_tensor_launch_names():
    """Per tensor: up to 1,024 groups the emit kernel forms the group bases
    itself (seven kernels); beyond that a scan kernel does (eight)."""
    p = tk.SparsifyPlan([10] * 5 + [40_000], mode=tk.PER_TENSOR, rho=0.1)
    assert p.nlaunch == 7
    assert p.launch_names() == ["stream", "pick1", "gather", "pick2", "hist3", "pick3", "emit"]
    q = tk.SparsifyPlan([3] * 1100, mode=tk.PER_TENSOR, rho=0.5)
    assert q.nlaunch == 8 and q.launch_names()[6:] == ["groupscan", "emit"]
    g = tk.SparsifyPlan([3] * 1100, mode=tk.GLOBAL, rho=0.5)
    assert g.launch_names() == ["stream", "collect", "finish"]


def test_approx_plan_host_side():
    """MSTopK plans: parameters, kernel count and names, and the errors the
    host can see (no GPU needed)."""
    L = tk.lib()
    assert _create([10, 20], mode=tk.APPROX) == tk.OK
    assert _create([10], mode=tk.APPROX, k=10, rho=0.0) == tk.OK
    assert _create([10], mode=tk.APPROX, k=11, rho=0.0) == tk.ERANGE
    p = tk.SparsifyPlan([1000, 8192 * 3 + 5], mode=tk.APPROX, rho=0.001)
    assert p.ngroups == 1 and p.k_total == tk.k_from_rho(1000 + 8192 * 3 + 5, 0.001)
    assert p.nlaunch == 3 + 2  # 30 rounds: 6 in the first pass, 12 in each later one
    names = p.launch_names()
    assert names[0] == "ms_stream" and names[1] == "ms_count" and names[-1] == "ms_emit"
    assert names[2:-1] == ["ms_refine1", "ms_refine2"]
    for n, launches in ((1, 3), (6, 3), (7, 4), (18, 4), (19, 5), (30, 5), (31, 6), (48, 7)):
        q = tk.SparsifyPlan([5000], mode=tk.APPROX, k=7, n_search=n)
        assert q.nlaunch == launches, n
    h = p._h
    assert L.tkef_sparsify_plan_set_approx(h, 0, 0) == tk.EINVAL
    assert L.tkef_sparsify_plan_set_approx(h, 49, 0) == tk.EINVAL
    assert L.tkef_sparsify_plan_set_approx(h, 30, 2**64 - 1) == tk.OK
    assert L.tkef_sparsify_plan_set_approx(None, 30, 0) == tk.EINVAL
    g = tk.SparsifyPlan([1000], rho=0.01)
    assert L.tkef_sparsify_plan_set_approx(g._h, 30, 0) == tk.EINVAL
    P = ctypes.c_void_p
    assert L.tkef_sparsify_approx_result(g._h, P(0x10000), None, None, None) == tk.EINVAL
    assert L.tkef_sparsify_approx_result(h, P(0x10000), None, None, None) == tk.ESTATE


def test_lars_host_side():
    """LARS entry points: the errors the host can see (no GPU needed)."""
    L = tk.lib()
    p = tk.UpdatePlan([100, 5000], P=2, stride=10)
    h = p._h
    P_ = ctypes.c_void_p
    ws = P_(0x10000)
    assert L.tkef_lars_update_execute(None, None, None, None, 1.0, 1.0, 0.0, 0.0, None, ws,
                                      10**9, None, None) == tk.EINVAL
    assert L.tkef_lars_update_execute(h, P_(0x100), P_(0x200), None, float("nan"), 1.0, 0.0,
                                      0.0, None, ws, 10**9, None, None) == tk.ERANGE
    assert L.tkef_lars_update_execute(h, P_(0x100), P_(0x200), None, 1.0, 1.0, 0.0, 0.0, None,
                                      ws, 10**9, None, None) == tk.ESTATE
    assert L.tkef_lars_update_execute(h, P_(0x100), P_(0x200), None, 1.0, 1.0, 0.0, 0.0, None,
                                      None, 10**9, None, None) == tk.EWORKSPACE
    g = (P_ * 2)(P_(0x1000), P_(0x2000))
    assert L.tkef_update_plan_bind_grads(h, g, ws, 10**9, None) == tk.ESTATE
    assert L.tkef_update_plan_bind_grads(h, None, ws, 10**9, None) == tk.EINVAL
    assert L.tkef_lars_rates_execute(h, 1.0, 1.0, 0.0, P_(0x3000), ws, 10**9, None) == tk.ESTATE
    assert L.tkef_lars_rates_execute(h, 1.0, float("inf"), 0.0, P_(0x3000), ws, 10**9,
                                     None) == tk.ERANGE
    # eps is a weight decay: negative values are refused (Eq. lars needs a
    # denominator that vanishes only with the gradient)
    assert L.tkef_lars_rates_execute(h, 1.0, 1.0, -1e-4, P_(0x3000), ws, 10**9,
                                     None) == tk.ERANGE
    assert L.tkef_lars_update_execute(h, P_(0x100), P_(0x200), None, 1.0, 1.0, -0.5, 0.0, None,
                                      ws, 10**9, None, None) == tk.ERANGE
    names = [L.tkef_lars_launch_name(0, i).decode() for i in range(4)]
    assert names == tk.LARS_LAUNCHES and L.tkef_lars_launch_name(0, 4) is None
    assert [L.tkef_lars_launch_name(1, i).decode() for i in range(2)] == tk.LARS_DENSE_LAUNCHES


def test_one_shot_sparsify_host_side():
    """tkef_sparsify writes counts_out (the k of each selection group) before
    any GPU work; tkef_sparsify1 checks d and k; both refuse a missing
    workspace without touching the GPU."""
    L = tk.lib()
    P_ = ctypes.c_void_p
    numels = [100, 8192 * 3 + 1, 0, 7]
    arr = (ctypes.c_int64 * 4)(*numels)
    g = (P_ * 4)(P_(0x1000), P_(0x100000), None, P_(0x300000))
    r = (P_ * 4)(P_(0x400000), P_(0x500000), None, P_(0x600000))
    counts = (ctypes.c_int64 * 4)(-1, -1, -1, -1)
    assert L.tkef_sparsify(g, r, arr, 4, tk.PER_TENSOR, 0.01, 0, tk.VAL_F32, P_(0x10), P_(0x20),
                           counts, None, 10**9, None, None) == tk.EWORKSPACE
    assert list(counts) == [1, 246, 0, 1]
    counts[0] = -1
    assert L.tkef_sparsify(g, r, arr, 4, tk.GLOBAL, 0.01, 0, tk.VAL_F16, P_(0x10), P_(0x20),
                           counts, None, 10**9, None, None) == tk.EWORKSPACE
    assert counts[0] == tk.k_from_rho(sum(numels), 0.01)
    assert L.tkef_sparsify(g, r, arr, 4, tk.GLOBAL, 0.01, 0, 7, P_(0x10), P_(0x20),
                           None, None, 10**9, None, None) == tk.EINVAL
    nb, kt = ctypes.c_size_t(), ctypes.c_int64()
    assert L.tkef_sparsify_workspace(arr, 4, tk.GLOBAL, 0.0, 5, ctypes.byref(nb),
                                     ctypes.byref(kt)) == tk.OK
    assert kt.value == 5 and nb.value % 256 == 0
    for d, k in ((0, 1), (10, 0), (10, 11), (2**31, 1), (-5, 1)):
        assert L.tkef_sparsify1(P_(0x1000), P_(0x100000), d, k, P_(0x10), P_(0x20), P_(0x10000),
                                10**9, None, None) == tk.ERANGE, (d, k)
    assert L.tkef_sparsify1(P_(0x1000), P_(0x100000), 10, 3, P_(0x10), P_(0x20), None, 10**9,
                            None, None) == tk.EWORKSPACE
    # g and r overlap
    assert L.tkef_sparsify1(P_(0x1000), P_(0x1000 + 8), 10, 3, P_(0x10), P_(0x20),
                            P_(0x10000), 10**9, None, None) == tk.EINVAL


def test_aggregate_update_host_side():
    """tkef_aggregate_update / tkef_aggregate_workspace: argument checks on
    the host, before any GPU work."""
    L = tk.lib()
    P_ = ctypes.c_void_p
    numels = (ctypes.c_int64 * 2)(100, 5000)
    nb, nb_g = ctypes.c_size_t(), ctypes.c_size_t()
    assert L.tkef_aggregate_workspace(numels, 2, 300, ctypes.byref(nb)) == tk.OK
    assert L.tkef_update_workspace(numels, 2, 300, 0, ctypes.byref(nb_g)) == tk.OK
    assert nb.value >= nb_g.value + 300 * 32 and nb.value % 256 == 0
    assert L.tkef_aggregate_workspace(numels, 2, 0, ctypes.byref(nb)) == tk.EINVAL
    w = (P_ * 2)(P_(0x1000), P_(0x2000))
    b = (P_ * 2)(P_(0x100000), P_(0x200000))
    ip = (P_ * 3)(P_(0x300000), None, P_(0x310000))
    vp = (P_ * 3)(P_(0x400000), None, P_(0x410000))
    nnz = (ctypes.c_int64 * 3)(10, 0, 5)
    ws = P_(0x10000)

    def call(params=w, mom=None, i=ip, v=vp, n=nnz, P=3, lr=0.1, mu=0.0, wd=0.0, ws=ws,
             wsb=10**9):
        return L.tkef_aggregate_update(params, mom, numels, 2, i, v, n, P, lr, mu, wd, ws, wsb,
                                       None, None)

    assert call(i=None) == tk.EINVAL
    assert call(v=None) == tk.EINVAL
    assert call(n=None) == tk.EINVAL
    assert call(P=0) == tk.EINVAL
    assert call(lr=float("nan")) == tk.ERANGE
    assert call(mu=0.9) == tk.EINVAL                     # momentum buffers needed
    bad_n = (ctypes.c_int64 * 3)(10, -1, 5)
    assert call(n=bad_n) == tk.EINVAL
    big_n = (ctypes.c_int64 * 3)(10, 2**31, 5)
    assert call(n=big_n) == tk.ERANGE
    null_list = (ctypes.c_int64 * 3)(10, 4, 5)            # list 1 has entries, no pointers
    assert call(n=null_list) == tk.EINVAL
    assert call(ws=None) == tk.EWORKSPACE
    assert call(ws=P_(0x10010)) == tk.EWORKSPACE
    assert call(wsb=16) == tk.EWORKSPACE
    assert call(params=(P_ * 2)(None, P_(0x2000))) == tk.EINVAL
    overlap = (P_ * 2)(P_(0x1000 + 4), P_(0x200000))
    assert call(mom=overlap, mu=0.9) == tk.EINVAL


def test_static_entry_point_host_side():
    """tkef_sparsify1_static (no workspace): its limits are refused on the
    host, and every single-tensor layout within them (each tile count up to
    2^26 elements, with the largest k allowed) fits the fixed scratch."""
    L = tk.lib()
    P_ = ctypes.c_void_p
    g, r, i, v = P_(0x1000), P_(0x40000000), P_(0x10), P_(0x20)
    for d, k in ((0, 1), (10, 0), (10, 11), (tk.STATIC_MAX_D + 1, 5),
                 (tk.STATIC_MAX_D, tk.STATIC_MAX_K + 1), (2**31, 1)):
        assert L.tkef_sparsify1_static(g, r, d, k, i, v, None, None) == tk.ERANGE, (d, k)
    assert L.tkef_sparsify1_static(None, r, 10, 1, i, v, None, None) == tk.EINVAL
    assert L.tkef_sparsify1_static(g, r, 10, 1, None, v, None, None) == tk.EINVAL
    assert L.tkef_sparsify1_static(g, P_(0x1000 + 4), 10, 1, i, v, None, None) == tk.EINVAL
    limit = 36 << 20
    worst = 0
    nb = ctypes.c_size_t()
    for ntiles in range(1, tk.STATIC_MAX_D // 8192 + 1):
        d = ntiles * 8192
        k = min(tk.STATIC_MAX_K, d)
        assert L.tkef_sparsify_workspace((ctypes.c_int64 * 1)(d), 1, tk.GLOBAL, 0.0, k,
                                         ctypes.byref(nb), None) == tk.OK
        worst = max(worst, nb.value)
    assert worst <= limit, worst


def test_header_is_plain_c(tmp_path):
    """include/tkef.h is a C header: a C11 program includes it, links the
    library and calls it (version and error strings; nothing reaches a GPU)."""
    import shutil
    import subprocess
    if shutil.which("gcc") is None:
        pytest.skip("gcc not available")
    src = tmp_path / "use.c"
    src.write_text(
        '#include <string.h>\n#include "tkef.h"\n'
        "int main(void) {\n"
        "  if (tkef_version() != TKEF_VERSION) return 1;\n"
        "  if (strlen(tkef_strerror(TKEF_EWORKSPACE)) == 0) return 2;\n"
        "  if (tkef_k_from_rho(1000, 0.01) != 10) return 3;\n"
        "  return 0;\n}\n")
    libdir = os.path.dirname(tk.LIB_PATH if os.path.isabs(tk.LIB_PATH)
                             else os.path.join(ROOT, tk.LIB_PATH))
    exe = tmp_path / "use"
    subprocess.run(["gcc", "-std=c11", "-Wall", "-Werror", "-D__HIP_PLATFORM_AMD__",
                    "-I/opt/rocm/include", "-I" + os.path.join(ROOT, "include"), str(src),
                    "-L" + libdir, "-ltkef", "-Wl,-rpath," + libdir, "-o", str(exe)],
                   check=True, capture_output=True, timeout=120)
    assert subprocess.run([str(exe)], timeout=120).returncode == 0
