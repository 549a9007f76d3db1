"""The allocation-free transform+quant entry point against the workspace
one: identical codes and scales on two calls in a row (the second with a
smaller input that leaves the first call's words in the shared scratch),
through the C ABI, on the single-pass and two-pass shapes, and captured
in a graph and replayed with new inputs."""
import numpy as np
import pytest

import paper_2603_04359_amd as cat
import workloads as wl
from oracle import cat_oracle as o
from paper_2603_04359_amd import binding as B

from gpu_common import check_codes, dev, host, say, torch_mod

pytestmark = pytest.mark.gpu


def _T(d, k, seed):
    rng = np.random.default_rng(seed)
    return o.round_storage(rng.standard_normal((d // k, k, k)) / np.sqrt(k), "bf16")


def _X(n, d, seed):
    rng = np.random.default_rng(seed)
    X = o.round_storage(rng.standard_normal((n, d)) * np.exp(rng.standard_normal(d)), "bf16")
    X[n // 2] = 0.0
    return X


def _pair(torch, X, T, k, bits):
    n, d = X.shape
    dX, dT = dev(X, "bf16"), dev(T, "bf16")
    shape = (n, d // 2) if bits == 4 else (n, d)
    ctype = torch.uint8 if bits == 4 else torch.int8
    c_ref = torch.empty(shape, dtype=ctype, device="cuda")
    s_ref = torch.empty(n, dtype=torch.float32, device="cuda")
    ws = torch.empty(cat.cat_transform_quant_workspace_bytes(n, d, k), dtype=torch.uint8,
                     device="cuda")
    cat.cat_transform_quant(dX, dT, k, c_ref, s_ref, ws, bits=bits)
    c_na = torch.full(shape, 0x55, dtype=ctype, device="cuda")
    s_na = torch.full((n,), -1.0, dtype=torch.float32, device="cuda")
    B.cat_transform_quant_noalloc(dX, dT, k, c_na, s_na, bits=bits)
    torch.cuda.synchronize()
    return host(c_ref), host(s_ref), host(c_na), host(s_na)


@pytest.mark.parametrize("d,n_first,n_second,bits", [(4096, 8192, 300, 4), (4096, 2049, 65, 8),
                                                     (2048, 3000, 17, 4)])
def test_noalloc_equals_workspace_entry_point_twice(d, n_first, n_second, bits):
    torch = torch_mod()
    k = 128
    assert cat.cat_transform_quant_workspace_bytes(n_first, d, k) <= \
        B.cat_transform_quant_noalloc_max_bytes()
    T = _T(d, k, seed=d)
    for i, n in enumerate((n_first, n_second)):
        say(f"noalloc d={d} n={n} bits={bits} (call {i + 1} of 2)")
        X = _X(n, d, seed=n + i)
        c_ref, s_ref, c_na, s_na = _pair(torch, X, T, k, bits)
        assert np.array_equal(c_na, c_ref), f"codes differ on call {i + 1}"
        assert np.array_equal(s_na, s_ref), f"scales differ on call {i + 1}"
        # and the workspace path itself is right, to the oracle's bar
        check_codes(c_na, X, T, bits, label=f"noalloc n={n}")


@pytest.mark.parametrize("d", [4096, 1024])
def test_noalloc_graph_replays_match_the_workspace_entry_point(d):
    # the callers this entry point is for capture it: a captured call
    # replayed with new activations, eager calls of both entry points in
    # between (the eager allocation-free ones share the captured call's
    # scratch), each replay bit for bit equal to the workspace entry point
    # (d = 4096: the single pass with its device-made tags; d = 1024: two
    # passes, whose words are cleared by a kernel, not a memset)
    say(f"noalloc graph capture d={d}: 3 replays with new X, eager calls between")
    torch = torch_mod()
    n, k = 300, 128
    T = _T(d, k, seed=d + 1)
    dT = dev(T, "bf16")
    Xs = [_X(n, d, seed=50 + i) for i in range(3)]
    dX = dev(Xs[0], "bf16")
    codes = torch.empty((n, d // 2), dtype=torch.uint8, device="cuda")
    s_x = torch.empty(n, dtype=torch.float32, device="cuda")
    B.cat_transform_quant_noalloc(dX, dT, k, codes, s_x)       # eager warm-up
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    side = torch.cuda.Stream()
    with torch.cuda.graph(g, stream=side):
        B.cat_transform_quant_noalloc(dX, dT, k, codes, s_x)
    c_e, s_e = torch.empty_like(codes), torch.empty_like(s_x)
    ws = torch.empty(cat.cat_transform_quant_workspace_bytes(n, d, k), dtype=torch.uint8,
                     device="cuda")
    for i, X in enumerate(Xs):
        dX.copy_(dev(X, "bf16"))
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        c, sx = host(codes), host(s_x)
        cat.cat_transform_quant(dX, dT, k, c_e, s_e, ws)
        torch.cuda.synchronize()
        assert np.array_equal(host(c_e), c) and np.array_equal(host(s_e), sx), f"replay {i}"
        B.cat_transform_quant_noalloc(dX, dT, k, c_e, s_e)   # eager, shared scratch
        torch.cuda.synchronize()
        assert np.array_equal(host(c_e), c) and np.array_equal(host(s_e), sx), f"eager {i}"


def test_noalloc_rejects_inputs_beyond_its_scratch():
    torch = torch_mod()
    n, d, k = 65536, 8192, 128
    assert cat.cat_transform_quant_workspace_bytes(n, d, k) > \
        B.cat_transform_quant_noalloc_max_bytes()
    X = torch.empty((n, d), dtype=torch.bfloat16, device="cuda")
    T = torch.empty((d // k, k, k), dtype=torch.bfloat16, device="cuda")
    codes = torch.empty((n, d // 2), dtype=torch.uint8, device="cuda")
    s_x = torch.empty(n, dtype=torch.float32, device="cuda")
    with pytest.raises(B.CatError) as e:
        B.cat_transform_quant_noalloc(X, T, k, codes, s_x)
    assert e.value.code == B.CAT_ERR_UNSUPPORTED
