"""Different entry points running at the same time on two streams give
their one-stream results bit for bit: the kernels keep no state outside
the buffers and workspaces the caller passes.  Stream 1 accumulates Sigma_x
and reduces an SQNR; stream 2 runs the single-pass transform+quant and the
W4A4 GEMM (one single-pass call at a time, as the ABI requires)."""
import numpy as np
import pytest

import paper_2603_04359_amd as cat
from oracle import cat_oracle as o
from paper_2603_04359_amd import binding as B
import workloads as wl

from gpu_common import dev, host, say, torch_mod

pytestmark = pytest.mark.gpu


def test_two_streams_match_one_stream():
    say("two streams: cov + sqnr against transform_quant + w4a4_linear")
    torch = torch_mod()
    rng = np.random.default_rng(61)
    n, d, k, d_out = 4096, 4096, 128, 2048
    X = dev(o.round_storage(rng.standard_normal((n, d)) * np.exp(rng.standard_normal(d)), "bf16"),
            "bf16")
    T = dev(o.round_storage(rng.standard_normal((d // k, k, k)) / np.sqrt(k), "bf16"), "bf16")
    qw = dev(o.pack_int4(wl.random_codes(d_out, d, 62)), "u8")
    sw = dev(rng.uniform(0.01, 1.0, d_out).astype(np.float32), "f32")
    y, yt = wl.random_pair(3_000_000, seed=63)
    dy, dyt = dev(y, "f32"), dev(yt, "f32")

    ws_c = torch.empty(max(16, cat.cat_cov_workspace_bytes(B.CAT_BF16, n, d, B.CAT_COV_FULL, k)),
                       dtype=torch.uint8, device="cuda")
    ws_s = torch.empty(cat.cat_sqnr_workspace_bytes(y.size), dtype=torch.uint8, device="cuda")
    ws_q = torch.empty(cat.cat_transform_quant_workspace_bytes(n, d, k), dtype=torch.uint8,
                       device="cuda")
    fo = cat.cat_transform_quant_flag_offset(n, d, k)

    def buffers():
        return dict(acc=torch.zeros((d, d), dtype=torch.float32, device="cuda"),
                    out=torch.empty(3, dtype=torch.float64, device="cuda"),
                    codes=torch.empty((n, d // 2), dtype=torch.uint8, device="cuda"),
                    s_x=torch.empty(n, dtype=torch.float32, device="cuda"),
                    yq=torch.empty((n, d_out), dtype=torch.float32, device="cuda"))

    def first(b, s):
        cat.cat_cov_accumulate(X, b["acc"], B.CAT_COV_FULL, k, ws_c, stream=s)
        cat.cat_sqnr(dy, dyt, ws_s, b["out"], stream=s)

    def second(b, s):
        cat.cat_transform_quant(X, T, k, b["codes"], b["s_x"], ws_q, stream=s)
        cat.cat_w4a4_linear(b["codes"], b["s_x"], qw, sw, b["yq"], stream=s)

    ref = buffers()
    ws_q[fo:fo + 4].zero_()
    cur = torch.cuda.current_stream()
    first(ref, cur)
    second(ref, cur)
    torch.cuda.synchronize()
    ref = {key: host(v) for key, v in ref.items()}
    s1, s2 = torch.cuda.Stream(), torch.cuda.Stream()
    for rep in range(3):
        got = buffers()
        torch.cuda.synchronize()
        with torch.cuda.stream(s1):
            first(got, s1)
        with torch.cuda.stream(s2):
            second(got, s2)
        torch.cuda.synchronize()
        for key, v in got.items():
            assert np.array_equal(host(v), ref[key]), f"{key} differs (repeat {rep})"
    assert int(host(ws_q[fo:fo + 4].view(torch.int32))[0]) == 0
