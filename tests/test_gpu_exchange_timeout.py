"""Forced timeouts of the single-pass transform+quant's exchange waits.

The single pass waits (bounded) for row maxima that other workgroups
publish; each workgroup reads a token's row maximum on its own.  A wait
that runs out must never yield a wrong scale: a workgroup whose read gave up
uses a NaN maximum, so the codes of its block of the token are zero
(symmetric codes) and, for block 0's workgroup, the token's s_x is NaN; the
workspace's timeout word is set.  Every other block and scale keeps its
exact result.  The host lowers the poll bound to one poll
(cat_set_exchange_spin_limit), so that reads of words not yet published
give up at once; every kernel still finishes normally.  Which reads time
out depends on timing, so the checks hold for any mix."""
import numpy as np
import pytest

import paper_2603_04359_amd as cat

from gpu_common import dev, host, say, torch_mod
from test_gpu_parity import _rand_T, _wide_X

pytestmark = pytest.mark.gpu


def _run(X, T, k, mode, ws, fo):
    torch = torch_mod()
    n, d = X.shape
    codes = torch.empty((n, d if mode == 8 else d // 2),
                        dtype=torch.int8 if mode == 8 else torch.uint8, device="cuda")
    s_x = torch.empty(n, dtype=torch.float32, device="cuda")
    zm = torch.empty(n, dtype=torch.float32, device="cuda")
    ws[fo:fo + 4].zero_()
    if mode == "asym":
        cat.cat_transform_quant_asym(X, T, k, codes, s_x, zm, ws)
    else:
        cat.cat_transform_quant(X, T, k, codes, s_x, ws, bits=mode)
    flag = int(host(ws[fo:fo + 4].view(torch.int32))[0])
    return host(codes), host(s_x), host(zm), flag


@pytest.mark.parametrize("d,mode", [(4096, 4), (2048, 8), (8192, 4), (4096, "asym")])
def test_forced_exchange_timeouts_are_loud(d, mode):
    say(f"tq forced exchange timeouts d={d} mode={mode}")
    torch = torch_mod()
    n, k = 8192, 128
    X = dev(_wide_X(n, d, seed=40), "bf16")
    T = dev(_rand_T(d, k, seed=41), "bf16")
    wsb = (cat.cat_transform_quant_asym_workspace_bytes if mode == "asym"
           else cat.cat_transform_quant_workspace_bytes)(n, d, k)
    ws = torch.zeros(wsb, dtype=torch.uint8, device="cuda")
    fo = cat.cat_transform_quant_flag_offset(n, d, k)
    ref_c, ref_s, ref_z, ref_flag = _run(X, T, k, mode, ws, fo)
    assert ref_flag == 0 and not np.isnan(ref_s).any()
    timed_out = 0
    try:
        cat.cat_set_exchange_spin_limit(1)
        for _ in range(3):
            c, s, z, flag = _run(X, T, k, mode, ws, fo)
            nan = np.isnan(s)
            # every scale is the exact one or NaN
            assert np.array_equal(s[~nan], ref_s[~nan])
            if mode == "asym":
                # the maximum and minimum keys are read apart: a lost
                # minimum makes both NaN, a lost maximum only the scale
                zn = np.isnan(z)
                assert not (zn & ~nan).any()
                assert np.array_equal(z[~zn], ref_z[~zn])
                changed = nan.any() or not np.array_equal(c, ref_c)
            else:
                # each 128-channel block of a token's codes is exact or zero
                seg = (k if mode == 8 else k // 2)
                cb, rb = c.reshape(n, d // k, seg), ref_c.reshape(n, d // k, seg)
                same = (cb == rb).all(axis=2)
                zero = (cb == 0).all(axis=2)
                assert (same | zero).all(), "a block of codes neither exact nor zeroed"
                changed = nan.any() or not same.all()
            if changed:
                assert flag != 0, "results changed without the timeout word set"
                timed_out += 1
    finally:
        cat.cat_set_exchange_spin_limit(0)
    # the default bound again: the same call is exact, with no timeout
    c, s, z, flag = _run(X, T, k, mode, ws, fo)
    assert flag == 0
    assert np.array_equal(c, ref_c) and np.array_equal(s, ref_s)
    if not timed_out:
        pytest.skip("no exchange read was early enough to time out at one poll")


def test_status_query_reports_and_clears_a_forced_timeout():
    # the status query returns CAT_ERR_TIMEOUT after a call whose waits ran
    # out and clears the word; after calls with the default bound it is
    # CAT_OK, on a caller workspace and on the allocation-free scratch
    say("tq status query: workspace and allocation-free scratch")
    torch = torch_mod()
    n, d, k = 8192, 4096, 128
    X = dev(_wide_X(n, d, seed=42), "bf16")
    T = dev(_rand_T(d, k, seed=43), "bf16")
    ws = torch.zeros(cat.cat_transform_quant_workspace_bytes(n, d, k), dtype=torch.uint8,
                     device="cuda")
    codes = torch.empty((n, d // 2), dtype=torch.uint8, device="cuda")
    s_x = torch.empty(n, dtype=torch.float32, device="cuda")
    fo = cat.cat_transform_quant_flag_offset(n, d, k)
    for noalloc in (False, True):
        def call():
            if noalloc:
                cat.cat_transform_quant_noalloc(X, T, k, codes, s_x)
            else:
                cat.cat_transform_quant(X, T, k, codes, s_x, ws)

        def status():
            if noalloc:
                cat.cat_transform_quant_noalloc_status(n, d, k)
            else:
                cat.cat_transform_quant_status(ws, n, d, k)

        status()                      # clears whatever earlier calls left
        call()
        status()                      # default bound: no timeout
        ref_s = host(s_x).copy()
        assert not np.isnan(ref_s).any()
        seen = False
        try:
            cat.cat_set_exchange_spin_limit(1)
            for _ in range(3):
                call()
                s = host(s_x)
                changed = np.isnan(s).any() or not np.array_equal(s, ref_s)
                try:
                    status()
                except cat.CatError as e:
                    assert e.code == cat.CAT_ERR_TIMEOUT
                    seen = True
                else:
                    assert not changed, "results changed but the status query saw no timeout"
        finally:
            cat.cat_set_exchange_spin_limit(0)
        # cleared by the query that reported it; exact again at the default bound
        if not noalloc:
            assert int(host(ws[fo:fo + 4].view(torch.int32))[0]) == 0
        call()
        status()
        assert np.array_equal(host(s_x), ref_s)
        if not seen:
            say(f"  noalloc={noalloc}: no read timed out at one poll")
