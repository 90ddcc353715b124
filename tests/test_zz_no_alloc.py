"""dm_route_batch_noalloc against dm_route_batch, through the C ABI (runs
last: its file name sorts after the other test files).

Two allocation-free calls in a row, the second with a smaller batch (the
static work area keeps the first call's contents), each compared element by
element with dm_route_batch on the same inputs and loads: ring keys,
candidates, matches, choices, TTFT, flags, final loads, and block keys when
the caller asks for them.  A batch whose work arrays do not fit the static
area is rejected on the host and changes nothing.
"""
import ctypes as C
import sys

import numpy as np
import pytest

import workloads

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


def _say(*a):
    print("[case]", *a, flush=True)


def _outputs(eng, n, nb=None):
    return eng.alloc_route_out(n, nb)


def _host(out, loads):
    r = {k: v.cpu().numpy() for k, v in out.items()}
    r["loads"] = loads.cpu().numpy()
    return r


def test_noalloc_matches_route_batch():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2602_06502_amd as pk
    import paper_2602_06502_amd.harness as gh
    wl = workloads.tiny(slo_us=20_000)
    g = gh.setup(wl, device="cuda:0")
    eng = g["eng"]
    dev = eng.device
    tok, off = g["tokens_np"], g["offsets_np"]
    for n, with_keys in ((1024, False), (300, False), (1024, True), (77, True)):
        _say("noalloc vs route_batch: requests", n, "block keys" if with_keys else "")
        t = gh.to_dev(tok[:off[n]], dev)
        f = gh.to_dev(off[:n + 1], dev)
        nb = int((np.diff(off[:n + 1]) // wl.route.block).sum()) if with_keys else None
        res = []
        for noalloc in (True, False):
            L = gh.to_dev(g["loads0"], dev)
            out = _outputs(eng, n, nb)
            eng.route_into(t, f, L, out, noalloc=noalloc)
            eng.sync()
            res.append(_host(out, L))
        for k in res[1]:
            assert np.array_equal(res[0][k], res[1][k]), (n, k)
    # a batch whose work arrays exceed the static area: rejected, no effect
    _say("noalloc: oversized batch rejected")
    lib = pk.load_library()
    n = 1024
    L = gh.to_dev(g["loads0"], dev)
    out = _outputs(eng, n)
    for v in out.values():
        v.zero_()
    ro = pk.dm_route_out(out["key"].data_ptr(), out["cand"].data_ptr(), out["match"].data_ptr(),
                         out["chosen"].data_ptr(), out["ttft"].data_ptr(), out["flags"].data_ptr(),
                         None)
    t = gh.to_dev(tok[:off[n]], dev)
    f = gh.to_dev(off[:n + 1], dev)
    st = lib.dm_route_batch_noalloc(eng._h, t.data_ptr(), 1 << 28, f.data_ptr(), n,
                                    L.data_ptr(), C.byref(ro))
    assert st == pk.DM_EINVAL
    assert b"static area" in lib.dm_last_error(eng._h)
    eng.sync()
    assert np.array_equal(L.cpu().numpy(), g["loads0"])
    assert not any(bool((v.view(torch.uint8) != 0).any().item()) for v in out.values())
    # and the next call works
    eng.route_into(t, f, L, out, noalloc=True)
    eng.sync()
