"""fpo_apply_update_noalloc (scratch in the library's static device array)
against fpo_apply_update (caller workspace), called through the C ABI with
ctypes: two calls in a row on one stream, the second on a smaller input with
another optimizer, each compared bit for bit with the workspace entry point
on identical copies of its inputs."""
import ctypes as C

import numpy as np
import pytest
import torch

from paper_2608_14563_amd import _lib as L

pytestmark = pytest.mark.gpu


def ptr_array(ts):
    a = (C.c_void_p * len(ts))(*[t.data_ptr() if t is not None else None for t in ts])
    return a, C.cast(a, L.PP)


def make_case(dev, numels, seed, grad_std):
    g = torch.Generator(device=dev)
    g.manual_seed(seed)
    W = [0.02 * torch.randn(n, generator=g, device=dev) for n in numels]
    G = [grad_std * torch.randn(n, generator=g, device=dev) for n in numels]
    S1 = [1e-3 * torch.randn(n, generator=g, device=dev) for n in numels]
    S2 = [1e-6 * torch.rand(n, generator=g, device=dev) for n in numels]
    return W, G, S1, S2


def run(lib, dev, opt, numels, W, G, S1, S2, adam, noalloc, ws=None):
    """One call on clones of the inputs; returns the buffers it wrote."""
    W = [w.clone() for w in W]
    S1 = [s.clone() for s in S1]
    S2 = [s.clone() for s in S2] if adam else None
    lp = [torch.empty(n, dtype=torch.bfloat16, device=dev) for n in numels]
    gsq = torch.tensor([float(g.double().pow(2).sum()) for g in G], dtype=torch.float64, device=dev)
    wsq = torch.tensor([float(w.double().pow(2).sum()) for w in W], dtype=torch.float64, device=dev)
    cs = torch.empty(len(numels), dtype=torch.float32, device=dev)
    keep = []
    arrs = {}
    for name, ts in (("W", W), ("G", G), ("S1", S1), ("S2", S2), ("lp", lp)):
        if ts is None:
            arrs[name] = None
            continue
        a, p = ptr_array(ts)
        keep.append(a)
        arrs[name] = p
    ub = L.UpdateBufs(arrs["W"], arrs["lp"], arrs["S1"], arrs["S2"], wsq.data_ptr(), cs.data_ptr())
    numel = (C.c_int64 * len(numels))(*numels)
    stream = torch.cuda.current_stream(dev).cuda_stream
    if noalloc:
        st = lib.fpo_apply_update_noalloc(C.byref(opt), len(numels), numel, arrs["G"], gsq.data_ptr(),
                                          C.byref(ub), L.FPO_BF16, stream)
    else:
        st = lib.fpo_apply_update(C.byref(opt), len(numels), numel, arrs["G"], gsq.data_ptr(), C.byref(ub),
                                  L.FPO_BF16, ws.data_ptr(), ws.numel(), stream)
    assert st == L.FPO_OK, lib.fpo_last_error().decode()
    return dict(W=W, S1=S1, S2=S2, lp=lp, wsq=wsq, cs=cs, keep=keep)


def same_bits(a, b, name):
    for k in ("W", "S1", "S2", "lp"):
        if a[k] is None:
            continue
        for m, (x, y) in enumerate(zip(a[k], b[k])):
            assert torch.equal(x.view(torch.int16) if x.dtype == torch.bfloat16 else x.view(torch.int32),
                               y.view(torch.int16) if y.dtype == torch.bfloat16 else y.view(torch.int32)), \
                f"{name}: {k}[{m}] differs"
    assert torch.equal(a["wsq"], b["wsq"]), f"{name}: ||W'||^2 differs"
    assert torch.equal(a["cs"], b["cs"]), f"{name}: clip factors differ"


def test_noalloc_update_matches_workspace_update_twice(dev):
    lib = L.load()
    # call 1: SGD-momentum (step 2, active clip) on three matrices, one with a
    # partial last block; call 2: AdamW (step 3) on one small matrix
    sgd = L.Opt(L.FPO_OPT_SGD, 1e-4, 0.9, 0.9, 0.999, 1e-8, 0.01, 0.01, 2, L.FPO_CLIP_GRADIENT)
    adam = L.Opt(L.FPO_OPT_ADAMW, 1e-4, 0.9, 0.9, 0.999, 1e-8, 0.01, 0.01, 3, L.FPO_CLIP_GRADIENT)
    n1 = [4096 * 300 + 12, 3100, 1_000_000]
    n2 = [8192]
    c1 = make_case(dev, n1, 1, 1e-3)
    c2 = make_case(dev, n2, 2, 1e-3)
    print("[no-alloc] two calls in a row: SGD-momentum on 3 matrices, then AdamW on 1", flush=True)
    got1 = run(lib, dev, sgd, n1, *c1, adam=False, noalloc=True)
    got2 = run(lib, dev, adam, n2, *c2, adam=True, noalloc=True)
    torch.cuda.synchronize()
    for numels, case, opt, is_adam, got, name in ((n1, c1, sgd, False, got1, "call 1"),
                                                   (n2, c2, adam, True, got2, "call 2")):
        nws = lib.fpo_apply_update_workspace(len(numels), (C.c_int64 * len(numels))(*numels))
        ws = torch.empty(max(nws, 256), dtype=torch.uint8, device=dev)
        ref = run(lib, dev, opt, numels, *case, adam=is_adam, noalloc=False, ws=ws)
        torch.cuda.synchronize()
        same_bits(got, ref, name)
        # the step really happened and the clip was active
        assert not torch.equal(got["W"][0], case[0][0])
        assert float(got["cs"].max()) < 1.0
