"""C-ABI surface of libfpo: loading, exported symbols, workspace queries and
every host-side validation error. Nothing here launches a kernel (each error
path returns before any HIP call), so it runs without a GPU."""
import ctypes as C
import os
import re

import pytest

from paper_2608_14563_amd import _lib as L
from paper_2608_14563_amd import inputs as I

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HDR = os.path.join(ROOT, "include", "fpo.h")
FAKE = 0x100000  # aligned, never dereferenced: every call below fails validation first


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(L.LIB_PATH):
        pytest.fail("libfpo.so is not built (run __graft_entry__.build())")
    return L.load()


def header_functions(path=HDR):
    txt = open(path).read()
    txt = re.sub(r"/\*.*?\*/", "", txt, flags=re.S)
    return sorted(set(re.findall(r"\b(fpo_[a-z_]+)\s*\(", txt)))


def all_header_functions():
    inc = os.path.join(ROOT, "include")
    names = []
    for f in sorted(os.listdir(inc)):
        if f.endswith(".h"):
            names += header_functions(os.path.join(inc, f))
    return sorted(set(names))


def test_header_declares_the_abi():
    names = header_functions()
    assert set(names) == set(L.EXPORTS), names


def test_library_exports_every_header_symbol(lib):
    """Every function the headers declare resolves in libfpo.so's dynamic
    symbol table (dlsym through ctypes; no child process)."""
    names = all_header_functions()
    assert "fpo_prof_read" in names
    for name in names:
        assert hasattr(lib, name), name
    assert not hasattr(lib, "fpo_no_such_symbol")


def test_abi_version(lib):
    assert lib.fpo_abi_version() == 7 == L.ABI_VERSION


def oe(T=128, d=256, V=4096, dtype=L.FPO_BF16, eps=1e-6, min_rms=0.5, chunk=0):
    return L.OeDesc(T, d, V, dtype, eps, min_rms, chunk)


def test_workspace_queries_for_every_workload(lib):
    for c in I.CONFIGS.values():
        dt = L.FPO_BF16 if c.dtype == "bf16" else L.FPO_F32
        ws = lib.fpo_output_error_workspace(C.byref(oe(c.T, c.d, c.V, dt)))
        assert ws >= c.T * c.d * (2 if dt else 4)
        pg = L.PgDesc(c.T, c.d, c.d_ff, c.L, dt, L.FPO_MODE_W3, 1.0 / c.T)
        assert lib.fpo_pseudograd_workspace(C.byref(pg)) >= c.d * c.T * (2 if dt else 4)
        pgf = L.PgDesc(c.T, c.d, c.d_ff, min(c.L, 21), dt, L.FPO_MODE_FULL_MLP, 1.0 / c.T)
        assert lib.fpo_pseudograd_workspace(C.byref(pgf)) > lib.fpo_pseudograd_workspace(C.byref(pg)) or c.L > 21
    n = (C.c_int64 * 2)(1024, 4096)
    assert lib.fpo_apply_update_workspace(2, n) >= 16
    assert lib.fpo_cosine_workspace(2, n) >= 48


def test_invalid_descriptions_give_zero_workspace(lib):
    assert lib.fpo_output_error_workspace(None) == 0
    assert lib.fpo_output_error_workspace(C.byref(oe(d=250))) == 0
    assert lib.fpo_output_error_workspace(C.byref(oe(dtype=7))) == 0


def call_oe(lib, desc, ws=FAKE, ws_bytes=1 << 40, **over):
    args = dict(h=FAKE, g=FAKE, W=FAKE, t=FAKE, gt=FAKE)
    args.update(over)
    return lib.fpo_output_error(C.byref(desc) if desc is not None else None, args["h"], args["g"], args["W"],
                                args["t"], args["gt"], None, None, None, None, None, None, ws, ws_bytes, None)


def test_output_error_validation(lib):
    assert call_oe(lib, None) == L.FPO_ERR_NULL
    assert call_oe(lib, oe(dtype=3)) == L.FPO_ERR_DTYPE
    assert call_oe(lib, oe(T=0)) == L.FPO_ERR_SHAPE     # empty batch: refused, not a no-op
    assert call_oe(lib, oe(d=0)) == L.FPO_ERR_SHAPE
    assert call_oe(lib, oe(V=0)) == L.FPO_ERR_SHAPE
    assert call_oe(lib, oe(d=12)) == L.FPO_ERR_SHAPE
    assert call_oe(lib, oe(V=4100)) == L.FPO_ERR_SHAPE
    assert call_oe(lib, oe(V=1 << 31)) == L.FPO_ERR_SHAPE
    assert call_oe(lib, oe(eps=-1.0)) == L.FPO_ERR_ARG
    assert call_oe(lib, oe(min_rms=float("nan"))) == L.FPO_ERR_ARG
    assert call_oe(lib, oe(chunk=-5)) == L.FPO_ERR_ARG
    assert call_oe(lib, oe(), h=None) == L.FPO_ERR_NULL
    assert call_oe(lib, oe(), gt=None) == L.FPO_ERR_NULL
    assert call_oe(lib, oe(), W=FAKE + 4) == L.FPO_ERR_ARG
    assert call_oe(lib, oe(), ws=None) == L.FPO_ERR_WORKSPACE
    assert call_oe(lib, oe(), ws=FAKE + 64) == L.FPO_ERR_WORKSPACE
    assert call_oe(lib, oe(), ws_bytes=100) == L.FPO_ERR_WORKSPACE
    msg = lib.fpo_last_error().decode()
    assert "workspace" in msg and "needed" in msg
    # bf16 operand bands are addressed through 32-bit buffer offsets
    assert call_oe(lib, oe(T=1 << 19, d=4096)) == L.FPO_ERR_UNSUPPORTED
    assert "2^31" in lib.fpo_last_error().decode()
    assert lib.fpo_output_error_workspace(C.byref(oe(T=1 << 19, d=4096, dtype=L.FPO_F32))) > 0  # fp32 unaffected
    assert lib.fpo_output_error_workspace(C.byref(oe(T=1 << 19, d=4096))) == 0
    # launch geometry: at most 2^23 tokens per call
    assert call_oe(lib, oe(T=(1 << 23) + 8, d=8, V=256, dtype=L.FPO_F32)) == L.FPO_ERR_SHAPE
    assert lib.fpo_output_error_workspace(C.byref(oe(T=1 << 23, d=8, V=256, dtype=L.FPO_F32))) > 0


def test_chunk_width_respects_operand_bands(lib):
    """The planner keeps a W_U chunk (Vc x d) and the staged p~ (T x Vc)
    within 2^30 elements: for d = 8192 the whole 128K vocabulary would not fit
    one chunk, so the workspace (dominated by T x Vc p~) is bounded."""
    T, d, V = 2048, 8192, 131072
    ws = lib.fpo_output_error_workspace(C.byref(oe(T=T, d=d, V=V)))
    vc_max = (1 << 30) // d
    assert 0 < ws
    assert ws <= T * vc_max * 2 + (T * d * 2) + 64 * T * d * 4 + (64 << 20)


def test_staged_p_pitch_padding_and_band(lib):
    """The staged p~ rows are padded by 256 bytes (a power-of-two pitch puts a
    tile's rows in one L2 set), and by default a chunk stages at most 128 MiB
    of p~ (half the Infinity Cache): the documented workspace layout exactly
    at T = 2048, V = 100352 (chunks in whole logits waves of 8192 entries:
    3 x 24576 + 26624, the widest sizing the staged p~; two projection
    splits)."""
    def a256(n):
        return (n + 255) // 256 * 256

    T, d, V, ns = 2048, 4096, 100352, 2
    vc = 26624
    nb = vc // 128
    # y, p~, block max / sum / argmax, seven per-token arrays (output factors, staging reference,
    # target logit, running max / partition / argmax), the projection's split accumulators
    want = (a256(T * d * 2) + a256(T * (vc + 128) * 2) + 3 * a256(T * nb * 4) + 7 * a256(T * 4)
            + a256(ns * T * d * 4))
    assert lib.fpo_output_error_workspace(C.byref(oe(T=T, d=d, V=V))) == want
    T, V = 8192, 131072
    ws = lib.fpo_output_error_workspace(C.byref(oe(T=T, d=d, V=V)))
    assert 0 < ws < T * V * 2


def test_default_chunk_keeps_staged_logits_cache_sized(lib):
    """For every workload the default plan stages at most 128 MiB of p~ per
    chunk (plus 256 bytes of padding per row), never the whole T x V logits:
    the workspace is bounded by y, that chunk, its block statistics, the
    per-token state and at most eight projection partials, and wherever the
    logits exceed the Infinity Cache it is smaller than the logits alone."""
    budget = 128 << 20
    for c in I.CONFIGS.values():
        dt = L.FPO_BF16 if c.dtype == "bf16" else L.FPO_F32
        esz = 2 if dt == L.FPO_BF16 else 4
        blkw = 128 if dt == L.FPO_BF16 else 64
        ws = lib.fpo_output_error_workspace(C.byref(oe(c.T, c.d, c.V, dt)))
        vc = min(budget // esz // c.T, c.V + 255)
        bound = (c.T * c.d * esz + budget + c.T * 256 + 3 * c.T * (vc // blkw + 1) * 4 + 6 * c.T * 4
                 + 8 * c.T * c.d * 4 + 16 * 256)
        assert ws <= bound, (c.name, ws, bound)
        if c.T * c.V * esz > (256 << 20):
            assert ws < c.T * c.V * esz, c.name


def arr(vals):
    a = (C.c_void_p * len(vals))(*vals)
    return C.cast(a, L.PP), a


def test_pseudograd_validation(lib):
    a, ka = arr([FAKE, FAKE])
    dw, kd = arr([FAKE, FAKE])

    def call(desc, A=a, dW3=dw, ref=None, ref_dot=None, opt=None, upd=None, ws_bytes=1 << 40, g=FAKE, pf=None,
             ref_cos=None, ov=None, pm=None):
        return lib.fpo_pseudograd(C.byref(desc) if desc is not None else None, g, A, None, None, None, None,
                                  dW3, None, None, None, ref, ref_dot, None, ref_cos, pf, pm, opt, upd, ov, FAKE,
                                  ws_bytes, None)

    good = L.PgDesc(128, 256, 688, 2, L.FPO_BF16, L.FPO_MODE_W3, 1 / 128)
    assert call(None) == L.FPO_ERR_NULL
    assert call(L.PgDesc(128, 256, 688, 2, 5, 0, 1.0)) == L.FPO_ERR_DTYPE
    assert call(L.PgDesc(128, 256, 688, 2, 1, 9, 1.0)) == L.FPO_ERR_ARG
    assert call(L.PgDesc(128, 256, 690, 2, 1, 0, 1.0)) == L.FPO_ERR_SHAPE
    assert call(L.PgDesc(128, 256, 688, 65, 1, 0, 1.0)) == L.FPO_ERR_SHAPE
    # empty inputs: the pseudogradient is a mean over the batch's tokens
    for T_, d_, f_, L_ in ((0, 256, 688, 2), (128, 0, 688, 2), (128, 256, 0, 2), (128, 256, 688, 0)):
        assert call(L.PgDesc(T_, d_, f_, L_, 1, 0, 1.0)) == L.FPO_ERR_SHAPE
    assert call(L.PgDesc(128, 256, 688, 2, 1, 0, float("inf"))) == L.FPO_ERR_ARG
    assert call(good, g=None) == L.FPO_ERR_NULL
    assert call(good, dW3=None) == L.FPO_ERR_NULL
    r, kr = arr([FAKE, FAKE])
    assert call(good, dW3=None, ref=r) == L.FPO_ERR_NULL  # ref needs ref_dot / ref_sumsq
    assert call(good, ref_cos=FAKE) == L.FPO_ERR_ARG          # a cosine needs a reference
    # a caller-owned overlap set must name its stream and both events
    for k in range(3):
        h = [FAKE, FAKE, FAKE]
        h[k] = None
        assert call(good, ov=C.byref(L.Overlap(*h))) == L.FPO_ERR_NULL, k
    assert call(good, ov=C.byref(L.Overlap(FAKE, FAKE, FAKE)), ws_bytes=16) == L.FPO_ERR_WORKSPACE
    o = L.Opt(0, 1e-4, 0.9, 0.9, 0.999, 1e-8, 0.01, 0.01, 1)
    assert call(good, opt=C.byref(o)) == L.FPO_ERR_ARG  # opt without upd
    full = L.PgDesc(128, 256, 688, 2, L.FPO_BF16, L.FPO_MODE_FULL_MLP, 1 / 128)
    assert call(full) == L.FPO_ERR_NULL
    assert call(good, ws_bytes=16) == L.FPO_ERR_WORKSPACE
    b, kb = arr([FAKE, None])
    assert call(good, A=b) == L.FPO_ERR_NULL
    # post-FFN composition (mode flag + argument): g_tilde_lp may then be NULL
    mo, kmo = arr([FAKE, FAKE])
    gm, kgm = arr([FAKE, FAKE])
    pmode = L.PgDesc(128, 256, 688, 2, L.FPO_BF16, L.FPO_MODE_POST_FFN, 1 / 128)
    pf = C.byref(L.PostFfn(FAKE, mo, gm, 1e-6, 0.5))
    assert call(pmode, g=None, pf=pf, ws_bytes=16) == L.FPO_ERR_WORKSPACE
    assert call(pmode, g=None) == L.FPO_ERR_ARG          # mode without the argument
    assert call(good, pf=pf) == L.FPO_ERR_ARG            # argument without the mode
    assert call(L.PgDesc(128, 256, 688, 2, 1, 16, 1.0)) == L.FPO_ERR_ARG  # unknown mode bit
    # pre-MLP composition (mode flag + argument), alone or after the post-FFN one
    qmode = L.PgDesc(128, 256, 688, 2, L.FPO_BF16, L.FPO_MODE_PRE_MLP, 1 / 128)
    pm = C.byref(L.PreMlp(FAKE, mo, gm, 1e-6, 0.5))
    assert call(qmode, g=None, pm=pm, ws_bytes=16) == L.FPO_ERR_WORKSPACE
    assert call(qmode, g=None) == L.FPO_ERR_ARG          # mode without the argument
    assert call(good, pm=pm) == L.FPO_ERR_ARG            # argument without the mode
    assert call(qmode, g=None, pm=C.byref(L.PreMlp(None, mo, gm, 1e-6, 0.5))) == L.FPO_ERR_NULL
    assert call(qmode, g=None, pm=C.byref(L.PreMlp(FAKE, mo, None, 1e-6, 0.5))) == L.FPO_ERR_NULL
    assert call(qmode, g=None, pm=C.byref(L.PreMlp(FAKE, mo, gm, -1.0, 0.5))) == L.FPO_ERR_ARG
    both = L.PgDesc(128, 256, 688, 2, L.FPO_BF16, L.FPO_MODE_POST_FFN | L.FPO_MODE_PRE_MLP, 1 / 128)
    assert call(both, g=None, pf=pf, pm=pm, ws_bytes=16) == L.FPO_ERR_WORKSPACE
    assert call(both, g=None, pf=pf, pm=C.byref(L.PreMlp(FAKE + 256, mo, gm, 1e-6, 0.5))) == L.FPO_ERR_ARG
    assert lib.fpo_pseudograd_workspace(C.byref(qmode)) == lib.fpo_pseudograd_workspace(C.byref(pmode))
    assert call(pmode, g=None, pf=C.byref(L.PostFfn(None, mo, gm, 1e-6, 0.5))) == L.FPO_ERR_NULL
    assert call(pmode, g=None, pf=C.byref(L.PostFfn(FAKE, None, gm, 1e-6, 0.5))) == L.FPO_ERR_NULL
    m1, km1 = arr([FAKE, None])
    assert call(pmode, g=None, pf=C.byref(L.PostFfn(FAKE, mo, m1, 1e-6, 0.5))) == L.FPO_ERR_NULL
    assert call(pmode, g=None, pf=C.byref(L.PostFfn(FAKE, mo, gm, -1.0, 0.5))) == L.FPO_ERR_ARG
    assert call(pmode, g=None, pf=C.byref(L.PostFfn(FAKE, mo, gm, 1e-6, float("nan")))) == L.FPO_ERR_ARG
    assert call(pmode, g=None, pf=C.byref(L.PostFfn(FAKE + 4, mo, gm, 1e-6, 0.5))) == L.FPO_ERR_ARG
    # the workspace holds every layer's composed signal
    w0 = lib.fpo_pseudograd_workspace(C.byref(good))
    w1 = lib.fpo_pseudograd_workspace(C.byref(pmode))
    assert w1 >= w0 + (2 - 1) * 256 * 128 * 2
    # bf16 staging of the pseudogradient for the fused update (W3-only bf16 path)
    stg = L.PgDesc(128, 256, 688, 2, L.FPO_BF16, L.FPO_MODE_GRAD_BF16, 1 / 128)
    assert call(L.PgDesc(128, 256, 688, 2, L.FPO_F32, L.FPO_MODE_GRAD_BF16, 1 / 128)) == L.FPO_ERR_UNSUPPORTED
    assert call(L.PgDesc(128, 256, 688, 2, L.FPO_BF16, L.FPO_MODE_GRAD_BF16 | L.FPO_MODE_FULL_MLP,
                         1 / 128)) == L.FPO_ERR_UNSUPPORTED
    assert lib.fpo_pseudograd_workspace(C.byref(L.PgDesc(128, 256, 688, 2, L.FPO_F32, L.FPO_MODE_GRAD_BF16,
                                                         1 / 128))) == 0
    assert call(stg) == L.FPO_ERR_ARG                    # dW3 given
    assert call(stg, dW3=None) == L.FPO_ERR_ARG          # no fused update
    w2 = lib.fpo_pseudograd_workspace(C.byref(stg))
    assert w2 >= w0 + 2 * 256 * 688 * 2                   # one staged bf16 matrix per layer
    # bf16 operand bands (T x d_ff activations) above 2^31 bytes are refused
    assert call(L.PgDesc(1 << 17, 256, 16384, 2, L.FPO_BF16, L.FPO_MODE_W3, 1.0)) == L.FPO_ERR_UNSUPPORTED
    # launch geometry: at most 2^23 tokens and d <= 2^22 per call
    assert call(L.PgDesc((1 << 23) + 64, 8, 8, 1, L.FPO_F32, L.FPO_MODE_W3, 1.0)) == L.FPO_ERR_SHAPE
    assert call(L.PgDesc(64, (1 << 22) + 8, 8, 1, L.FPO_F32, L.FPO_MODE_W3, 1.0)) == L.FPO_ERR_SHAPE
    assert lib.fpo_pseudograd_workspace(C.byref(L.PgDesc(64, 1 << 22, 8, 1, L.FPO_F32, L.FPO_MODE_W3, 1.0))) > 0


def test_pseudograd_operand_alignment(lib):
    """Reference gradients and the full-MLP operands are read 16 bytes per
    lane: a pointer off 16-byte alignment is refused before any launch (the
    well-aligned call fails only at the workspace check)."""
    good = [FAKE, FAKE]
    bad = [FAKE, FAKE + 4]

    def ref_call(ref):
        r, kr = arr(ref)
        desc = L.PgDesc(128, 256, 688, 2, L.FPO_BF16, L.FPO_MODE_W3, 1 / 128)
        a, ka = arr(good)
        return lib.fpo_pseudograd(C.byref(desc), FAKE, a, None, None, None, None, None, None, None, None, r,
                                  FAKE, FAKE, None, None, None, None, None, None, FAKE, 16, None)

    assert ref_call(good) == L.FPO_ERR_WORKSPACE
    assert ref_call(bad) == L.FPO_ERR_ARG

    def full_call(which):
        bufs = [arr(bad if k == which else good) for k in range(7)]
        p = [b[0] for b in bufs]
        desc = L.PgDesc(128, 256, 688, 2, L.FPO_BF16, L.FPO_MODE_FULL_MLP, 1 / 128)
        return lib.fpo_pseudograd(C.byref(desc), FAKE, p[0], p[1], p[2], p[3], p[4], p[5], p[6], p[6], None,
                                  None, None, None, None, None, None, None, None, None, FAKE, 16, None)

    assert full_call(-1) == L.FPO_ERR_WORKSPACE
    for k in range(1, 7):  # W3_init, gate, up, x_in, dW3 / dW1, dW2
        assert full_call(k) == L.FPO_ERR_ARG, k


def test_apply_update_validation(lib):
    g, kg = arr([FAKE])
    W, kw = arr([FAKE])
    s1, k1 = arr([FAKE])
    n = (C.c_int64 * 1)(1024)
    ub = L.UpdateBufs(W, None, s1, None, FAKE, None)

    def call(o, n_mats=1, numel=n, upd=ub, lp=L.FPO_BF16, ws_bytes=1 << 20):
        return lib.fpo_apply_update(C.byref(o) if o is not None else None, n_mats, numel, g, FAKE,
                                    C.byref(upd) if upd is not None else None, lp, FAKE, ws_bytes, None)

    sgd = L.Opt(0, 1e-4, 0.9, 0.9, 0.999, 1e-8, 0.01, 0.01, 1)
    assert call(None) == L.FPO_ERR_NULL
    assert call(L.Opt(4, 1e-4, 0.9, 0.9, 0.999, 1e-8, 0.01, 0.01, 1)) == L.FPO_ERR_ARG
    assert call(L.Opt(0, -1.0, 0.9, 0.9, 0.999, 1e-8, 0.01, 0.01, 1)) == L.FPO_ERR_ARG
    assert call(L.Opt(0, 1e-4, 0.9, 0.9, 0.999, 1e-8, 0.01, 0.01, 0)) == L.FPO_ERR_ARG
    assert call(L.Opt(0, 1e-4, 0.9, 0.9, 0.999, 1e-8, 0.01, 0.01, 1, 2)) == L.FPO_ERR_ARG  # unknown clip target
    assert call(L.Opt(1, 1e-4, 0.9, 1.0, 0.999, 1e-8, 0.01, 0.01, 1)) == L.FPO_ERR_ARG
    assert call(L.Opt(1, 1e-4, 0.9, 0.9, 0.999, 1e-8, 0.01, 0.01, 1)) == L.FPO_ERR_NULL  # AdamW needs state2
    assert call(sgd, upd=None) == L.FPO_ERR_NULL
    assert call(sgd, n_mats=0) == L.FPO_ERR_SHAPE
    assert call(sgd, numel=(C.c_int64 * 1)(0)) == L.FPO_ERR_SHAPE  # empty matrix: no relative clip
    assert call(sgd, numel=(C.c_int64 * 1)(1022)) == L.FPO_ERR_SHAPE
    assert call(sgd, lp=9) == L.FPO_ERR_DTYPE
    assert call(sgd, ws_bytes=8) == L.FPO_ERR_WORKSPACE
    # no state buffer: allowed only for SGD with momentum 0 (plain SGD)
    nostate = L.UpdateBufs(W, None, None, None, FAKE, None)
    assert call(sgd, upd=nostate) == L.FPO_ERR_NULL
    assert "momentum 0" in lib.fpo_last_error().decode()
    plain = L.Opt(0, 1e-4, 0.0, 0.9, 0.999, 1e-8, 0.01, 0.01, 1)
    assert call(plain, upd=nostate, ws_bytes=8) == L.FPO_ERR_WORKSPACE  # passes the state check
    # operand alignment: 16 bytes, except a bf16 copy of the weights (8)
    lp8, k8 = arr([FAKE + 8])
    with_lp = L.UpdateBufs(W, lp8, s1, None, FAKE, None)
    assert call(sgd, upd=with_lp, ws_bytes=8) == L.FPO_ERR_WORKSPACE
    assert call(sgd, upd=with_lp, lp=L.FPO_F32) == L.FPO_ERR_ARG
    s2b, k2 = arr([FAKE + 4])
    adam = L.Opt(1, 1e-4, 0.9, 0.9, 0.999, 1e-8, 0.01, 0.01, 1)
    assert call(adam, upd=L.UpdateBufs(W, None, s1, s2b, FAKE, None)) == L.FPO_ERR_ARG
    s1b, k1b = arr([FAKE + 8])
    assert call(sgd, upd=L.UpdateBufs(W, None, s1b, None, FAKE, None)) == L.FPO_ERR_ARG


def test_apply_update_noalloc_validation(lib):
    """The no-allocation update validates like fpo_apply_update and refuses,
    before any HIP call, matrices whose scratch exceeds its static array."""
    g, kg = arr([FAKE])
    W, kw = arr([FAKE])
    s1, k1 = arr([FAKE])
    ub = L.UpdateBufs(W, None, s1, None, FAKE, None)
    sgd = L.Opt(0, 1e-4, 0.9, 0.9, 0.999, 1e-8, 0.01, 0.01, 1)

    def call(o, numel, n_mats=1, upd=ub, lp=L.FPO_BF16):
        return lib.fpo_apply_update_noalloc(C.byref(o) if o is not None else None, n_mats, numel, g, FAKE,
                                            C.byref(upd) if upd is not None else None, lp, None)

    n = (C.c_int64 * 1)(1024)
    assert call(None, n) == L.FPO_ERR_NULL
    assert call(sgd, n, upd=None) == L.FPO_ERR_NULL
    assert call(sgd, n, n_mats=0) == L.FPO_ERR_SHAPE
    assert call(sgd, (C.c_int64 * 1)(1022)) == L.FPO_ERR_SHAPE
    assert call(sgd, n, lp=9) == L.FPO_ERR_DTYPE
    # one double of scratch per 4096 parameters: just past the array's capacity
    too_many = (L.NOALLOC_SCRATCH_BYTES // 8 + 1) * 4096
    assert call(sgd, (C.c_int64 * 1)(too_many)) == L.FPO_ERR_WORKSPACE
    assert "static array" in lib.fpo_last_error().decode()


def test_cosine_validation(lib):
    A, ka = arr([FAKE])
    n = (C.c_int64 * 1)(1024)
    assert lib.fpo_cosine(0, n, A, None, 0, None, None, None, None, FAKE, 1 << 20, None) == L.FPO_ERR_SHAPE
    assert lib.fpo_cosine(1, (C.c_int64 * 1)(0), A, None, 0, None, None, None, None, FAKE, 1 << 20,
                          None) == L.FPO_ERR_SHAPE
    assert lib.fpo_cosine(1, None, A, None, 0, None, None, None, None, FAKE, 1 << 20, None) == L.FPO_ERR_NULL
    assert lib.fpo_cosine(1, n, A, None, 3, None, None, None, None, FAKE, 1 << 20, None) == L.FPO_ERR_DTYPE
    assert lib.fpo_cosine(1, (C.c_int64 * 1)(6), A, None, 0, None, None, None, None, FAKE, 1 << 20, None) == L.FPO_ERR_SHAPE
    assert lib.fpo_cosine(1, n, A, None, 0, None, None, None, None, FAKE, 8, None) == L.FPO_ERR_WORKSPACE


def test_binding_rejects_host_tensors():
    """The binding hands the library device pointers only: host tensors are
    refused before any call (no GPU needed)."""
    import torch

    from paper_2608_14563_amd import api
    T, d, V = 4, 8, 16
    x = torch.zeros(T, d)
    with pytest.raises(ValueError, match="GPU tensors"):
        api.fpo_output_error(x, torch.ones(d), torch.zeros(V, d), torch.zeros(T, dtype=torch.int32),
                             torch.empty(T, d), ws=torch.empty(1 << 20, dtype=torch.uint8))
    with pytest.raises(ValueError, match="GPU tensors"):
        api.fpo_cosine([torch.zeros(8)], [torch.zeros(8)], ws=torch.empty(4096, dtype=torch.uint8))
