"""GPU parity of fpo_output_error against the fp64 oracle: error, projection
through W_U, clamped final-RMSNorm VJP, lse / loss / argmax and the
out-of-range-target counter, on seeded inputs (several tiles, ragged tails,
several vocabulary chunks) and the stress cases of the parity contract."""
import numpy as np
import pytest
import torch

import oracle as O
from paper_2608_14563_amd import api
from paper_2608_14563_amd import inputs as I
from tests._util import TOL, assert_close, dev_tensor, host64

pytestmark = pytest.mark.gpu


def run_gpu(x, gamma, W, y, dtype, dev, eps=1e-6, min_rms=0.5, chunk=0):
    T, d = x.shape
    tx = dev_tensor(x, dev)
    tdt = tx.dtype
    out = dict(
        g_tilde=torch.empty(T, d, dtype=torch.float32, device=dev), g_tilde_lp=torch.empty(T, d, dtype=tdt, device=dev),
        g_pre=torch.empty(T, d, dtype=torch.float32, device=dev), lse=torch.empty(T, dtype=torch.float32, device=dev), loss=torch.empty(T, dtype=torch.float32, device=dev),
        argmax=torch.empty(T, dtype=torch.int32, device=dev), bad_targets=torch.full((1,), -7, dtype=torch.int32, device=dev))
    api.fpo_output_error(tx, dev_tensor(gamma, dev), dev_tensor(W, dev), dev_tensor(y, dev), eps=eps,
                         min_rms=min_rms, vocab_chunk=chunk, **out)
    torch.cuda.synchronize()
    return {k: (v.cpu().numpy() if v.dtype == torch.int32 else host64(v)) for k, v in out.items()}


def check_against_oracle(x, gamma, W, y, dtype, got, eps=1e-6, min_rms=0.5):
    ref = O.output_error(x, gamma, W, y, eps=eps, min_rms=min_rms)
    errs = {}
    for k in ("g_pre", "g_tilde", "lse", "loss"):
        errs[k] = assert_close(k, got[k], ref[k], dtype)
    assert_close("g_tilde_lp", got["g_tilde_lp"], ref["g_tilde"], dtype)
    assert int(got["bad_targets"][0]) == ref["bad"]
    # argmax: exact above the margin, otherwise any near-maximal index
    rel = 1e-5 if dtype == "f32" else 1e-2
    xs, Ws = x, W
    for t in range(x.shape[0]):
        ga = int(got["argmax"][t])
        if ga == int(ref["argmax"][t]):
            continue
        delta = rel * max(abs(ref["zmax"][t]), 1.0)
        zg = O.logit(xs, gamma, Ws, t, ga, eps)
        assert zg >= ref["zmax"][t] - delta, f"argmax row {t}: {ga} vs {ref['argmax'][t]}"
    return errs, ref


def small_case(cfg, T, d, V, seed_layer=0):
    c = cfg.shrink(T=T, d=d, V=V)
    return c, I.hidden(c), I.gain(c), I.unembedding(c), I.targets(c)


@pytest.mark.parametrize("chunk", [0, 1024])
def test_tiny_fp32_config(dev, chunk):
    c = I.CONFIGS[0]
    x, g, W, y = I.hidden(c), I.gain(c), I.unembedding(c), I.targets(c)
    got = run_gpu(x, g, W, y, "f32", dev, chunk=chunk)
    check_against_oracle(x, g, W, y, "f32", got)


@pytest.mark.parametrize("T,d,V,chunk", [(300, 264, 4104, 1024), (517, 512, 8200, 0), (64, 256, 2048, 256),
                                         (5, 8200, 264, 0), (16, 64, 100000, 0)])
def test_fp32_ragged(dev, T, d, V, chunk):
    c, x, g, W, y = small_case(I.CONFIGS[0], T, d, V)
    got = run_gpu(x, g, W, y, "f32", dev, chunk=chunk)
    check_against_oracle(x, g, W, y, "f32", got)


# (512, 512, 4224, 1024) and (512, 256, 2048, 0) are whole 256 x 256 tiles (the
# GEMM core's copy form without bounds), the first with a ragged last chunk
@pytest.mark.parametrize("T,d,V,chunk", [(300, 264, 4104, 1024), (600, 512, 10000, 0), (256, 256, 4096, 2048), (1, 128, 1024, 0),
                                         (5, 8200, 264, 0), (16, 64, 200000, 0), (512, 512, 4224, 1024),
                                         (512, 256, 2048, 0)])
def test_bf16_ragged(dev, T, d, V, chunk):
    c, x, g, W, y = small_case(I.CONFIGS[1], T, d, V)
    got = run_gpu(x, g, W, y, "bf16", dev, chunk=chunk)
    check_against_oracle(x, g, W, y, "bf16", got)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_more_tokens_than_a_second_grid_dimension_holds(dev, dtype):
    """T = 65600, above the 65536 cap of a second grid dimension: the
    per-token kernels run on flat grids."""
    print(f"[oe] T=65600 d=16 V=520 {dtype}", flush=True)
    c, x, g, W, y = small_case(I.CONFIGS[0] if dtype == "f32" else I.CONFIGS[1], 65600, 16, 520)
    got = run_gpu(x, g, W, y, dtype, dev)
    check_against_oracle(x, g, W, y, dtype, got)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_low_rms_rows_activate_clamp(dev, dtype):
    base = I.CONFIGS[0] if dtype == "f32" else I.CONFIGS[1]
    c = base.shrink(T=200, d=256, V=4096)
    x = I.hidden(c)
    xf = x.astype(np.float32) if dtype == "f32" else I.bf16_to_f32(x)
    rows = np.arange(0, 200, 50)  # ~1% BOS-like rows scaled x0.1 -> rho ~ 0.1 < 0.5
    xf = xf.copy()
    xf[rows] *= 0.1
    x = I.to_storage(xf, c.dtype)
    g, W, y = I.gain(c), I.unembedding(c), I.targets(c)
    rho, _ = O.rmsnorm_forward(x, g, 1e-6)
    assert np.all(rho[rows] < 0.5)
    got = run_gpu(x, g, W, y, dtype, dev, chunk=1024)
    check_against_oracle(x, g, W, y, dtype, got)


@pytest.mark.parametrize("chunk", [0, 2048])
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_argmax_ties_take_the_lowest_index(dev, dtype, chunk):
    """Identical unembedding rows that dominate every token's logits (as with
    duplicated or padded vocabulary rows): the kernels compute identical rows
    identically, so the tie is exact and the argmax is the lowest tied index,
    across 128-entry blocks, 256-wide tiles and vocabulary chunks. The fp64
    oracle's matrix product may round the tied entries differently (its edge
    columns take another summation order), so it only has to pick one of
    them."""
    base = I.CONFIGS[0] if dtype == "f32" else I.CONFIGS[1]
    c = base.shrink(T=300, d=256, V=10000)
    xf = I.storage_to_f64(I.hidden(c)) + 3.0  # a common direction in every row
    x = I.to_storage(xf.astype(np.float32), c.dtype)
    g, y = I.gain(c), I.targets(c)
    Wf = I.storage_to_f64(I.unembedding(c)).astype(np.float32)
    tied = [4001, 130, 2500, 2049, 9999]
    Wf[tied] = 1.0 / 16.0  # logit ~15 against a random-row maximum ~1.3
    W = I.to_storage(Wf, c.dtype)
    got = run_gpu(x, g, W, y, dtype, dev, chunk=chunk)
    ref = O.output_error(x, g, W, y)
    assert np.all(np.isin(ref["argmax"], tied))
    assert np.all(got["argmax"] == 130)
    check_against_oracle(x, g, W, y, dtype, got)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_peaky_logits_and_planted_targets(dev, dtype):
    """W_U x8 makes softmax peaky (online max rescaling across chunks and the
    p_y -> 1 cancellation); half the targets are set to the oracle argmax."""
    base = I.CONFIGS[0] if dtype == "f32" else I.CONFIGS[1]
    c = base.shrink(T=256, d=256, V=8192)
    x, g = I.hidden(c), I.gain(c)
    Wf = (I.unembedding(c).astype(np.float32) if dtype == "f32" else I.bf16_to_f32(I.unembedding(c))) * 8
    W = I.to_storage(Wf, c.dtype)
    y = I.targets(c)
    ref0 = O.output_error(x, g, W, y)
    y = y.copy()
    y[::2] = ref0["argmax"][::2]
    got = run_gpu(x, g, W, y, dtype, dev, chunk=1024)
    _, ref = check_against_oracle(x, g, W, y, dtype, got)
    # planted: a boosted row wins by far more than the margin
    y2 = y.copy()
    Wp = Wf.copy()
    _, yy = O.rmsnorm_forward(x, g, 1e-6)
    for t in range(0, 256, 37):
        v = 4000 + t
        Wp[v] = (4.0 * yy[t] / np.linalg.norm(yy[t])).astype(np.float32)
        y2[t] = v
    W2 = I.to_storage(Wp, c.dtype)
    got2 = run_gpu(x, g, W2, y2, dtype, dev, chunk=1024)
    check_against_oracle(x, g, W2, y2, dtype, got2)
    for t in range(0, 256, 37):
        assert int(got2["argmax"][t]) == 4000 + t


@pytest.mark.parametrize("chunk", [0, 1024])
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_staging_reference_far_below_the_row_maximum(dev, dtype, chunk):
    """p~ is staged against a per-token reference (the target logit for the
    first chunk, then the running maximum); a block more than the margin above
    it is staged in its own scale and the statistics kernel brings that row to
    one scale. W_U x64 puts a random target's logit ~80 below its row maximum
    (rows whose target is the argmax stay on the common path), and planted
    rows in a later chunk exceed the maximum of the earlier chunks by ~200,
    with their targets left elsewhere."""
    base = I.CONFIGS[0] if dtype == "f32" else I.CONFIGS[1]
    c = base.shrink(T=300, d=256, V=8200)
    x, g = I.hidden(c), I.gain(c)
    Wf = I.storage_to_f64(I.unembedding(c)).astype(np.float32) * 64
    y = I.targets(c).copy()
    W = I.to_storage(Wf, c.dtype)
    ref0 = O.output_error(x, g, W, y)
    y[::2] = ref0["argmax"][::2]
    _, yy = O.rmsnorm_forward(x, g, 1e-6)
    far = ref0["zmax"] - np.array([O.logit(x, g, W, t, int(y[t])) for t in range(c.T)])
    assert np.sum(far > 70) > c.T // 4  # many rows take the own-scale path
    got = run_gpu(x, g, W, y, dtype, dev, chunk=chunk)
    check_against_oracle(x, g, W, y, dtype, got)
    Wp = Wf.copy()
    for t in range(1, c.T, 29):
        Wp[6200 + t] = (300.0 * yy[t] / np.dot(yy[t], yy[t])).astype(np.float32)
    W2 = I.to_storage(Wp, c.dtype)
    got2 = run_gpu(x, g, W2, y, dtype, dev, chunk=chunk)
    check_against_oracle(x, g, W2, y, dtype, got2)
    for t in range(1, c.T, 29):
        assert int(got2["argmax"][t]) == 6200 + t


def test_out_of_range_targets_counted_and_zeroed(dev):
    c, x, g, W, y = small_case(I.CONFIGS[1], 128, 256, 4096)
    y = y.copy()
    y[3] = 4096
    y[77] = -1
    y[100] = 2 ** 31 - 1
    got = run_gpu(x, g, W, y, "bf16", dev)
    assert int(got["bad_targets"][0]) == 3
    for t in (3, 77, 100):
        assert np.all(got["g_tilde"][t] == 0) and got["loss"][t] == 0
    check_against_oracle(x, g, W, y, "bf16", got)


def test_deterministic(dev):
    c, x, g, W, y = small_case(I.CONFIGS[1], 300, 512, 8192)
    a = run_gpu(x, g, W, y, "bf16", dev, chunk=2048)
    b = run_gpu(x, g, W, y, "bf16", dev, chunk=2048)
    for k in a:
        assert np.array_equal(a[k], b[k]), k


@pytest.mark.slow
@pytest.mark.parametrize("cid", [1, 2, 3])
def test_full_size_sampled_rows(dev, cid):
    """Full workload (bench launch configuration) with oracle rows sampled."""
    c = I.CONFIGS[cid]
    x, g, W, y = I.hidden(c), I.gain(c), I.unembedding(c), I.targets(c)
    got = run_gpu(x, g, W, y, "bf16", dev)
    rows = np.unique(np.concatenate([np.arange(4), np.random.default_rng(cid).choice(c.T, 8, replace=False), [c.T - 1]]))
    ref = O.output_error(x[rows], g, W, y[rows], vocab_chunk=16384)
    for k in ("g_pre", "g_tilde", "lse", "loss"):
        assert_close(k, got[k][rows], ref[k], "bf16")
    assert int(got["bad_targets"][0]) == 0
