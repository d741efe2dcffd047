"""GPU parity of the second-order HLA library against the fp64 oracle.

Every call goes through the C ABI (paper_2510_27258_amd.capi via the torch
helpers).  Inputs come from the seeded generator; expected values come from
the oracle only.  Bars: 1e-5 (fp32 inputs) and 2e-3 (bf16 inputs) on the
row-wise relative error max_t ||o_t - ref_t||_inf / ||ref_t||_inf.  The ratio
normalised output is judged on rows whose denominator is well away from zero
(|den_t + eps| >= 0.05 D_t, D_t the sum of |terms| of den_t); its numerator
and denominator are judged separately everywhere.
"""
import ctypes
import sys

import numpy as np
import pytest
import torch

import paper_2510_27258_amd as hla
from paper_2510_27258_amd import capi
from paper_2510_27258_amd import inputs as I
from oracle import hla2 as O
from oracle import native
from tests.helpers import dev, gen, rowwise_err, tol_for

pytestmark = pytest.mark.gpu

ALGOS = [capi.HLA_ALGO_CHUNKED, capi.HLA_ALGO_FUSED]
FUSED_SHAPES = [(64, 64, 64), (32, 32, 32), (64, 32, 32), (32, 64, 64), (64, 64, 32), (64, 32, 64), (64, 128, 128),
                (32, 128, 128)]


def _say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def _oracle(q, k, v, masked, state=None):
    num, den, fin, _ = native.hla2_serial_c(q, k, v, masked=masked, state=state, threads=16)
    return num, den, fin


def _supported(algo, n, d, dv, chunk, code, masked):
    return bool(capi.hla2_algo_supported(algo, n, d, dv, chunk, code, masked))


def _check_forward(B, H, n, d, dv, chunk, dist, masked, normalized, algo, seed=0, eps=1e-6):
    code = I.HLA_BF16 if dist == "unit" else I.HLA_FP32
    if not _supported(algo, n, d, dv, chunk, code, masked):
        return False
    q, k, v, code = gen(B, H, n, d, dv, dist, seed)
    _say(f"case B={B} H={H} n={n} d={d} dv={dv} chunk={chunk} dist={dist} masked={masked} "
         f"normalized={normalized} algo={algo}")
    qd, kd, vd = dev(q, code), dev(k, code), dev(v, code)
    num_ref, den_ref, _ = _oracle(q, k, v, masked)
    tol = tol_for(code)
    num = hla.forward(qd, kd, vd, chunk, masked=masked, normalized=False, algo=algo).cpu().numpy()
    err = rowwise_err(num, num_ref)
    assert err <= tol, f"num row-wise error {err:.3e} > {tol}"
    if normalized:
        out = hla.forward(qd, kd, vd, chunk, masked=masked, normalized=True, eps=eps, algo=algo).cpu().numpy()
        ones = torch.ones(B, H, n, dv, dtype=vd.dtype, device="cuda")
        den = hla.forward(qd, kd, ones, chunk, masked=masked, normalized=False, algo=algo)[..., 0].cpu().numpy()
        D = O.hla2_den_scale(q, k, masked=bool(masked))
        e_den = float((np.abs(den - den_ref) / D).max())
        assert e_den <= tol, f"den error {e_den:.3e} > {tol}"
        good = np.abs(den_ref + eps) >= 0.05 * D
        assert good.mean() > 0.3
        ref = num_ref / (den_ref + eps)[..., None]
        e_out = rowwise_err(out[good], ref[good])
        assert e_out <= tol, f"normalised output error {e_out:.3e} > {tol}"
    return True


@pytest.mark.parametrize("algo", ALGOS)
@pytest.mark.parametrize("shape", [
    (1, 2, 256, 32, 32, 64),      # the small fp32 workload (B1 H2 n256 d32, chunk 64)
    (2, 3, 200, 32, 64, 64),      # d != dv, ragged tail
    (1, 2, 77, 16, 16, 16),
    (1, 1, 1, 16, 16, 16),        # a single token
    (1, 2, 300, 128, 128, 128),
    (1, 2, 130, 64, 128, 32),
    (2, 2, 257, 128, 16, 64),
    (1, 1, 50, 64, 64, 128),      # n < chunk
])
@pytest.mark.parametrize("dist", ["scaled", "unit"])
def test_forward_small(shape, dist, algo):
    B, H, n, d, dv, chunk = shape
    for masked in (1, 0):
        _check_forward(B, H, n, d, dv, chunk, dist, masked, normalized=False, algo=algo)


@pytest.mark.parametrize("algo", ALGOS)
@pytest.mark.parametrize("dist", ["scaled", "unit"])
def test_forward_normalized_small(dist, algo):
    for masked in (1, 0):
        _check_forward(2, 2, 190, 32, 32, 64, dist, masked, normalized=True, algo=algo)


@pytest.mark.parametrize("algo", ALGOS)
def test_forward_every_chunk(algo):
    if algo == capi.HLA_ALGO_FUSED:
        pytest.skip("the fused path has its own shape tests")
    for chunk in (16, 32, 64, 128):
        _check_forward(1, 2, 203, 64, 64, chunk, "unit", 1, normalized=False, algo=algo)


@pytest.mark.parametrize("algo", ALGOS)
def test_bf16_d64_workload_all_heads(algo):
    """B4 H16 n4096 d=dv=64 bf16, chunk 64: the full GPU run against the C
    oracle on every one of the 64 heads."""
    w = I.WORKLOADS["hla2-masked-bf16-B4H16-n4096-d64-C64"]
    if not _supported(algo, w["n"], w["d"], w["dv"], w["chunk"], I.HLA_BF16, 1):
        pytest.skip("algorithm does not cover this shape")
    q, k, v, code = gen(w["B"], w["H"], w["n"], w["d"], w["dv"], w["dist"], w["seed"])
    _say(f"case bf16 B4H16 n4096 d64 full size, all heads, algo={algo}")
    out = hla.forward(dev(q, code), dev(k, code), dev(v, code), w["chunk"], masked=True, algo=algo).cpu().numpy()
    num_ref, _, _ = _oracle(q, k, v, True)
    err = rowwise_err(out, num_ref)
    _say(f"row-wise error over all heads {err:.3e}")
    assert err <= 2e-3


@pytest.mark.parametrize("algo", ALGOS)
def test_bf16_d128_normalized_workload(algo):
    """B2 H32 n16384 d=dv=128 bf16, chunk 128, ratio-normalised.  The
    numerator of every one of the 64 heads against the C oracle; on 16 seeded
    heads the denominator, taken from the normalised launch itself (its den
    output), against the oracle's den scaled by D_t, and the normalised
    output on the rows whose denominator is away from zero."""
    w = I.WORKLOADS["hla2-masked-normalized-bf16-B2H32-n16384-d128-C128"]
    if not _supported(algo, w["n"], w["d"], w["dv"], w["chunk"], I.HLA_BF16, 1):
        pytest.skip("algorithm does not cover this shape")
    B, H, n = w["B"], w["H"], w["n"]
    q, k, v, code = gen(B, H, n, w["d"], w["dv"], w["dist"], w["seed"])
    _say(f"case bf16 B2H32 n16384 d128 normalized full size, algo={algo}")
    qd, kd, vd = dev(q, code), dev(k, code), dev(v, code)
    eps = w["eps"]
    den_d = torch.empty(B, H, n, dtype=torch.float32, device="cuda")
    out = hla.forward(qd, kd, vd, w["chunk"], masked=True, normalized=True, eps=eps, algo=algo,
                      den=den_d).cpu().numpy()
    den = den_d.cpu().numpy()
    num = hla.forward(qd, kd, vd, w["chunk"], masked=True, normalized=False, algo=algo).cpu().numpy()
    num_ref, den_ref, _ = _oracle(q, k, v, True)
    e_num = rowwise_err(num, num_ref)
    _say(f"num over all 64 heads {e_num:.3e}")
    assert e_num <= 2e-3
    sel = sorted(np.random.default_rng(7).choice(B * H, size=16, replace=False).tolist())
    bs, hs = np.array(sel) // H, np.array(sel) % H
    D = O.hla2_den_scale(q[bs, hs], k[bs, hs])
    e_den = float((np.abs(den[bs, hs] - den_ref[bs, hs]) / D).max())
    good = np.abs(den_ref[bs, hs] + eps) >= 0.05 * D
    ref = num_ref[bs, hs] / (den_ref[bs, hs] + eps)[..., None]
    e_out = rowwise_err(out[bs, hs][good], ref[good])
    _say(f"den {e_den:.3e} out {e_out:.3e} on 16 heads; rows kept {good.mean():.3f} "
         f"negative den {float((den_ref[bs, hs] < 0).mean()):.3f}")
    assert e_den <= 2e-3 and e_out <= 2e-3
    # the normalised launch's rows are num / (den + eps) of its own den everywhere
    recon = num / (den + eps)[..., None]
    fin = np.isfinite(recon).all(-1) & (np.abs(den + eps) >= 1e-3)
    assert rowwise_err(out[fin], recon[fin]) <= 1e-5


# ----------------------------------------------------------------- fused path specifics
@pytest.mark.parametrize("shape", FUSED_SHAPES)
def test_fused_shapes(shape):
    C, d, dv = shape
    for (B, H, n) in ((1, 2, 5 * C + 7), (2, 3, 3 * C), (1, 1, C - 3)):
        for normalized in (False, True):
            assert _check_forward(B, H, n, d, dv, C, "unit", 1, normalized, capi.HLA_ALGO_FUSED, seed=n)


@pytest.mark.parametrize("segments", [1, 2, 3, 7, 100])
def test_fused_segment_counts(segments, monkeypatch):
    """The result must not depend on how chunks are grouped into segments."""
    monkeypatch.setenv("HLA_FUSED_SEGMENTS", str(segments))
    assert _check_forward(1, 2, 64 * 9 + 20, 64, 64, 64, "unit", 1, True, capi.HLA_ALGO_FUSED, seed=11)


@pytest.mark.parametrize("segments", [1, 2, 3, 7, 100])
def test_fused_d128_segment_counts(segments, monkeypatch):
    """The d = 128 pipeline (segment 0's output walk beside the summary walks
    of the later segments from a zero state, their brackets and carries, then
    the other segments' output walks from their true carries) must not
    depend on the segment plan either; ragged tail, normalised."""
    monkeypatch.setenv("HLA_FUSED_SEGMENTS", str(segments))
    assert _check_forward(2, 1, 64 * 9 + 20, 128, 128, 128, "unit", 1, True, capi.HLA_ALGO_FUSED, seed=13)


@pytest.mark.parametrize("B,H,n", [
    (1, 1, 64),        # one tile: a single output walk
    (1, 3, 130),       # three one-tile segments
    (2, 5, 777),       # 13 segments of one tile
    (1, 100, 200),     # two walks per head: segments of 1, 2 and 1 tiles
    (3, 50, 300),      # more than 128 heads: a single walk per head
    (1, 40, 2000),     # seven segments, segment 0 shorter than the others
    (4, 16, 640),      # four segments of 2, 3, 3 and 2 tiles
])
def test_fused_d128_plan_sweep(B, H, n):
    """The d = 128 two-pass plan over head counts and lengths that give
    every plan shape (the plan query reports each); normalised, num and den
    against the oracle on every head."""
    assert _check_forward(B, H, n, 128, 128, 128, "unit", 1, True, capi.HLA_ALGO_FUSED, seed=29)


@pytest.mark.parametrize("ratio", ["0.2", "1.0", "2.5"])
def test_fused_d128_first_segment_length(ratio, monkeypatch):
    """Nor on the length of segment 0 against the others (HLA_WS_RATIO), at
    the plan of a 64-head launch; ragged tail, normalised."""
    monkeypatch.setenv("HLA_WS_RATIO", ratio)
    monkeypatch.setenv("HLA_FUSED_SEGMENTS", "5")
    assert _check_forward(1, 2, 64 * 23 + 9, 128, 128, 128, "unit", 1, True, capi.HLA_ALGO_FUSED, seed=19)


def test_fused_d128_pipelines_agree(monkeypatch):
    """The d = 128 forward's two pipelines (every output row written once
    from the true carry, and the earlier walk + carry fix-up, which prefill
    with states still uses) agree to the bf16 bar, num and den."""
    q, k, v, code = gen(2, 3, 64 * 11 + 5, 128, 128, "unit", 17)
    qd, kd, vd = dev(q, code), dev(k, code), dev(v, code)
    res = []
    for legacy in ("0", "1"):
        monkeypatch.setenv("HLA_FUSED_LEGACY", legacy)
        den = torch.empty(2, 3, q.shape[2], device="cuda")
        out = hla.forward(qd, kd, vd, 128, normalized=True, algo=capi.HLA_ALGO_FUSED, den=den)
        num = hla.forward(qd, kd, vd, 128, algo=capi.HLA_ALGO_FUSED)
        res.append((num.cpu().numpy(), den.cpu().numpy(), out.cpu().numpy()))
    (n0, d0, o0), (n1, d1, o1) = res
    assert rowwise_err(n0, n1) <= 2e-3
    D = O.hla2_den_scale(q, k)
    assert float((np.abs(d0 - d1) / D).max()) <= 2e-3


@pytest.mark.parametrize("segments", [3, 14])
def test_fused_d128_legacy_segments(segments, monkeypatch):
    """The d = 128 walk + carry fix-up pipeline at a few segments per head,
    where each walk sums its S prefix from the moment records itself, and at
    more, where a prefix launch forms it; normalised, against the oracle."""
    monkeypatch.setenv("HLA_FUSED_LEGACY", "1")
    monkeypatch.setenv("HLA_FUSED_SEGMENTS", str(segments))
    n = 64 * 13 + 9
    assert capi.hla2_fused_plan(1, 2, n, 128, 128, 128)[0] == segments
    assert _check_forward(1, 2, n, 128, 128, 128, "unit", 1, True, capi.HLA_ALGO_FUSED, seed=23)


def test_fused_long_single_head():
    """One head of 262 144 tokens: 4096 tiles cut into the plan's largest
    segment count (one head), so the longest carry chains and the largest
    moment prefixes; every row against the oracle."""
    assert _check_forward(1, 1, 262144, 64, 64, 64, "unit", 1, False, capi.HLA_ALGO_FUSED, seed=5)


def test_fused_long_single_head_d128():
    """One d = 128 head of 65 536 tokens: 1024 tiles cut into 257 segments of
    the two-pass plan (segment 0 of 3 tiles, 255 of 4 and the last of 1), so
    the longest bracket and carry chains of that plan; every row against the
    oracle.
    (Unnormalised: at this length too few rows' denominators stand clear of
    their cancellation scale for the ratio test.)"""
    assert capi.hla2_fused_plan(1, 1, 65536, 128, 128, 128, tiles=True) == (257, 64, 3, 4)
    assert _check_forward(1, 1, 65536, 128, 128, 128, "unit", 1, False, capi.HLA_ALGO_FUSED, seed=23)


def test_fused_matches_chunked_closely():
    q, k, v, code = gen(2, 4, 1000, 64, 64, "unit", 21)
    qd, kd, vd = dev(q, code), dev(k, code), dev(v, code)
    a = hla.forward(qd, kd, vd, 64, algo=capi.HLA_ALGO_FUSED).cpu().numpy()
    b = hla.forward(qd, kd, vd, 64, algo=capi.HLA_ALGO_CHUNKED).cpu().numpy()
    assert rowwise_err(a, b) <= 2e-3


@pytest.mark.parametrize("d", [64, 128])
def test_fused_chunk128_walks_64_token_tiles(d):
    """chunk=128 is walked in 64-token tiles; the result is the chunk=128 result
    up to rounding (the scan is exact for any chunking)."""
    for (B, H, n) in ((1, 2, 3 * 128 + 50), (2, 1, 128)):
        for normalized in (False, True):
            assert _check_forward(B, H, n, d, d, 128, "unit", 1, normalized, capi.HLA_ALGO_FUSED, seed=n + d)


def test_fused_rejects_unsupported():
    q = torch.zeros(1, 1, 64, 64, dtype=torch.bfloat16, device="cuda")
    with pytest.raises(capi.HLAError) as ei:
        hla.forward(q, q, q, 16, algo=capi.HLA_ALGO_FUSED)
    assert ei.value.code == capi.HLA_ERR_UNSUPPORTED
    qf = torch.zeros(1, 1, 64, 64, device="cuda")
    with pytest.raises(capi.HLAError):
        hla.forward(qf, qf, qf, 64, algo=capi.HLA_ALGO_FUSED)


# ----------------------------------------------------------------- summaries and scan
@pytest.mark.parametrize("dist", ["scaled", "unit"])
def test_chunk_summaries_and_scan(dist):
    B, H, n, d, dv, chunk = 2, 2, 150, 32, 16, 32
    q, k, v, code = gen(B, H, n, d, dv, dist, 3)
    _say(f"case summaries+scan {dist}")
    st = hla.chunk_summaries(dev(q, code), dev(k, code), dev(v, code), chunk)
    ref = O.chunk_summaries(q, k, v, chunk)
    S, C, m, G, h = (x.cpu().numpy() for x in hla.split_state(st, d, dv))
    for got, exp in zip((S, C, m, G, h), ref):
        scale = np.abs(exp).max()
        assert np.abs(got - exp).max() <= 1e-5 * scale
    # scan with an initial state
    init_q, init_k, init_v, _ = gen(B, H, 40, d, dv, dist, 4)
    _, init = O.hla2_serial(init_q, init_k, init_v)
    init_dev = torch.cat([torch.from_numpy(np.ascontiguousarray(x, np.float32)).reshape(B, H, -1) for x in init],
                         dim=-1).cuda()
    prefix, total = hla.scan(st, d, dv, init=init_dev)
    pre_ref, tot_ref = O.exclusive_scan_states(ref)
    pre_ref = tuple(np.stack([O.combine(tuple(x[:, :] for x in init),
                                        tuple(y[:, :, c] for y in pre_ref))[i] for c in range(st.shape[2])],
                             axis=2) for i in range(5))
    tot_ref = O.combine(init, tot_ref)
    for got, exp in zip(hla.split_state(prefix, d, dv), pre_ref):
        got = got.cpu().numpy()
        assert np.abs(got - exp).max() <= 1e-5 * max(np.abs(exp).max(), 1.0)
    for got, exp in zip(hla.split_state(total, d, dv), tot_ref):
        got = got.cpu().numpy()
        assert np.abs(got - exp).max() <= 1e-5 * max(np.abs(exp).max(), 1.0)


@pytest.mark.parametrize("d,dv,chunk", [
    (128, 128, 128),   # Q and V of the chunk exceed LDS: the block-restaging kernel
    (128, 64, 128),
    (64, 64, 128),     # one pass over four 32-token blocks
    (16, 128, 16),     # a single 16-token block (block-restaging kernel)
    (32, 16, 64),
])
def test_chunk_summaries_shapes(d, dv, chunk):
    """Per-chunk summaries (S, C, m, G, h) of both summary kernels against
    the oracle, ragged last chunk."""
    B, H, n = 1, 2, 2 * chunk + 37
    q, k, v, code = gen(B, H, n, d, dv, "scaled", 31)
    _say(f"case summaries d={d} dv={dv} chunk={chunk}")
    st = hla.chunk_summaries(dev(q, code), dev(k, code), dev(v, code), chunk)
    ref = O.chunk_summaries(q, k, v, chunk)
    for got, exp in zip((x.cpu().numpy() for x in hla.split_state(st, d, dv)), ref):
        assert np.abs(got - exp).max() <= 1e-5 * np.abs(exp).max()


@pytest.mark.parametrize("d", [16, 32, 64, 128])
@pytest.mark.parametrize("with_init", [False, True])
def test_scan_square_states(d, with_init):
    """The d == dv scan (row blocks on fp32 MFMA) against sequential (+) in
    fp64 over random records: segment counts around its prefetch depth and
    unroll, three heads (a partial group of eight), with and without an
    initial state.  Random S is not symmetric, so S_c C_acc must use S_c's
    rows as stored."""
    rng = np.random.default_rng(d + 7 * with_init)
    B, H = 1, 3
    F = d * d + 2 * d * d + 2 * d
    for M in (1, 2, 3, 6, 7, 12):
        _say(f"case scan d={d} M={M} init={with_init}")
        x = rng.standard_normal((B, H, M, F)).astype(np.float32)
        init = rng.standard_normal((B, H, F)).astype(np.float32) if with_init else None
        prefix, total = hla.scan(torch.from_numpy(x).cuda(), d, d,
                                 init=torch.from_numpy(init).cuda() if with_init else None)
        parts = [(0, d * d, (d, d)), (d * d, d * d, (d, d)), (2 * d * d, d, (d,)), (2 * d * d + d, d * d, (d, d)),
                 (3 * d * d + d, d, (d,))]
        split = lambda r: tuple(r[..., o:o + c].reshape(r.shape[:-1] + sh).astype(np.float64) for o, c, sh in parts)
        acc = split(init) if with_init else tuple(np.zeros((B, H) + sh) for _, _, sh in parts)
        got_pre, got_tot = prefix.cpu().numpy(), total.cpu().numpy()
        for c in range(M + 1):
            got = split(got_pre[:, :, c]) if c < M else split(got_tot)
            for name, gv, ev in zip("SCmGh", got, acc):
                err = np.abs(gv - ev).max() / max(np.abs(ev).max(), 1.0)
                assert err <= 1e-5, f"M={M} segment {c} {name}: {err:.3e}"
            if c < M:
                acc = O.combine(acc, split(x[:, :, c]))


@pytest.mark.parametrize("d,B,H,M", [(128, 2, 32, 128), (64, 4, 16, 64)])
def test_scan_full_size_sampled_heads(d, B, H, M):
    """The scan at the benchmark's full sizes and launch configuration (8192
    records at d = 128 for B2 H32, 4096 at d = 64 for B4 H16) over seeded
    random records: the prefixes and the total of three heads against a
    sequential (+) in fp64."""
    F = 3 * d * d + 2 * d
    rng = np.random.default_rng(100 + d)
    x = rng.standard_normal((B, H, M, F), dtype=np.float32)
    _say(f"case scan full size d={d} B={B} H={H} M={M}")
    prefix, total = hla.scan(torch.from_numpy(x).cuda(), d, d)
    heads = [0, (B * H) // 2 + 1, B * H - 1]
    idx = torch.tensor(heads, device="cuda")
    got_pre = prefix.reshape(B * H, M, F).index_select(0, idx).cpu().numpy()
    got_tot = total.reshape(B * H, F).index_select(0, idx).cpu().numpy()
    del prefix, total
    parts = [(0, d * d, (d, d)), (d * d, d * d, (d, d)), (2 * d * d, d, (d,)), (2 * d * d + d, d * d, (d, d)),
             (3 * d * d + d, d, (d,))]
    split = lambda r: tuple(r[..., o:o + c].reshape(r.shape[:-1] + sh).astype(np.float64) for o, c, sh in parts)
    for j, hd in enumerate(heads):
        b, h = divmod(hd, H)
        acc = tuple(np.zeros(sh) for _, _, sh in parts)
        for c in range(M + 1):
            got = split(got_pre[j, c]) if c < M else split(got_tot[j])
            for name, gv, ev in zip("SCmGh", got, acc):
                err = np.abs(gv - ev).max() / max(np.abs(ev).max(), 1.0)
                assert err <= 1e-5, f"head {hd} segment {c} {name}: {err:.3e}"
            if c < M:
                acc = O.combine(acc, split(x[b, h, c]))


# ----------------------------------------------------------------- prefill and decode
def _state_to_np(state, d, dv):
    return tuple(x.cpu().numpy().astype(np.float64) for x in hla.split_state(state.export(), d, dv))


def _tdtype(code):
    return torch.bfloat16 if code == I.HLA_BF16 else torch.float32


@pytest.mark.parametrize("dist", ["scaled", "unit"])
@pytest.mark.parametrize("masked,normalized", [(1, 0), (0, 0), (1, 1)])
def test_prefill_then_steps(dist, masked, normalized):
    B, H, d, dv, n1, steps, chunk = 2, 3, 32, 64, 100, 20, 32
    q, k, v, code = gen(B, H, n1 + steps, d, dv, dist, 5)
    _say(f"case prefill+steps {dist} masked={masked} normalized={normalized}")
    eps = 0.5 if normalized else 1e-6
    num_ref, den_ref, fin_ref = _oracle(q, k, v, masked)
    ref = num_ref / (den_ref + eps)[..., None] if normalized else num_ref
    state = hla.State(B, H, d, dv, masked=bool(masked), normalized=bool(normalized), eps=eps, dtype=_tdtype(code))
    out1 = hla.prefill(state, dev(q[:, :, :n1], code), dev(k[:, :, :n1], code), dev(v[:, :, :n1], code),
                       chunk).cpu().numpy()
    outs = [out1]
    for t in range(n1, n1 + steps):
        o = hla.step(state, dev(q[:, :, t], code), dev(k[:, :, t], code), dev(v[:, :, t], code))
        outs.append(o.cpu().numpy()[:, :, None])
    got = np.concatenate(outs, axis=2)
    if normalized:
        good = np.abs(den_ref + eps) >= 0.05 * O.hla2_den_scale(q, k, masked=bool(masked))
        assert rowwise_err(got[good], ref[good]) <= 1e-4
    else:
        assert rowwise_err(got, ref) <= 1e-5
    for g, e in zip(_state_to_np(state, d, dv), fin_ref):
        assert np.abs(g - e).max() <= 1e-5 * np.abs(e).max()


@pytest.mark.parametrize("d,chunk", [(64, 64), (128, 128)])
@pytest.mark.parametrize("normalized", [0, 1])
def test_prefill_chain_fused_shape(normalized, d, chunk):
    """Two chained prefills on a shape the fused path covers (init state in,
    total state out), then decode steps; all against one serial oracle run."""
    B, H, dv = 2, 3, d
    n1, n2, steps = 5 * 64 + 9, 7 * 64 + 40, 6
    q, k, v, code = gen(B, H, n1 + n2 + steps, d, dv, "unit", 31)
    assert _supported(capi.HLA_ALGO_FUSED, n1, d, dv, chunk, code, 1)
    _say(f"case fused-shape prefill chain d={d} chunk={chunk} normalized={normalized}")
    eps = 0.5 if normalized else 1e-6
    num_ref, den_ref, fin_ref = _oracle(q, k, v, True)
    ref = num_ref / (den_ref + eps)[..., None] if normalized else num_ref
    state = hla.State(B, H, d, dv, masked=True, normalized=bool(normalized), eps=eps, dtype=_tdtype(code))
    outs = []
    for a, b in ((0, n1), (n1, n1 + n2)):
        outs.append(hla.prefill(state, dev(q[:, :, a:b], code), dev(k[:, :, a:b], code), dev(v[:, :, a:b], code),
                                chunk).cpu().numpy())
    for t in range(n1 + n2, n1 + n2 + steps):
        outs.append(hla.step(state, dev(q[:, :, t], code), dev(k[:, :, t], code),
                             dev(v[:, :, t], code)).cpu().numpy()[:, :, None])
    got = np.concatenate(outs, axis=2)
    if normalized:
        good = np.abs(den_ref + eps) >= 0.05 * O.hla2_den_scale(q, k)
        assert rowwise_err(got[good], ref[good]) <= 2e-3
    else:
        assert rowwise_err(got, ref) <= 2e-3
    for g, e in zip(_state_to_np(state, d, dv), fin_ref):
        assert np.abs(g - e).max() <= 1e-4 * np.abs(e).max()


def test_decode_workload_sampled_heads():
    """B64 H32 d=dv=128: prefill 2048 bf16 tokens, then 1024 steps; 16 sampled
    heads vs the oracle over all 3072 tokens, including the final states."""
    w = I.WORKLOADS["hla2-decode-bf16-B64H32-d128-prefix2048-steps1024"]
    B, H, d, dv = w["B"], w["H"], w["d"], w["dv"]
    q, k, v, code = gen(B, H, w["n"], d, dv, w["dist"], w["seed"])
    qs, ks, vs, _ = gen(B, H, w["steps"], d, dv, w["dist"], w["step_seed"])
    _say("case decode B64 H32 d128 prefix 2048 + 1024 steps")
    rng = np.random.default_rng(123)
    sel = sorted(rng.choice(B * H, size=16, replace=False).tolist())
    bsel, hsel = np.array(sel) // H, np.array(sel) % H
    bsel_d, hsel_d = torch.as_tensor(bsel, device="cuda"), torch.as_tensor(hsel, device="cuda")
    state = hla.State(B, H, d, dv, dtype=_tdtype(code))
    hla.prefill(state, dev(q, code), dev(k, code), dev(v, code), w["chunk"], want_out=False)
    qsd, ksd, vsd = dev(qs, code), dev(ks, code), dev(vs, code)
    got = []
    for t in range(w["steps"]):
        o = hla.step(state, qsd[:, :, t].contiguous(), ksd[:, :, t].contiguous(), vsd[:, :, t].contiguous())
        got.append(o[bsel_d, hsel_d])
    got = torch.stack(got, dim=1).cpu().numpy()
    qa = np.concatenate([q[bsel, hsel], qs[bsel, hsel]], axis=1)
    ka = np.concatenate([k[bsel, hsel], ks[bsel, hsel]], axis=1)
    va = np.concatenate([v[bsel, hsel], vs[bsel, hsel]], axis=1)
    num_ref, _, fin_ref = _oracle(qa, ka, va, True)
    err = rowwise_err(got, num_ref[:, w["n"]:])
    _say(f"decode row-wise error {err:.3e}")
    assert err <= 2e-3
    for g, e in zip(_state_to_np(state, d, dv), fin_ref):
        g = g[bsel, hsel]
        assert np.abs(g - e).max() <= 2e-3 * np.abs(e).max()


# ----------------------------------------------------------------- ABI behaviour
def test_abi_errors_leave_outputs_untouched():
    q = torch.zeros(1, 1, 8, 16, device="cuda")
    out = torch.full((1, 1, 8, 16), 7.0, device="cuda")
    ws = torch.empty(1 << 20, dtype=torch.uint8, device="cuda")
    s = torch.cuda.current_stream().cuda_stream
    L = capi.lib()
    rc = L.hla2_forward(q.data_ptr(), q.data_ptr(), q.data_ptr(), out.data_ptr(), 1, 1, 8, 24, 16, 16, 1, 0,
                        1e-6, 0, ws.data_ptr(), ws.numel(), s)
    assert rc == capi.HLA_ERR_UNSUPPORTED and "d and dv" in capi.hla_last_error()
    rc = L.hla2_forward(None, q.data_ptr(), q.data_ptr(), out.data_ptr(), 1, 1, 8, 16, 16, 16, 1, 0, 1e-6, 0,
                        ws.data_ptr(), ws.numel(), s)
    assert rc == capi.HLA_ERR_INVALID
    rc = L.hla2_forward(q.data_ptr(), q.data_ptr(), q.data_ptr(), out.data_ptr(), 1, 1, 8, 16, 16, 16, 1, 0, 1e-6,
                        0, ws.data_ptr(), 16, s)
    assert rc == capi.HLA_ERR_WORKSPACE
    rc = L.hla2_forward(q.data_ptr(), q.data_ptr(), q.data_ptr(), out.data_ptr(), 1, 1, 8, 16, 16, 16, 2, 0, 1e-6,
                        0, ws.data_ptr(), ws.numel(), s)
    assert rc == capi.HLA_ERR_INVALID
    rc = L.hla2_forward(q.data_ptr(), q.data_ptr(), q.data_ptr(), out.data_ptr(), 1, 1, 8, 16, 16, 16, 1, 0,
                        float("nan"), 0, ws.data_ptr(), ws.numel(), s)
    assert rc == capi.HLA_ERR_INVALID
    rc = L.hla2_forward(q.data_ptr() + 4, q.data_ptr(), q.data_ptr(), out.data_ptr(), 1, 1, 8, 16, 16, 16, 1, 0,
                        1e-6, 0, ws.data_ptr(), ws.numel(), s)
    assert rc == capi.HLA_ERR_INVALID
    torch.cuda.synchronize()
    assert bool((out == 7.0).all())


def test_deterministic():
    q, k, v, code = gen(1, 4, 500, 64, 64, "unit", 9)
    qd, kd, vd = dev(q, code), dev(k, code), dev(v, code)
    for algo in ALGOS:
        a = hla.forward(qd, kd, vd, 64, algo=algo)
        b = hla.forward(qd, kd, vd, 64, algo=algo)
        assert torch.equal(a, b)


def _packed_s_from_full(S):
    """The decode state's packed S as include/hla.h describes it, from a full
    [..., d, d] S: for p < d/2, row p from column p, then row d-1-p from
    column d-1-p."""
    d = S.shape[-1]
    parts = []
    for p in range(d // 2):
        parts += [S[..., p, p:], S[..., d - 1 - p, d - 1 - p:]]
    return np.concatenate(parts, axis=-1)


@pytest.mark.parametrize("d,dv", [(16, 32), (64, 64), (128, 128)])
def test_state_packed_layout(d, dv):
    """The state buffer holds S's upper triangle in the documented folded
    order (d(d+1)/2 floats), then C, m, G, h; hla2_state_export gives the full
    records with S symmetric, equal to the oracle's state after the same
    tokens (prefill, then steps)."""
    B, H, n = 1, 3, 40
    q, k, v, code = gen(B, H, n + 2, d, dv, "unit", 43 + d)
    _say(f"case packed state layout d={d} dv={dv}")
    st = hla.State(B, H, d, dv, dtype=torch.bfloat16)
    hla.prefill(st, dev(q[:, :, :n], code), dev(k[:, :, :n], code), dev(v[:, :, :n], code), 32, want_out=False)
    for t in (n, n + 1):
        hla.step(st, dev(q[:, :, t], code), dev(k[:, :, t], code), dev(v[:, :, t], code))
    full = st.export().cpu().numpy()
    raw = st.data.cpu().numpy()
    nS = d * (d + 1) // 2
    assert raw.shape[-1] == nS + 2 * d * dv + 2 * d
    S = full[..., :d * d].reshape(B, H, d, d)
    assert np.array_equal(S, np.swapaxes(S, -1, -2))
    assert np.array_equal(raw[..., :nS], _packed_s_from_full(S))
    assert np.array_equal(raw[..., nS:], full[..., d * d:])
    _, _, fin_ref = _oracle(q, k, v, True)
    for g, e in zip(_state_to_np(st, d, dv), fin_ref):
        assert np.abs(g - e).max() / max(np.abs(e).max(), 1.0) <= 2e-3


def test_state_descriptor_fixes_the_operator():
    """hla2_state_init zeroes the caller's buffer (the identity segment) and
    fixes the operator: a descriptor edited after init (a prefill with one
    flag, then a step with another) is rejected through the C ABI before
    anything is enqueued, and the state is left as the prefill made it."""
    B, H, d, dv, n = 1, 2, 32, 32, 70
    q, k, v, code = gen(B, H, n + 1, d, dv, "unit", 41)
    _say("case state descriptor checks")
    st = hla.State(B, H, d, dv, masked=True, normalized=False, dtype=torch.bfloat16)
    st.data.fill_(3.0)
    L = capi.lib()
    nbytes = capi.hla2_state_bytes(B, H, d, dv)
    assert L.hla2_state_init(ctypes.byref(st.desc), st.data.data_ptr(), nbytes, B, H, d, dv, 1, 0,
                             ctypes.c_float(1e-6), capi.HLA_BF16, torch.cuda.current_stream().cuda_stream) == 0
    torch.cuda.synchronize()
    assert bool((st.data == 0).all())
    hla.prefill(st, dev(q[:, :, :n], code), dev(k[:, :, :n], code), dev(v[:, :, :n], code), 32, want_out=False)
    torch.cuda.synchronize()
    before = st.data.clone()
    qt, kt, vt = (dev(x[:, :, n], code) for x in (q, k, v))
    out = torch.empty(B, H, dv, device="cuda")
    s = torch.cuda.current_stream().cuda_stream
    st.desc.masked = 0
    rc = L.hla2_step(ctypes.byref(st.desc), qt.data_ptr(), kt.data_ptr(), vt.data_ptr(), out.data_ptr(), s)
    assert rc == capi.HLA_ERR_INVALID and "changed" in capi.hla_last_error()
    st.desc.masked = 1
    st.desc.eps = 0.5
    rc = L.hla2_step(ctypes.byref(st.desc), qt.data_ptr(), kt.data_ptr(), vt.data_ptr(), out.data_ptr(), s)
    assert rc == capi.HLA_ERR_INVALID
    torch.cuda.synchronize()
    assert torch.equal(st.data, before)
    st.desc.eps = 1e-6
    got = hla.step(st, qt, kt, vt).cpu().numpy()
    num_ref, _, _ = _oracle(q, k, v, True)
    assert rowwise_err(got, num_ref[:, :, n]) <= 2e-3
    with pytest.raises(ValueError):
        hla.step(st, qt.float(), kt.float(), vt.float())
