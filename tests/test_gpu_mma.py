"""Batched decode on the matrix cores (wsr_decode_sweep_mma): unit activation vectors return the
dequantised weights bit for bit (which pins the decoders, the lane transposes and the operand
orders), every token of a mixed-format sweep matches the oracle and the vector-ALU sweep, outputs
outside the tokens and rows asked for stay untouched, and the full-size models agree on sampled rows."""
import numpy as np
import pytest
import torch

import oracle
import synth
from synth import device as dv
from synth import workloads as wl
from gpu_util import TOL, f32_bits, needs_gpu, rel_l2, stream, zeros_u8

from paper_2608_12114_amd import wsr

pytestmark = [pytest.mark.gpu, needs_gpu]
CODE = {wl.F16: wsr.WSR_F16, wl.BF16: wsr.WSR_BF16, wl.Q4: wsr.WSR_Q4, wl.I8: wsr.WSR_I8}
# K past a whole number of steps (128 elements; 64 for int8) and M past whole 64-row groups
SHAPES = {wl.F16: (100, 520), wl.BF16: (77, 4104), wl.Q4: (100, 2080), wl.I8: (130, 2064)}
# Matrix-core against vector-ALU outputs: both form every product exactly and sum in fp32, in
# different orders, so they differ by fp32 rounding only (worst measured on these seeded inputs:
# 7.5e-6 rel-L2 per matrix, the 8B q4 down projection with K = 14336, whose q4 products enter the
# matrix core as (q + 8) x 2^-24 with the bias as accumulator input; 1e-6 or less for 16-bit and
# int8).
MMA_VS_VALU = 1e-5


def host_matrix(fmt, M, K, seed):
    if fmt == wl.Q4:
        return synth.q4_codes(M, K, seed=seed, stream=601), synth.q4_scales(M, K, seed=seed, stream=602)
    if fmt == wl.I8:
        return synth.i8_codes(M, K, seed=seed, stream=601), synth.i8_scales(M, seed=seed, stream=602)
    return synth.normal16((M, K), wl.W_SIGMA, fmt, seed=seed, stream=601), None


def run_mma(fmt, W, S, X, M, K, T, y_rows=None):
    """X: (tokens, K) fp16/bf16 bits on the host; returns y (tokens_alloc, y_rows) after one call."""
    y_rows = y_rows or M
    w, s, x = dv.to_device(W), (dv.to_device(S) if S is not None else None), dv.to_device(X)
    y = torch.full((X.shape[0], y_rows), float("nan"), dtype=torch.float32, device="cuda")
    mats = wsr.make_mats([dict(fmt=CODE[fmt], M=M, K=K, w=w, scales=s, x=x, x_tok_stride=K * 2, y=y,
                               y_tok_stride=y_rows * 4)])
    ws = zeros_u8(wsr.wsr_sweep_workspace_bytes(mats))
    wsr.wsr_decode_sweep_mma(mats, T, ws, ws.numel(), stream())
    torch.cuda.synchronize()
    return y.cpu().numpy()


@pytest.mark.parametrize("fmt", [wl.F16, wl.BF16, wl.Q4, wl.I8])
def test_mma_unit_vectors_exact(fmt):
    M, K = SHAPES[fmt]
    W, S = host_matrix(fmt, M, K, seed=7)
    xfmt = wl.BF16 if fmt == wl.BF16 else wl.F16
    zero, one = synth.encode16([0.0, 1.0], xfmt)
    cols = [0, 1, 4, 5, 7, 8, 15, 16, 31, 32, 33, 63, 64, 127, 128, K - 1]
    X = np.full((16, K), zero, np.uint16)
    for t, j in enumerate(cols):
        X[t, j] = one
    y = run_mma(fmt, W, S, X, M, K, 16)
    ora = oracle.get()
    for t, j in enumerate(cols):
        if fmt in (wl.Q4, wl.I8):
            want = ora.gemv(dict(fmt=fmt, w=W, s=S), X[t])
        else:
            want = ora.gemv16(W, X[t], fmt)
        assert np.array_equal(f32_bits(y[t]), f32_bits(want)), (fmt, j)


@pytest.mark.parametrize("fmt", [wl.F16, wl.BF16, wl.Q4, wl.I8])
@pytest.mark.parametrize("T", [1, 3, 16, 17, 21])
def test_mma_matrix_parity_and_bounds(fmt, T):
    """T tokens in passes of 16; rows in a strided output (gaps after each token's M rows) and the
    tokens past T stay NaN."""
    M, K = SHAPES[fmt]
    W, S = host_matrix(fmt, M, K, seed=8)
    xfmt = wl.BF16 if fmt == wl.BF16 else wl.F16
    X = synth.normal16((T + 2, K), wl.X_SIGMA, xfmt, seed=8, stream=603)
    y = run_mma(fmt, W, S, X, M, K, T, y_rows=M + 5)
    assert np.isnan(y[:, M:]).all() and np.isnan(y[T:]).all()
    ora = oracle.get()
    for t in range(T):
        want = ora.gemv(dict(fmt=fmt, w=W, s=S), X[t]) if fmt in (wl.Q4, wl.I8) else ora.gemv16(W, X[t], fmt)
        assert rel_l2(y[t, :M], want) <= TOL, (fmt, t)


# groups of 128 rows (eight tiles: 16-bit at any token count, q4 from 8 tokens, int8 from 12) over
# several whole groups and a ragged last one, against four tiles where the token count picks them
GROUPS128 = [(wl.BF16, 300, 1000), (wl.F16, 129, 512), (wl.Q4, 300, 2048), (wl.Q4, 260, 2080), (wl.I8, 300, 1024)]


@pytest.mark.parametrize("fmt,M,K", GROUPS128, ids=lambda v: str(v))
@pytest.mark.parametrize("T", [2, 8, 12, 16])
def test_mma_row_groups_parity_and_bounds(fmt, M, K, T):
    W, S = host_matrix(fmt, M, K, seed=13)
    xfmt = wl.BF16 if fmt == wl.BF16 else wl.F16
    X = synth.normal16((T + 1, K), wl.X_SIGMA, xfmt, seed=13, stream=607)
    y = run_mma(fmt, W, S, X, M, K, T, y_rows=M + 3)
    assert np.isnan(y[:, M:]).all() and np.isnan(y[T:]).all()
    ora = oracle.get()
    for t in range(T):
        want = ora.gemv(dict(fmt=fmt, w=W, s=S), X[t]) if fmt in (wl.Q4, wl.I8) else ora.gemv16(W, X[t], fmt)
        assert rel_l2(y[t, :M], want) <= TOL, (fmt, t)


# q4 rows of a whole number of 8-block steps take their scales in blocks of four steps; rows of 1,
# 2, 3, 5, 6 and 7 steps end in a partial block (one step: every group's only unit carries its
# scales across the next group's block), over several row groups with a ragged last one
@pytest.mark.parametrize("K", [256, 512, 768, 1280, 1536, 1792])
@pytest.mark.parametrize("T", [3, 16])
def test_mma_q4_scale_blocks(K, T):
    M = 150
    W, S = host_matrix(wl.Q4, M, K, seed=14)
    X = synth.normal16((T + 1, K), wl.X_SIGMA, wl.F16, seed=14, stream=608)
    y = run_mma(wl.Q4, W, S, X, M, K, T, y_rows=M + 3)
    assert np.isnan(y[:, M:]).all() and np.isnan(y[T:]).all()
    ora = oracle.get()
    for t in range(T):
        assert rel_l2(y[t, :M], ora.gemv(dict(fmt=wl.Q4, w=W, s=S), X[t])) <= TOL, (K, t)


def sweep_pair(inp, tokens, chained=False):
    """(vector-ALU sweep outputs, matrix-core sweep outputs) for the same inputs."""
    mats = wsr.make_mats(inp.specs(chained=chained))
    ws = zeros_u8(wsr.wsr_sweep_workspace_bytes(mats))
    for y in inp.y:
        y.fill_(float("nan"))
    wsr.wsr_decode_sweep(mats, tokens, ws, ws.numel(), stream())
    torch.cuda.synchronize()
    valu = [y.clone() for y in inp.y]
    for y in inp.y:
        y.fill_(float("nan"))
    wsr.wsr_decode_sweep_mma(mats, tokens, ws, ws.numel(), stream())
    torch.cuda.synchronize()
    return valu, [y.clone() for y in inp.y]


@pytest.mark.parametrize("chained", [False, True], ids=["one_launch", "chained"])
def test_mma_mixed_sweep(chained):
    """Chained: each layer's activation slots depend on earlier outputs, so every pass is several
    launches (one per run of independent matrices)."""
    mats = wl.decode_matrices(dv.small_model(layers=4, d=512, ffn=1536, vocab=3000))
    fmts = [(wl.I8, wl.Q4, wl.BF16, wl.F16, wl.Q4)[m.layer] for m in mats]
    inp = dv.SweepInputs(mats, fmts, tokens=19)
    valu, mma = sweep_pair(inp, 19, chained)
    ora = oracle.get()
    for i, (m, fmt) in enumerate(zip(mats, fmts)):
        a, b = valu[i].cpu().numpy(), mma[i].cpu().numpy()
        for t in range(19):
            assert rel_l2(b[t], a[t]) <= MMA_VS_VALU, (m.name, m.layer, t)
        for t in (0, 15, 16, 18):
            hw = inp.host_weights(i)
            x = inp.host_x(i, t)
            want = ora.gemv(dict(fmt=fmt, w=hw[0], s=hw[1]), x) if fmt in (wl.Q4, wl.I8) else ora.gemv16(hw, x, fmt)
            assert rel_l2(b[t], want) <= TOL, (m.name, m.layer, t)


@pytest.mark.parametrize("name", ["llama3-8b-q4", "llama-70b-bf16", "protocol-i8"])
def test_mma_full_size(name):
    """The full models, 16 tokens in one pass: every matrix against the vector-ALU sweep, and
    sampled rows of every matrix against the oracle for the first and last token."""
    if name == "protocol-i8":
        mats, fmt = wl.protocol_matrices(), wl.I8
    else:
        _, shape, fmt = {"llama3-8b-q4": wl.LLAMA8B_Q4, "llama-70b-bf16": wl.LLAMA70B_BF16}[name]
        mats = wl.decode_matrices(shape)
    inp = dv.SweepInputs(mats, [fmt] * len(mats), tokens=16)
    valu, mma = sweep_pair(inp, 16)
    ora = oracle.get()
    for i, m in enumerate(mats):
        assert rel_l2(mma[i].cpu().numpy(), valu[i].cpu().numpy()) <= MMA_VS_VALU, (m.name, m.layer)
        rows = np.unique(np.linspace(0, m.M - 1, 4).astype(np.int64))
        for t in (0, 15):
            x = inp.host_x(i, t)
            got = mma[i][t].cpu().numpy()[rows]
            want = []
            for r in rows:
                hw = inp.host_weights(i, int(r), 1)
                want.append((ora.gemv(dict(fmt=fmt, w=hw[0], s=hw[1]), x) if fmt in (wl.Q4, wl.I8)
                             else ora.gemv16(hw, x, fmt))[0])
            assert rel_l2(got, np.array(want)) <= TOL, (m.name, m.layer, t)
    del inp, valu, mma
    torch.cuda.empty_cache()


# rows shorter than one step of K (one clamped step: a step is 64 weights of 16-bit rows, 128 of
# int8, 256 of q4), a 16-bit row one step plus a moved-back partial one, and a q4 shape whose
# scales load 8 at a time
SHORT = [(wl.F16, 33, 40), (wl.BF16, 20, 56), (wl.F16, 9, 8), (wl.BF16, 20, 120), (wl.Q4, 40, 96),
         (wl.I8, 50, 48), (wl.I8, 17, 16), (wl.Q4, 70, 4096)]


@pytest.mark.parametrize("fmt,M,K", SHORT, ids=lambda v: str(v))
@pytest.mark.parametrize("T", [1, 7, 16])
def test_mma_short_rows_parity_and_bounds(fmt, M, K, T):
    W, S = host_matrix(fmt, M, K, seed=9)
    xfmt = wl.BF16 if fmt == wl.BF16 else wl.F16
    X = synth.normal16((T + 1, K), wl.X_SIGMA, xfmt, seed=9, stream=604)
    y = run_mma(fmt, W, S, X, M, K, T, y_rows=M + 3)
    assert np.isnan(y[:, M:]).all() and np.isnan(y[T:]).all()
    ora = oracle.get()
    for t in range(T):
        want = ora.gemv(dict(fmt=fmt, w=W, s=S), X[t]) if fmt in (wl.Q4, wl.I8) else ora.gemv16(W, X[t], fmt)
        assert rel_l2(y[t, :M], want) <= TOL, (fmt, t)


@pytest.mark.parametrize("fmt,M,K", SHORT, ids=lambda v: str(v))
def test_mma_short_rows_unit_vectors_exact(fmt, M, K):
    W, S = host_matrix(fmt, M, K, seed=10)
    xfmt = wl.BF16 if fmt == wl.BF16 else wl.F16
    zero, one = synth.encode16([0.0, 1.0], xfmt)
    cols = sorted({0, 1, 7, 8, K // 2, K - 9, K - 1} & set(range(K)))[:16]
    X = np.full((len(cols), K), zero, np.uint16)
    for t, j in enumerate(cols):
        X[t, j] = one
    y = run_mma(fmt, W, S, X, M, K, len(cols))
    ora = oracle.get()
    for t, j in enumerate(cols):
        want = ora.gemv(dict(fmt=fmt, w=W, s=S), X[t]) if fmt in (wl.Q4, wl.I8) else ora.gemv16(W, X[t], fmt)
        assert np.array_equal(f32_bits(y[t]), f32_bits(want)), (fmt, j)


def test_mma_edge_cases():
    """No tokens: rejected (WSR_E_ARG) before anything is enqueued.  An empty matrix (M = 0) inside the table, an activation shared
    by every token (x_tok_stride = 0), and 33 tokens (passes of 16, 16 and 1): every token within
    2e-3 of the oracle, outputs past each token's M rows untouched."""
    ora = oracle.get()
    M, K = 40, 520
    W, _ = host_matrix(wl.F16, M, K, seed=11)
    Wq, Sq = host_matrix(wl.Q4, 24, 2048, seed=12)
    T = 33
    X = synth.normal16((T, K), wl.X_SIGMA, wl.F16, seed=11, stream=605)
    xq = synth.normal16((1, 2048), wl.X_SIGMA, wl.F16, seed=12, stream=606)
    w, x = dv.to_device(W), dv.to_device(X)
    wq, sq, xqd = dv.to_device(Wq), dv.to_device(Sq), dv.to_device(xq)
    y = torch.full((T, M + 2), float("nan"), dtype=torch.float32, device="cuda")
    yq = torch.full((T, 24 + 2), float("nan"), dtype=torch.float32, device="cuda")
    y0 = torch.full((T, 4), float("nan"), dtype=torch.float32, device="cuda")
    mats = wsr.make_mats([
        dict(fmt=wsr.WSR_F16, M=M, K=K, w=w, scales=None, x=x, x_tok_stride=K * 2, y=y, y_tok_stride=(M + 2) * 4),
        dict(fmt=wsr.WSR_BF16, M=0, K=K, w=w, scales=None, x=x, x_tok_stride=K * 2, y=y0, y_tok_stride=16),
        dict(fmt=wsr.WSR_Q4, M=24, K=2048, w=wq, scales=sq, x=xqd, x_tok_stride=0, y=yq, y_tok_stride=26 * 4)])
    ws = zeros_u8(wsr.wsr_sweep_workspace_bytes(mats))
    with pytest.raises(wsr.WsrError) as e:
        wsr.wsr_decode_sweep_mma(mats, 0, ws, ws.numel(), stream())
    assert e.value.status == wsr.WSR_E_ARG
    torch.cuda.synchronize()
    assert torch.isnan(y).all() and torch.isnan(yq).all()
    wsr.wsr_decode_sweep_mma(mats, T, ws, ws.numel(), stream())
    torch.cuda.synchronize()
    a, b = y.cpu().numpy(), yq.cpu().numpy()
    assert np.isnan(a[:, M:]).all() and np.isnan(b[:, 24:]).all() and torch.isnan(y0).all()
    want_q = ora.gemv(dict(fmt=wl.Q4, w=Wq, s=Sq), xq[0])
    for t in range(T):
        assert rel_l2(a[t, :M], ora.gemv16(W, X[t], wl.F16)) <= TOL, t
        assert rel_l2(b[t, :24], want_q) <= TOL, t


def test_mma_q4_extreme_values():
    """q4 codes at both ends of their range, block scales from the smallest fp16 subnormal to the
    largest fp16, activations at +-65504, at the smallest subnormal and mixed: the codes enter the
    matrix cores as fp16 subnormals (q + 8) 2^-24 and the bias leaves through the accumulator
    input, which must neither flush nor overflow.  Every token finite and within 2e-3 of the
    oracle, and every row within the first-order bound of fp32 summation: products are exact, and
    a result passes through at most 33 roundings in a block (32 products and the bias) and one per
    block in the row's running sum, each of a partial sum no larger than the sum of the absolute
    terms, bias terms included (s (|q| + 16) |x| per weight); twice that count of unit roundoffs
    times that sum bounds the error.  Rows here cancel terms near 65504^2 against each other, so a
    relative comparison with the vector-ALU sweep means nothing for them (the two paths differ by
    1.5e-5 rel-L2 on token 5, each within 1.5e-5 of the oracle)."""
    M, K, T = 64, 1024, 16
    rng = np.random.default_rng(21)
    W = synth.q4_codes(M, K, seed=21, stream=611)
    W[:16] = 0x88                                   # every code -8
    W[16:32] = 0x77                                 # every code +7
    svals = synth.encode16([65504.0, 1.0, 2.0 ** -14, 2.0 ** -24, 1e-3], wl.F16)
    S = svals[rng.integers(0, len(svals), size=(M, K // 32))]
    X = synth.normal16((T, K), wl.X_SIGMA, wl.F16, seed=21, stream=612)
    big, nbig, tiny = synth.encode16([65504.0, -65504.0, 2.0 ** -24], wl.F16)
    X[0], X[1], X[2] = big, nbig, tiny
    X[3] = synth.encode16(np.where(np.arange(K) % 2 == 0, 1.0, -1.0), wl.F16)
    for t in range(4, T):
        idx = rng.permutation(K)[: K // 8]
        X[t, idx[: K // 16]] = rng.choice(np.array([big, nbig]), size=K // 16)
        X[t, idx[K // 16:]] = tiny
    y = run_mma(wl.Q4, W, S, X, M, K, T)
    nib = np.stack([W & 0xF, W >> 4], axis=-1).reshape(M, K).astype(np.int64)   # even k low nibble
    q = (nib ^ 8) - 8
    sk = np.repeat(S.view(np.float16).astype(np.float64), 32, axis=1)
    mag = sk * (np.abs(q) + 16)                       # per weight: s (|q| + 16)
    rounds = 2 * (33 + K // 32)
    ora = oracle.get()
    for t in range(T):
        want = ora.gemv(dict(fmt=wl.Q4, w=W, s=S), X[t])
        assert np.isfinite(y[t]).all(), t
        assert rel_l2(y[t], want) <= TOL, t
        bound = rounds * 2.0 ** -24 * (mag @ np.abs(X[t].view(np.float16).astype(np.float64)))
        bound += 2.0 ** -24 * np.abs(want.astype(np.float64))           # the oracle's fp32 result
        assert (np.abs(y[t].astype(np.float64) - want.astype(np.float64)) <= bound).all(), t


def test_mma_mixed_full_size_tail():
    """Four int8 and four bf16 matrices of 12288 x 7168 (1.06 GB), interleaved, 16 tokens: about 1,150
    spans of the largest 64-row group, just past one round of the mixed-format kernel's wave slots,
    so the stream ends in a tail of 16-row groups.  Every matrix against the vector-ALU sweep, and
    sampled rows against the oracle for the first and last token."""
    mats = wl.protocol_matrices(n=8)
    fmts = [wl.I8 if i % 2 == 0 else wl.BF16 for i in range(8)]
    inp = dv.SweepInputs(mats, fmts, tokens=16)
    valu, mma = sweep_pair(inp, 16)
    ora = oracle.get()
    for i, (m, fmt) in enumerate(zip(mats, fmts)):
        assert rel_l2(mma[i].cpu().numpy(), valu[i].cpu().numpy()) <= MMA_VS_VALU, (m.name, fmt)
        rows = np.unique(np.linspace(0, m.M - 1, 4).astype(np.int64))
        for t in (0, 15):
            x = inp.host_x(i, t)
            got = mma[i][t].cpu().numpy()[rows]
            want = []
            for r in rows:
                hw = inp.host_weights(i, int(r), 1)
                want.append((ora.gemv(dict(fmt=fmt, w=hw[0], s=hw[1]), x) if fmt == wl.I8 else ora.gemv16(hw, x, fmt))[0])
            assert rel_l2(got, np.array(want)) <= TOL, (m.name, fmt, t)
    del inp, valu, mma
    torch.cuda.empty_cache()


def test_mma_single_token_passes_equal_the_sweep():
    """A pass of one token (n_tokens = 1, or the last of 17) runs the vector-ALU loop: those outputs
    equal wsr_decode_sweep's bit for bit; the 16-token pass stays within rounding of them."""
    mats = wl.decode_matrices(dv.small_model(layers=3, d=512, ffn=1536, vocab=3000))
    fmts = [(wl.Q4, wl.BF16, wl.I8, wl.F16)[m.layer] for m in mats]
    inp = dv.SweepInputs(mats, fmts, tokens=17)
    valu, mma = sweep_pair(inp, 17)
    for i in range(len(mats)):
        a, b = valu[i].cpu().numpy(), mma[i].cpu().numpy()
        assert np.array_equal(f32_bits(a[16]), f32_bits(b[16])), i
        assert rel_l2(b[:16], a[:16]) <= MMA_VS_VALU, i
    one = dv.SweepInputs([m for m, f in zip(mats, fmts) if f == wl.Q4], [wl.Q4] * 7, tokens=1)
    valu, mma = sweep_pair(one, 1)
    for a, b in zip(valu, mma):
        assert np.array_equal(f32_bits(a.cpu().numpy()), f32_bits(b.cpu().numpy()))
