"""Decode weight sweep on the GPU against the oracle, plus its structural properties: the fused,
chained and per-matrix paths give bitwise-identical outputs, and every token reads its own
activation and writes its own outputs."""
import numpy as np
import pytest
import torch

import oracle
from synth import device as dv
from synth import workloads as wl
from gpu_util import TOL, f32_bits, needs_gpu, rel_l2, stream, zeros_u8

from paper_2608_12114_amd import wsr

pytestmark = [pytest.mark.gpu, needs_gpu]


def run_sweep(inp, tokens, chained=False):
    for y in inp.y:
        y.fill_(float("nan"))
    mats = wsr.make_mats(inp.specs(chained=chained))
    ws = zeros_u8(wsr.wsr_sweep_workspace_bytes(mats))
    wsr.wsr_decode_sweep(mats, tokens, ws, ws.numel(), stream())
    torch.cuda.synchronize()
    return [y.cpu().numpy().copy() for y in inp.y]


def oracle_y(inp, i, t, rows=None):
    ora = oracle.get()
    fmt = inp.fmts[i]
    x = inp.host_x(i, t)
    if rows is None:
        hw = inp.host_weights(i)
        return ora.gemv_q4(*hw, x, threads=8) if fmt == wl.Q4 else ora.gemv16(hw, x, fmt, threads=8)
    out = []
    for r in rows:
        hw = inp.host_weights(i, int(r), 1)
        out.append((ora.gemv_q4(*hw, x) if fmt == wl.Q4 else ora.gemv16(hw, x, fmt))[0])
    return np.array(out)


@pytest.fixture(scope="module")
def mixed():
    mats = wl.decode_matrices(dv.small_model(layers=3, d=512, ffn=1536, vocab=4000))
    fmts = [(wl.Q4, wl.BF16, wl.F16, wl.BF16)[m.layer] for m in mats]
    return dv.SweepInputs(mats, fmts, tokens=3)


def test_sweep_mixed_parity(mixed):
    ys = run_sweep(mixed, 3)
    for i in range(len(mixed.mats)):
        for t in range(3):
            assert rel_l2(ys[i][t], oracle_y(mixed, i, t)) <= TOL, (i, t)


def test_sweep_arena_layout_bitwise_identical(mixed):
    """Weights and scales as views into one device buffer (the benchmark's layout) give the same
    outputs, bit for bit, as one allocation per tensor; int8 matrices included."""
    mats = list(mixed.mats)
    fmts = [(wl.Q4, wl.BF16, wl.I8, wl.F16)[m.layer] for m in mats]
    own = dv.SweepInputs(mats, fmts, tokens=3)
    one = dv.SweepInputs(mats, fmts, tokens=3, arena=True)
    assert all(w.data_ptr() % (2 << 20) == 0 for w in one.w)
    assert one.w[0].data_ptr() == one.arena.data_ptr()
    for a, b in zip(run_sweep(own, 3), run_sweep(one, 3)):
        assert np.array_equal(f32_bits(a), f32_bits(b))


def test_sweep_paths_bitwise_identical(mixed):
    fused = run_sweep(mixed, 3)
    chained = run_sweep(mixed, 3, chained=True)
    for a, b in zip(fused, chained):
        assert np.array_equal(f32_bits(a), f32_bits(b))
    # the standalone GEMVs of each matrix and token give the same bits
    for i, (m, fmt) in enumerate(zip(mixed.mats, mixed.fmts)):
        xt, _ = mixed.x[(m.layer, m.slot)]
        for t in (0, 2):
            y = torch.empty(m.M, dtype=torch.float32, device="cuda")
            if fmt == wl.Q4:
                wsr.wsr_gemv_q4(mixed.w[i], mixed.s[i], xt[t], y, m.M, m.K, stream())
            else:
                wsr.wsr_gemv_f16(mixed.w[i], xt[t], y, m.M, m.K, dv.WSR_FMT[fmt], stream())
            assert np.array_equal(f32_bits(y.cpu().numpy()), f32_bits(fused[i][t])), (i, t)


def test_sweep_same_activation_every_token(mixed):
    specs = mixed.specs()
    for s in specs:
        s["x_tok_stride"] = 0
    for y in mixed.y:
        y.fill_(float("nan"))
    mats = wsr.make_mats(specs)
    ws = zeros_u8(wsr.wsr_sweep_workspace_bytes(mats))
    wsr.wsr_decode_sweep(mats, 3, ws, ws.numel(), stream())
    for y in mixed.y:
        a = y.cpu().numpy()
        assert np.array_equal(f32_bits(a[0]), f32_bits(a[1])) and np.array_equal(f32_bits(a[0]), f32_bits(a[2]))


@pytest.mark.parametrize("layers,d,ffn", [(1, 64, 96), (2, 128, 4160)])
@pytest.mark.parametrize("fmt", [wl.Q4, wl.BF16])
def test_sweep_ragged_shapes(layers, d, ffn, fmt):
    """Shapes whose rows do not fill whole 64-lane steps, one and several layers."""
    mats = wl.decode_matrices(dv.small_model(layers=layers, d=d, ffn=ffn, vocab=333, n_q=2, n_kv=1,
                                             head_dim=32 if d == 64 else 64))
    inp = dv.SweepInputs(mats, [fmt] * len(mats), tokens=2)
    ys = run_sweep(inp, 2)
    for i in range(len(mats)):
        for t in range(2):
            assert rel_l2(ys[i][t], oracle_y(inp, i, t)) <= TOL, (i, t)


def _check_sampled(inp, tokens, nrows=6):
    """Sampled rows (first, last, spread) of every matrix against the oracle, row by row."""
    worst = 0.0
    for i, m in enumerate(inp.mats):
        rows = np.unique(np.linspace(0, m.M - 1, nrows).astype(np.int64))
        ys = inp.y[i][tokens].cpu().numpy()
        for t_i, t in enumerate(tokens):
            got = ys[t_i][rows]
            want = oracle_y(inp, i, t, rows)
            err = rel_l2(got, want)
            assert err <= TOL, (m.layer, m.name, t, err)
            worst = max(worst, err)
    return worst


@pytest.mark.parametrize("name", ["llama3-8b-q4", "llama-70b-bf16"])
def test_sweep_full_size(name):
    """The decode sweeps at their full shapes, in the launch configuration bench.py times: every
    matrix checked on sampled rows for the first and last of four tokens."""
    _, shape, fmt = {"llama3-8b-q4": wl.LLAMA8B_Q4, "llama-70b-bf16": wl.LLAMA70B_BF16}[name]
    mats = wl.decode_matrices(shape)
    inp = dv.SweepInputs(mats, [fmt] * len(mats), tokens=4)
    assert inp.weight_bytes() == wl.bytes_per_token(shape, fmt)
    ys = run_sweep(inp, 4)
    del ys
    _check_sampled(inp, [0, 3])
    del inp
    torch.cuda.empty_cache()


@pytest.mark.parametrize("n", [32, 33, 288, 289])
@pytest.mark.parametrize("fmt", [wl.BF16, wl.Q4, wl.I8])
def test_sweep_table_sizes(n, fmt):
    """Tables on both sides of the by-value limits of a span-scheduled sweep (up to 32 and up to 288
    matrices carried in the launch arguments, more read from the workspace): every matrix, with
    ragged row counts, against the oracle for both tokens and bit for bit against its standalone
    GEMV."""
    K = 512
    mats = [wl.Mat(i, f"m{i}", i, 1 + (37 * i) % 70, K, "attn") for i in range(n)]
    inp = dv.SweepInputs(mats, [fmt] * n, tokens=2)
    ys = run_sweep(inp, 2)
    ora = oracle.get()
    gemv = {wl.BF16: None, wl.Q4: wsr.wsr_gemv_q4, wl.I8: wsr.wsr_gemv_i8}[fmt]
    for i, m in enumerate(mats):
        hw = inp.host_weights(i)
        xt, _ = inp.x[(m.layer, m.slot)]
        for t in range(2):
            x = inp.host_x(i, t)
            want = ora.gemv(dict(fmt=fmt, w=hw[0], s=hw[1]), x) if fmt in (wl.Q4, wl.I8) else ora.gemv16(hw, x, fmt)
            assert rel_l2(ys[i][t], want) <= TOL, (n, i, t)
        y = torch.empty(m.M, dtype=torch.float32, device="cuda")
        if gemv is None:
            wsr.wsr_gemv_f16(inp.w[i], xt[1], y, m.M, K, wsr.WSR_BF16, stream())
        else:
            gemv(inp.w[i], inp.s[i], xt[1], y, m.M, K, stream())
        assert np.array_equal(f32_bits(y.cpu().numpy()), f32_bits(ys[i][1])), (n, i)
