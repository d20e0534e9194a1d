"""Workload recipes: the shapes, distributions and stream ids of every synthetic input.

A decode sweep reads every projection matrix of every layer once per token, then the output head
(paper Sec. 6.2, RQ1, matched dense model: a batch-1 token reads the model's full weight set, and
the logical rate is tokens/s times the bytes read per token).  The byte count per token covers projections, the head and any scales, and
excludes the embedding table, of which a token gathers a single row; with that rule the int8
Qwen2.5-72B shape the paper evaluates reads 71.48 GB per token, the figure the paper prints.

Activations are independent synthetic vectors, one per (layer, input slot, token): q, k and v
share the attention input, o has its own, gate and up share the MLP input, down has its own, and
the head reads the final hidden state.  No attention or normalisation runs between them.
"""
from __future__ import annotations

from dataclasses import dataclass, field

# storage formats of a weight matrix
F16, BF16, Q4, I8 = "f16", "bf16", "q4", "i8"      # i8: int8 codes with one fp16 scale per row

# Distribution parameters of the synthetic inputs.
W_SIGMA = 0.02          # 16-bit weights ~ N(0, 0.02), 0.02 the standard deviation
X_SIGMA = 1.0           # activations ~ N(0, 1)
Q4_SCALE_LO, Q4_SCALE_HI = 0.005, 0.02   # q4 block scales ~ U[0.005, 0.02], rounded to fp16
Q4_BLOCK = 32
SEED = 0

# Stream-id layout: weights, q4 scales and activations of matrix m never share a stream.
def w_stream(m: int) -> int:
    return m + 1


def s_stream(m: int) -> int:
    return (1 << 20) + m + 1


def x_stream(layer: int, slot: int) -> int:
    return (2 << 20) + layer * 8 + slot


X_SLOTS = {"attn": 0, "o": 1, "mlp": 2, "down": 3, "head": 4}


@dataclass(frozen=True)
class ModelShape:
    name: str
    layers: int
    d: int
    n_q: int
    n_kv: int
    head_dim: int
    ffn: int
    vocab: int


LLAMA3_8B = ModelShape("llama3-8b", 32, 4096, 32, 8, 128, 14336, 128256)
LLAMA_70B = ModelShape("llama-70b", 80, 8192, 64, 8, 128, 28672, 128256)
# Shape of the dense model of the paper's matched decode evaluation (used for byte accounting).
QWEN25_72B = ModelShape("qwen2.5-72b", 80, 8192, 64, 8, 128, 29568, 152064)


@dataclass(frozen=True)
class Mat:
    index: int          # position in the per-token sweep order
    name: str
    layer: int          # == model.layers for the head
    M: int              # output rows
    K: int              # reduction length
    slot: str           # activation slot feeding it


def decode_matrices(m: ModelShape) -> list[Mat]:
    """Every matrix a batch-1 decode token reads, in layer order: q, k, v, o, gate, up, down; head last."""
    out: list[Mat] = []
    qd, kvd = m.n_q * m.head_dim, m.n_kv * m.head_dim
    for l in range(m.layers):
        for name, M, K, slot in (("q", qd, m.d, "attn"), ("k", kvd, m.d, "attn"),
                                 ("v", kvd, m.d, "attn"), ("o", m.d, qd, "o"),
                                 ("gate", m.ffn, m.d, "mlp"), ("up", m.ffn, m.d, "mlp"),
                                 ("down", m.d, m.ffn, "down")):
            out.append(Mat(len(out), name, l, M, K, slot))
    out.append(Mat(len(out), "lm_head", m.layers, m.vocab, m.d, "head"))
    return out


def matrix_bytes(M: int, K: int, fmt: str) -> int:
    """Bytes one read of the matrix streams: weights plus their scales."""
    if fmt in (F16, BF16):
        return M * K * 2
    if fmt == Q4:
        assert K % Q4_BLOCK == 0
        return M * K // 2 + M * (K // Q4_BLOCK) * 2
    if fmt == I8:
        return M * K + M * 2
    raise ValueError(fmt)


def bytes_per_token(m: ModelShape, fmt: str, extra_vectors: int = 0) -> int:
    """Weight (+ scale) bytes one decode token reads; extra_vectors adds fp16 per-layer vectors
    of length d (biases, norms) when a model has them."""
    b = sum(matrix_bytes(x.M, x.K, fmt) for x in decode_matrices(m))
    return b + extra_vectors * 2


def embedding_bytes(m: ModelShape, fmt: str) -> int:
    per = {F16: 2, BF16: 2, Q4: 0.5625, I8: 1}[fmt]
    return int(m.vocab * m.d * per)


def footprint_bytes(m: ModelShape, fmt: str) -> int:
    return bytes_per_token(m, fmt) + embedding_bytes(m, fmt)


# ---- the standalone configurations --------------------------------------------------------------

@dataclass(frozen=True)
class GemvConfig:
    M: int = 4096
    K: int = 4096
    fmt: str = F16
    rotate: int = 32    # distinct W buffers visited per pass (1 GiB at 32 MiB each)


PROBE_N = 1 << 28       # fp32 elements: 1 GiB

# bf16 size sweep with reduction length 4096 and N output rows: 2 MiB ... 1100 MiB, covering the
# stated 576 MiB point (N = 73728) and the largest stated column count (N = 140800).
SWEEP_K = 4096
SWEEP_N = (256, 512, 1024, 2048, 4096, 8192, 16384, 32768, 65536, 73728, 131072, 140800)


@dataclass
class SweepSpec:
    model: ModelShape
    fmt: str
    tokens: int
    mats: list = field(default_factory=list)

    def __post_init__(self):
        if not self.mats:
            self.mats = decode_matrices(self.model)


LLAMA8B_Q4 = ("llama3-8b-q4", LLAMA3_8B, Q4)
LLAMA70B_BF16 = ("llama-70b-bf16", LLAMA_70B, BF16)

# The matched protocol of Sec. 3.1 (Table 2): a single-token int8 GEMV with fp16 row scales over a
# 12288 x 7168 matrix (88.1 MB with its scales), a pass visiting 12 such matrices.  Each matrix has
# its own weights and its own activation vector.
PROTOCOL_M, PROTOCOL_K, PROTOCOL_MATRICES = 12288, 7168, 12


def protocol_matrices(n: int = PROTOCOL_MATRICES, M: int = PROTOCOL_M, K: int = PROTOCOL_K) -> list[Mat]:
    return [Mat(i, f"w{i}", i, M, K, "attn") for i in range(n)]
