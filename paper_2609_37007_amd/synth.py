"""Seeded synthetic inputs: the weight blob, frame inputs and pre-drawn uniforms.

This module holds data generation only -- no part of the model or of the
speculative decoding rule.  The same bytes feed the GPU library and the CPU
oracle, so both sides see bit-identical weights and uniforms.

Weight blob layout (little endian, no padding between tensors)::

    header, 64 bytes:
        char[8]  magic "RVQSDW1\\0"
        u32      version (1)
        u32      dtype of the matrices: 0 = float32, 1 = bfloat16
        u32 x 9  n_layers, hidden, n_q_heads, n_kv_heads, head_dim, ffn,
                 n_codes, vocab, max_draft
        u32 x 3  reserved (0)
    for each layer:
        attn_norm f32[H]
        Wq  [nq*d][H]   Wk [nkv*d][H]   Wv [nkv*d][H]      (matrix dtype)
        q_norm f32[d]   k_norm f32[d]
        Wo  [H][nq*d]
        mlp_norm f32[H]
        Wgate [F][H]    Wup [F][H]      Wdown [H][F]
    final_norm f32[H]
    E_0 .. E_{n_codes-1}      [V][H]   (E_i embeds code c_i)
    LMH_1 .. LMH_{n_codes}    [V][H]   (LMH_s emits code c_s)
    b_1 .. b_{max_draft}      f32[H]   (position-aware draft offsets)

All matrices are [out][in] row-major.  With dtype 2 (int8, the W8A16 weights of
Sec. 3.4) every matrix is stored as int8 codes q [out][in] followed by its fp32
per-row (output channel) scales s [out], then zero bytes up to the next 16-byte
boundary; the weight is s[o] * q[o][i]: s = max_i |w[o][i]| / 127 (fp32, computed
in fp64), q = round-half-even(w / s) in [-127, 127], w being the fp32 value the
other dtypes store (a row of zeros has s = 0 and q = 0).  Values: N(0, std) from
``numpy.random.default_rng(seed).standard_normal`` drawn tensor by tensor in
the order above (norm gains are 1.0 and draw nothing); the LM heads are
multiplied by ``head_scale`` before rounding; the offsets are drawn last (N(0,
offset_std)).  Matrices are rounded float64 -> float32 (round to nearest even)
and, for bfloat16, float32 -> bfloat16 (round to nearest even).
"""
from __future__ import annotations

import dataclasses
import struct

import numpy as np

MAGIC = b"RVQSDW1\0"
VERSION = 1
DTYPE_F32 = 0
DTYPE_BF16 = 1
DTYPE_I8 = 2
HEADER_BYTES = 64


@dataclasses.dataclass(frozen=True)
class ModelShape:
    n_layers: int
    hidden: int
    n_q_heads: int
    n_kv_heads: int
    head_dim: int
    ffn: int
    n_codes: int
    vocab: int
    max_draft: int
    dtype: int  # DTYPE_F32 or DTYPE_BF16

    @property
    def q_dim(self) -> int:
        return self.n_q_heads * self.head_dim

    @property
    def kv_dim(self) -> int:
        return self.n_kv_heads * self.head_dim


# The tiny 2-layer fp32 model (hidden 256, 4 heads of 64, FFN 512, 64 codes).
TINY = ModelShape(n_layers=2, hidden=256, n_q_heads=4, n_kv_heads=4, head_dim=64,
                  ffn=512, n_codes=15, vocab=64, max_draft=14, dtype=DTYPE_F32)
# The Qwen3-TTS-0.6B-shaped MultiCodeDecoder (5 layers, hidden 1024, GQA 16/8 x 128,
# FFN 3072, codebook 2048, bf16 weights).
MCD_1024 = ModelShape(n_layers=5, hidden=1024, n_q_heads=16, n_kv_heads=8, head_dim=128,
                      ffn=3072, n_codes=15, vocab=2048, max_draft=14, dtype=DTYPE_BF16)
# The same model with W8A16 weights (int8 per output channel), the precision of Sec. 3.4.
MCD_1024_W8 = ModelShape(n_layers=5, hidden=1024, n_q_heads=16, n_kv_heads=8, head_dim=128,
                         ffn=3072, n_codes=15, vocab=2048, max_draft=14, dtype=DTYPE_I8)


# The outer CodeDecoder of the full pipeline (Fig. 1): 28 layers of the same block, one
# code table (E_0 over its 3072-entry codebook) and one head in the blob layout above
# (n_codes = 1, max_draft = 0); the 15 tables of the residual codes come separately
# (make_outer_tables).
OUTER_1024 = ModelShape(n_layers=28, hidden=1024, n_q_heads=16, n_kv_heads=8, head_dim=128,
                        ffn=3072, n_codes=1, vocab=3072, max_draft=0, dtype=DTYPE_BF16)


def make_outer_tables(s: ModelShape, n_tables: int, vocab: int, seed: int = 5, std: float = 0.02) -> bytes:
    """Embedding tables E_1..E_n of the residual codes for the outer decoder's input:
    [n_tables][vocab][hidden] in the matrix dtype of s, N(0, std) drawn in that order."""
    v = (np.random.default_rng(seed).standard_normal((n_tables, vocab, s.hidden)) * std).astype(np.float32)
    return v.tobytes() if s.dtype == DTYPE_F32 else f32_to_bf16_bits(v).tobytes()


def unpack_outer_tables(s: ModelShape, blob: bytes, n_tables: int, vocab: int) -> np.ndarray:
    if s.dtype == DTYPE_F32:
        return np.frombuffer(blob, dtype=np.float32).reshape(n_tables, vocab, s.hidden).copy()
    return bf16_bits_to_f32(np.frombuffer(blob, dtype=np.uint16)).reshape(n_tables, vocab, s.hidden)


def pipeline_inputs(s: ModelShape, frames: int, seed_t: int = 3, seed_u: int = 4):
    """Per-frame text-side input vectors t_i ~ N(0,1) [frames, H] float32 and the uniform of
    each frame's c_0 draw [frames] float32 (prefix-stable)."""
    t = np.random.default_rng(seed_t + 1000).standard_normal((frames, s.hidden)).astype(np.float32)
    u = np.minimum(np.random.default_rng(seed_u).random(frames), 1.0 - 2.0 ** -24).astype(np.float32)
    return t, u


def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round float32 to bfloat16 (nearest even); returns the uint16 bit patterns."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32).astype(np.uint64)
    lsb = (u >> np.uint64(16)) & np.uint64(1)
    r = (u + np.uint64(0x7FFF) + lsb) >> np.uint64(16)
    return r.astype(np.uint16)


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    return (b.astype(np.uint32) << np.uint32(16)).view(np.float32)


def tensor_list(s: ModelShape):
    """(name, shape, kind) in blob order; kind is 'vec' (f32, gain or offset) or 'mat'."""
    H, d, F, V = s.hidden, s.head_dim, s.ffn, s.vocab
    out = []
    for l in range(s.n_layers):
        out += [
            (f"l{l}.attn_norm", (H,), "vec"),
            (f"l{l}.wq", (s.q_dim, H), "mat"),
            (f"l{l}.wk", (s.kv_dim, H), "mat"),
            (f"l{l}.wv", (s.kv_dim, H), "mat"),
            (f"l{l}.q_norm", (d,), "vec"),
            (f"l{l}.k_norm", (d,), "vec"),
            (f"l{l}.wo", (H, s.q_dim), "mat"),
            (f"l{l}.mlp_norm", (H,), "vec"),
            (f"l{l}.wgate", (F, H), "mat"),
            (f"l{l}.wup", (F, H), "mat"),
            (f"l{l}.wdown", (H, F), "mat"),
        ]
    out.append(("final_norm", (H,), "vec"))
    out += [(f"emb{i}", (V, H), "mat") for i in range(s.n_codes)]
    out += [(f"lmh{t}", (V, H), "mat") for t in range(1, s.n_codes + 1)]
    out.append(("offsets", (s.max_draft, H), "vec"))
    return out


def mat_bytes(s: ModelShape, shape) -> int:
    """Bytes of one matrix in the blob (int8: codes, row scales, padding to 16 bytes)."""
    cnt = int(np.prod(shape))
    if s.dtype == DTYPE_I8:
        raw = cnt + 4 * shape[0]
        return (raw + 15) // 16 * 16
    return cnt * (4 if s.dtype == DTYPE_F32 else 2)


def blob_size(s: ModelShape) -> int:
    n = HEADER_BYTES
    for _, shape, kind in tensor_list(s):
        n += mat_bytes(s, shape) if kind == "mat" else 4 * int(np.prod(shape))
    return n


def quantize_rows(w32: np.ndarray):
    """Symmetric per-row int8: (q int8 [rows][cols], s float32 [rows])."""
    w = np.asarray(w32, dtype=np.float32).astype(np.float64)
    s = (np.abs(w).max(axis=1) / 127.0).astype(np.float32)
    sd = s.astype(np.float64)
    q = np.zeros(w.shape, dtype=np.float64)
    nz = sd > 0
    q[nz] = np.rint(w[nz] / sd[nz, None])
    return np.clip(q, -127, 127).astype(np.int8), s


def dequantize_rows(q: np.ndarray, s: np.ndarray) -> np.ndarray:
    """The weights an int8 matrix stands for, exactly (float64)."""
    return q.astype(np.float64) * np.asarray(s, dtype=np.float32).astype(np.float64)[:, None]


def make_header(s: ModelShape) -> bytes:
    h = MAGIC + struct.pack("<11I", VERSION, s.dtype, s.n_layers, s.hidden, s.n_q_heads,
                            s.n_kv_heads, s.head_dim, s.ffn, s.n_codes, s.vocab, s.max_draft)
    h += b"\0" * (HEADER_BYTES - len(h))
    return h


def make_weights(s: ModelShape, seed: int = 0, std: float = 0.02, head_scale: float = 1.0,
                 offset_std: float | None = None, offsets: np.ndarray | None = None) -> bytes:
    """Build the weight blob.  ``offsets`` (shape [max_draft, H]) overrides the drawn offsets."""
    rng = np.random.default_rng(seed)
    parts = [make_header(s)]
    for name, shape, kind in tensor_list(s):
        if name == "offsets":
            continue
        if kind == "vec":  # RMSNorm gains
            parts.append(np.ones(shape, dtype=np.float32).tobytes())
            continue
        v = rng.standard_normal(shape) * std
        if name.startswith("lmh"):
            v = v * head_scale
        v32 = v.astype(np.float32)
        if s.dtype == DTYPE_F32:
            parts.append(v32.tobytes())
        elif s.dtype == DTYPE_I8:
            q, sc = quantize_rows(v32)
            raw = q.tobytes() + sc.tobytes()
            parts.append(raw + b"\0" * (mat_bytes(s, shape) - len(raw)))
        else:
            parts.append(f32_to_bf16_bits(v32).tobytes())
    ostd = std if offset_std is None else offset_std
    ofs = rng.standard_normal((s.max_draft, s.hidden)) * ostd
    if offsets is not None:
        ofs = np.asarray(offsets, dtype=np.float64).reshape(s.max_draft, s.hidden)
    parts.append(ofs.astype(np.float32).tobytes())
    blob = b"".join(parts)
    assert len(blob) == blob_size(s), (len(blob), blob_size(s))
    return blob


def unpack_weights(s: ModelShape, blob: bytes) -> dict:
    """Decode the blob into float32 numpy arrays (bf16 matrices widened exactly; int8
    matrices dequantized exactly into float64)."""
    wb = 4 if s.dtype == DTYPE_F32 else 2
    off = HEADER_BYTES
    out = {}
    for name, shape, kind in tensor_list(s):
        cnt = int(np.prod(shape))
        if kind == "mat" and s.dtype == DTYPE_I8:
            q = np.frombuffer(blob, dtype=np.int8, count=cnt, offset=off).reshape(shape)
            sc = np.frombuffer(blob, dtype=np.float32, count=shape[0], offset=off + cnt)
            out[name] = dequantize_rows(q, sc)
            off += mat_bytes(s, shape)
        elif kind == "mat" and s.dtype == DTYPE_BF16:
            a = np.frombuffer(blob, dtype=np.uint16, count=cnt, offset=off)
            out[name] = bf16_bits_to_f32(a).reshape(shape)
            off += cnt * 2
        else:
            out[name] = np.frombuffer(blob, dtype=np.float32, count=cnt, offset=off).reshape(shape).copy()
            off += cnt * 4
    assert off == len(blob)
    return out


def frame_inputs(s: ModelShape, frames: int, seed_hidden: int = 2, seed_c0: int = 3):
    """Frame hidden vectors f ~ N(0,1) [frames, H] float32 and c0 ~ U{0..V-1} int32.

    Frame i's values do not depend on ``frames`` (prefix-stable draws)."""
    f = np.random.default_rng(seed_hidden).standard_normal((frames, s.hidden)).astype(np.float32)
    c0 = np.random.default_rng(seed_c0).integers(0, s.vocab, size=frames).astype(np.int32)
    return f, c0


def uniforms(frames: int, n_codes: int = 15, seed: int = 1) -> np.ndarray:
    """Pre-drawn uniforms [frames, n_codes, 3] float32 in [0, 1).

    Slot 0 = u_draft, 1 = u_acc, 2 = u_samp, for code positions s = 1..n_codes."""
    u = np.random.default_rng(seed).random((frames, n_codes, 3)).astype(np.float32)
    return np.minimum(u, np.float32(np.nextafter(np.float32(1.0), np.float32(0.0))))
