"""Seeded generators (SplitMix64 counter streams, see csrc/synth_gen.c).

Streams are numbered per purpose so that any tensor can be regenerated alone,
e.g. one layer at a time for models that do not fit in host memory.
"""
import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "csrc", "synth_gen.c")
_LIB_PATH = os.path.join(_HERE, "libsynth.so")
_lib = None

# Stream numbering (purpose -> stream id).
S_EMBED, S_LM_HEAD = 1, 2
S_PREFIX, S_DRAFT, S_CONF, S_CONTEXT, S_DRAFT_LOGITS, S_KV, S_PLANT, S_LOGITS = 10, 11, 12, 13, 14, 15, 17, 18
LAYER_KINDS = {"wq": 1, "wk": 2, "wv": 3, "wo": 4, "wg": 5, "wu": 6, "wd": 7, "attn_norm": 8, "ffn_norm": 9}
S_FINAL_NORM = 20


def layer_stream(layer: int, kind: str) -> int:
    return ((layer + 1) << 8) | LAYER_KINDS[kind]


def build(force: bool = False) -> str:
    if force or not os.path.exists(_LIB_PATH) or os.path.getmtime(_LIB_PATH) < os.path.getmtime(_SRC):
        tmp = _LIB_PATH + ".tmp"
        subprocess.check_call(["gcc", "-O2", "-fopenmp", "-shared", "-fPIC", _SRC, "-o", tmp, "-lm"])
        os.replace(tmp, _LIB_PATH)
    return _LIB_PATH


def _L():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB_PATH):
            build()
        lib = ctypes.CDLL(_LIB_PATH)
        u64, sz, dbl, vp = ctypes.c_uint64, ctypes.c_size_t, ctypes.c_double, ctypes.c_void_p
        for name in ("synth_normal_f64", "synth_normal_f32", "synth_normal_bf16"):
            getattr(lib, name).argtypes = [u64, u64, u64, sz, dbl, dbl, vp]
        lib.synth_randint.argtypes = [u64, u64, u64, sz, u64, vp]
        lib.synth_uniform_f64.argtypes = [u64, u64, u64, sz, vp]
        lib.synth_words.argtypes = [u64, u64, u64, sz, vp]
        lib.synth_stream_key.argtypes = [u64, u64]
        lib.synth_stream_key.restype = u64
        _lib = lib
    return _lib


def normal(seed, stream, n, std=1.0, dtype="f64", offset=0, mean=0.0, out=None):
    """n normal draws; dtype "f64" | "f32" | "bf16" (bf16 returned as uint16 bit patterns)."""
    npdt = {"f64": np.float64, "f32": np.float32, "bf16": np.uint16}[dtype]
    if out is None:
        out = np.empty(n, dtype=npdt)
    assert out.dtype == npdt and out.size == n and out.flags.c_contiguous
    fn = {"f64": _L().synth_normal_f64, "f32": _L().synth_normal_f32, "bf16": _L().synth_normal_bf16}[dtype]
    fn(seed, stream, offset, n, float(mean), float(std), out.ctypes.data)
    return out


def randint(seed, stream, n, high, offset=0):
    out = np.empty(n, dtype=np.int32)
    _L().synth_randint(seed, stream, offset, n, int(high), out.ctypes.data)
    return out


def uniform(seed, stream, n, offset=0):
    out = np.empty(n, dtype=np.float64)
    _L().synth_uniform_f64(seed, stream, offset, n, out.ctypes.data)
    return out


def words(seed, stream, n, offset=0):
    out = np.empty(n, dtype=np.uint64)
    _L().synth_words(seed, stream, offset, n, out.ctypes.data)
    return out


def numpy_rng(seed, stream):
    """numpy Generator for small draws that need a named distribution (e.g. Beta)."""
    return np.random.Generator(np.random.Philox(key=[int(seed), int(stream)]))


# ---------------------------------------------------------------- bf16 helpers
def bf16_to_f32(bits: np.ndarray) -> np.ndarray:
    return (bits.astype(np.uint32) << 16).view(np.float32)


def f32_to_bf16(x: np.ndarray) -> np.ndarray:
    """Round-to-nearest-even fp32 -> bf16 bit patterns (NaN kept quiet)."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32).astype(np.uint64)
    nan = (u & 0x7F800000) == 0x7F800000
    nan &= (u & 0x007FFFFF) != 0
    r = ((u + 0x7FFF + ((u >> 16) & 1)) >> 16).astype(np.uint16)
    r[nan] = ((u[nan] >> 16) | 0x40).astype(np.uint16)
    return r


# ---------------------------------------------------------------- model tensors
def tensor_shapes(m):
    d, hd, F = m.d_model, m.head_dim, m.d_ff
    return {
        "wq": (m.n_q_heads * hd, d), "wk": (m.n_kv_heads * hd, d), "wv": (m.n_kv_heads * hd, d),
        "wo": (d, m.n_q_heads * hd), "wg": (F, d), "wu": (F, d), "wd": (d, F),
    }


def _gain(m, seed, stream, gains):
    """RMSNorm gain vector in the storage dtype: ones, or (gains="random") 0.5 + U(0, 1) per
    column, so that tests see gains that differ from column to column."""
    g = np.ones(m.d_model, np.float32) if gains == "ones" else (0.5 + uniform(seed, stream, m.d_model)).astype(np.float32)
    return g if m.dtype == "f32" else f32_to_bf16(g)


def layer_weights(m, seed, layer, gains="ones"):
    """Row-major [out_features, in_features] matrices (torch.nn.Linear layout) of one layer,
    in the storage dtype (np.float32, or np.uint16 bf16 bits), and its two norm gains."""
    assert gains in ("ones", "random")
    out = {}
    for kind, shp in tensor_shapes(m).items():
        n = shp[0] * shp[1]
        out[kind] = normal(seed, layer_stream(layer, kind), n, m.init_std, m.dtype).reshape(shp)
    out["attn_norm"] = _gain(m, seed, layer_stream(layer, "attn_norm"), gains)
    out["ffn_norm"] = _gain(m, seed, layer_stream(layer, "ffn_norm"), gains)
    return out


def embed_weights(m, seed):
    return normal(seed, S_EMBED, m.vocab * m.d_model, m.init_std, m.dtype).reshape(m.vocab, m.d_model)


def lm_head_weights(m, seed):
    return normal(seed, S_LM_HEAD, m.vocab * m.d_model, m.init_std, m.dtype).reshape(m.vocab, m.d_model)


def final_norm_weights(m, seed=0, gains="ones"):
    return _gain(m, seed, S_FINAL_NORM, gains)


def model_weights(m, seed, gains="ones"):
    """Every tensor of a model.  gains: "ones" (the workloads) or "random" (tests of the
    norm gains: 0.5 + U(0, 1) per column, seeded)."""
    return {
        "embed": embed_weights(m, seed),
        "final_norm": final_norm_weights(m, seed, gains),
        "lm_head": lm_head_weights(m, seed),
        "layers": [layer_weights(m, seed, l, gains) for l in range(m.n_layers)],
    }


# ---------------------------------------------------------------- workload inputs
def contexts(wl, seed=None):
    seed = wl.seed if seed is None else seed
    kind = wl.context[0]
    if kind == "fixed":
        return np.full(wl.batch, wl.context[1], dtype=np.int32)
    lo, hi = wl.context[1], wl.context[2]
    return (lo + randint(seed, S_CONTEXT, wl.batch, hi - lo + 1)).astype(np.int32)


def confidences(wl, seed=None, batch=None):
    """Drafter confidences q_i, i = 1..G, per sequence (float32 [B, G]).
    ("uniform", r): U(0,1) * r**i ;  ("beta", a, b, r): Beta(a, b) * r**i."""
    seed = wl.seed if seed is None else seed
    B = wl.batch if batch is None else batch
    i = np.arange(1, wl.G + 1, dtype=np.float64)
    rng = numpy_rng(seed, S_CONF)
    if wl.conf[0] == "uniform":
        base = rng.random((B, wl.G))
        decay = wl.conf[1]
    else:
        base = rng.beta(wl.conf[1], wl.conf[2], size=(B, wl.G))
        decay = wl.conf[3]
    return (base * decay ** i).astype(np.float32)


def prefix_ids(seed, batch, ctx_len, vocab):
    return [randint(seed, S_PREFIX + 1000 * b, int(ctx_len[b]), vocab) for b in range(batch)]


def draft_ids(seed, batch, G, vocab):
    return randint(seed, S_DRAFT, batch * G, vocab).reshape(batch, G)


def draft_probs(seed, n_rows, vocab):
    """Draft distributions q_v = softmax(z), z ~ N(0,1)^V, as float32 [n_rows, V].
    (The softmax here builds an *input* distribution; it is not part of the verify path.)"""
    z = normal(seed, S_DRAFT_LOGITS, n_rows * vocab, 1.0, "f64").reshape(n_rows, vocab)
    z -= z.max(axis=1, keepdims=True)
    e = np.exp(z)
    return (e / e.sum(axis=1, keepdims=True)).astype(np.float32)


def synthetic_kv(m, seed, layer, batch, ctx, std=1.0):
    """KV-cache contents for positions [0, ctx) in the storage dtype, shape [B, n_kv, ctx, hd] each."""
    n = batch * m.n_kv_heads * ctx * m.head_dim
    k = normal(seed, S_KV + 1000 * (2 * layer), n, std, m.dtype).reshape(batch, m.n_kv_heads, ctx, m.head_dim)
    v = normal(seed, S_KV + 1000 * (2 * layer + 1), n, std, m.dtype).reshape(batch, m.n_kv_heads, ctx, m.head_dim)
    return k, v


def synthetic_logits(seed, n_rows, vocab, std=1.0):
    return normal(seed, S_LOGITS, n_rows * vocab, std, "f32").reshape(n_rows, vocab)
