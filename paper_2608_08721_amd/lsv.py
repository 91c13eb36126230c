"""ctypes binding of liblsv (include/lsv.h): argument marshalling only.

Every function has the C name and argument order.  Device buffers may be given as
torch tensors (their data_ptr() is passed) or as raw integer addresses; ``stream``
defaults to torch's current stream.  A non-zero status raises LsvError carrying
the code and lsv_last_error().  Nothing here computes: each call enqueues HIP work.
"""
import ctypes
import os

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "liblsv.so")

LSV_OK, LSV_ERR_INVALID_ARG, LSV_ERR_UNSUPPORTED, LSV_ERR_HIP, LSV_ERR_CAPACITY, LSV_ERR_NONFINITE = 0, -1, -2, -3, -4, -5
LSV_DTYPE_F32, LSV_DTYPE_BF16 = 0, 1
LSV_MAX_BATCH, LSV_MAX_ROWS, LSV_MAX_G, LSV_MAX_SEQ_ROWS, LSV_WIDE_ROWS = 64, 512, 64, 64, 272
LSV_KV_ALIGN = LSV_KV_PAGE = 64
LSV_ACCEPT_NOALLOC_BYTES = 512 * 1024
LSV_ACC_GREEDY, LSV_ACC_SAMPLE = 0, 1
LSV_SEL_MARGINAL, LSV_SEL_EXHAUSTIVE, LSV_SEL_ALG1 = 0, 1, 2
LSV_SEL_BONUS = 1
LSV_SEL_DRAFTED = 2

EXPORTED = (
    "lsv_status_string", "lsv_last_error", "lsv_abi_version", "lsv_packed_model_bytes", "lsv_pack_globals",
    "lsv_pack_layer", "lsv_kv_cache_bytes", "lsv_verify_workspace_bytes", "lsv_workspace_clear",
    "lsv_verify_block", "lsv_verify_tree", "lsv_accept_tree", "lsv_commit_tree", "lsv_kv_pool_bytes",
    "lsv_verify_paged", "lsv_commit_tree_paged", "lsv_accept_workspace_bytes", "lsv_accept", "lsv_accept_noalloc", "lsv_select_length", "lsv_select_joint", "lsv_next_length_g4", "lsv_pack_block", "lsv_next_roots",
    "lsv_set_timing_events",
)
LSV_KERNEL_QKV, LSV_KERNEL_O, LSV_KERNEL_GATEUP, LSV_KERNEL_DOWN, LSV_KERNEL_LMHEAD, LSV_KERNEL_ATTENTION = range(6)
LSV_MAX_TIMING_SLOTS = 256


class LsvError(RuntimeError):
    def __init__(self, code, msg):
        super().__init__(f"lsv status {code}: {msg}")
        self.code = code


class ModelConfig(ctypes.Structure):
    _fields_ = [
        ("n_layers", ctypes.c_int32), ("d_model", ctypes.c_int32), ("n_q_heads", ctypes.c_int32),
        ("n_kv_heads", ctypes.c_int32), ("head_dim", ctypes.c_int32), ("d_ff", ctypes.c_int32),
        ("vocab", ctypes.c_int32), ("dtype", ctypes.c_int32), ("rms_eps", ctypes.c_float),
        ("reserved0", ctypes.c_float), ("rope_base", ctypes.c_double),
    ]


_lib = None


def load(path=LIB_PATH):
    """Load liblsv.so; raises (never falls back) when the HIP library is missing."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise ImportError(f"{path} is not built: run __graft_entry__.build() (hipcc, gfx950)")
    try:  # torch first, so the process holds exactly one HIP runtime (torch's), matched by soname
        import torch  # noqa: F401
    except ImportError:
        pass
    lib = ctypes.CDLL(path)
    P, I32, U32, U64, SZ, F32, F64 = (ctypes.c_void_p, ctypes.c_int32, ctypes.c_uint32, ctypes.c_uint64,
                                      ctypes.c_size_t, ctypes.c_float, ctypes.c_double)
    CP = ctypes.POINTER(ModelConfig)
    sig = {
        "lsv_status_string": (ctypes.c_char_p, [ctypes.c_int]),
        "lsv_last_error": (ctypes.c_char_p, []),
        "lsv_abi_version": (ctypes.c_int, []),
        "lsv_packed_model_bytes": (SZ, [CP]),
        "lsv_pack_globals": (ctypes.c_int, [CP, P, P, P, P, P]),
        "lsv_pack_layer": (ctypes.c_int, [CP, I32, P, P, P, P, P, P, P, P, P, P, P]),
        "lsv_kv_cache_bytes": (SZ, [CP, I32, I32]),
        "lsv_verify_workspace_bytes": (SZ, [CP, I32, I32, I32]),
        "lsv_workspace_clear": (ctypes.c_int, [P, SZ, P]),
        "lsv_verify_block": (ctypes.c_int, [CP, P, P, I32, I32, P, P, P, I32, I32, P, P, P, SZ, P]),
        "lsv_verify_tree": (ctypes.c_int, [CP, P, P, I32, I32, P, P, P, P, I32, I32, P, P, P, SZ, P]),
        "lsv_accept_tree": (ctypes.c_int, [I32, I32, P, P, P, P, I32, I32, P, P, P, P, P, P, SZ, P]),
        "lsv_commit_tree": (ctypes.c_int, [CP, P, I32, I32, P, P, P, I32, P, P]),
        "lsv_kv_pool_bytes": (SZ, [CP, I32]),
        "lsv_verify_paged": (ctypes.c_int, [CP, P, P, I32, P, I32, I32, P, P, P, P, I32, I32, P, P, P, SZ, P]),
        "lsv_commit_tree_paged": (ctypes.c_int, [CP, P, I32, P, I32, I32, P, P, P, I32, P, P]),
        "lsv_accept_workspace_bytes": (SZ, [I32, I32, I32]),
        "lsv_accept": (ctypes.c_int, [I32, I32, I32, P, P, I32, I32, P, P, F32, U64, U64, P, P, P, P, P, SZ, P]),
        "lsv_accept_noalloc": (ctypes.c_int, [I32, I32, I32, P, P, I32, I32, P, P, F32, U64, U64, P, P, P, P, P]),
        "lsv_select_length": (ctypes.c_int, [I32, I32, I32, P, P, I32, I32, F64, I32, U32, P, P, P, P, P]),
        "lsv_select_joint": (ctypes.c_int, [I32, I32, P, P, I32, U32, P, P, P, P, P]),
        "lsv_next_length_g4": (ctypes.c_int, [I32, P, P, P, I32, I32, P, P, P, P]),
        "lsv_pack_block": (ctypes.c_int, [I32, I32, P, I32, P, P, P, P, P]),
        "lsv_next_roots": (ctypes.c_int, [I32, P, P, I32, P, P, P]),
        "lsv_set_timing_events": (ctypes.c_int, [I32, ctypes.POINTER(ctypes.c_void_p), I32, U32]),
    }
    for name, (res, args) in sig.items():
        fn = getattr(lib, name)
        fn.restype = res
        fn.argtypes = args
    _lib = lib
    return lib


def _ptr(x):
    if x is None:
        return None
    if isinstance(x, int):
        return x
    return x.data_ptr()


def _stream(s):
    if s is None:
        import torch
        return torch.cuda.current_stream().cuda_stream
    if isinstance(s, int):
        return s
    return s.cuda_stream


def _need(t, name, n, dtype):
    """Marshalling check of a tensor argument the kernels read n elements of: a device tensor
    of the expected dtype and length (raw integer addresses are passed through unchecked)."""
    if t is None or isinstance(t, int):
        return
    import torch
    if t.device.type != "cuda" or t.dtype != dtype or t.numel() < n or not t.is_contiguous():
        raise LsvError(LSV_ERR_INVALID_ARG, f"{name}: need a contiguous cuda {dtype} tensor of >= {n} elements, got "
                                            f"{t.dtype} {tuple(t.shape)} on {t.device}")


def _check(rc):
    if rc != LSV_OK:
        raise LsvError(rc, load().lsv_last_error().decode())


def lsv_status_string(code):
    return load().lsv_status_string(code).decode()


def lsv_last_error():
    return load().lsv_last_error().decode()


def lsv_abi_version():
    return load().lsv_abi_version()


def lsv_packed_model_bytes(cfg):
    return load().lsv_packed_model_bytes(ctypes.byref(cfg))


def lsv_pack_globals(cfg, embed, final_norm, lm_head, packed, stream=None):
    _check(load().lsv_pack_globals(ctypes.byref(cfg), _ptr(embed), _ptr(final_norm), _ptr(lm_head), _ptr(packed),
                                   _stream(stream)))


def lsv_pack_layer(cfg, layer, wq, wk, wv, wo, wg, wu, wd, attn_norm, ffn_norm, packed, stream=None):
    _check(load().lsv_pack_layer(ctypes.byref(cfg), layer, *(_ptr(t) for t in (wq, wk, wv, wo, wg, wu, wd, attn_norm,
                                                                                  ffn_norm, packed)), _stream(stream)))


def lsv_kv_cache_bytes(cfg, batch, capacity):
    return load().lsv_kv_cache_bytes(ctypes.byref(cfg), batch, capacity)


def lsv_verify_workspace_bytes(cfg, batch, max_rows, max_ctx):
    return load().lsv_verify_workspace_bytes(ctypes.byref(cfg), batch, max_rows, max_ctx)


def lsv_workspace_clear(ws, nbytes, stream=None):
    _check(load().lsv_workspace_clear(_ptr(ws), nbytes, _stream(stream)))


def lsv_verify_block(cfg, packed, kv, capacity, batch, seq_len, tokens, row_offsets, max_rows, max_ctx, logits,
                     status, ws, ws_bytes, stream=None):
    _check(load().lsv_verify_block(ctypes.byref(cfg), _ptr(packed), _ptr(kv), capacity, batch, _ptr(seq_len),
                                   _ptr(tokens), _ptr(row_offsets), max_rows, max_ctx, _ptr(logits), _ptr(status),
                                   _ptr(ws), ws_bytes, _stream(stream)))


def lsv_verify_tree(cfg, packed, kv, capacity, batch, seq_len, tokens, row_offsets, parents, max_rows, max_ctx, logits,
                    status, ws, ws_bytes, stream=None):
    _check(load().lsv_verify_tree(ctypes.byref(cfg), _ptr(packed), _ptr(kv), capacity, batch, _ptr(seq_len),
                                  _ptr(tokens), _ptr(row_offsets), _ptr(parents), max_rows, max_ctx, _ptr(logits),
                                  _ptr(status), _ptr(ws), ws_bytes, _stream(stream)))


def lsv_accept_tree(batch, vocab, logits, row_offsets, parents, tokens, max_rows, width, accept_len, out_tokens, path,
                    seq_len, status, ws, ws_bytes, stream=None):
    _check(load().lsv_accept_tree(batch, vocab, _ptr(logits), _ptr(row_offsets), _ptr(parents), _ptr(tokens), max_rows,
                                  width, _ptr(accept_len), _ptr(out_tokens), _ptr(path), _ptr(seq_len), _ptr(status),
                                  _ptr(ws), ws_bytes, _stream(stream)))


def lsv_commit_tree(cfg, kv, capacity, batch, seq_len, accept_len, path, width, status, stream=None):
    _check(load().lsv_commit_tree(ctypes.byref(cfg), _ptr(kv), capacity, batch, _ptr(seq_len), _ptr(accept_len),
                                  _ptr(path), width, _ptr(status), _stream(stream)))


def lsv_kv_pool_bytes(cfg, n_pages):
    return load().lsv_kv_pool_bytes(ctypes.byref(cfg), n_pages)


def lsv_verify_paged(cfg, packed, kv_pool, n_pages, page_table, max_pages, batch, seq_len, tokens, row_offsets, parents,
                     max_rows, max_ctx, logits, status, ws, ws_bytes, stream=None):
    _check(load().lsv_verify_paged(ctypes.byref(cfg), _ptr(packed), _ptr(kv_pool), n_pages, _ptr(page_table), max_pages,
                                   batch, _ptr(seq_len), _ptr(tokens), _ptr(row_offsets), _ptr(parents), max_rows,
                                   max_ctx, _ptr(logits), _ptr(status), _ptr(ws), ws_bytes, _stream(stream)))


def lsv_commit_tree_paged(cfg, kv_pool, n_pages, page_table, max_pages, batch, seq_len, accept_len, path, width, status,
                          stream=None):
    _check(load().lsv_commit_tree_paged(ctypes.byref(cfg), _ptr(kv_pool), n_pages, _ptr(page_table), max_pages, batch,
                                        _ptr(seq_len), _ptr(accept_len), _ptr(path), width, _ptr(status),
                                        _stream(stream)))


def lsv_accept_workspace_bytes(batch, max_rows, vocab):
    return load().lsv_accept_workspace_bytes(batch, max_rows, vocab)


def lsv_accept(mode, batch, vocab, logits, row_offsets, max_rows, max_rows_per_seq, tokens, draft_probs, temperature,
               seed, round, accept_len, out_tokens, seq_len, status, ws, ws_bytes, stream=None):
    _check(load().lsv_accept(mode, batch, vocab, _ptr(logits), _ptr(row_offsets), max_rows, max_rows_per_seq,
                             _ptr(tokens), _ptr(draft_probs), temperature, seed, round, _ptr(accept_len),
                             _ptr(out_tokens), _ptr(seq_len), _ptr(status), _ptr(ws), ws_bytes, _stream(stream)))


def lsv_accept_noalloc(mode, batch, vocab, logits, row_offsets, max_rows, max_rows_per_seq, tokens, draft_probs,
                       temperature, seed, round, accept_len, out_tokens, seq_len, status, stream=None):
    _check(load().lsv_accept_noalloc(mode, batch, vocab, _ptr(logits), _ptr(row_offsets), max_rows, max_rows_per_seq,
                                     _ptr(tokens), _ptr(draft_probs), temperature, seed, round, _ptr(accept_len),
                                     _ptr(out_tokens), _ptr(seq_len), _ptr(status), _stream(stream)))


def lsv_select_length(mode, batch, G, conf, cost, d_init, d_max, alpha, block_n, flags, gamma, aux, row_offsets,
                      status, stream=None):
    import torch
    _need(conf, "conf", batch * G, torch.float32)
    if mode != LSV_SEL_ALG1:
        _need(cost, "cost", d_max + 1, torch.float64)
    _check(load().lsv_select_length(mode, batch, G, _ptr(conf), _ptr(cost), d_init, d_max, alpha, block_n, flags,
                                    _ptr(gamma), _ptr(aux), _ptr(row_offsets), _ptr(status), _stream(stream)))


def lsv_select_joint(batch, G, conf, cost, d_max, flags, gamma, total, row_offsets, status, stream=None):
    import torch
    _need(conf, "conf", batch * G, torch.float32)
    _need(cost, "cost", batch * d_max + 1, torch.float64)
    _check(load().lsv_select_joint(batch, G, _ptr(conf), _ptr(cost), d_max, flags, _ptr(gamma), _ptr(total),
                                   _ptr(row_offsets), _ptr(status), _stream(stream)))


def lsv_next_length_g4(batch, gamma, accept_len, status, d_min, d_max, gamma_next, row_offsets, err, stream=None):
    _check(load().lsv_next_length_g4(batch, _ptr(gamma), _ptr(accept_len), _ptr(status), d_min, d_max,
                                     _ptr(gamma_next), _ptr(row_offsets), _ptr(err), _stream(stream)))


def lsv_pack_block(batch, G, row_offsets, max_rows, roots, drafts, tokens, status, stream=None):
    _check(load().lsv_pack_block(batch, G, _ptr(row_offsets), max_rows, _ptr(roots), _ptr(drafts), _ptr(tokens),
                                 _ptr(status), _stream(stream)))


def lsv_next_roots(batch, accept_len, out_tokens, width, status, roots, stream=None):
    _check(load().lsv_next_roots(batch, _ptr(accept_len), _ptr(out_tokens), width, _ptr(status), _ptr(roots),
                                 _stream(stream)))


def lsv_set_timing_events(kernel, events, n_slots, record_flags=0):
    """events: sequence of 2 * n_slots hipEvent_t handles (ints); record_flags 1 = external
    (use while capturing a graph)."""
    arr = (ctypes.c_void_p * max(1, 2 * n_slots))(*[int(e) for e in events][:2 * n_slots])
    _check(load().lsv_set_timing_events(kernel, arr, n_slots, record_flags))


def hip_runtime():
    """ctypes handle of the HIP runtime already loaded in this process (for events)."""
    load()
    for line in open("/proc/self/maps"):
        parts = line.split()
        if parts and "libamdhip64" in parts[-1]:
            return ctypes.CDLL(parts[-1])
    raise RuntimeError("HIP runtime not loaded")
