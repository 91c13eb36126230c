"""Device buffers for the verify path: packed model, KV cache, workspaces.

torch provides device memory and streams; all compute is in liblsv.so."""
import numpy as np
import torch

from . import lsv


def model_config(shape):
    """lsv.ModelConfig from any object with the usual fields (n_layers, d_model, ...)."""
    return lsv.ModelConfig(
        n_layers=shape.n_layers, d_model=shape.d_model, n_q_heads=shape.n_q_heads, n_kv_heads=shape.n_kv_heads,
        head_dim=shape.head_dim, d_ff=shape.d_ff, vocab=shape.vocab,
        dtype=lsv.LSV_DTYPE_BF16 if shape.dtype == "bf16" else lsv.LSV_DTYPE_F32,
        rms_eps=shape.rms_eps, reserved0=0.0, rope_base=shape.rope_base)


def storage_dtype(cfg):
    return torch.bfloat16 if cfg.dtype == lsv.LSV_DTYPE_BF16 else torch.float32


def to_device(arr, device="cuda"):
    """numpy array in storage form (float32, or uint16 bf16 bit patterns) -> device tensor."""
    a = np.ascontiguousarray(arr)
    if a.dtype == np.uint16:
        return torch.from_numpy(a.view(np.int16)).to(device).view(torch.bfloat16)
    return torch.from_numpy(a).to(device)


class DeviceModel:
    """Packed weights of one model in a single device buffer."""

    def __init__(self, cfg, device="cuda"):
        self.cfg = cfg
        self.device = device
        self.nbytes = lsv.lsv_packed_model_bytes(cfg)
        if self.nbytes == 0:
            raise lsv.LsvError(lsv.LSV_ERR_INVALID_ARG, lsv.lsv_last_error())
        self.buf = torch.empty(self.nbytes, dtype=torch.uint8, device=device)

    def pack_globals(self, embed, final_norm, lm_head):
        t = [to_device(x, self.device) for x in (embed, final_norm, lm_head)]
        lsv.lsv_pack_globals(self.cfg, *t, self.buf)
        torch.cuda.current_stream().synchronize()

    def pack_layer(self, layer, w):
        keys = ("wq", "wk", "wv", "wo", "wg", "wu", "wd", "attn_norm", "ffn_norm")
        t = [to_device(w[k], self.device) for k in keys]
        lsv.lsv_pack_layer(self.cfg, layer, *t, self.buf)
        torch.cuda.current_stream().synchronize()

    @classmethod
    def from_weights(cls, cfg, weights, device="cuda"):
        """weights: {"embed", "final_norm", "lm_head", "layers": [dict per layer]} in storage form."""
        dm = cls(cfg, device)
        dm.pack_globals(weights["embed"], weights["final_norm"], weights["lm_head"])
        for l, w in enumerate(weights["layers"]):
            dm.pack_layer(l, w)
        return dm


def kv_capacity(positions):
    """Smallest valid cache capacity (a multiple of LSV_KV_ALIGN) holding `positions`."""
    a = lsv.LSV_KV_ALIGN
    return max(a, (int(positions) + a - 1) // a * a)


def v_column(pos):
    """Column of cache position `pos` in a transposed V row (lsv.h, LSV_V_COLUMN)."""
    return (pos & ~31) | ((pos & 12) << 1) | ((pos & 16) >> 2) | (pos & 3)


class KVCache:
    """The library's KV cache (lsv.h): per layer and K|V, each sequence's 64-position blocks in
    order, the kv heads of a block side by side; K row-major, V transposed with permuted columns."""

    def __init__(self, cfg, batch, capacity, device="cuda"):
        self.cfg, self.batch, self.capacity = cfg, batch, capacity
        nbytes = lsv.lsv_kv_cache_bytes(cfg, batch, capacity)
        if nbytes == 0:
            raise lsv.LsvError(lsv.LSV_ERR_INVALID_ARG, f"invalid KV cache shape (capacity {capacity} must be a "
                                                        f"positive multiple of {lsv.LSV_KV_ALIGN})")
        self.buf = torch.zeros(nbytes, dtype=torch.uint8, device=device)

    def _blocks(self):
        c, P = self.cfg, lsv.LSV_KV_ALIGN
        return self.buf.view(storage_dtype(c)).view(c.n_layers, 2, self.batch, self.capacity // P, c.n_kv_heads,
                                                    P * c.head_dim)

    def k_view(self):
        """[layer][batch][block][kv_head][j][head_dim] view of the K blocks (position 64 block + j)."""
        c, P = self.cfg, lsv.LSV_KV_ALIGN
        return self._blocks()[:, 0].view(c.n_layers, self.batch, self.capacity // P, c.n_kv_heads, P, c.head_dim)

    def vt_view(self):
        """[layer][batch][block][kv_head][head_dim][column] view of the transposed V blocks."""
        c, P = self.cfg, lsv.LSV_KV_ALIGN
        return self._blocks()[:, 1].view(c.n_layers, self.batch, self.capacity // P, c.n_kv_heads, c.head_dim, P)

    def _index(self, start, n):
        pos = torch.arange(start, start + n, device=self.buf.device)
        j = pos % lsv.LSV_KV_ALIGN
        return pos // lsv.LSV_KV_ALIGN, j, v_column(j)

    def write(self, layer, b, start, k, v):
        """Store K and V of positions start.. (device tensors [kv_head][n][head_dim])."""
        blk, j, col = self._index(start, k.shape[1])
        # the indexed views put the position first: [n][kv_head][head_dim]
        self.k_view()[layer, b][blk, :, j] = k.transpose(0, 1)
        self.vt_view()[layer, b][blk, :, :, col] = v.transpose(0, 1)

    def read(self, layer, b, start, n):
        """(K, V) of positions start..start+n-1 as [kv_head][n][head_dim] tensors."""
        blk, j, col = self._index(start, n)
        k = self.k_view()[layer, b][blk, :, j].transpose(0, 1)
        v = self.vt_view()[layer, b][blk, :, :, col].transpose(0, 1)
        return k, v


class PagedKVCache:
    """A paged KV cache (lsv.h, lsv_kv_pool_bytes): n_pages pages of LSV_KV_PAGE positions per
    layer and K|V, and a page table [batch][max_pages] (int32, device) mapping each sequence's
    64-position blocks to pages."""

    def __init__(self, cfg, n_pages, page_table, device="cuda"):
        self.cfg, self.n_pages = cfg, n_pages
        nbytes = lsv.lsv_kv_pool_bytes(cfg, n_pages)
        if nbytes == 0:
            raise lsv.LsvError(lsv.LSV_ERR_INVALID_ARG, "invalid KV pool shape")
        self.buf = torch.zeros(nbytes, dtype=torch.uint8, device=device)
        self.table_np = np.ascontiguousarray(page_table, dtype=np.int32)
        self.batch, self.max_pages = self.table_np.shape
        self.table = torch.tensor(self.table_np, device=device)

    def _pages(self):
        c, P = self.cfg, lsv.LSV_KV_PAGE
        return self.buf.view(storage_dtype(c)).view(c.n_layers, 2, self.n_pages, c.n_kv_heads, P * c.head_dim)

    def _views(self, layer):
        c, P = self.cfg, lsv.LSV_KV_PAGE
        kp = self._pages()[layer, 0].view(self.n_pages, c.n_kv_heads, P, c.head_dim)
        vp = self._pages()[layer, 1].view(self.n_pages, c.n_kv_heads, c.head_dim, P)
        return kp, vp

    def _runs(self, b, start, n):
        """(page, first slot in the page, offset in the run, length) of each run of positions
        start..start+n-1 inside one page."""
        P, pos, out = lsv.LSV_KV_PAGE, start, []
        while pos < start + n:
            ln = min(P - pos % P, start + n - pos)
            out.append((int(self.table_np[b, pos // P]), pos % P, pos - start, ln))
            pos += ln
        return out

    def write(self, layer, b, start, k, v):
        """Store K and V of positions start.. (device tensors [kv_head][n][head_dim])."""
        kp, vp = self._views(layer)
        for pg, j0, t0, ln in self._runs(b, start, k.shape[1]):
            kp[pg, :, j0:j0 + ln] = k[:, t0:t0 + ln]
            cols = v_column(torch.arange(j0, j0 + ln, device=self.buf.device))
            vp[pg][:, :, cols] = v[:, t0:t0 + ln].transpose(1, 2)

    def read(self, layer, b, start, n):
        """(K, V) of positions start..start+n-1 as [kv_head][n][head_dim] tensors."""
        kp, vp = self._views(layer)
        ks, vs = [], []
        for pg, j0, t0, ln in self._runs(b, start, n):
            ks.append(kp[pg, :, j0:j0 + ln])
            cols = v_column(torch.arange(j0, j0 + ln, device=self.buf.device))
            vs.append(vp[pg][:, :, cols].transpose(1, 2))
        return torch.cat(ks, dim=1), torch.cat(vs, dim=1)


class Workspace:
    """Zero-initialised device scratch (the library keeps its counters at zero)."""

    def __init__(self, nbytes, device="cuda"):
        self.nbytes = max(256, (int(nbytes) + 255) // 256 * 256)
        self.buf = torch.zeros(self.nbytes, dtype=torch.uint8, device=device)


def row_offsets_of(rows_per_seq):
    return np.concatenate([[0], np.cumsum(rows_per_seq)]).astype(np.int32)
