"""A cache, its workspace and the calls of one decode loop, with torch
providing device memory and the stream.  Every computation runs in
libpask.so's kernels through the C ABI binding.
"""

from __future__ import annotations

import math
import struct

import torch

from . import pask


class PaskSession:
    """One cache of `max_batch` sequences x `n_layers` layers on one GPU."""

    def __init__(self, policy_blob: bytes, *, max_batch: int, n_layers: int, n_q_heads: int, n_kv_heads: int,
                 head_dim: int, max_tokens_per_seq: int, hi_pages: int, lo_pages: int,
                 max_ctx_hint: int | None = None, device: str = "cuda:0", extra_bytes: int = 0,
                 prefill: int | None = None):
        self.device = torch.device(device)
        # the recent window W is the table's (blob header word at byte 24)
        self.window = struct.unpack_from("<I", bytes(policy_blob[:28]), 24)[0] if len(policy_blob) >= 28 else 0
        self.geom = pask.make_geom(max_batch=max_batch, n_layers=n_layers, n_q_heads=n_q_heads,
                                   n_kv_heads=n_kv_heads, head_dim=head_dim,
                                   max_tokens_per_seq=max_tokens_per_seq, hi_pages=hi_pages, lo_pages=lo_pages,
                                   recent_window=self.window)
        self.policy = pask.pask_policy_load(policy_blob, self.geom)
        self.nbytes = pask.pask_cache_bytes(self.geom)
        if self.nbytes == 0:
            raise pask.PaskError(pask.PASK_E_SHAPE, "pask_cache_bytes")
        self.layout = pask.pask_cache_layout_query(self.geom)
        # extra_bytes: room after the cache for out-of-bounds canaries in tests.
        # prefill: a byte written over the whole buffer and the workspace before
        # pask_cache_init (tests: no result may depend on bytes the library has
        # not written).
        self.buf = torch.empty(self.nbytes + extra_bytes, dtype=torch.uint8, device=self.device)
        if prefill is not None:
            self.buf.fill_(prefill)
        self.cache = pask.pask_cache()
        pask.pask_cache_init(self.cache, self.geom, self.buf, self.nbytes, self.stream)
        self.max_ctx_hint = max_ctx_hint or max_tokens_per_seq
        self.ws_bytes = pask.pask_workspace_bytes(self.geom, max_batch, self.max_ctx_hint)
        self.ws = torch.empty(self.ws_bytes, dtype=torch.uint8, device=self.device)
        if prefill is not None:
            self.ws.fill_(prefill)
        self.softmax_scale = float(torch.tensor(1.0 / math.sqrt(head_dim), dtype=torch.float32))

    @property
    def stream(self) -> int:
        return torch.cuda.current_stream(self.device).cuda_stream

    # -- the hot path ------------------------------------------------------
    def append(self, layer: int, tags, k, v, n_new=None, keep_all: bool = False, batch: int | None = None,
               states=None):
        """k, v: bf16 [batch, max_new, Hkv, D]; tags, states (parser states
        for the online controller, optional): uint8 [batch, max_new]."""
        b = batch or k.shape[0]
        pask.pask_kv_append(self.policy, self.cache, layer, b, n_new, k.shape[1], tags, k, v,
                            pask.PASK_APPEND_KEEP_ALL if keep_all else 0, self.stream, states=states)

    def budget_init(self, t_max: int, batch: int | None = None):
        """Online controller: tables into the cache, R_0 for every layer."""
        pask.pask_budget_init(self.policy, self.cache, batch or self.geom.max_batch, t_max, self.stream)

    def decode(self, layer: int, q, out, lse=None, tags_new=None, k_new=None, v_new=None,
               batch: int | None = None, max_ctx_hint: int | None = None, states_new=None):
        """q, out: bf16 [batch, Hq, D]; optional fused append of one token per
        sequence (tags_new, states_new uint8 [batch], k_new / v_new bf16
        [batch, Hkv, D])."""
        b = batch or q.shape[0]
        hint = max_ctx_hint or self.max_ctx_hint
        pask.pask_decode_attn(self.policy, self.cache, layer, b, q, out, lse, tags_new, k_new, v_new,
                              self.softmax_scale, hint, self.ws, self.ws_bytes, self.stream, states_new=states_new)

    def decode_noalloc(self, layer: int, q, out, lse=None, tags_new=None, k_new=None, v_new=None,
                       batch: int | None = None, max_ctx_hint: int | None = None, states_new=None):
        """decode() through pask_decode_attn_noalloc: no workspace argument,
        the partials go to the library's own device scratch."""
        b = batch or q.shape[0]
        hint = max_ctx_hint or self.max_ctx_hint
        pask.pask_decode_attn_noalloc(self.policy, self.cache, layer, b, q, out, lse, tags_new, k_new, v_new,
                                      self.softmax_scale, hint, self.stream, states_new=states_new)

    def budgets(self):
        """Remaining budget R of every (sequence, layer), int64 [max_batch, n_layers]."""
        c = self.counters()
        return c[:, :, 6:8].contiguous().view(torch.int64)[:, :, 0]

    def stats(self, batch: int | None = None, per_seq: bool = False):
        import numpy as np
        b = batch or self.geom.max_batch
        arr = None
        if per_seq:
            arr = np.zeros(b * self.policy.n_groups * self.geom.n_kv_heads * 3, dtype=np.int64)
        st, status = pask.pask_cache_stats(self.policy, self.cache, b, arr, self.stream)
        if arr is not None:
            arr = arr.reshape(b, self.policy.n_groups, self.geom.n_kv_heads, 3)
        return st, status, arr

    def reset(self):
        pask.pask_cache_reset(self.cache, self.stream)

    # -- views of the cache buffer (inspection) ----------------------------
    def _i32(self, off: int, shape):
        n = 1
        for s in shape:
            n *= s
        return self.buf[off:off + 4 * n].view(torch.int32).view(*shape)

    def status_words(self):
        return self._i32(self.layout.status_off, (4,))

    def counters(self):
        g = self.geom
        return self._i32(self.layout.counters_off, (g.max_batch, g.n_layers, self.layout.counter_stride))

    def block_tables(self):
        g = self.geom
        return self._i32(self.layout.block_table_off, (g.max_batch, g.n_layers, 2, self.layout.max_pages))

    def index_lists(self):
        g = self.geom
        return self._i32(self.layout.index_list_off, (g.max_batch, g.n_layers, 2, g.max_tokens_per_seq))

    def hi_pool(self):
        """Every page of the HIGH pool: the recent windows, then the HIGH store."""
        L = self.layout
        n = L.ring_pages + self.geom.hi_pages
        return self.buf[L.hi_pool_off:L.hi_pool_off + n * L.hi_page_bytes].view(n, L.hi_page_bytes)

    def lo_pool(self):
        L = self.layout
        return self.buf[L.lo_pool_off:L.lo_pool_off + self.geom.lo_pages * L.lo_page_bytes].view(
            self.geom.lo_pages, L.lo_page_bytes)

    def _decode_hi(self, raw, pages, n: int):
        """(k bits, v bits) int64 [n, Hkv, D] of the first n slots of HIGH-layout pages."""
        import numpy as np
        D, H = self.geom.head_dim, self.geom.n_kv_heads
        t = np.arange(16)[:, None]
        d = np.arange(D)[None, :]
        x = raw.view(np.uint16).reshape(-1, H, 2, 16 * D).astype(np.int64)
        kidx = ((d // 32 * 64 + (d % 32) // 8 * 16 + t) * 8 + d % 8)
        vidx = ((((d // 16) // 2) * 64 + t // 4 * 16 + d % 16) * 2 + (d // 16) % 2) * 4 + t % 4
        x = x[np.arange(x.shape[0])[:, None], (np.arange(H)[None, :] + pages[:, None]) % H]   # head slots
        k = x[:, :, 0][:, :, kidx].transpose(0, 2, 1, 3).reshape(-1, H, D)[:n]
        v = x[:, :, 1][:, :, vidx].transpose(0, 2, 1, 3).reshape(-1, H, D)[:n]
        return k, v

    def gather_window(self, b: int, layer: int):
        """The recent window of (b, layer): (positions int64 [m], k bits, v bits
        int64 [m, Hkv, D]) in position order, m = min(n_pos, W); position p
        sits in window slot p mod W."""
        import numpy as np
        W = self.window
        n_pos = int(self.counters()[b, layer, 2].item())
        m = min(n_pos, W)
        if m == 0:
            z = np.zeros((0, self.geom.n_kv_heads, self.geom.head_dim), np.int64)
            return np.zeros(0, np.int64), z, z
        pp = (W + 15) // 16
        pages = (b * self.geom.n_layers + layer) * pp + np.arange(pp)
        raw = self.hi_pool()[torch.as_tensor(pages, dtype=torch.long, device=self.device)].cpu().numpy()
        k, v = self._decode_hi(raw, pages, W)
        pos = np.arange(n_pos - m, n_pos)
        return pos, k[pos % W], v[pos % W]

    def gather_store(self, b: int, layer: int, store: int):
        """Host copies of one store's entries, by slot, read through the block
        table and decoded from the page layout (KV head g of page P sits in
        head slot (g + P) mod Hkv).  HIGH: (k bits, v bits) int64
        [n, Hkv, D].  LOW: (k codes int8 [n, Hkv, D], k scale bits [n, Hkv, D/32],
        v codes, v scale bits); the pages hold each code c as the nibble c + 8."""
        import numpy as np
        g = self.geom
        D, H = g.head_dim, g.n_kv_heads
        NG, NM = D // 32, D // 16
        cnt = self.counters()[b, layer].cpu().numpy()
        n = int(cnt[store])
        bt = self.block_tables()[b, layer, store].cpu().numpy()
        pages = bt[: (n + 15) // 16]
        pool = self.hi_pool() if store == 0 else self.lo_pool()
        nbytes = self.layout.hi_page_bytes if store == 0 else self.layout.lo_page_bytes
        raw = pool[torch.as_tensor(pages, dtype=torch.long, device=self.device)].cpu().numpy() if n else \
            np.zeros((0, nbytes), np.uint8)
        t = np.arange(16)[:, None]
        d = np.arange(D)[None, :]
        # LOW K: word ((d%32)//8*16 + t)*NG + d//32, element j = d%8 in byte j%4, nibble j//4
        kbyte = (((d % 32) // 8 * 16 + t) * NG + d // 32) * 4 + (d % 8) % 4                  # [16, D]
        khalf = (d % 8) // 4
        if store == 0:
            return self._decode_hi(raw, pages, n)
        head = 16 * D + 64 * NG
        r = raw.reshape(-1, H, head)
        r = r[np.arange(r.shape[0])[:, None], (np.arange(H)[None, :] + pages[:, None]) % H]       # head slots
        unbias = lambda c: (c.astype(np.int16) - 8).astype(np.int8)                          # offset binary
        kc = unbias((r[:, :, :8 * D][..., kbyte] >> (4 * khalf)) & 0xF)                   # [P, H, 16, D]
        ks = r[:, :, 8 * D:8 * D + 32 * NG].copy().view(np.uint16).reshape(-1, H, 16, NG)
        vbyte = ((t // 4 * 16 + d % 16) * (NM // 2) + d // 32) * 4 + t % 4
        vhalf = (d % 32) // 16
        vb = r[:, :, 8 * D + 32 * NG:16 * D + 32 * NG]
        vc = unbias((vb[..., vbyte] >> (4 * vhalf)) & 0xF)
        vs = r[:, :, 16 * D + 32 * NG:].copy().view(np.uint16).reshape(-1, H, 16, NG)
        fix = lambda a: a.transpose(0, 2, 1, 3).reshape(-1, H, a.shape[-1])[:n]
        return fix(kc), fix(ks).astype(np.int64), fix(vc), fix(vs).astype(np.int64)
