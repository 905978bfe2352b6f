"""Shared pieces of the GPU parity tests: a scenario that feeds the same
seeded inputs to the HIP path (through the C ABI) and to the CPU oracle, and
the comparisons (bit-exact for decisions, lists, counters, codes, scales and
bf16 copies; attention within |gpu - ref| <= 2e-3 + 1e-2 |ref|)."""

from __future__ import annotations

import math
import sys

import numpy as np
import torch

import oracle
from workload.policy import pack_blob
from workload.tensors import bf16_normal, sub_seed

ATOL, RTOL = 2e-3, 1e-2


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def bits16(t: torch.Tensor) -> np.ndarray:
    return t.detach().contiguous().cpu().view(torch.int16).numpy().view(np.uint16)


def bf16_f64(t: torch.Tensor) -> np.ndarray:
    return t.detach().float().cpu().double().numpy()


def assert_attn_close(gpu: np.ndarray, ref: np.ndarray, what: str):
    err = np.abs(gpu - ref)
    bound = ATOL + RTOL * np.abs(ref)
    bad = err > bound
    assert not bad.any(), (f"{what}: {int(bad.sum())} of {bad.size} outside tolerance; "
                           f"max err {err.max():.3e} at {np.unravel_index(err.argmax(), err.shape)}")


def policy_dict(pol):
    d = dict(action=pol.action, floor=pol.floor, group_of_layer=pol.group_of_layer, n_sink=pol.n_sink,
             rho_up=pol.rho_up, recent_window=pol.recent_window)
    if pol.n_states:
        d.update(n_states=pol.n_states, beta_q=pol.beta_q, reserve_q=pol.reserve_q, crit=pol.crit)
    return d


def budgets(cnt: np.ndarray) -> np.ndarray:
    """Remaining budget R (int64) from host counters [..., 8] (words 6, 7)."""
    return np.ascontiguousarray(cnt[..., 6:8]).view(np.int64)[..., 0]


class Scenario:
    """B sequences x L layers: a prompt (kept HIGH, or tagged), then generated
    tokens with tags, appended step by step or in bulk, with fused decode
    attention at chosen steps.  Inputs are generated on the CPU."""

    def __init__(self, pol, *, B, L, Hq, Hkv, D, prompt_lens, gen_tags, seed, prompt_tags=None,
                 max_ctx_hint=None, hi_pages=None, lo_pages=None, extra_bytes=0, outliers=0, gen_states=None,
                 expect_flags=0, q_scale=1.0, v_scale=1.0, prefill=None):
        from paper_2608_28276_amd.session import PaskSession
        self.pol, self.B, self.L, self.Hq, self.Hkv, self.D = pol, B, L, Hq, Hkv, D
        self.P = np.asarray(prompt_lens, dtype=np.int64)
        self.gen_tags = np.asarray(gen_tags, dtype=np.uint8).reshape(B, -1)
        # parser states of the generated tokens: the online controller decides
        self.gen_states = None if gen_states is None else np.asarray(gen_states, dtype=np.uint8).reshape(B, -1)
        self.expect_flags = expect_flags
        self.T = self.gen_tags.shape[1]
        self.prompt_tags = prompt_tags
        self.seed = seed
        self.max_tok = int(self.P.max()) + self.T
        pages = lambda n: int(np.sum((np.asarray(n, dtype=np.int64) + 15) // 16))
        if hi_pages is None:
            hi_pages = L * pages(self.P + self.T)
        if lo_pages is None:
            lo_pages = L * pages((self.P if prompt_tags is not None else np.zeros(B, np.int64)) + self.T)
        self.sess = PaskSession(pack_blob(pol), max_batch=B, n_layers=L, n_q_heads=Hq, n_kv_heads=Hkv,
                                head_dim=D, max_tokens_per_seq=self.max_tok, hi_pages=hi_pages,
                                lo_pages=lo_pages, max_ctx_hint=max_ctx_hint, extra_bytes=extra_bytes,
                                prefill=prefill)
        self.oc = oracle.OracleCache(policy_dict(pol), Hkv, D)
        self.scale = self.sess.softmax_scale
        self.outliers = outliers
        # powers of two scale q and V exactly in bf16 (stress inputs: large
        # scores, small V scales)
        for x in (q_scale, v_scale):
            assert x > 0 and math.frexp(x)[0] == 0.5, "q_scale and v_scale must be powers of two"
        self.q_scale, self.v_scale = q_scale, v_scale
        self.dev = self.sess.device

    # -- inputs ----------------------------------------------------------
    def prompt_kv(self, layer):
        shape = (self.B, int(self.P.max()), self.Hkv, self.D)
        k = bf16_normal(shape, sub_seed(self.seed, "prompt_k", layer), outlier_channels=self.outliers)
        v = bf16_normal(shape, sub_seed(self.seed, "prompt_v", layer)) * self.v_scale
        return k, v

    def gen_kv(self, layer, t0, t1):
        """K/V of generated tokens t0..t1-1: [B, t1 - t0, Hkv, D]."""
        k = torch.stack([bf16_normal((self.B, self.Hkv, self.D), sub_seed(self.seed, "gen_k", layer, t),
                                     outlier_channels=self.outliers) for t in range(t0, t1)], dim=1)
        v = torch.stack([bf16_normal((self.B, self.Hkv, self.D), sub_seed(self.seed, "gen_v", layer, t))
                         for t in range(t0, t1)], dim=1) * self.v_scale
        return k, v

    def q(self, layer, t):
        return bf16_normal((self.B, self.Hq, self.D), sub_seed(self.seed, "q", layer, t)) * self.q_scale

    # -- driving both sides ---------------------------------------------
    def budget_init(self, t_max: int):
        self.sess.budget_init(t_max, batch=self.B)
        for b in range(self.B):
            self.oc.budget_init(b, range(self.L), t_max)

    def _states(self, t0, t1):
        return None if self.gen_states is None else np.ascontiguousarray(self.gen_states[:, t0:t1])

    def fill_prompt(self, layers=None):
        for layer in (range(self.L) if layers is None else layers):
            k, v = self.prompt_kv(layer)
            n_new = torch.as_tensor(self.P, dtype=torch.int32, device=self.dev)
            kd, vd = k.to(self.dev), v.to(self.dev)
            if self.prompt_tags is None:
                self.sess.append(layer, None, kd, vd, n_new=n_new, keep_all=True)
            else:
                tg = torch.as_tensor(self.prompt_tags, dtype=torch.uint8, device=self.dev)
                self.sess.append(layer, tg, kd, vd, n_new=n_new)
            for b in range(self.B):
                p = int(self.P[b])
                tags = np.zeros(p, np.uint8) if self.prompt_tags is None else self.prompt_tags[b, :p]
                self.oc.append(layer, b, tags, bits16(k[b, :p]), bits16(v[b, :p]),
                               keep_all=self.prompt_tags is None)

    def append_steps(self, t0, t1, layers=None):
        """Bulk-append generated tokens t0..t1-1 (no attention)."""
        if t1 <= t0:
            return
        for layer in (range(self.L) if layers is None else layers):
            k, v = self.gen_kv(layer, t0, t1)
            tg = torch.as_tensor(np.ascontiguousarray(self.gen_tags[:, t0:t1]), device=self.dev)
            st = self._states(t0, t1)
            sd = None if st is None else torch.as_tensor(st, device=self.dev)
            self.sess.append(layer, tg, k.to(self.dev), v.to(self.dev), states=sd)
            for b in range(self.B):
                self.oc.append(layer, b, self.gen_tags[b, t0:t1], bits16(k[b]), bits16(v[b]),
                               states=None if st is None else st[b])

    def decode_step(self, t, layers=None, check=True, seqs=None, noalloc=False):
        """Fused append of token t + attention, on every layer; compare.  The
        outputs and log-sum-exps of the last call per layer stay in
        self.last[layer]; noalloc: through pask_decode_attn_noalloc."""
        worst = 0.0
        self.last = getattr(self, "last", {})
        for layer in (range(self.L) if layers is None else layers):
            k, v = self.gen_kv(layer, t, t + 1)
            q = self.q(layer, t)
            out = torch.empty((self.B, self.Hq, self.D), dtype=torch.bfloat16, device=self.dev)
            lse = torch.empty((self.B, self.Hq), dtype=torch.float32, device=self.dev)
            tg = torch.as_tensor(np.ascontiguousarray(self.gen_tags[:, t]), device=self.dev)
            st = self._states(t, t + 1)
            sd = None if st is None else torch.as_tensor(np.ascontiguousarray(st[:, 0]), device=self.dev)
            call = self.sess.decode_noalloc if noalloc else self.sess.decode
            call(layer, q.to(self.dev), out, lse, tg, k[:, 0].contiguous().to(self.dev),
                 v[:, 0].contiguous().to(self.dev), states_new=sd)
            self.last[layer] = (out, lse)
            for b in range(self.B):
                self.oc.append(layer, b, self.gen_tags[b, t:t + 1], bits16(k[b]), bits16(v[b]),
                               states=None if st is None else st[b])
            if not check:
                continue
            self.check_state(layers=[layer], seqs=seqs)
            o_gpu = bf16_f64(out)
            l_gpu = lse.cpu().double().numpy()
            for b in (range(self.B) if seqs is None else seqs):
                o_ref, lse_ref = self.oc.attend(layer, b, bits16(q[b]), self.scale)
                assert_attn_close(o_gpu[b], o_ref, f"attention step {t} layer {layer} seq {b}")
                if self.v_scale != 1.0:   # the same bound in units of the V scale
                    assert_attn_close(o_gpu[b] / self.v_scale, o_ref / self.v_scale,
                                      f"attention / v_scale, step {t} layer {layer} seq {b}")
                fin = np.isfinite(lse_ref)
                assert (np.isneginf(l_gpu[b]) == ~fin).all()
                assert np.abs(l_gpu[b][fin] - lse_ref[fin]).max(initial=0) <= 1e-4 + 1e-5 * np.abs(lse_ref[fin]).max(initial=0)
                worst = max(worst, float(np.abs(o_gpu[b] - o_ref).max(initial=0)))
        return worst

    # -- bit-exact state comparison --------------------------------------
    def check_state(self, layers=None, seqs=None):
        cnt = self.sess.counters().cpu().numpy()
        il = self.sess.index_lists().cpu().numpy()
        for layer in (range(self.L) if layers is None else layers):
            for b in (range(self.B) if seqs is None else seqs):
                c = self.oc.counts(b, layer)
                got = cnt[b, layer]
                assert (got[0], got[1], got[2], got[3], got[4], got[5]) == \
                    (c["hi"], c["lo"], c["pos"], c["drop"], c["forced"], 0), (layer, b, got, c)
                if self.gen_states is not None:
                    assert int(budgets(got)) == c["R"], ("remaining budget", layer, b, int(budgets(got)), c["R"])
                hi, lo = self.oc.lists(b, layer)
                assert (il[b, layer, 0, :hi.size] == hi).all(), ("HIGH list", layer, b)
                assert (il[b, layer, 1, :lo.size] == lo).all(), ("LOW list", layer, b)
                gk, gv = self.sess.gather_store(b, layer, 0)
                ok, ov = self.oc.hi_entries(b, layer)
                assert (gk == ok).all() and (gv == ov).all(), ("HIGH bf16 copies", layer, b)
                kc, ks, vc, vs = self.sess.gather_store(b, layer, 1)
                okc, oks, ovc, ovs = self.oc.lo_entries(b, layer)
                assert (kc == okc).all(), ("LOW K codes", layer, b)
                assert (vc == ovc).all(), ("LOW V codes", layer, b)
                assert (ks == oks).all() and (vs == ovs).all(), ("LOW scales", layer, b)
                if self.sess.window:
                    wpos, wk, wv = self.sess.gather_window(b, layer)
                    sl = self.oc.sl(b, layer)
                    assert (wpos == sl.w_pos).all(), ("window positions", layer, b)
                    if wpos.size:
                        assert (wk == sl.w_k).all() and (wv == sl.w_v).all(), ("window bf16 bits", layer, b)
        st, status, _ = self.sess.stats(batch=self.B)
        sw = self.sess.status_words().cpu().numpy()
        assert st.device_flags == self.expect_flags, (
            f"device flags {st.device_flags:#x}; cursors {sw[2]}, {sw[3]} of pools "
            f"{self.sess.geom.hi_pages}, {self.sess.geom.lo_pages}; lost {st.n_lost}")
