#!/usr/bin/env python3
"""Decode-attention throughput of the PASK hot path on one MI355X.

One step = one decode step of every sequence through every layer: per layer
pask_kv_append persists the step's token (table lookup, compaction,
quantise-and-pack or bf16 copy) and pask_decode_attn runs grouped-query
attention over the layer's mixed bf16 / int4 cache.  Prints one JSON line.

Workload (default): Qwen3-4B attention geometry (36 layers in 4 groups,
32 query / 8 KV heads, head_dim 128), batch 64, prompts U{1024..8192} kept
RETAIN-HIGH, function-call tag streams read by the tagger from seeded tool-call output, a
6 x 4 policy table at budget 0.33.  512 generated tokens are persisted
before timing; the timed steps continue the same streams.  Synthetic data,
random values; inputs are resident in HBM before the timed region.
"""

from __future__ import annotations

import argparse
import json
import math
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

import numpy as np  # noqa: E402

METRIC = "decode-attn tokens/s at KV budget 0.33; achieved HBM GB/s vs MI355X peak"
HBM_PEAK_GBS = 8000.0


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def build_workload(cfg_idx: int, beta: float | None = None):
    """Workload shapes, generated-token tags [B, T], the policy table and,
    for the prompt-side workload, the prompt labels [B, max P] (else None)."""
    from workload import CONFIGS, make_policy, prompt_lengths, schema_prompt_tags, tag_mix, function_call_tags
    from workload.tags import iid_tags
    from workload.tensors import sub_seed
    cfg = CONFIGS[cfg_idx]
    P = prompt_lengths(cfg)
    if beta is None:
        beta = cfg.budgets[0] if len(cfg.budgets) == 1 else 0.33
    if cfg.tag_source == "calls":
        tags = np.stack([function_call_tags(cfg.gen_tokens, sub_seed(cfg.seed, "tags", b))
                         for b in range(cfg.batch)])
        probs = tag_mix(function_call_tags(200000, sub_seed(cfg.seed, "tags", 1 << 20)), 6)
    else:
        tags = np.stack([iid_tags(cfg.gen_tokens, sub_seed(cfg.seed, "tags", b)) for b in range(cfg.batch)])
        probs = None
    ptags = None
    if cfg.prompt_tagged:
        # prompt-side companion: prompt labels under the same table (12 tags), sinks kept HIGH
        ptags = np.zeros((cfg.batch, int(P.max())), np.uint8)
        for b, p in enumerate(P):
            ptags[b, :p] = schema_prompt_tags(int(p), sub_seed(cfg.seed, "prompt_tags", b))
        probs = tag_mix(np.concatenate([ptags[b, :P[b]] for b in range(cfg.batch)] + [tags.ravel()]), 12)
        pol = make_policy(12, cfg.n_groups, cfg.n_layers, beta, cfg.seed, tag_probs=probs, n_sink=cfg.n_sink)
    else:
        pol = make_policy(6, cfg.n_groups, cfg.n_layers, beta, cfg.seed, tag_probs=probs)
    return cfg, P, tags.astype(np.uint8), pol, ptags


def controller_inputs(cfg, tags, pol):
    """Parser states of the tagged tool-call streams (the same seeds give the same tags)
    and the table with the controller's reserve, calibrated on eight tagged
    traces of the generation length."""
    from workload.policy import with_budget_controller
    from workload.tags import CRITICAL_STATES, PARSER_STATES, function_call_tags_with_states
    from workload.tensors import sub_seed
    ts = [function_call_tags_with_states(cfg.gen_tokens, sub_seed(cfg.seed, "tags", b)) for b in range(cfg.batch)]
    assert all((t == tags[b]).all() for b, (t, _) in enumerate(ts)), "controller runs need tagger tags"
    cal = [function_call_tags_with_states(cfg.gen_tokens, sub_seed(cfg.seed, "tags", 1000 + i)) for i in range(8)]
    pol = with_budget_controller(pol, cal, len(PARSER_STATES), CRITICAL_STATES)
    return np.stack([s for _, s in ts]).astype(np.uint8), pol


class HipEvent:
    """A HIP event recorded on the launch stream, created with
    hipEventDisableSystemFence: recording it does not write back and
    invalidate the caches, so it costs the timed step about 1% where a
    default event (torch.cuda.Event) leaves the GPU idle for about 5 us.
    The runtime is the one torch loaded (same soname), so torch's stream
    handles are valid here."""

    _hip = None
    DISABLE_SYSTEM_FENCE = 0x20000000

    def __init__(self):
        import ctypes as C
        if HipEvent._hip is None:
            hip = C.CDLL("libamdhip64.so.7")
            hip.hipEventCreateWithFlags.argtypes = [C.POINTER(C.c_void_p), C.c_uint]
            hip.hipEventRecord.argtypes = [C.c_void_p, C.c_void_p]
            hip.hipEventElapsedTime.argtypes = [C.POINTER(C.c_float), C.c_void_p, C.c_void_p]
            hip.hipEventDestroy.argtypes = [C.c_void_p]
            HipEvent._hip = hip
        self._e = C.c_void_p()
        self._lib = HipEvent._hip      # kept for __del__, which may run after module teardown
        if HipEvent._hip.hipEventCreateWithFlags(C.byref(self._e), self.DISABLE_SYSTEM_FENCE) != 0:
            raise RuntimeError("hipEventCreateWithFlags failed")

    def record(self, stream_handle: int):
        import ctypes as C
        if HipEvent._hip.hipEventRecord(self._e, C.c_void_p(stream_handle)) != 0:
            raise RuntimeError("hipEventRecord failed")

    def elapsed_ms(self, end: "HipEvent") -> float:
        import ctypes as C
        ms = C.c_float()
        if HipEvent._hip.hipEventElapsedTime(C.byref(ms), self._e, end._e) != 0:
            raise RuntimeError("hipEventElapsedTime failed")
        return ms.value

    def __del__(self):
        lib = getattr(self, "_lib", None)
        if lib is not None and self._e:
            lib.hipEventDestroy(self._e)


def plan_pool_pages(cfg, P, tags, pol, ptags, online: bool):
    """Pages of the HIGH and LOW pools for the whole run (memory planning on
    the host, as a server holding the table and the tag streams would do):
    the frozen table's action of every (token, layer group) - the higher of
    selected action and floor, sinks and keep-all prompts HIGH - counted per
    (sequence, layer) store.  Under the online controller the actions move
    with the budget, so every token gets room in both pools."""
    B, L, T = cfg.batch, cfg.layers_resident, cfg.gen_tokens
    pages = lambda n: int(np.sum((np.asarray(n) + 15) // 16))
    if online:
        return L * pages(P + T), L * pages((P if ptags is not None else 0) + np.full(B, T))
    act = np.maximum(np.asarray(pol.action), np.asarray(pol.floor))          # [tags, groups]
    gol = np.asarray(pol.group_of_layer)[:L]
    hi = lo = 0
    for b in range(B):
        z = np.concatenate([ptags[b, :P[b]] if ptags is not None else np.zeros(P[b], np.uint8), tags[b, :T]])
        forced = np.arange(z.size) < (pol.n_sink if ptags is not None else P[b])   # sinks / kept prompt
        for c in np.unique(gol):
            a = np.where(forced, 2, act[z, c])
            n_layers_c = int(np.sum(gol == c))
            hi += n_layers_c * pages(int(np.sum(a == 2)))
            lo += n_layers_c * pages(int(np.sum(a == 1)))
    return hi + L * B, lo + L * B                                            # + one spare page per store


def gpu_leg(cfg, P, tags, pol, steps: int, warmup: int, positions, states=None, ptags=None, graph=False):
    """Times the decode step at each position t of `positions` (generated
    tokens persisted before the first warm-up step; ascending): the tokens up
    to t are bulk-appended untimed, then `warmup` steps, then `steps` timed
    steps.  With `graph`, `steps` more steps follow, each a replay of one HIP
    graph holding the whole step (every layer's append and attention
    launches), the step's tags copied into the graph's input buffer first.
    Returns one result per position."""
    import torch

    from paper_2608_28276_amd import pask
    from paper_2608_28276_amd.session import PaskSession
    from workload.policy import pack_blob

    dev = torch.device("cuda:0")
    B, L, Hq, Hkv, D = cfg.batch, cfg.layers_resident, cfg.n_q_heads, cfg.n_kv_heads, cfg.head_dim
    T = cfg.gen_tokens
    positions = sorted(positions)
    per_pos = warmup + steps * (2 if graph else 1)
    assert positions[0] >= 0 and positions[-1] + per_pos <= T, "not enough generated tokens for the steps"
    assert all(b >= a + per_pos for a, b in zip(positions, positions[1:])), "timed ranges overlap"
    hi_pages, lo_pages = plan_pool_pages(cfg, P, tags, pol, ptags, online=states is not None)
    max_tok = int(P.max()) + T
    sess = PaskSession(pack_blob(pol), max_batch=B, n_layers=cfg.n_layers, n_q_heads=Hq, n_kv_heads=Hkv,
                       head_dim=D, max_tokens_per_seq=max_tok, hi_pages=hi_pages, lo_pages=lo_pages,
                       max_ctx_hint=max_tok)
    log(f"cache {sess.nbytes / 2**30:.1f} GiB, workspace {sess.ws_bytes / 2**20:.1f} MiB")
    if states is not None:
        sess.budget_init(T, batch=B)                     # online controller: R_0 for T_max = T
        states_dev = torch.as_tensor(states, dtype=torch.uint8, device=dev)
    g = torch.Generator(device=dev)
    g.manual_seed(cfg.seed)
    n_new = torch.as_tensor(P, dtype=torch.int32, device=dev)
    tags_dev = torch.as_tensor(tags, device=dev)
    ptags_dev = None if ptags is None else torch.as_tensor(ptags, device=dev)
    t0 = time.time()
    sptr = torch.cuda.current_stream(dev).cuda_stream
    fill_ev = [(HipEvent(), HipEvent()) for _ in range(L)]
    after_prompt = []                                    # counters of each layer right after its prompt
    for layer in range(L):
        k = torch.randn((B, int(P.max()), Hkv, D), generator=g, device=dev, dtype=torch.bfloat16)
        v = torch.randn((B, int(P.max()), Hkv, D), generator=g, device=dev, dtype=torch.bfloat16)
        fill_ev[layer][0].record(sptr)
        if ptags_dev is None:                            # decode workloads: the prompt stays HIGH
            sess.append(layer, None, k, v, n_new=n_new, keep_all=True)
        else:                                            # prompt-side companion: labelled prompt, sinks HIGH
            sess.append(layer, ptags_dev, k, v, n_new=n_new)
        fill_ev[layer][1].record(sptr)
        after_prompt.append(sess.counters()[:B, layer, :2].clone())
        del k, v
    torch.cuda.synchronize()
    log(f"prompts persisted in {time.time() - t0:.1f} s")
    # The prompt's bulk append per layer (plan + pack kernels): algorithmic bytes = the K / V rows
    # of the persisted tokens read (bf16; a released token's row is never read), tags read, the
    # stored forms and index-list entries written.
    mH = 2 * Hkv * D * 2
    mL = 2 * Hkv * (D // 2 + 2 * (D // 32))
    n_prompt = int(P.sum())
    ap = torch.stack(after_prompt).cpu().numpy().astype(np.int64)        # [L, B, 2]: n_hi, n_lo
    kept = ap[..., 0].sum(1) + ap[..., 1].sum(1)                          # [L]
    pa_bytes = (kept * mH + n_prompt * (1 if ptags is not None else 0) + ap[..., 0].sum(1) * (mH + 4)
                + ap[..., 1].sum(1) * (mL + 4))                          # [L]
    pa_ms = np.array([e0.elapsed_ms(e1) for e0, e1 in fill_ev])
    prompt_append = dict(tokens_per_layer=n_prompt, us_per_layer=round(float(pa_ms.mean()) * 1e3, 1),
                         algorithmic_gb_per_layer=round(float(pa_bytes.mean()) / 1e9, 4),
                         achieved_gbs=round(float((pa_bytes / (pa_ms / 1e3)).mean()) / 1e9, 1))
    log(f"prompt append: {prompt_append}")

    q = torch.randn((L, B, Hq, D), generator=g, device=dev, dtype=torch.bfloat16)
    kn = torch.randn((L, B, Hkv, D), generator=g, device=dev, dtype=torch.bfloat16)
    vn = torch.randn((L, B, Hkv, D), generator=g, device=dev, dtype=torch.bfloat16)
    out = torch.empty((L, B, Hq, D), dtype=torch.bfloat16, device=dev)
    tags_t = tags_dev.t().contiguous()                   # [T, B]
    states_t = None if states is None else states_dev.t().contiguous()
    pol_c, cache_c = sess.policy, sess.cache
    ws, ws_bytes, hint, scale = sess.ws.data_ptr(), sess.ws_bytes, sess.max_ctx_hint, sess.softmax_scale
    qp = [q[i].data_ptr() for i in range(L)]
    op = [out[i].data_ptr() for i in range(L)]
    kp = [kn[i].data_ptr() for i in range(L)]
    vp = [vn[i].data_ptr() for i in range(L)]
    lib = pask.library()
    import ctypes as C
    pol_ref, cache_ref = C.byref(pol_c), C.byref(cache_c)

    def step(t, events=None, stream=None, tp=None, sp=None):
        # One decode step: per layer, one pask_decode_attn call that persists the
        # step's token and attends the layer's history including it (the
        # attention and merge kernels persist the token themselves for at most
        # 256 sequences without a recent window or parser states; otherwise the
        # one-token append kernel runs first, inside the same call).
        sptr_ = sptr if stream is None else stream
        if tp is None:
            tp = tags_t[t].data_ptr()
            sp = None if states_t is None else states_t[t].data_ptr()
        for layer in range(L):
            if events is not None:
                events[layer][0].record(sptr_)
            st = lib.pask_decode_attn(pol_ref, cache_ref, layer, B, qp[layer], op[layer], None, tp, sp, kp[layer],
                                      vp[layer], C.c_float(scale), hint, ws, ws_bytes, sptr_)
            if st != 0:
                raise pask.PaskError(st, "pask_decode_attn")
            if events is not None:
                events[layer][1].record(sptr_)

    def graph_steps(t0):
        """`steps` decode steps from t0 as replays of one captured step."""
        tags_cur = torch.empty(B, dtype=torch.uint8, device=dev)
        states_cur = None if states_t is None else torch.empty(B, dtype=torch.uint8, device=dev)
        tags_cur.copy_(tags_t[t0])
        if states_cur is not None:
            states_cur.copy_(states_t[t0])
        gr = torch.cuda.CUDAGraph()
        with torch.cuda.graph(gr):
            cap = torch.cuda.current_stream(dev).cuda_stream
            step(None, stream=cap, tp=tags_cur.data_ptr(),
                 sp=None if states_cur is None else states_cur.data_ptr())
        torch.cuda.synchronize()
        w0 = time.perf_counter()
        for i in range(steps):
            tags_cur.copy_(tags_t[t0 + i])
            if states_cur is not None:
                states_cur.copy_(states_t[t0 + i])
            gr.replay()
        torch.cuda.synchronize()
        wall = time.perf_counter() - w0
        del gr
        return wall

    W = int(pol.recent_window)
    kv_bytes = lambda c: c[..., 0] * mH + c[..., 1] * mL + np.minimum(c[..., 2], W) * mH   # stores + window
    results = []
    t = 0                                                # generated tokens persisted so far
    for pos in positions:
        if pos > t:                                      # untimed bulk append of tokens t..pos-1
            for layer in range(L):
                k = torch.randn((B, pos - t, Hkv, D), generator=g, device=dev, dtype=torch.bfloat16)
                v = torch.randn((B, pos - t, Hkv, D), generator=g, device=dev, dtype=torch.bfloat16)
                sess.append(layer, tags_dev[:, t:pos].contiguous(), k, v,
                            states=None if states is None else states_dev[:, t:pos].contiguous())
                del k, v
            t = pos
        for i in range(warmup):
            step(t + i)
        torch.cuda.synchronize()
        cnt0 = sess.counters()[:B, :L].cpu().numpy().astype(np.int64)
        events = [[[HipEvent(), HipEvent()] for _ in range(L)] for _ in range(steps)]
        torch.cuda.synchronize()
        w0 = time.perf_counter()
        for i in range(steps):
            step(t + warmup + i, events[i])
        torch.cuda.synchronize()
        wall = time.perf_counter() - w0
        t += warmup + steps
        cnt1 = sess.counters()[:B, :L].cpu().numpy().astype(np.int64)
        graph_res = None
        if graph:
            gwall = graph_steps(t)
            t += steps
            graph_res = dict(tokens_per_s=round(B * steps / gwall, 1), ms_per_step=round(gwall / steps * 1e3, 4),
                             us_per_layer=round(gwall / steps / L * 1e6, 2))
            log(f"t={t - steps}: HIP graph of the step: {graph_res}")
        call_ms = np.array([[e[0].elapsed_ms(e[1]) for e in ev] for ev in events])   # [steps, L]
        st, status, _ = sess.stats(batch=B)
        if status != 0:
            raise RuntimeError(f"device flags set: {st.device_flags:#x}")

        # Algorithmic bytes of one call, averaged over the timed ones: every
        # persisted entry read once (counts grow linearly over the region, each
        # call sees its step's token), q read, o written; and the append of the
        # step's token: its K and V rows read, its stored form and one list
        # entry written.
        read = 0.5 * (kv_bytes(cnt0) + kv_bytes(cnt1)).sum(axis=0)      # per layer, summed over seqs
        qo = 2 * 2 * B * Hq * D
        attn_bytes = read + qo                                             # [L]
        new_tok = (kv_bytes(cnt1) - kv_bytes(cnt0)).sum(axis=0) / steps  # per layer per step
        stored = ((cnt1[..., 0] + cnt1[..., 1]) - (cnt0[..., 0] + cnt0[..., 1])).sum(axis=0) / steps
        if W:                                    # the token entering the window and the one leaving it
            new_tok = new_tok + 2 * B * mH
        append_bytes = new_tok + 4 * stored + 2 * B * Hkv * D * 2         # stored form + lists + k/v read
        call_bytes = attn_bytes + append_bytes                             # [L]
        bytes_per_step = float(call_bytes.sum())
        avg_call_s = float(call_ms.mean()) / 1e3
        achieved = float(call_bytes.mean()) / avg_call_s / 1e9
        res = dict(
            t=pos, tokens_per_s=B * steps / wall, ms_per_step=wall / steps * 1e3, achieved=achieved,
            avg_call_us=avg_call_s * 1e6, bytes_per_step=bytes_per_step, per_call_bytes=float(call_bytes.mean()),
            c_kv_governed=st.c_kv_governed, c_kv_all=st.c_kv_all,
            step_gbs=bytes_per_step / (wall / steps) / 1e9,
            mean_entries=float((cnt1[..., 0] + cnt1[..., 1]).mean()), prompt_append=prompt_append,
            graph=graph_res,
        )
        log(f"t={pos}: {res['tokens_per_s']:.0f} tokens/s, call {res['avg_call_us']:.1f} us, "
            f"{achieved:.0f} GB/s algorithmic")
        results.append(res)
    return results


def probe_leg(read_gib: float = 4.0, copy_gib: float = 2.0, reps: int = 5):
    """On-device ceilings measured on the same box in the same run: the
    streaming read and copy probes (paper_2608_28276_amd/csrc/probe.hip),
    HIP events around `reps` back-to-back launches after a warm-up."""
    import ctypes as C

    import torch
    lib = C.CDLL(os.path.join(ROOT, "paper_2608_28276_amd", "libpask_probe.so"))
    lib.pask_probe_read.argtypes = [C.c_void_p, C.c_size_t, C.c_void_p, C.c_int, C.c_void_p]
    lib.pask_probe_copy.argtypes = [C.c_void_p, C.c_void_p, C.c_size_t, C.c_int, C.c_void_p]
    dev = torch.device("cuda:0")
    sptr = torch.cuda.current_stream(dev).cuda_stream
    nr, nc = int(read_gib * 2**30), int(copy_gib * 2**30)
    x = torch.empty(nr, dtype=torch.uint8, device=dev).fill_(3)
    outw = torch.empty(65536, dtype=torch.int32, device=dev)
    y = torch.empty(nc, dtype=torch.uint8, device=dev)

    def timed(fn):
        if fn() != 0:
            raise RuntimeError("probe launch failed")
        e0, e1 = HipEvent(), HipEvent()
        e0.record(sptr)
        for _ in range(reps):
            if fn() != 0:
                raise RuntimeError("probe launch failed")
        e1.record(sptr)
        torch.cuda.synchronize()
        return e0.elapsed_ms(e1) / 1e3 / reps

    rd = timed(lambda: lib.pask_probe_read(x.data_ptr(), nr, outw.data_ptr(), 0, sptr))
    cp = timed(lambda: lib.pask_probe_copy(x.data_ptr(), y.data_ptr(), nc, 0, sptr))
    del x, y
    return dict(read_gbs=round(nr / rd / 1e9, 1), copy_gbs=round(2 * nc / cp / 1e9, 1),
                read_bytes=nr, copy_bytes=nc)


def distortion_leg(cfg, P, tags, pol, steps: int, warmup: int, t_start: int, bucket):
    """Attention-output distortion (Eq. 4) of bucket (z, c) with action a on
    the workload's trajectories: a reference cache (every bucket HIGH) and an
    intervened cache (bucket (z, c) -> a) hold the same tokens of the layers
    of group c.  One step appends each sequence's next token to both caches
    in every such layer, then pask_attn_distortion adds max_h ||o_ref - o_int||^2
    of every layer for the sequences whose bucket has occurred (S(q))."""
    import ctypes as C
    from dataclasses import replace

    import torch

    from paper_2608_28276_amd import pask
    from paper_2608_28276_amd.session import PaskSession
    from workload.policy import pack_blob

    z, c, act = bucket
    dev = torch.device("cuda:0")
    B, Hq, Hkv, D, T = cfg.batch, cfg.n_q_heads, cfg.n_kv_heads, cfg.head_dim, cfg.gen_tokens
    layers = [l for l in range(cfg.layers_resident) if int(pol.group_of_layer[l]) == c]
    full = np.full_like(np.asarray(pol.action), 2)
    inter = full.copy()
    inter[z, c] = act
    pol_ref = replace(pol, action=full, floor=np.zeros_like(full))
    pol_int = replace(pol, action=inter, floor=np.zeros_like(full))
    pages = lambda n: int(np.sum((np.asarray(n) + 15) // 16))
    hi = len(layers) * (pages(P + T) + B)
    lo = len(layers) * (pages(np.full(B, T)) + B) if act == 1 else len(layers) * B
    max_tok = int(P.max()) + T
    mk = lambda pl, lo_pages: PaskSession(pack_blob(pl), max_batch=B, n_layers=cfg.n_layers, n_q_heads=Hq,
                                          n_kv_heads=Hkv, head_dim=D, max_tokens_per_seq=max_tok, hi_pages=hi,
                                          lo_pages=lo_pages, max_ctx_hint=max_tok)
    ref, itv = mk(pol_ref, B), mk(pol_int, lo)
    log(f"distortion of bucket (tag {z}, group {c}) -> action {act}: layers {layers[0]}..{layers[-1]}, "
        f"caches {ref.nbytes / 2**30:.1f} + {itv.nbytes / 2**30:.1f} GiB")
    g = torch.Generator(device=dev)
    g.manual_seed(cfg.seed)
    n_new = torch.as_tensor(P, dtype=torch.int32, device=dev)
    tags_dev = torch.as_tensor(tags, device=dev)
    for layer in layers:
        k = torch.randn((B, int(P.max()), Hkv, D), generator=g, device=dev, dtype=torch.bfloat16)
        v = torch.randn((B, int(P.max()), Hkv, D), generator=g, device=dev, dtype=torch.bfloat16)
        for sess in (ref, itv):
            sess.append(layer, None, k, v, n_new=n_new, keep_all=True)
        k = torch.randn((B, t_start, Hkv, D), generator=g, device=dev, dtype=torch.bfloat16)
        v = torch.randn((B, t_start, Hkv, D), generator=g, device=dev, dtype=torch.bfloat16)
        for sess in (ref, itv):
            sess.append(layer, tags_dev[:, :t_start].contiguous(), k, v)
        del k, v
    seen = np.cumsum(tags == z, axis=1) > 0                                 # [B, T]: bucket occurred by step t
    in_s = torch.as_tensor(seen.T.astype(np.uint8).copy(), device=dev)      # [T, B]
    nL = len(layers)
    q = torch.randn((nL, B, Hq, D), generator=g, device=dev, dtype=torch.bfloat16)
    kn = torch.randn((nL, B, Hkv, D), generator=g, device=dev, dtype=torch.bfloat16)
    vn = torch.randn((nL, B, Hkv, D), generator=g, device=dev, dtype=torch.bfloat16)
    tags_t = tags_dev.t().contiguous()
    ws_bytes = 2 * ref.ws_bytes
    ws = torch.empty(ws_bytes, dtype=torch.uint8, device=dev)
    dist = torch.zeros(B, dtype=torch.float32, device=dev)
    sptr = torch.cuda.current_stream(dev).cuda_stream
    lib = pask.library()
    r_pol, r_cache, i_pol, i_cache = (C.byref(ref.policy), C.byref(ref.cache), C.byref(itv.policy),
                                      C.byref(itv.cache))
    scale, hint = C.c_float(ref.softmax_scale), ref.max_ctx_hint

    def step(t, events=None):
        tp = tags_t[t].data_ptr()
        for i, layer in enumerate(layers):
            for pp, cc in ((r_pol, r_cache), (i_pol, i_cache)):
                st = lib.pask_kv_append(pp, cc, layer, B, None, 1, tp, None, kn[i].data_ptr(), vn[i].data_ptr(), 0,
                                        sptr)
                if st != 0:
                    raise pask.PaskError(st, "pask_kv_append")
            if events is not None:
                events[i][0].record(sptr)
            st = lib.pask_attn_distortion(r_cache, i_cache, layer, B, q[i].data_ptr(), in_s[t].data_ptr(), scale,
                                          hint, ws.data_ptr(), ws_bytes, dist.data_ptr(), sptr)
            if st != 0:
                raise pask.PaskError(st, "pask_attn_distortion")
            if events is not None:
                events[i][1].record(sptr)

    for i in range(warmup):
        step(t_start + i)
    torch.cuda.synchronize()
    cnt0 = [s.counters()[:B, layers].cpu().numpy().astype(np.int64) for s in (ref, itv)]
    events = [[[HipEvent(), HipEvent()] for _ in layers] for _ in range(steps)]
    dist.zero_()
    torch.cuda.synchronize()
    w0 = time.perf_counter()
    for i in range(steps):
        step(t_start + warmup + i, events[i])
    torch.cuda.synchronize()
    wall = time.perf_counter() - w0
    cnt1 = [s.counters()[:B, layers].cpu().numpy().astype(np.int64) for s in (ref, itv)]
    call_ms = np.array([[e[0].elapsed_ms(e[1]) for e in ev] for ev in events])
    n_s = int(seen[:, t_start + warmup:t_start + warmup + steps].sum())
    d = float(dist.sum().item()) / max(1, n_s)
    mH = 2 * Hkv * D * 2
    mL = 2 * Hkv * (D // 2 + 2 * (D // 32))
    kvb = lambda cn: cn[..., 0] * mH + cn[..., 1] * mL
    read = sum(0.5 * (kvb(a) + kvb(b)).sum() for a, b in zip(cnt0, cnt1)) / nL     # both caches, per call
    call_bytes = float(read + 2 * 2 * B * Hq * D)                                   # + q read by both passes
    return dict(steps_per_s=B * steps / wall, ms_per_step=wall / steps * 1e3, avg_call_us=float(call_ms.mean()) * 1e3,
                call_bytes=call_bytes, achieved=call_bytes / (float(call_ms.mean()) / 1e3) / 1e9, D=d, n_s=n_s,
                layers=nL)


def cpu_leg(cfg, P, tags, pol, t_start: int, n_seq: int, states=None, ptags=None):
    """The oracle as it stands, on a bounded sample: n_seq sequences of the
    same workload (their prompt lengths and tag streams, seeded CPU inputs),
    history built untimed, then one timed decode step through all layers."""
    import threadpoolctl
    import torch

    import oracle
    from workload.tensors import bf16_normal, sub_seed
    L, Hq, Hkv, D = cfg.layers_resident, cfg.n_q_heads, cfg.n_kv_heads, cfg.head_dim
    pd = dict(action=pol.action, floor=pol.floor, group_of_layer=pol.group_of_layer, n_sink=pol.n_sink,
              rho_up=pol.rho_up, recent_window=pol.recent_window)
    if states is not None:
        pd.update(n_states=pol.n_states, beta_q=pol.beta_q, reserve_q=pol.reserve_q, crit=pol.crit)
    oc = oracle.OracleCache(pd, Hkv, D)
    st_of = (lambda b, t0, t1: None) if states is None else (lambda b, t0, t1: states[b, t0:t1])
    bits = lambda t: t.contiguous().view(torch.int16).numpy().view(np.uint16)
    seqs = list(range(min(n_seq, cfg.batch)))
    for b in seqs:
        if states is not None:
            oc.budget_init(b, range(L), cfg.gen_tokens)
        for layer in range(L):
            p = int(P[b])
            k = bf16_normal((p + t_start, Hkv, D), sub_seed(cfg.seed, "prompt_k", layer, b))
            v = bf16_normal((p + t_start, Hkv, D), sub_seed(cfg.seed, "prompt_v", layer, b))
            if ptags is None:
                oc.append(layer, b, np.zeros(p, np.uint8), bits(k[:p]), bits(v[:p]), keep_all=True)
            else:
                oc.append(layer, b, ptags[b, :p], bits(k[:p]), bits(v[:p]))
            oc.append(layer, b, tags[b, :t_start], bits(k[p:]), bits(v[p:]), states=st_of(b, 0, t_start))
    q = bf16_normal((L, Hq, D), sub_seed(cfg.seed, "q", 0))
    kn = bf16_normal((L, Hkv, D), sub_seed(cfg.seed, "gen_k", 0))
    vn = bf16_normal((L, Hkv, D), sub_seed(cfg.seed, "gen_v", 0))
    scale = float(np.float32(1.0 / math.sqrt(D)))
    # The oracle is a per-head loop of small products: timed with its BLAS pool
    # held to one thread, it runs on one core (torch's own pool too).
    torch_threads = torch.get_num_threads()
    torch.set_num_threads(1)
    try:
        with threadpoolctl.threadpool_limits(1):
            t0 = time.perf_counter()
            for b in seqs:
                for layer in range(L):
                    oc.append(layer, b, tags[b, t_start:t_start + 1], bits(kn[layer][None]), bits(vn[layer][None]),
                              states=st_of(b, t_start, t_start + 1))
                    oc.attend(layer, b, bits(q[layer]), scale)
            el = time.perf_counter() - t0
    finally:
        torch.set_num_threads(torch_threads)
    return dict(value=len(seqs) / el, unit="tokens/s", cores=1, kind="oracle",
                sample=f"{len(seqs)} sequences (prompts {', '.join(str(int(P[b])) for b in seqs)} + {t_start} "
                       f"generated tokens) x 1 decode step x {L} layers, fp64 numpy on one thread, {el:.1f} s",
                threads=1, nproc=os.cpu_count(), cpu_model=cpu_model())


def cpu_model() -> str:
    """The host CPU's model name (first 'model name' line of /proc/cpuinfo)."""
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def kernel_source_digest() -> str:
    """Digest of the attention kernels' code (the kernels the traffic
    counters measure): pask_internal.h (their tuning constants), pask_device.h,
    pask_plan.h (the work split), then pask_attn.hip, each with its //
    comments, trailing blanks and empty lines removed, so that a change of
    comments alone keeps the counters valid."""
    import hashlib
    import re
    h = hashlib.sha256()
    for name in ("pask_internal.h", "pask_device.h", "pask_plan.h", "pask_attn.hip"):
        text = open(os.path.join(ROOT, "paper_2608_28276_amd", "csrc", name)).read()
        code = [re.sub(r"//.*$", "", line).rstrip() for line in text.splitlines()]
        h.update("\n".join(line for line in code if line).encode())
    return h.hexdigest()[:16]


def attn_kernels(cfg, window: int = 0, controller: bool = False) -> str:
    """The kernels of one pask_decode_attn call with its step's token: calls
    with at most 64 (sequence, KV head) segments use the equal-range attention
    and the sliced merge, larger ones the per-XCD weighted attention and the
    merge; the one-token append kernel comes first when the call cannot
    persist the token in those (more than 256 sequences, a recent window or
    parser states)."""
    D, G = cfg.head_dim, cfg.group_size
    if cfg.batch * cfg.n_kv_heads <= 64:
        k = f"attn_kernel<{D}, {G}, false> + attn_merge_sliced_kernel<{D}, {G}>"
    else:
        k = f"attn_kernel<{D}, {G}, true> + attn_merge_kernel<{D}, {G}>"
    if cfg.batch > 256 or window or controller:
        k = f"append_step{'_window' if window else ''}_kernel<{D}> + " + k
    return k


def prompt_desc(cfg) -> str:
    if cfg.prompt_dist == "fixed":
        return str(cfg.prompt_min)
    return f"{'logU' if cfg.prompt_dist == 'loguniform' else 'U'}{{{cfg.prompt_min}..{cfg.prompt_max}}}"


def traffic_record(workload: str):
    """HBM bytes per attention launch from the committed rocprofv3 counter
    summary of this workload (options included in its name), or None when the
    kernel source has changed since the counters were taken (or no summary
    exists)."""
    path = os.path.join(ROOT, "profiles", f"attn_kernel_{workload}.md")
    if not os.path.exists(path):
        return None
    for line in open(path):
        if line.startswith("<!-- traffic "):
            rec = json.loads(line[len("<!-- traffic "):line.rindex("-->")])
            if rec.get("source_digest") == kernel_source_digest():
                return rec["bytes_per_launch"]
    return None


def copy_probe(gib: float):
    """A plain copy kernel of known size: reads and writes n bytes, 3 times.
    rocprofv3 counter readings of it calibrate FETCH_SIZE / WRITE_SIZE.  Also
    reports the copy's and a read-only reduction's bandwidth (HIP events), an
    on-box reference for what a streaming kernel reaches."""
    import torch
    n = int(gib * 2**30)
    x = torch.empty(n, dtype=torch.uint8, device="cuda:0").fill_(1)
    y = torch.empty_like(x)
    torch.cuda.synchronize()
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(4)]
    for _ in range(3):
        y.copy_(x)
    ev[0].record()
    for _ in range(5):
        y.copy_(x)
    ev[1].record()
    xf = x.view(torch.bfloat16)
    xf.float().sum() if False else xf.sum(dtype=torch.float32)
    ev[2].record()
    for _ in range(5):
        xf.sum(dtype=torch.float32)
    ev[3].record()
    torch.cuda.synchronize()
    copy_gbs = 2 * n * 5 / (ev[0].elapsed_time(ev[1]) / 1e3) / 1e9
    read_gbs = n * 5 / (ev[2].elapsed_time(ev[3]) / 1e3) / 1e9
    print(json.dumps({"copy_probe_bytes": n, "copy_gbs": round(copy_gbs, 1),
                      "sum_read_gbs": round(read_gbs, 1)}), flush=True)


def main():
    ap = argparse.ArgumentParser(description=__doc__.splitlines()[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--config", type=int, default=2, help="workload index (default: the B=64 serving batch)")
    ap.add_argument("--t-start", type=int, default=None,
                    help="time only this decode position: generated tokens persisted before the warm-up "
                         "(default: three positions, 0, min(512, half the generation) and the last steps; "
                         "the line's value is the middle one)")
    ap.add_argument("--budget", type=float, default=None,
                    help="KV budget of the policy table (default: the workload's; 0.33 for the budget sweep)")
    ap.add_argument("--cpu-seqs", type=int, default=3, help="sequences in the oracle's timed sample")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--window", type=int, default=0, metavar="W",
                    help="protected recent window of W positions (Section 3.1); default 0")
    ap.add_argument("--controller", action="store_true",
                    help="parser states drive the online budget controller (Alg. 2)")
    ap.add_argument("--distortion", type=str, default=None, metavar="TAG,GROUP,ACTION",
                    help="measure the attention-output distortion (Eq. 4) of one bucket instead "
                         "(ACTION 0 = DROP, 1 = RETAIN-LOW)")
    ap.add_argument("--no-probe", action="store_true", help="skip the on-device read / copy probes")
    ap.add_argument("--graph", action="store_true",
                    help="also time the step as replays of one HIP graph (after the eager steps; one position)")
    ap.add_argument("--copy-probe", type=float, default=0.0, metavar="GIB",
                    help="only run a plain device-to-device copy of this many GiB (counter calibration)")
    args = ap.parse_args()
    if args.copy_probe:
        copy_probe(args.copy_probe)
        return
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only: the PASK hot path here has no cross-GPU part "
              f"(--gpus {args.gpus} requested)", file=sys.stderr)
        sys.exit(2)
    from workload import CONFIGS
    cfg0 = CONFIGS[args.config]
    beta = args.budget if args.budget is not None else (cfg0.budgets[0] if len(cfg0.budgets) == 1 else 0.33)
    t_default = min(512, cfg0.gen_tokens // 2)
    if args.t_start is None and not args.graph:
        args.t_start = t_default
        positions = sorted({0, t_default, cfg0.gen_tokens - args.warmup - args.steps})
    else:
        args.t_start = t_default if args.t_start is None else args.t_start
        positions = [args.t_start]
    cfg, P, tags, pol, ptags = build_workload(args.config, beta)
    pol.recent_window = args.window
    workload = (cfg.name + (f"_beta{beta:g}" if len(cfg.budgets) > 1 or beta not in cfg.budgets else "") +
                (f"+window{args.window}" if args.window else "") + ("+controller" if args.controller else "") +
                (f"+t{args.t_start}" if args.t_start != t_default else ""))
    states = None
    if args.controller:
        states, pol = controller_inputs(cfg, tags, pol)
    log(f"workload {cfg.name}: B={cfg.batch} L={cfg.n_layers} prompts {int(P.min())}..{int(P.max())}, "
        f"policy expected cost {pol.expected_cost:.3f}")
    if args.distortion:
        z, c, a = (int(x) for x in args.distortion.split(","))
        if a not in (0, 1) or not 0 <= z < pol.n_tags or not 0 <= c < pol.n_groups:
            raise SystemExit("--distortion TAG,GROUP,ACTION: tag and group of the table, action 0 or 1")
        d = distortion_leg(cfg, P, tags, pol, args.steps, args.warmup, args.t_start, (z, c, a))
        log(f"distortion: {d['steps_per_s']:.0f} sequence-steps/s, call {d['avg_call_us']:.1f} us, "
            f"{d['achieved']:.0f} GB/s, D = {d['D']:.4e} over |S| = {d['n_s']}")
        print(json.dumps({
            "metric": "attention-output distortion (Eq. 4) sequence-steps/s; achieved HBM GB/s vs MI355X peak",
            "value": round(d["steps_per_s"], 1), "unit": "sequence-steps/s", "n_gpus": 1, "steps": args.steps,
            "warmup": args.warmup, "ms_per_step": round(d["ms_per_step"], 4), "higher_is_better": True,
            "scaling": "weak", "vs_baseline": None, "dtype": "bf16", "data": "synthetic",
            "config": {"workload": f"{workload}+distortion(tag {z}, group {c}, action {a})", "batch": cfg.batch,
                       "layers_of_group": d["layers"], "q_heads": cfg.n_q_heads, "kv_heads": cfg.n_kv_heads,
                       "head_dim": cfg.head_dim, "prompt_tokens": prompt_desc(cfg),
                       "generated_before_timing": args.t_start, "D": d["D"], "S_size": d["n_s"]},
            "roofline": {"bound": "hbm", "achieved": round(d["achieved"], 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                         "frac": round(d["achieved"] / HBM_PEAK_GBS, 4), "traffic": None,
                         "kernel": f"2 x attn_kernel<{cfg.head_dim}, {cfg.group_size}, true> + distortion_kernel "
                                   "(one pask_attn_distortion call)",
                         "bytes_per_launch": round(d["call_bytes"]), "avg_launch_us": round(d["avg_call_us"], 2)},
            "cpu_baseline": None}), flush=True)
        return
    runs = gpu_leg(cfg, P, tags, pol, args.steps, args.warmup, positions, states, ptags, graph=args.graph)
    g = next(r for r in runs if r["t"] == args.t_start)
    log(f"gpu: {g['tokens_per_s']:.0f} tokens/s, {g['ms_per_step']:.2f} ms/step, call {g['avg_call_us']:.1f} us, "
        f"{g['achieved']:.0f} GB/s algorithmic")
    probe = None if args.no_probe else probe_leg()
    if probe:
        log(f"probes: read {probe['read_gbs']} GB/s, copy {probe['copy_gbs']} GB/s")
    cpu = None
    if not args.no_cpu_baseline:
        cpu = cpu_leg(cfg, P, tags, pol, args.t_start, args.cpu_seqs, states, ptags)
        log(f"cpu oracle: {cpu['value']:.3f} tokens/s on {cpu['cores']} threads")
    line = {
        "metric": METRIC,
        "value": round(g["tokens_per_s"], 1),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(g["ms_per_step"], 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {
            "workload": workload, "batch": cfg.batch, "layers": cfg.n_layers, "layer_groups": cfg.n_groups,
            "resident_layers": cfg.layers_resident,
            "q_heads": cfg.n_q_heads, "kv_heads": cfg.n_kv_heads, "head_dim": cfg.head_dim,
            "prompt_tokens": prompt_desc(cfg), "prompt_tagged": cfg.prompt_tagged, "n_sink": int(pol.n_sink),
            "generated_before_timing": args.t_start,
            "budget": beta, "realised_c_kv_governed": round(g["c_kv_governed"], 4),
            "realised_c_kv_all": round(g["c_kv_all"], 4), "page_tokens": 16,
            "mean_persisted_entries": round(g["mean_entries"], 1),
            "hbm_gb_per_step": round(g["bytes_per_step"] / 1e9, 3),
            "step_gbs": round(g["step_gbs"], 1),
            "recent_window": args.window, "online_controller": bool(args.controller),
            "prompt_append": g["prompt_append"],
        },
        "roofline": {
            "bound": "hbm", "achieved": round(g["achieved"], 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
            "frac": round(g["achieved"] / HBM_PEAK_GBS, 4), "traffic": traffic_record(workload),
            "kernel": attn_kernels(cfg, args.window, bool(args.controller)) + " (one pask_decode_attn call)",
            "bytes_per_launch": round(g["per_call_bytes"]), "avg_launch_us": round(g["avg_call_us"], 2),
            "read_probe_gbs": probe["read_gbs"] if probe else None,
            "frac_of_read_probe": round(g["achieved"] / probe["read_gbs"], 4) if probe else None,
            "copy_probe_gbs": probe["copy_gbs"] if probe else None,
        },
        "graph": g["graph"],
        "positions": [dict(t=r["t"], tokens_per_s=round(r["tokens_per_s"], 1), ms_per_step=round(r["ms_per_step"], 4),
                           avg_call_us=round(r["avg_call_us"], 2), bytes_per_call=round(r["per_call_bytes"]),
                           achieved_gbs=round(r["achieved"], 1), frac=round(r["achieved"] / HBM_PEAK_GBS, 4))
                      for r in runs],
        "cpu_baseline": cpu,
    }
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
