"""The C ABI on the host (no GPU): the library loads, exports every entry
point include/pask.h declares, parses and validates policy blobs, lays out
caches and rejects bad arguments before any HIP call."""

import os
import re
import struct

import numpy as np
import pytest

from workload.policy import fnv1a32, make_policy, pack_blob, with_budget_controller

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
pask = pytest.importorskip("paper_2608_28276_amd.pask", reason="libpask.so not built")


def header_functions():
    text = open(os.path.join(ROOT, "include", "pask.h")).read()
    return sorted(set(re.findall(r"^\s*(?:int|size_t|const char\*)\s+(pask_\w+)\s*\(", text, re.M)))


def test_exports_every_declared_symbol():
    names = header_functions()
    assert len(names) == 13
    lib = pask.library()
    for n in names:
        assert hasattr(lib, n), n
    assert set(names) == set(pask.EXPORTS)


def geom(**kw):
    d = dict(max_batch=4, n_layers=2, n_q_heads=8, n_kv_heads=2, head_dim=64, max_tokens_per_seq=512,
             hi_pages=64, lo_pages=64)
    d.update(kw)
    return pask.make_geom(**d)


def blob_for(T=6, C=2, L=2, beta=0.33, seed=1, **over):
    pol = make_policy(T, C, L, beta, seed)
    for k, v in over.items():
        setattr(pol, k, v)
    return pol, pack_blob(pol)


def test_policy_load_roundtrip():
    pol, blob = blob_for()
    p = pask.pask_policy_load(blob, geom())
    assert (p.n_tags, p.n_groups, p.n_layers, p.n_sink, p.recent_window) == (6, 2, 2, 0, 0)
    got_a = np.array([[p.action[z][c] for c in range(2)] for z in range(6)])
    got_f = np.array([[p.floor_[z][c] for c in range(2)] for z in range(6)])
    got_r = np.array([[[p.rho_up[z][c][i] for i in range(2)] for c in range(2)] for z in range(6)], np.float32)
    assert (got_a == pol.action).all() and (got_f == pol.floor).all() and (got_r == pol.rho_up).all()
    assert list(p.group_of_layer[:2]) == pol.group_of_layer.tolist()
    assert list(p.entry_bytes) == [0, 144, 512]


def blob_v2(T=6, C=2, L=2, S=7, beta=0.33, seed=1):
    pol = make_policy(T, C, L, beta, seed)
    rng = np.random.default_rng(seed)
    traces = [(rng.integers(0, T, 200), rng.integers(0, S, 200)) for _ in range(3)]
    pol = with_budget_controller(pol, traces, S, critical=(1, 2))
    return pol, pack_blob(pol)


def test_policy_load_v2_roundtrip():
    pol, blob = blob_v2()
    assert struct.unpack_from("<H", blob, 4)[0] == 2
    p = pask.pask_policy_load(blob, geom())
    assert (p.n_states, p.beta_q) == (7, pol.beta_q)
    assert list(p.reserve_q[:7]) == pol.reserve_q.tolist() and list(p.crit[:7]) == pol.crit.tolist()
    assert list(p.reserve_q[7:]) == [0] * 57 and list(p.crit[7:]) == [0] * 57
    got_a = np.array([[p.action[z][c] for c in range(2)] for z in range(6)])
    assert (got_a == pol.action).all()
    p1 = pask.pask_policy_load(pack_blob(pol, version=1), geom())      # the table without the controller
    assert p1.n_states == 0 and p1.beta_q == 0


@pytest.mark.parametrize("case", ["states0", "states65", "crit2", "pad", "short", "long"])
def test_policy_load_v2_rejects(case):
    pol, blob = blob_v2()
    L, T, C, S = 2, 6, 2, 7
    ctl = 32 + ((L + 2 * T * C + 3) // 4) * 4 + 8 * T * C        # n_states, beta_q, reserve_q, crit
    crit_at = ctl + 8 + 4 * S
    if case == "states0":
        bad = _patch(blob, ctl, "<I", 0)
    elif case == "states65":
        bad = _patch(blob, ctl, "<I", 65)
    elif case == "crit2":
        bad = _patch(blob, crit_at + 3, "<B", 2)
    elif case == "pad":
        bad = _patch(blob, crit_at + S, "<B", 1)
    elif case == "short":                      # body one word short of what n_states needs
        b = bytearray(blob[:-8] + blob[-4:])
        struct.pack_into("<I", b, 28, struct.unpack_from("<I", b, 28)[0] - 4)
        bad = _rehash(bytes(b))
    else:                                      # n_states claims more than the body holds
        bad = _patch(blob, ctl, "<I", 8)
    with pytest.raises(pask.PaskError) as e:
        pask.pask_policy_load(bad, geom())
    assert e.value.status == pask.PASK_E_POLICY


def _rehash(b: bytes) -> bytes:
    return b[:-4] + struct.pack("<I", fnv1a32(b[:-4]))


def _patch(blob: bytes, off: int, fmt: str, val) -> bytes:
    b = bytearray(blob)
    struct.pack_into(fmt, b, off, val)
    return _rehash(bytes(b))


@pytest.mark.parametrize("case,code", [
    ("magic", pask.PASK_E_POLICY), ("version", pask.PASK_E_POLICY), ("hash", pask.PASK_E_POLICY),
    ("truncated", pask.PASK_E_POLICY), ("action3", pask.PASK_E_POLICY), ("group_oob", pask.PASK_E_POLICY),
    ("rho_nan", pask.PASK_E_POLICY), ("rho_neg", pask.PASK_E_POLICY), ("n_tags0", pask.PASK_E_POLICY),
    ("window", pask.PASK_E_SHAPE), ("layers_mismatch", pask.PASK_E_SHAPE), ("pad", pask.PASK_E_POLICY),
])
def test_policy_load_rejects(case, code):
    pol, blob = blob_for()
    L, T, C = 2, 6, 2
    rho_off = 32 + ((L + 2 * T * C + 3) // 4) * 4
    if case == "magic":
        bad = b"XASK" + blob[4:]
    elif case == "version":
        bad = _patch(blob, 4, "<H", 3)
    elif case == "hash":
        bad = blob[:-1] + bytes([blob[-1] ^ 1])
    elif case == "truncated":
        bad = blob[:-8]
    elif case == "action3":
        bad = _patch(blob, 32 + L + 3, "<B", 3)
    elif case == "group_oob":
        bad = _patch(blob, 32, "<B", 2)
    elif case == "rho_nan":
        bad = _patch(blob, rho_off, "<f", float("nan"))
    elif case == "rho_neg":
        bad = _patch(blob, rho_off + 4, "<f", -1.0)
    elif case == "n_tags0":
        bad = _patch(blob, 8, "<I", 0)
    elif case == "window":
        bad = _patch(blob, 24, "<I", 4)
    elif case == "layers_mismatch":
        with pytest.raises(pask.PaskError) as e:
            pask.pask_policy_load(blob, geom(n_layers=4))
        assert e.value.status == code
        return
    else:  # non-zero padding byte between the u8 tables and rho
        pad_at = 32 + L + 2 * T * C
        assert pad_at < rho_off
        bad = _patch(blob, pad_at, "<B", 1)
    with pytest.raises(pask.PaskError) as e:
        pask.pask_policy_load(bad, geom())
    assert e.value.status == code


def test_recent_window_geometry_and_layout():
    """The table's recent window W must equal the geometry's; the HIGH pool
    starts with ceil(W/16) window pages per (sequence, layer) and the staging
    rows grow by W + 2 words."""
    pol, _ = blob_for()
    pol.recent_window = 20
    blob = pack_blob(pol)
    p = pask.pask_policy_load(blob, geom(recent_window=20))
    assert p.recent_window == 20
    with pytest.raises(pask.PaskError) as e:
        pask.pask_policy_load(blob, geom())
    assert e.value.status == pask.PASK_E_SHAPE
    L0 = pask.pask_cache_layout_query(geom())
    L = pask.pask_cache_layout_query(geom(recent_window=20))
    assert (L0.ring_pages, L0.staging_stride) == (0, 512 + 4)
    assert (L.ring_pages, L.staging_stride) == (4 * 2 * 2, 512 + 20 + 4)
    assert L.lo_pool_off - L.hi_pool_off >= (16 + 64) * L.hi_page_bytes
    assert L.hi_pool_off - L.ring_act_off >= 4 * 2 * 20 and L.ring_act_off >= L.budget_off + 11232
    assert pask.pask_cache_bytes(geom(recent_window=513)) == 0       # W <= max_tokens_per_seq
    assert pask.pask_cache_bytes(geom(recent_window=-1)) == 0
    c = _fake_cache(geom())
    with pytest.raises(pask.PaskError) as e:                          # a W = 20 table on a W = 0 cache
        pask.pask_kv_append(pask.pask_policy_load(blob, geom(recent_window=20)), c, 0, 1, None, 4, 1 << 41,
                            1 << 41, 1 << 41, 0, 0)
    assert e.value.status == pask.PASK_E_SHAPE


def test_layout_and_sizes():
    g = geom()
    L = pask.pask_cache_layout_query(g)
    assert L.hi_page_bytes == 2 * 2 * 16 * 64 * 2
    assert L.lo_page_bytes == 2 * 2 * (16 * 32 + 16 * 2 * 2)
    assert L.max_pages == 32 and L.counter_stride == 8
    offs = [L.status_off, L.counters_off, L.block_table_off, L.index_list_off, L.staging_off, L.budget_off,
            L.hi_pool_off, L.lo_pool_off, L.total_bytes]
    assert offs == sorted(offs) and all(o % 256 == 0 for o in offs)
    assert L.counters_off - L.status_off >= 16
    assert L.block_table_off - L.counters_off >= 4 * 2 * 8 * 4
    assert L.index_list_off - L.block_table_off >= 4 * 2 * 2 * 32 * 4
    assert L.budget_off - L.staging_off >= 4 * 512 * 4
    assert L.hi_pool_off - L.budget_off >= 11232 and L.hi_pool_off % 4096 == 0
    assert L.lo_pool_off - L.hi_pool_off >= 64 * L.hi_page_bytes
    assert L.total_bytes - L.lo_pool_off >= 64 * L.lo_page_bytes
    assert pask.pask_cache_bytes(g) == L.total_bytes
    g4 = geom(n_q_heads=64, n_kv_heads=8, head_dim=128)
    L4 = pask.pask_cache_layout_query(g4)
    assert L4.hi_page_bytes == 65536 and L4.lo_page_bytes == 8 * 2 * (16 * 64 + 16 * 4 * 2)


@pytest.mark.parametrize("bad", [dict(head_dim=96), dict(n_q_heads=6), dict(n_q_heads=32, n_kv_heads=2),
                                 dict(page_tokens=32), dict(max_batch=0), dict(n_layers=200),
                                 dict(hi_pages=-1), dict(max_tokens_per_seq=0)])
def test_unsupported_geometry(bad):
    g = geom(**bad)
    assert pask.pask_cache_bytes(g) == 0
    with pytest.raises(pask.PaskError) as e:
        pask.pask_cache_layout_query(g)
    assert e.value.status == pask.PASK_E_SHAPE


def _ws_want(g, batch, hint):
    # splits = ceil(hint / 128) + 2; with at most 64 (sequence, KV head) segments, pieces down to
    # one page while the call holds at most 4096 partials: max(that, min(ceil(hint / 16) + 2,
    # 4096 // segments)).  Per (sequence, KV head, piece) a block of G4 = max(G, 4) rows:
    # o: blocks*G4*D*4, ml: blocks*G4*2*4, then 8 int32 per sequence (each 256-aligned)
    # a hint above max_tokens_per_seq counts as max_tokens_per_seq
    hint = min(hint, g.max_tokens_per_seq)
    segs = batch * g.n_kv_heads
    splits = -(-hint // 128) + 2
    if segs <= 64:
        splits = max(splits, min(-(-hint // 16) + 2, 4096 // segs))
    G4 = max(4, g.n_q_heads // g.n_kv_heads)
    blocks = segs * splits
    want = ((blocks * G4 * g.head_dim * 4 + 255) // 256) * 256
    want = ((want + blocks * G4 * 8 + 255) // 256) * 256
    return ((want + batch * 32 + 255) // 256) * 256


@pytest.mark.parametrize("batch,hint", [(4, 512), (8, 512), (9, 512), (1, 100000), (32, 100000), (64, 9000)])
def test_workspace_bytes(batch, hint):
    g = geom(max_batch=64)
    assert pask.pask_workspace_bytes(g, batch, hint) == _ws_want(g, batch, hint)
    g = geom(max_batch=64, max_tokens_per_seq=200000)
    assert pask.pask_workspace_bytes(g, batch, hint) == _ws_want(g, batch, hint)


def test_workspace_bytes_hint_and_batch_edges():
    """A hint at the int32 limit sizes as max_tokens_per_seq (no overflow); a
    batch outside 1..max_batch gets 0."""
    g = geom(max_batch=64)
    top = pask.pask_workspace_bytes(g, 64, g.max_tokens_per_seq)
    assert pask.pask_workspace_bytes(g, 64, 2**31 - 1) == top == pask.pask_workspace_bytes(g, 64, 0)
    assert pask.pask_workspace_bytes(g, 65, 512) == 0 and pask.pask_workspace_bytes(g, 0, 512) == 0


def test_distortion_validation_before_any_hip_call():
    g = geom()
    ref, itv = _fake_cache(g), _fake_cache(g)
    A = 1 << 41
    ws_need = 2 * pask.pask_workspace_bytes(g, 2, 512)
    other = _fake_cache(geom(n_kv_heads=4))
    cases = [
        (dict(layer=2), pask.PASK_E_SHAPE), (dict(batch=0), pask.PASK_E_SHAPE), (dict(batch=5), pask.PASK_E_SHAPE),
        (dict(itv=other), pask.PASK_E_SHAPE), (dict(q=0), pask.PASK_E_ARG), (dict(q=A + 8), pask.PASK_E_ARG),
        (dict(dist=0), pask.PASK_E_ARG), (dict(dist=A + 2), pask.PASK_E_ARG), (dict(ws=A + 128), pask.PASK_E_ARG),
        (dict(ws_bytes=ws_need - 1), pask.PASK_E_CAPACITY), (dict(scale=float("nan")), pask.PASK_E_ARG),
    ]
    for over, code in cases:
        kw = dict(itv=itv, layer=0, batch=2, q=A, dist=A, ws=A, ws_bytes=ws_need, scale=0.125)
        kw.update(over)
        with pytest.raises(pask.PaskError) as e:
            pask.pask_attn_distortion(ref, kw["itv"], kw["layer"], kw["batch"], kw["q"], None, kw["scale"], 512,
                                      kw["ws"], kw["ws_bytes"], kw["dist"], 0)
        assert e.value.status == code, over
    small = _fake_cache(g)
    small.bytes = ref.bytes - 1
    with pytest.raises(pask.PaskError) as e:
        pask.pask_attn_distortion(ref, small, 0, 2, A, None, 0.125, 512, A, ws_need, A, 0)
    assert e.value.status == pask.PASK_E_CAPACITY


def _fake_cache(g):
    c = pask.pask_cache()
    c.geom = g
    c.base = 1 << 40       # never dereferenced: every call below fails validation first
    c.bytes = pask.pask_cache_bytes(g)
    return c


def test_append_and_attn_validation_before_any_hip_call():
    g = geom()
    _, blob = blob_for()
    p = pask.pask_policy_load(blob, g)
    c = _fake_cache(g)
    A = 1 << 41
    cases = [
        (dict(layer=2), pask.PASK_E_SHAPE), (dict(layer=-1), pask.PASK_E_SHAPE),
        (dict(batch=0), pask.PASK_E_SHAPE), (dict(batch=5), pask.PASK_E_SHAPE),
        (dict(max_new=513), pask.PASK_E_SHAPE), (dict(k=A + 2), pask.PASK_E_ARG),
        (dict(k=0), pask.PASK_E_ARG), (dict(tags=0), pask.PASK_E_ARG), (dict(flags=2), pask.PASK_E_ARG),
    ]
    for over, code in cases:
        kw = dict(layer=0, batch=1, n_new=None, max_new=4, tags=A, k=A, v=A, flags=0)
        kw.update(over)
        with pytest.raises(pask.PaskError) as e:
            pask.pask_kv_append(p, c, kw["layer"], kw["batch"], kw["n_new"], kw["max_new"], kw["tags"], kw["k"],
                                kw["v"], kw["flags"], 0, states=kw.get("states"))
        assert e.value.status == code, over
    # parser states need a table that carries the controller (version 2)
    with pytest.raises(pask.PaskError) as e:
        pask.pask_kv_append(p, c, 0, 1, None, 4, A, A, A, 0, 0, states=A)
    assert e.value.status == pask.PASK_E_POLICY
    small = _fake_cache(g)
    small.bytes = c.bytes - 1
    with pytest.raises(pask.PaskError) as e:
        pask.pask_kv_append(p, small, 0, 1, None, 4, A, A, A, 0, 0)
    assert e.value.status == pask.PASK_E_CAPACITY
    ws_need = pask.pask_workspace_bytes(g, 1, 512)
    acases = [
        (dict(q=A + 8), pask.PASK_E_ARG), (dict(out=0), pask.PASK_E_ARG), (dict(ws=A + 128), pask.PASK_E_ARG),
        (dict(ws_bytes=ws_need - 1), pask.PASK_E_CAPACITY), (dict(scale=float("inf")), pask.PASK_E_ARG),
        (dict(tags=A, k=0), pask.PASK_E_ARG), (dict(layer=9), pask.PASK_E_SHAPE),
    ]
    for over, code in acases:
        kw = dict(layer=0, q=A, out=A, tags=None, k=None, ws=A, ws_bytes=ws_need, scale=0.125)
        kw.update(over)
        with pytest.raises(pask.PaskError) as e:
            pask.pask_decode_attn(p, c, kw["layer"], 1, kw["q"], kw["out"], None, kw["tags"], kw["k"], kw["k"],
                                  kw["scale"], 512, kw["ws"], kw["ws_bytes"], 0)
        assert e.value.status == code, over
    with pytest.raises(pask.PaskError) as e:
        pask.pask_decode_attn(p, c, 0, 1, A, A, None, A, A, A, 0.125, 512, A, ws_need, 0, states_new=A)
    assert e.value.status == pask.PASK_E_POLICY
    # the controller's set-up
    for args, code in [((p, c, 1, 100), pask.PASK_E_POLICY), ((p2 := pask.pask_policy_load(blob_v2()[1], g), c, 0, 100),
                                                                 pask.PASK_E_SHAPE),
                       ((p2, c, 5, 100), pask.PASK_E_SHAPE), ((p2, c, 1, -1), pask.PASK_E_ARG)]:
        with pytest.raises(pask.PaskError) as e:
            pask.pask_budget_init(*args, 0)
        assert e.value.status == code, args[2:]
    bad_act = pask.pask_policy_load(blob_v2()[1], g)
    bad_act.action[1][0] = 3
    with pytest.raises(pask.PaskError) as e:
        pask.pask_budget_init(bad_act, c, 1, 100, 0)
    assert e.value.status == pask.PASK_E_POLICY
    # R_0 = beta_q * t_max * sum_c m(H, c) / 65536 must stay below 2^62
    gb = geom(n_layers=128, n_q_heads=8, n_kv_heads=8, head_dim=128)
    pb = pask.pask_policy_load(blob_v2(L=128)[1], gb)
    pb.beta_q = 0xFFFFFFFF
    with pytest.raises(pask.PaskError) as e:
        pask.pask_budget_init(pb, _fake_cache(gb), 1, (1 << 31) - 1, 0)
    assert e.value.status == pask.PASK_E_ARG
    other = pask.pask_policy_load(blob_for(L=4, C=2)[1], geom(n_layers=4))
    with pytest.raises(pask.PaskError) as e:
        pask.pask_kv_append(other, c, 0, 1, None, 4, A, A, A, 0, 0)
    assert e.value.status == pask.PASK_E_SHAPE


def test_noalloc_attn_validation_before_any_hip_call():
    """pask_decode_attn_noalloc: the checks of pask_decode_attn, and a batch
    whose partials cannot fit the library's scratch even at two pieces per
    (sequence, KV head) (505 sequences x 8 KV heads at group 8, head_dim 128)."""
    A = 1 << 41
    g = geom()
    p = pask.pask_policy_load(blob_for()[1], g)
    c = _fake_cache(g)
    for over, code in [(dict(q=A + 8), pask.PASK_E_ARG), (dict(out=0), pask.PASK_E_ARG),
                       (dict(scale=float("nan")), pask.PASK_E_ARG), (dict(layer=2), pask.PASK_E_SHAPE),
                       (dict(batch=5), pask.PASK_E_SHAPE), (dict(tags=A, k=0), pask.PASK_E_ARG)]:
        kw = dict(layer=0, batch=1, q=A, out=A, tags=None, k=None, scale=0.125)
        kw.update(over)
        with pytest.raises(pask.PaskError) as e:
            pask.pask_decode_attn_noalloc(p, c, kw["layer"], kw["batch"], kw["q"], kw["out"], None, kw["tags"],
                                          kw["k"], kw["k"], kw["scale"], 512, 0)
        assert e.value.status == code, over
    gb = geom(max_batch=600, n_q_heads=64, n_kv_heads=8, head_dim=128, max_tokens_per_seq=64)
    pb = pask.pask_policy_load(blob_for()[1], gb)
    cb = _fake_cache(gb)
    with pytest.raises(pask.PaskError) as e:
        pask.pask_decode_attn_noalloc(pb, cb, 0, 505, A, A, None, None, None, None, 0.125, 64, 0)
    assert e.value.status == pask.PASK_E_CAPACITY


def test_status_strings():
    assert pask.pask_status_string(0) == "ok"
    assert "policy" in pask.pask_status_string(pask.PASK_E_POLICY)
    assert pask.pask_status_string(-99) == "unknown status"


def test_debug_mode_keeps_the_validation_codes():
    """PASK_DEBUG=1 adds checks after launches only: every argument check
    still returns its code before any HIP call (the library reads the
    variable once, hence a process of its own)."""
    import subprocess
    import sys
    env = dict(os.environ, PASK_DEBUG="1")
    p = subprocess.run([sys.executable, "-m", "pytest", "-q", "-p", "no:cacheprovider", "-m", "not gpu",
                        os.path.join(ROOT, "tests", "test_abi_host.py"), "-k", "validation_before_any_hip_call"],
                       cwd=ROOT, env=env, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True, timeout=300)
    assert p.returncode == 0, p.stdout[-3000:]
    assert re.search(r"\b3 passed\b", p.stdout), p.stdout[-1000:]
