"""CPU tests of the C ABI: symbols, host-side method steps against the oracle,
and argument errors.  No device call is made here."""
import ctypes
import os
import re

import numpy as np
import pytest

from oracle import blockgtq_oracle as o
from paper_2606_24033_amd import blockgtq as bg
from paper_2606_24033_amd import synth

HEADER = os.path.join(os.path.dirname(os.path.dirname(__file__)), "include", "blockgtq.h")


def test_library_exports_every_declared_symbol():
    names = set(re.findall(r"\b(blockgtq_\w+)\s*\(", open(HEADER).read()))
    assert names == set(bg.EXPORTED)
    L = ctypes.CDLL(bg.LIB_PATH)
    for n in names:
        assert getattr(L, n) is not None


@pytest.mark.parametrize("b", range(1, 9))
def test_codebook_bit_exact_vs_oracle(b):
    c16, thr = bg.blockgtq_codebook(b)
    oc, ot = o.codebook(b)
    np.testing.assert_array_equal(c16.astype(np.float64), oc)
    np.testing.assert_array_equal(thr.astype(np.float64), ot)


def test_energy_scores_vs_oracle():
    sig = synth.sigma_profile(1, 0, 0)
    q, k = synth.calibration(1, 0, 0, 256, 4, sig)
    q, k = q.astype(np.float32), k.astype(np.float32)
    np.testing.assert_allclose(bg.blockgtq_energy_scores(q, k), o.energy_scores(q, k), rtol=1e-13)


def test_allocator_bit_exact_vs_oracle():
    g = np.random.default_rng(3)
    rows = [np.exp(2 * g.standard_normal(64)) for _ in range(40)]
    rows += [np.ones(64), np.zeros(64), np.array([4.0 ** (i % 5) for i in range(64)]),
             np.repeat([1.0, 16.0], 32), np.array([0.0] * 63 + [1.0])]
    s = np.stack(rows)
    for budget in (64, 100, 128, 192, 256, 511, 512):
        got = bg.blockgtq_allocate(s, budget)
        for r in range(len(rows)):
            np.testing.assert_array_equal(got[r], o.allocate(s[r], budget))


def test_allocator_small_blocks_and_bounds():
    g = np.random.default_rng(8)
    for _ in range(50):
        s = np.exp(g.standard_normal(4))
        for B in range(4, 33):
            np.testing.assert_array_equal(bg.blockgtq_allocate(s, B, 1, 8)[0], o.allocate(s, B, 1, 8))
        for B in range(8, 17):
            np.testing.assert_array_equal(bg.blockgtq_allocate(s, B, 2, 4)[0], o.allocate(s, B, 2, 4))


def test_allocator_degenerate_scores_vs_oracle():
    """Scores that stress the tie rules: subnormal and huge values (4^-b
    scalings that lose bits or underflow to zero), exact power-of-4 ladders
    (equal gains across blocks at different levels), many zeros, and bounds
    other than [1, 8]; the library's selection of the largest gains must give
    the oracle's greedy schedule bit for bit."""
    g = np.random.default_rng(21)
    tiny = np.finfo(np.float64).tiny
    rows = [np.full(64, 5e-324), np.full(64, tiny * 3.0), np.geomspace(5e-324, 1e300, 64),
            np.array([4.0 ** -(i % 9) for i in range(64)]), np.array([tiny * 4.0 ** (i % 4) for i in range(64)]),
            np.where(g.random(64) < 0.5, 0.0, np.exp(3 * g.standard_normal(64))),
            np.repeat([7.0, 7.0 / 4, 7.0 / 16, 7.0 / 64], 16), np.full(64, 1e308)]
    s = np.stack(rows)
    for bmin, bmax in ((1, 8), (2, 6), (3, 3), (1, 2)):
        cands = {64 * bmin, 64 * bmin + 1, 64 * bmin + 37, 32 * (bmin + bmax), 64 * bmax - 1, 64 * bmax}
        for budget in sorted(b for b in cands if 64 * bmin <= b <= 64 * bmax):
            got = bg.blockgtq_allocate(s, budget, bmin, bmax)
            for r in range(len(rows)):
                np.testing.assert_array_equal(got[r], o.allocate(s[r], budget, bmin, bmax), err_msg=f"row {r} B {budget}")


def test_allocator_errors():
    s = np.ones((1, 64))
    with pytest.raises(bg.BlockGTQError) as e:
        bg.blockgtq_allocate(s, 63)
    assert e.value.code == -2
    with pytest.raises(bg.BlockGTQError) as e:
        bg.blockgtq_allocate(-s, 128)
    assert e.value.code == -1
    with pytest.raises(bg.BlockGTQError):
        bg.blockgtq_allocate(s * np.nan, 128)
    with pytest.raises(bg.BlockGTQError):
        bg.blockgtq_allocate(s, 128, 0, 8)


def test_sizes_and_config_errors():
    cfg = bg.Config(n_layers=32, batch=1, n_kv_heads=8, group=4, capacity=131072 + 64, k_budget=128, v_bits=2)
    kc, kn, vc, vn = bg.cache_bytes(cfg)
    rows = 32 * 8 * cfg.capacity
    assert kc == rows * 32 and vc == rows * 32 and vn == rows * 2 and kn == rows * 16
    ws = bg.workspace_bytes(cfg, 32, 0, 131072)
    assert ws > 0
    bad = bg.Config(n_layers=1, batch=1, n_kv_heads=1, group=4, capacity=100, k_budget=128, v_bits=2)
    with pytest.raises(bg.BlockGTQError):
        bg.cache_bytes(bad)
    bad = bg.Config(n_layers=1, batch=1, n_kv_heads=1, group=9, capacity=128, k_budget=128, v_bits=2)
    with pytest.raises(bg.BlockGTQError) as e:
        bg.cache_bytes(bad)
    assert e.value.code == -5
    with pytest.raises(bg.BlockGTQError) as e:
        bg.workspace_bytes(cfg, 32, 0, cfg.capacity + 1)
    assert e.value.code == -3


def test_prefill_sizes_and_argument_errors():
    """Host-side checks of the prefill entry point (rejected before any launch:
    the pointers are never dereferenced)."""
    cfg = bg.Config(n_layers=2, batch=3, n_kv_heads=2, group=8, capacity=1024, k_budget=192, v_bits=3)
    assert bg.prefill_workspace_bytes(cfg, 100) == ((3 * 100 * 16 * 128 * 4 + 255) // 256) * 256
    assert bg.prefill_workspace_bytes(cfg, 0) == 0
    with pytest.raises(bg.BlockGTQError) as e:
        bg.prefill_workspace_bytes(cfg, -1)
    assert e.value.code == -1
    L = bg.lib()
    c = cfg.c()
    fake = ctypes.c_void_p(256)
    cache = bg._Cache(256, 256, 256, 256)

    def call(layer=0, n_q=10, max_pos=100, ws=10 ** 9, q=fake):
        return L.blockgtq_prefill_attn(ctypes.byref(c), fake, layer, q, n_q, fake, max_pos, ctypes.byref(cache),
                                       fake, fake, ws, None)
    assert call(layer=-1) == -1            # all-layer calls are decode-only
    assert call(layer=2) == -1
    assert call(n_q=-3) == -1
    assert call(n_q=0) == 0                # nothing to do, nothing launched
    assert call(max_pos=1024) == -3        # must stay below the capacity
    assert call(max_pos=-1) == -3
    assert call(ws=16) == -4
    assert call(q=ctypes.c_void_p(258)) == -1   # 4-byte alignment
    assert b"aligned" in L.blockgtq_last_error()


def test_window_sizes_and_argument_errors():
    """Host-side checks of the protected-window entry points (rejected before
    any launch: the pointers are never dereferenced)."""
    cfg = bg.Config(n_layers=2, batch=3, n_kv_heads=2, group=4, capacity=1024, k_budget=128, v_bits=2)
    assert bg.window_bytes(cfg, 4, 128) == 2 * 3 * 2 * 2 * 132 * 128 * 2
    assert bg.window_bytes(cfg, 0, 0) == 0
    for ns, nr in [(64, 128), (-1, 0), (4, 1025), (0, -2)]:
        with pytest.raises(bg.BlockGTQError) as e:
            bg.window_bytes(cfg, ns, nr)
        assert e.value.code == -1
    base = bg.workspace_bytes(cfg, 2, 0, 1000)
    assert bg.protected_workspace_bytes(cfg, 2, 0, 1000) == base + ((2 * 3 * 8 * 130 * 4 + 255) // 256) * 256
    L = bg.lib()
    c = cfg.c()
    fake = ctypes.c_void_p(256)
    cache = bg._Cache(256, 256, 256, 256)

    def dec(layer=-1, ns=4, nr=128, ws=10 ** 9, max_ctx=1000, win=fake):
        return L.blockgtq_decode_attn_protected(ctypes.byref(c), fake, layer, fake, fake, max_ctx,
                                                ctypes.byref(cache), win, ns, nr, fake, fake, ws, 0, None)
    assert dec(ns=64) == -1
    assert dec(nr=2000) == -1
    assert dec(layer=2) == -1
    assert dec(max_ctx=1025) == -3
    assert dec(win=None) == -1
    assert dec(win=None, ns=0, nr=0, ws=16) == -4   # an empty window needs no buffer
    assert dec(ws=base) == -4              # the window partials need room past the split partials

    def app(layer=0, n_new=5, ns=4, nr=128, win=fake):
        return L.blockgtq_window_append(ctypes.byref(c), layer, fake, fake, n_new, fake, ns, nr, win, None)
    assert app(layer=5) == -1
    assert app(n_new=-1) == -1
    assert app(n_new=2000) == -3
    assert app(ns=70) == -1
    assert app(n_new=0) == 0               # nothing to write
    assert app(ns=0, nr=0) == 0            # no window
    assert app(win=None) == -1


def test_rope_step_sizes_and_argument_errors():
    """Host-side checks of the pre-RoPE decode step (rejected before any launch)."""
    cfg = bg.Config(n_layers=2, batch=3, n_kv_heads=2, group=4, capacity=1024, k_budget=128, v_bits=2)
    dec = bg.workspace_bytes(cfg, 2, 0, 1000)
    a = lambda x: (x + 255) // 256 * 256
    assert bg.rope_step_workspace_bytes(cfg, 1000) == dec + a(12) + a(2 * 3 * 8 * 512) + 2 * a(2 * 3 * 2 * 512)
    L = bg.lib()
    c = cfg.c()
    fake = ctypes.c_void_p(256)
    cache = bg._Cache(256, 256, 256, 256)

    def call(base=1e4, max_ctx=1000, ws=10 ** 9, splits=0, q=fake):
        return L.blockgtq_rope_decode_step(ctypes.byref(c), fake, base, q, fake, fake, fake, max_ctx,
                                           ctypes.byref(cache), fake, fake, ws, splits, None)
    assert call(base=1.0) == -1
    assert call(base=float("inf")) == -1
    assert call(base=float("nan")) == -1
    assert call(max_ctx=0) == -3
    assert call(max_ctx=1025) == -3
    assert call(splits=5000) == -1
    assert call(ws=dec) == -4
    assert call(q=None) == -1


def test_bench_refuses_more_than_one_gpu():
    """bench.py measures one GPU; --gpus above 1 exits with a message, before
    touching a device."""
    import subprocess
    import sys
    root = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
    r = subprocess.run([sys.executable, os.path.join(root, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr


def test_cache_buffers_must_be_16_byte_aligned():
    """Every entry point that reads or writes the packed cache rejects a cache
    buffer that is not 16-byte aligned (the kernels use 16-byte loads) before
    any launch: the fake pointers are never dereferenced."""
    cfg = bg.Config(n_layers=1, batch=1, n_kv_heads=1, group=4, capacity=128, k_budget=128, v_bits=2)
    L = bg.lib()
    c = cfg.c()
    f = ctypes.c_void_p(256)
    big = 1 << 30
    for field in ("k_codes", "k_norms", "v_codes", "v_norms"):
        ptrs = dict(k_codes=256, k_norms=256, v_codes=256, v_norms=256)
        ptrs[field] = 264
        cache = ctypes.byref(bg._Cache(**ptrs))
        calls = {
            "quantize_append": lambda: L.blockgtq_quantize_append(ctypes.byref(c), f, 0, f, f, 3, f, cache, None),
            "decode_attn": lambda: L.blockgtq_decode_attn(ctypes.byref(c), f, 0, f, f, 10, cache, f, f, big, 0, None),
            "decode_attn_protected": lambda: L.blockgtq_decode_attn_protected(ctypes.byref(c), f, 0, f, f, 10, cache,
                                                                              f, 4, 8, f, f, big, 0, None),
            "rope_decode_step": lambda: L.blockgtq_rope_decode_step(ctypes.byref(c), f, 1e4, f, f, f, f, 10, cache,
                                                                    f, f, big, 0, None),
            "prefill_attn": lambda: L.blockgtq_prefill_attn(ctypes.byref(c), f, 0, f, 10, f, 100, cache, f, f, big,
                                                            None),
        }
        for name, call in calls.items():
            assert call() == -1, (field, name)
            assert b"16-byte aligned" in L.blockgtq_last_error(), (field, name)
