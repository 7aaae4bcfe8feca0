"""The decode entry point that allocates nothing (blockgtq_decode_attn_noalloc)
against blockgtq_decode_attn with a caller-owned workspace: two calls in a
row, the second smaller (one layer, shorter contexts), each bit-identical to
the workspace entry point and within 2e-3 of the oracle; a call whose
workspace exceeds the static array is rejected on the host."""
import numpy as np
import pytest

from oracle import blockgtq_oracle as o  # noqa: F401  (the oracle side of the parity check)
from paper_2606_24033_amd import synth
from tests import _parity as P

pytestmark = pytest.mark.gpu
torch = pytest.importorskip("torch")


def _dev(x):
    t = torch.from_numpy(np.ascontiguousarray(x, dtype=np.float32))
    return t.to(device="cuda", dtype=torch.bfloat16).contiguous()


@pytest.mark.parametrize("G,v_bits", [(4, 2), (8, 3)])
def test_noalloc_decode_matches_workspace_entry_point(G, v_bits):
    """K3V2 with one query set of 4 heads, and K3V3 with two sets of 8 (the
    12-bit table of 3-bit codes)."""
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2606_24033_amd import blockgtq as bg
    bg.lib()
    L, B, H = 2, 2, 2
    lens = [1400, 300]
    st = P.make_setup(61, L, B, H, G, 1408, 192, v_bits, 5e5, "bf16")
    assert np.array_equal(st.bits, st.bits_oracle)
    layout = bg.Layout(st.cfg, st.bits, synth.flat_rot_k(st.rot_k), st.rot_v)
    cache = bg.Cache(st.cfg)
    kv = {(l, b, h): P.keys_values(st, l, h, 3000 * b, lens[0]) for l in range(L) for b in range(B) for h in range(H)}
    for l in range(L):
        K = np.stack([np.stack([kv[l, b, h][0] for h in range(H)], 1) for b in range(B)])   # [B, n, H, 128]
        V = np.stack([np.stack([kv[l, b, h][1] for h in range(H)], 1) for b in range(B)])
        bg.blockgtq_quantize_append(st.cfg, layout, l, _dev(K), _dev(V), torch.zeros(B, dtype=torch.int32,
                                                                                  device="cuda"), cache)
    qs = np.stack([np.stack([np.concatenate([synth.cast(synth.queries(st.seed, l, h, lens[b] - 1, G, st.base, step=b),
                                                        "bf16") for h in range(H)]) for b in range(B)])
                   for l in range(L)])                                    # [L, B, H G, 128]
    q_all = _dev(qs)

    def check(layer, ctxl, n_splits):
        ctx = torch.tensor(ctxl, dtype=torch.int32, device="cuda")
        q = q_all if layer < 0 else q_all[layer].contiguous()
        ref = bg.blockgtq_decode_attn(st.cfg, layout, layer, q, ctx, max(ctxl), cache, n_splits=n_splits)
        out = torch.full_like(ref, float("nan"))
        bg.blockgtq_decode_attn_noalloc(st.cfg, layout, layer, q, ctx, max(ctxl), cache, out, n_splits=n_splits)
        torch.cuda.synchronize()
        np.testing.assert_array_equal(out.cpu().numpy(), ref.cpu().numpy())
        got = out.cpu().numpy().astype(np.float64)
        layers = range(L) if layer < 0 else [layer]
        for li, lay in enumerate(layers):
            for b in range(B):
                for h in range(H):
                    rows = P.oracle_rows(st, lay, h, kv[lay, b, h][0][:ctxl[b]], kv[lay, b, h][1][:ctxl[b]])
                    oref = P.oracle_attention(st, lay, h, qs[lay, b, h * G:(h + 1) * G], rows, ctxl[b])
                    g = got[li, b] if layer < 0 else got[b]
                    assert P.rel_err(g[h * G:(h + 1) * G], oref) <= P.tol_attention(), (layer, lay, b, h)

    check(-1, lens, 0)            # all layers, 1400 / 300 rows, default split plan
    check(1, [200, 77], 3)        # then a smaller call: one layer, fewer rows and splits
    # a workspace beyond the static array: rejected before anything is enqueued
    big = bg.Config(n_layers=64, batch=16, n_kv_heads=8, group=8, capacity=1 << 20, k_budget=128, v_bits=2)
    with pytest.raises(bg.BlockGTQError) as e:
        bg.blockgtq_decode_attn_noalloc(big, layout, -1, q_all, torch.tensor([5] * 16, dtype=torch.int32,
                                                                            device="cuda"),
                                        1 << 20, cache, torch.empty(1, device="cuda"), n_splits=64)
    assert e.value.code == -4
